// kernels_metrics.hip -- per-round metrics, off the hot path.
//
// Appendix A states the goal as minimising the sum of the private objectives
// at a common point and bounds the distance to consensus by sigma_2(P)^t.
// These kernels report, in fp64 with fixed summation orders:
//   mean_i f_i(w_i), F(w_bar) = (1/n) sum_i f_i(w_bar), ||W - 1 w_bar^T||_F and
//   the mean of all model entries (which a doubly-stochastic reduce keeps).
#include <cmath>
#include <mutex>

#include "asap_launch.h"

namespace asap {
namespace {

constexpr int kColBlocksMax = kMetricColBlocks;  // partials 0 .. 2*kColBlocksMax

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return __shfl(v, 0, 64);
}

// fixed-order tree over the 256 threads of a block
__device__ double block_sum_d(double v, double* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

__device__ __forceinline__ double model_at(const MetricArgs& a, int i, int64_t c) {
  const double s = a.scale ? double(a.scale[i]) : 1.0;
  return s * double(a.W[int64_t(i) * a.ld + c]);
}

// column pass: w_bar, consensus partial, mean partial
__global__ __launch_bounds__(256) void cols_kernel(MetricArgs a) {
  __shared__ double sh[256];
  double cons = 0.0, msum = 0.0;
  for (int64_t c = int64_t(blockIdx.x) * 256 + threadIdx.x; c < a.dim; c += int64_t(gridDim.x) * 256) {
    double m = 0.0;
    for (int i = 0; i < a.n; ++i) m += model_at(a, i, c);
    m /= double(a.n);
    double d2 = 0.0;
    for (int i = 0; i < a.n; ++i) {
      const double d = model_at(a, i, c) - m;
      d2 += d * d;
    }
    a.wbar[c] = m;
    cons += d2;
    msum += m;
  }
  cons = block_sum_d(cons, sh);
  msum = block_sum_d(msum, sh);
  if (threadIdx.x == 0) {
    a.part[2 * blockIdx.x] = cons;
    a.part[2 * blockIdx.x + 1] = msum;
  }
}

__device__ __forceinline__ double loss_of(double ym, int loss) {
  if (loss == 1) return fmax(0.0, 1.0 - ym);
  return fmax(-ym, 0.0) + log1p(exp(-fabs(ym)));  // softplus(-ym)
}

// block (i, c): worker i's samples and model entries of chunk c (contiguous
// ranges); loss at its own model, loss at w_bar, and its part of ||w_i||^2
__global__ __launch_bounds__(256) void loss_kernel(MetricArgs a, int64_t base, int nch) {
  __shared__ double sh[256];
  const int i = blockIdx.x / nch, ch = blockIdx.x % nch, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t r0 = a.S * ch / nch, r1 = a.S * (ch + 1) / nch;
  const int64_t c0 = a.dim * ch / nch, c1 = a.dim * (ch + 1) / nch;
  double lown = 0.0, lbar = 0.0, nrm = 0.0;
  for (int64_t r = r0 + wave; r < r1; r += 4) {
    const int64_t g = int64_t(i) * a.S + r;
    double mo = 0.0, mb = 0.0;
    if (a.row_ptr) {
      const int64_t p0 = a.row_ptr[g], p1 = a.row_ptr[g + 1];
      for (int64_t p = p0 + lane; p < p1; p += 64) {
        const double v = a.val[p];
        mo += v * model_at(a, i, a.col[p]);
        mb += v * a.wbar[a.col[p]];
      }
    } else {
      const float* x = a.X + g * a.ldx;
      for (int64_t c = lane; c < a.dim; c += 64) {
        const double v = x[c];
        mo += v * model_at(a, i, c);
        mb += v * a.wbar[c];
      }
    }
    mo = wave_sum_d(mo);
    mb = wave_sum_d(mb);
    if (lane == 0) {
      const double y = a.y[g];
      lown += loss_of(y * mo, a.loss);
      lbar += loss_of(y * mb, a.loss);
    }
  }
  for (int64_t c = c0 + threadIdx.x; c < c1; c += 256) {
    const double w = model_at(a, i, c);
    nrm += w * w;
  }
  lown = block_sum_d(lown, sh);
  lbar = block_sum_d(lbar, sh);
  nrm = block_sum_d(nrm, sh);
  if (threadIdx.x == 0) {
    double* q = a.part + base + 3 * (int64_t(i) * nch + ch);
    q[0] = lown;
    q[1] = lbar;
    q[2] = nrm;
  }
}

__global__ __launch_bounds__(256) void finish_kernel(MetricArgs a, int ncb, int64_t base, int nch) {
  __shared__ double sh[256];
  double cons = 0.0, msum = 0.0, wb2 = 0.0;
  for (int b = threadIdx.x; b < ncb; b += 256) {
    cons += a.part[2 * b];
    msum += a.part[2 * b + 1];
  }
  for (int64_t c = threadIdx.x; c < a.dim; c += 256) wb2 += a.wbar[c] * a.wbar[c];
  cons = block_sum_d(cons, sh);
  msum = block_sum_d(msum, sh);
  wb2 = block_sum_d(wb2, sh);
  double own = 0.0, bar = 0.0;
  if (a.S > 0) {
    for (int i = threadIdx.x; i < a.n; i += 256) {
      const double* q = a.part + base + 3 * int64_t(i) * nch;
      double lo = 0.0, lb = 0.0, nr = 0.0;
      for (int ch = 0; ch < nch; ++ch) {  // chunk order
        lo += q[3 * ch];
        lb += q[3 * ch + 1];
        nr += q[3 * ch + 2];
      }
      own += lo / double(a.S) + 0.5 * double(a.l2) * nr;
      bar += lb / double(a.S);
    }
  }
  own = block_sum_d(own, sh);
  bar = block_sum_d(bar, sh);
  if (threadIdx.x == 0) {
    const double nan = __longlong_as_double(0x7ff8000000000000ll);
    a.out[0] = a.S > 0 ? own / double(a.n) : nan;
    a.out[1] = a.S > 0 ? bar / double(a.n) + 0.5 * double(a.l2) * wb2 : nan;
    a.out[2] = sqrt(cons);
    a.out[3] = msum / double(a.dim);
  }
}

}  // namespace

hipError_t launch_metrics(const MetricArgs& a, hipStream_t s) {
  const int ncb = int(std::min<int64_t>((a.dim + 255) / 256, kColBlocksMax));
  const int64_t base = 2 * kColBlocksMax;
  const int nch = metric_chunks(a.n, a.S);
  hipLaunchKernelGGL(cols_kernel, dim3(ncb), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.S > 0) {
    hipLaunchKernelGGL(loss_kernel, dim3(uint32_t(a.n) * uint32_t(nch)), dim3(256), 0, s, a, base, nch);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(256), 0, s, a, ncb, base, nch);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Static scratch for callers that cannot allocate (asap_metrics_noalloc):
// w_bar, the partial sums and the four results live in this file-scope
// device array, one copy per GPU, kept until the process ends.  Host code
// never passes the array's name to a kernel or a copy: it uses the device
// address hipGetSymbolAddress returns for the current device.
// ---------------------------------------------------------------------------
namespace {

// n * metric_chunks(n, S) <= max(2048, n), so the partial sums of at most
// kStaticMetricMaxWorkers workers fit in kStaticPartMax bytes
constexpr size_t kStaticWbarBytes = size_t(kStaticMetricMaxDim) * 8;
constexpr size_t kStaticPartMax = (size_t(2 * kMetricColBlocks) + 3 * size_t(kStaticMetricMaxWorkers)) * 8;
constexpr size_t kStaticScratchBytes = kStaticWbarBytes + kStaticPartMax + 256;  // 8.4 MiB

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// device address of this GPU's copy of `scratch`, looked up once per device
// with that device current
hipError_t scratch_for_current_device(unsigned char** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = p;
  }
  *ptr = static_cast<unsigned char*>(g_scratch_dev[dev]);
  return hipSuccess;
}

}  // namespace

hipError_t metrics_static_scratch(MetricArgs a, hipStream_t s, double* out_host) {
  if (a.dim < 1 || a.dim > kStaticMetricMaxDim || a.n < 1 || a.n > kStaticMetricMaxWorkers)
    return hipErrorInvalidValue;
  if (metric_part_doubles(a.n, a.S) * 8 > kStaticPartMax) return hipErrorInvalidValue;
  unsigned char* base = nullptr;
  hipError_t e = scratch_for_current_device(&base);
  if (e != hipSuccess) return e;
  // every word the kernels read is written by them first in this call
  // (w_bar by the column pass, the partials by the column and loss passes,
  // the results by the final pass), so nothing needs clearing
  a.wbar = reinterpret_cast<double*>(base);
  a.part = reinterpret_cast<double*>(base + kStaticWbarBytes);
  a.out = reinterpret_cast<double*>(base + kStaticWbarBytes + kStaticPartMax);
  if ((e = launch_metrics(a, s)) != hipSuccess) return e;
  if ((e = hipMemcpyAsync(out_host, a.out, 4 * sizeof(double), hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

}  // namespace asap
