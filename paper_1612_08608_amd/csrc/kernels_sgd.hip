// kernels_sgd.hip -- the sample schedule, the local half-step of (A.2)
// (Appendix A) on dense shards, and the bind-time scan of CSR shards.
//
// Every worker runs one pass of minibatch SGD over its own shard (Section 5)
// in the order of this round's sample schedule.  One workgroup owns one
// worker for the whole pass, because the steps of a pass form a dependency
// chain (step k+1's margins read step k's model) and a workgroup barrier is
// the cheapest way to order them.  The work inside a step is a batched GEMV
// with a rank-B' update: HBM- and latency-bound, no dense contraction, so
// MFMA is not used.
//
// Determinism: margins reduce across lanes with a fixed butterfly and across
// waves in wave order; the gradient sums over the batch in batch order.
#include <cmath>

#include "asap_common.h"
#include "asap_launch.h"
#include "rounds_device.h"

namespace asap {
namespace {

// d loss(y m) / d m: logistic -y / (1 + e^{y m}); hinge -y if y m < 1 else 0.
// Margins are accumulated in fp64 (a 4096-term fp32 dot product with a
// wide dynamic range loses more than the 1e-5 the models are held to), and
// the coefficient -- including the hinge decision -- is taken in fp64.
__device__ __forceinline__ double loss_coef(double m, double y, int loss) {
  const double ym = y * m;
  if (loss == ASAP_LOSS_HINGE) return ym < 1.0 ? -y : 0.0;
  return -y / (1.0 + exp(ym));
}

__device__ __forceinline__ double step_size(int lr_kind, float lr0, int64_t t) {
  return lr_kind == 0 ? double(lr0) : double(lr0) / sqrt(double(t));
}

// N independent butterfly sums over the wave, level by level, so that the N
// shuffles of a level are in flight together; every lane ends with lane 0's
// association order.
template <int N>
__device__ __forceinline__ void wave_sums(double (&v)[N]) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    double o[N];
#pragma unroll
    for (int s = 0; s < N; ++s) o[s] = __shfl_xor(v[s], off, 64);
#pragma unroll
    for (int s = 0; s < N; ++s) v[s] += o[s];
  }
#pragma unroll
  for (int s = 0; s < N; ++s) v[s] = __shfl(v[s], 0, 64);
}

// ----------------------------------------------------------------------------
// schedule
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void schedule_kernel(uint64_t seed, int64_t round, int64_t S,
                                                       uint32_t blocks_per_worker, int32_t* out) {
  const int worker = int(blockIdx.x / blocks_per_worker);
  const Perm p = perm_make(seed, worker, round, uint32_t(S));
  const int64_t pos = int64_t(blockIdx.x % blocks_per_worker) * 256 + threadIdx.x;
  if (pos < S) out[int64_t(worker) * S + pos] = int32_t(perm_at(p, uint32_t(pos)));
}

// ----------------------------------------------------------------------------
// dense SGD: thread t owns columns t, t+T, ..., t+(CPT-1)T and keeps that
// slice of w in registers for the whole pass.  Samples of a step are taken
// SB at a time: each thread loads its columns of the SB rows, the SB margins
// are reduced over the block, and the rows (still in registers) are folded
// into the thread's gradient slice.
// ----------------------------------------------------------------------------
// samples per block reduction: keep SB * CPT row values within 32 registers
template <int CPT>
constexpr int dense_sb() { return CPT >= 16 ? 2 : CPT >= 8 ? 4 : 8; }

template <int CPT>
__device__ __forceinline__ void dense_pass(const SgdArgs& a, int i) {
  constexpr int SB = dense_sb<CPT>();
  __shared__ double part[16 * SB];
  const int T = blockDim.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = T >> 6;
  float* wrow = a.models + int64_t(i) * a.ld;
  const float* Xi = a.X + int64_t(i) * a.S * a.ldx;
  const float* yi = a.y + int64_t(i) * a.S;
  // sample order of the pass: every lane evaluates the keyed permutation at
  // one position of the step (64 at a time) and each sub-batch takes its row
  // indices from those lanes, so no index is read from memory on the chain
  const Perm P = perm_make(a.seed, i, a.round, uint32_t(a.S));
  float wr[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int64_t c = tid + int64_t(q) * T;
    wr[q] = c < a.dim ? wrow[c] : 0.f;
  }
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  for (int64_t k = a.k0; k < a.k1; ++k) {
    const int64_t b0 = k * a.batch;
    const int Bp = int(min(int64_t(a.batch), a.S - b0));
    const double eta = step_size(a.lr_kind, a.lr0, a.round * K + k + 1);
    double gr[CPT];
#pragma unroll
    for (int q = 0; q < CPT; ++q) gr[q] = 0.0;
    int rows = 0;      // lane l: the sample at position b0 + (sb & ~63) + l ...
    float labels = 0.f;  // ... and its label, loaded with the rows' first loads
    for (int sb = 0; sb < Bp; sb += SB) {
      if ((sb & 63) == 0) {
        const int u = sb + lane;
        rows = u < Bp ? int(perm_at(P, uint32_t(b0 + u))) : 0;
        labels = u < Bp ? yi[rows] : 0.f;
      }
      float xr[SB][CPT];
      double d[SB];
      int rix[SB];
#pragma unroll
      for (int s = 0; s < SB; ++s) rix[s] = __builtin_amdgcn_readlane(rows, (sb & 63) + s);  // SB divides 64
      // every load is issued (out-of-range ones read row 0 / column 0 and
      // are replaced by 0), so the sub-batch's loads are in flight together
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const bool ok = sb + s < Bp;
        const float* row = Xi + int64_t(ok ? rix[s] : 0) * a.ldx;
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
          const int64_t c = tid + int64_t(q) * T;
          const bool in = ok && c < a.dim;
          const float v = row[in ? c : 0];
          xr[s][q] = in ? v : 0.f;
        }
      }
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        d[s] = 0.0;
#pragma unroll
        for (int q = 0; q < CPT; ++q) d[s] = fma(double(wr[q]), double(xr[s][q]), d[s]);
      }
      // margins: butterfly within the wave, then waves in order
      wave_sums<SB>(d);
      if (lane == 0) {
#pragma unroll
        for (int s = 0; s < SB; ++s) part[wave * SB + s] = d[s];
      }
      __syncthreads();
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        double m = 0.0;
        for (int w = 0; w < nw; ++w) m += part[w * SB + s];
        d[s] = m;
      }
      __syncthreads();
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        if (sb + s < Bp) {
          const float ys = __builtin_bit_cast(
              float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, labels), (sb & 63) + s));
          const double cf = loss_coef(d[s], double(ys), a.loss);
#pragma unroll
          for (int q = 0; q < CPT; ++q) gr[q] = fma(cf, double(xr[s][q]), gr[q]);
        }
      }
    }
    const double inv = 1.0 / double(Bp);
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      const double w = wr[q];
      wr[q] = float(w - eta * fma(gr[q], inv, double(a.l2) * w));
    }
  }
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int64_t c = tid + int64_t(q) * T;
    if (c < a.dim) wrow[c] = wr[q];
  }
  if (tid == 0) {
    a.scale[i] = 1.0f;
    if (a.tag) a.tag[i] = a.tag_value;
  }
}

template <int CPT>
__global__ __launch_bounds__(1024) void sgd_dense_kernel(SgdArgs a) {
  dense_pass<CPT>(a, int(blockIdx.x));
}

// Several rounds in one launch (rounds_device.h): one workgroup per worker
// runs its passes and reduces its own row.
template <int CPT>
__global__ __launch_bounds__(1024) void rounds_dense_kernel(SgdArgs a, RoundsArgs ra) {
  const int i = int(blockIdx.x);
  rounds::drive(
      a, ra, i, 0, 1, [](int64_t) {},  // the pass evaluates its sample order itself
      [&](const SgdArgs& ar) {
        dense_pass<CPT>(ar, i);
        return true;
      });
}

// ----------------------------------------------------------------------------
// bind-time scan of the CSR shards
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void csr_scan_kernel(const int64_t* row_ptr, const int32_t* col,
                                                       const float* val, const float* y, int64_t S,
                                                       int64_t dim, float* vmax, int64_t* out) {
  const int i = blockIdx.x;
  __shared__ float smax[256];
  __shared__ int slen[256];
  float m = 0.f;
  int maxlen = 0;
  unsigned long long badcol = 0, bady = 0, badorder = 0, badptr = 0;
  if (i == 0 && threadIdx.x == 0 && row_ptr[0] != 0) ++badptr;
  for (int64_t r = threadIdx.x; r < S; r += 256) {
    const int64_t g = int64_t(i) * S + r;
    const int64_t p0 = row_ptr[g], p1 = row_ptr[g + 1];
    if (p1 < p0 || p0 < 0) {  // entries are only read from well-formed rows
      ++badptr;
      continue;
    }
    maxlen = max(maxlen, int(min<int64_t>(p1 - p0, 1 << 30)));
    const float yy = y[g];
    bady += (yy != 1.0f && yy != -1.0f);
    int prev = -1;
    for (int64_t p = p0; p < p1; ++p) {
      const int c = col[p];
      badcol += (c < 0 || c >= dim);
      badorder += (c <= prev);
      prev = c;
      m = fmaxf(m, fabsf(val[p]));
    }
  }
  smax[threadIdx.x] = m;
  slen[threadIdx.x] = maxlen;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      smax[threadIdx.x] = fmaxf(smax[threadIdx.x], smax[threadIdx.x + o]);
      slen[threadIdx.x] = max(slen[threadIdx.x], slen[threadIdx.x + o]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    vmax[i] = smax[0];
    atomicMax(reinterpret_cast<unsigned long long*>(&out[0]), static_cast<unsigned long long>(slen[0]));
    const long long seg = row_ptr[int64_t(i + 1) * S] - row_ptr[int64_t(i) * S];
    atomicMax(reinterpret_cast<unsigned long long*>(&out[5]), static_cast<unsigned long long>(seg < 0 ? 0 : seg));
  }
  if (badcol) atomicAdd(reinterpret_cast<unsigned long long*>(&out[1]), badcol);
  if (bady) atomicAdd(reinterpret_cast<unsigned long long*>(&out[2]), bady);
  if (badorder) atomicAdd(reinterpret_cast<unsigned long long*>(&out[3]), badorder);
  if (badptr) atomicAdd(reinterpret_cast<unsigned long long*>(&out[4]), badptr);
}

}  // namespace

hipError_t launch_schedule(uint64_t seed, int64_t round, int32_t n, int64_t S, int32_t* out,
                           hipStream_t s) {
  if (S <= 0 || n <= 0) return hipSuccess;
  const uint64_t bx = uint64_t((S + 255) / 256);
  if (bx * uint64_t(n) >= (1ull << 31)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(schedule_kernel, dim3(uint32_t(bx * uint64_t(n))), dim3(256), 0, s, seed, round, S,
                     uint32_t(bx), out);
  return hipGetLastError();
}

hipError_t launch_sgd_dense(const SgdArgs& a, hipStream_t s) {
  int T = int(std::min<int64_t>(1024, (a.dim + 63) / 64 * 64));
  const int64_t need = (a.dim + T - 1) / T;
  const dim3 grid{uint32_t(a.n)}, block{uint32_t(T)};
  if (need <= 1)
    hipLaunchKernelGGL(sgd_dense_kernel<1>, grid, block, 0, s, a);
  else if (need <= 2)
    hipLaunchKernelGGL(sgd_dense_kernel<2>, grid, block, 0, s, a);
  else if (need <= 4)
    hipLaunchKernelGGL(sgd_dense_kernel<4>, grid, block, 0, s, a);
  else if (need <= 8)
    hipLaunchKernelGGL(sgd_dense_kernel<8>, grid, block, 0, s, a);
  else if (need <= 16)
    hipLaunchKernelGGL(sgd_dense_kernel<16>, grid, block, 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

namespace {
template <int CPT>
hipError_t launch_rounds_dense_t(const SgdArgs& a, const RoundsArgs& ra, int T, int n_cu, hipStream_t s) {
  const void* fn = reinterpret_cast<const void*>(&rounds_dense_kernel<CPT>);
  int per = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, rounds_dense_kernel<CPT>, T, 0);
  if (e != hipSuccess) return e;
  if (int64_t(per) * n_cu < a.n) return hipErrorCooperativeLaunchTooLarge;
  SgdArgs aa = a;
  RoundsArgs rr = ra;
  void* args[] = {&aa, &rr};
  return hipLaunchCooperativeKernel(fn, dim3(uint32_t(a.n)), dim3(uint32_t(T)), args, 0, s);
}
}  // namespace

hipError_t launch_rounds_dense(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s) {
  const int T = int(std::min<int64_t>(1024, (a.dim + 63) / 64 * 64));
  const int64_t need = (a.dim + T - 1) / T;
  if (need <= 1) return launch_rounds_dense_t<1>(a, ra, T, n_cu, s);
  if (need <= 2) return launch_rounds_dense_t<2>(a, ra, T, n_cu, s);
  if (need <= 4) return launch_rounds_dense_t<4>(a, ra, T, n_cu, s);
  if (need <= 8) return launch_rounds_dense_t<8>(a, ra, T, n_cu, s);
  if (need <= 16) return launch_rounds_dense_t<16>(a, ra, T, n_cu, s);
  return hipErrorInvalidValue;
}

hipError_t launch_csr_scan(const int64_t* row_ptr, const int32_t* col, const float* val,
                           const float* y, int32_t n, int64_t S, int64_t dim, float* vmax,
                           int64_t* out, hipStream_t s) {
  hipLaunchKernelGGL(csr_scan_kernel, dim3(uint32_t(n)), dim3(256), 0, s, row_ptr, col, val, y, S, dim,
                     vmax, out);
  return hipGetLastError();
}

}  // namespace asap
