// kernels_mix.hip -- the stochastic reduce (Appendix A, update equation
// (A.2), second line): W'[i] = sum_{j in N_in(i)} P_ij W[j].
//
// The reduce is a low fan-in streaming product: every output element is
// deg+1 fused multiply-adds over rows that are each read by deg+1 outputs.
// It is bound by HBM bandwidth (arithmetic intensity < 1 flop/byte), so MFMA
// has no role here.  What matters is that every model byte crosses HBM
// once: a tile is one 1 KiB segment of 16 consecutive output rows, one wave
// per row segment with 16-byte loads, and the tiles of one column range are
// handed to a single XCD so that the deg+1 re-reads of a neighbour's segment
// hit that XCD's L2 instead of HBM.
//
// NOTIFY-ACK (Section 4) on one device: a prologue kernel (the WAIT) checks,
// one thread per worker, that every in-neighbour carries the tag "published
// in this round" in buffer e and records the verdict in row_ok; a row with a
// stale neighbour is not reduced and the mismatch is counted in the device
// error words.  Rows that are reduced get the next round's tag in buffer e^1.
#include "asap_launch.h"

namespace asap {
namespace {

constexpr int kSegFloats = 256;  // one wave x float4
constexpr int kTileRows = 16;
constexpr int kMixThreads = 256;

// Blocks are dealt round-robin to the 8 XCDs (blockIdx % 8).  Give XCD x the
// contiguous tile range [x*T/8, (x+1)*T/8) so that consecutive tiles of a
// column range stay in one L2.
__device__ __forceinline__ uint32_t xcd_tile(uint32_t bid, uint32_t total) {
  if (total % 8u) return bid;
  return (bid % 8u) * (total / 8u) + bid / 8u;
}

__device__ __forceinline__ void fma4(float4& acc, float w, const float4& x) {
  acc.x = fmaf(w, x.x, acc.x);
  acc.y = fmaf(w, x.y, acc.y);
  acc.z = fmaf(w, x.z, acc.z);
  acc.w = fmaf(w, x.w, acc.w);
}

__device__ __forceinline__ void store_tail(float* d, const float4& v, int64_t c, int64_t dim) {
  if (c + 4 <= dim) {
    *reinterpret_cast<float4*>(d) = v;
  } else {
    d[0] = v.x;
    if (c + 1 < dim) d[1] = v.y;
    if (c + 2 < dim) d[2] = v.z;
  }
}

__global__ __launch_bounds__(256) void epoch_check_kernel(MixArgs a) {
  const int r = int(blockIdx.x) * 256 + int(threadIdx.x);
  if (r >= a.n) return;
  int ok = 1;
  const int p0 = a.nbr_ptr[r], p1 = a.nbr_ptr[r + 1];
  for (int p = p0; p < p1; ++p) ok &= (a.tag_src[a.nbr_idx[p]] == a.expect);
  a.row_ok[r] = ok;
  if (!ok) {
    atomicAdd(&a.err[kErrEpochCount], 1);
    atomicMin(&a.err[kErrEpochWorker], r);
  }
}

__global__ __launch_bounds__(kMixThreads) void mix_kernel(MixArgs a, uint32_t nseg, uint32_t nrg) {
  const uint32_t tile = xcd_tile(blockIdx.x, nseg * nrg);
  const uint32_t seg = tile / nrg, rg = tile % nrg;
  const int row0 = int(rg) * kTileRows;
  const int row1 = min(row0 + kTileRows, a.n);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t c = int64_t(seg) * kSegFloats + lane * 4;
  for (int r = row0 + wave; r < row1; r += kMixThreads / 64) {
    if (!a.row_ok[r]) continue;
    if (c < a.dim) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      const int p0 = a.nbr_ptr[r], p1 = a.nbr_ptr[r + 1];
      for (int p = p0; p < p1; ++p) {
        const int j = a.nbr_idx[p];
        float wt = a.nbr_w[p];
        if (a.scale) wt *= a.scale[j];
        const float4 x = *reinterpret_cast<const float4*>(a.src + int64_t(j) * a.ld + c);
        fma4(acc, wt, x);
      }
      store_tail(a.dst + int64_t(r) * a.ld + c, acc, c, a.dim);
    }
    if (seg == 0 && lane == 0) a.tag_dst[r] = a.next;
  }
}

// Complete graph with uniform weights (all-reduce, Figure 2a): every output
// row is the same weighted column sum, so compute it once per column and
// broadcast it: n reads and n writes per column instead of n^2 reads.  The
// sum runs over j ascending with the same fused multiply-adds as mix_kernel,
// so both kernels produce identical bits on this graph.  On the complete
// graph one stale worker makes every row stale.
__global__ __launch_bounds__(64) void mean_kernel(MixArgs a, uint32_t nseg) {
  const uint32_t seg = xcd_tile(blockIdx.x, nseg);
  const int lane = threadIdx.x;
  int stale = 0;
  for (int j = lane; j < a.n; j += 64) stale |= !a.row_ok[j];
  if (__ballot(stale) != 0ull) return;
  const int64_t c = int64_t(seg) * kSegFloats + lane * 4;
  if (c < a.dim) {
    const float w0 = a.nbr_w[0];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
    for (int j = 0; j < a.n; ++j) {
      float wt = w0;
      if (a.scale) wt *= a.scale[j];
      const float4 x = *reinterpret_cast<const float4*>(a.src + int64_t(j) * a.ld + c);
      fma4(acc, wt, x);
    }
#pragma unroll 4
    for (int j = 0; j < a.n; ++j) store_tail(a.dst + int64_t(j) * a.ld + c, acc, c, a.dim);
  }
  if (seg == 0)
    for (int j = lane; j < a.n; j += 64) a.tag_dst[j] = a.next;
}

template <class T>
__global__ void fill_kernel(T* p, int64_t count, T value) {
  for (int64_t k = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; k < count;
       k += int64_t(gridDim.x) * blockDim.x)
    p[k] = value;
}

template <class T>
hipError_t fill(T* p, int64_t count, T value, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_kernel<T>, dim3(uint32_t(blocks)), dim3(256), 0, s, p, count, value);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_epoch_check(const MixArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(epoch_check_kernel, dim3(uint32_t((a.n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mix(const MixArgs& a, hipStream_t s) {
  const uint32_t nseg = uint32_t((a.dim + kSegFloats - 1) / kSegFloats);
  const uint32_t nrg = uint32_t((a.n + kTileRows - 1) / kTileRows);
  const uint64_t total = uint64_t(nseg) * nrg;
  if (total >= (1ull << 31)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mix_kernel, dim3(uint32_t(total)), dim3(kMixThreads), 0, s, a, nseg, nrg);
  return hipGetLastError();
}

hipError_t launch_mean(const MixArgs& a, hipStream_t s) {
  const uint32_t nseg = uint32_t((a.dim + kSegFloats - 1) / kSegFloats);
  hipLaunchKernelGGL(mean_kernel, dim3(nseg), dim3(64), 0, s, a, nseg);
  return hipGetLastError();
}

hipError_t launch_fill_i64(int64_t* p, int64_t count, int64_t value, hipStream_t s) {
  return fill<int64_t>(p, count, value, s);
}
hipError_t launch_fill_f32(float* p, int64_t count, float value, hipStream_t s) {
  return fill<float>(p, count, value, s);
}
hipError_t launch_fill_i32(int32_t* p, int64_t count, int32_t value, hipStream_t s) {
  return fill<int32_t>(p, count, value, s);
}

}  // namespace asap
