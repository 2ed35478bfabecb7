// kernels_dense.hip -- local SGD pass on dense shards for wide models
// (Appendix A, update (A.2), first line; Section 5: each replica trains on its
// own data partition), dim in (1024, 8192].
//
// A pass is a chain of minibatch steps, and a step reads B rows of 4*dim
// bytes: HBM-bound, no dense contraction (batched GEMV + rank-B' update), so
// MFMA is not used.  One workgroup per worker would leave most of the chip
// idle when workers are few, so K workgroups share a worker: each holds the
// whole model slice in registers, takes a contiguous K-th of every
// minibatch, and the K partial gradients are exchanged once per step through
// the workspace (written, counted in, read back and summed in member order).
// The launch is cooperative, so every member is resident and the rendezvous
// cannot wait on a workgroup that has not started; the wait is bounded
// anyway and reports a timeout instead of spinning for ever.
//
// Inside a workgroup (512 threads), thread t owns the float4 columns
// 4(t + 512 q), q < CPQ.  Rows go SR at a time ("sub-batch"); the next sub-batch's rows are
// loaded while the current one is reduced, and one LDS barrier per sub-batch
// suffices (per-wave partial margins are double-buffered in LDS).
//
// Determinism: a thread's partial dot is an fp32 sum of its 4*CPQ products;
// partials are summed in fp64 by a fixed lane tree, then over the rows of a
// wave and over waves in index order; the gradient is accumulated in fp64 in
// batch order and the K partials are added in member order.  Every member
// applies the same update, so the K copies of the model stay identical.
#include <cmath>

#include "asap_launch.h"

namespace asap {
namespace {

constexpr int kThreads = 512;  // 8 waves: 256 registers per lane for the row prefetch
constexpr int kWaves = kThreads / 64;
constexpr int kMaxBatch = 512;  // minibatch limit of asap_sgd_params

__device__ __forceinline__ double loss_coef(double m, double y, int loss) {
  const double ym = y * m;
  if (loss == 1) return ym < 1.0 ? -y : 0.0;  // hinge
  return -y / (1.0 + exp(ym));                // logistic
}

__device__ __forceinline__ double step_size(int lr_kind, float lr0, int64_t t) {
  return lr_kind == 0 ? double(lr0) : double(lr0) / sqrt(double(t));
}

// sum over the 16 lanes of a DPP row; every lane of the row gets the same
// bits (the four stages pair lanes symmetrically and fp addition commutes)
__device__ __forceinline__ double row16_sum(double v) {
#define ASAP_DPP_STAGE(ctrl)                                                                  \
  {                                                                                           \
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), ctrl, 0xF, 0xF, false); \
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), ctrl, 0xF, 0xF, false); \
    v += __hiloint2double(hi, lo);                                                            \
  }
  ASAP_DPP_STAGE(0xB1)   // quad_perm [1,0,3,2]
  ASAP_DPP_STAGE(0x4E)   // quad_perm [2,3,0,1]
  ASAP_DPP_STAGE(0x141)  // row_half_mirror
  ASAP_DPP_STAGE(0x140)  // row_mirror
#undef ASAP_DPP_STAGE
  return v;
}

__device__ __forceinline__ double lane_value(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
  return __hiloint2double(hi, lo);
}

// wave total, uniform: rows summed as ((r0 + r1) + r2) + r3
__device__ __forceinline__ double wave_total(double v) {
  v = row16_sum(v);
  return ((lane_value(v, 0) + lane_value(v, 16)) + lane_value(v, 32)) + lane_value(v, 48);
}

__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float dot4(const float4& a, const float4& b) {
  return fmaf(a.w, b.w, fmaf(a.z, b.z, fmaf(a.y, b.y, a.x * b.x)));
}

template <int CPQ, int SR>
__global__ __launch_bounds__(kThreads) void sgd_dense_wide_kernel(SgdArgs a, DenseSync ds) {
  __shared__ double red[2][kWaves][SR];
  __shared__ int ridx[2][kMaxBatch];  // this member's row indices of steps t, t+1 (slot t & 1)
  __shared__ int abort_flag;
  const int K = ds.K;
  // members of one worker on one XCD when the grid allows it (blocks are
  // dealt to the 8 XCDs round-robin), so the exchange stays in one L2
  int i, k;
  {
    const int bid = int(blockIdx.x), nb = int(gridDim.x);
    if (nb % 8 == 0 && a.n % 8 == 0) {
      const int j = bid / 8;
      i = (bid % 8) * (a.n / 8) + j / K;
      k = j % K;
    } else {
      i = bid / K;
      k = bid % K;
    }
  }
  const int tid = int(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  if (tid == 0) abort_flag = 0;
  float* wrow = a.models + int64_t(i) * a.ld;
  const float* Xi = a.X + int64_t(i) * a.S * a.ldx;
  const float* yi = a.y + int64_t(i) * a.S;
  const int32_t* si = a.sched + int64_t(i) * a.S;

  // model slice; entries past dim are 0 and stay 0 (their rows entries are 0)
  float4 w[CPQ];
#pragma unroll
  for (int q = 0; q < CPQ; ++q) {
    const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c + 4 <= a.dim) {
      v = *reinterpret_cast<const float4*>(wrow + c);
    } else if (c < a.dim) {
      v.x = wrow[c];
      if (c + 1 < a.dim) v.y = wrow[c + 1];
      if (c + 2 < a.dim) v.z = wrow[c + 2];
    }
    w[q] = v;
  }

  const int B = a.batch, S = int(a.S);  // S < 2^31 (checked at bind)
  const int KS = (S + B - 1) / B;
  // valid components of the thread's last float4 of each q (entries of X
  // past dim are never used)
  int nv[CPQ];
#pragma unroll
  for (int q = 0; q < CPQ; ++q) {
    const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
    nv[q] = int(max<int64_t>(0, min<int64_t>(4, a.dim - c)));
  }

  // Position of a sub-batch: step t, first sample sb, this member's samples
  // [lo, hi) of step t.  Member k takes [b0 + Bp*k/K, b0 + Bp*(k+1)/K).
  struct Pos {
    int t, sb, lo, hi;
  };
  auto share = [&](int t, int& lo_, int& hi_) {
    const int b0 = t * B, Bp = min(B, S - b0);
    lo_ = b0 + int((int64_t(Bp) * k) / K);
    hi_ = b0 + int((int64_t(Bp) * (k + 1)) / K);
  };
  auto settle = [&](Pos p) {  // move past steps in which this member has no samples
    while (p.t < KS && p.sb >= p.hi) {
      ++p.t;
      if (p.t < KS) {
        share(p.t, p.lo, p.hi);
        p.sb = p.lo;
      }
    }
    return p;
  };
  // Row indices of a step are staged in LDS two steps ahead: thread j <
  // (samples of step t) holds index j of step t in pi between issuing its
  // load and writing it to slot t & 1.
  int pi = 0;
  auto fetch = [&](int t) {
    if (t >= KS) return;
    int lo_, hi_;
    share(t, lo_, hi_);
    if (tid < hi_ - lo_) pi = si[lo_ + tid];
  };
  auto stage = [&](int t) {
    if (t >= KS) return;
    int lo_, hi_;
    share(t, lo_, hi_);
    if (tid < hi_ - lo_) ridx[t & 1][tid] = pi;
  };

  // load the SR rows of sub-batch p (rows past p.hi are 0); lane s < SR also
  // loads row s's label
  auto load = [&](float4 (&x)[SR][CPQ], float& yl, Pos p) {
    const int base = p.sb - p.lo, slot = p.t & 1, cnt = p.hi - p.sb;
#pragma unroll
    for (int s = 0; s < SR; ++s) {
      const bool ok = s < cnt;
      const int r = ok ? __builtin_amdgcn_readfirstlane(ridx[slot][base + s]) : 0;
      const float* row = Xi + int64_t(r) * a.ldx;
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
        float4 v = (ok && nv[q] > 0) ? *reinterpret_cast<const float4*>(row + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        if (nv[q] < 4) {
          if (nv[q] <= 1) v.y = 0.f;
          if (nv[q] <= 2) v.z = 0.f;
          v.w = 0.f;
        }
        x[s][q] = v;
      }
    }
    yl = lane < min(cnt, SR) ? yi[ridx[slot][base + lane]] : 0.f;
  };

  double g[CPQ][4];
#pragma unroll
  for (int q = 0; q < CPQ; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) g[q][e] = 0.0;
  int par = 0;

  // margins, coefficients and gradient of the sub-batch held in xc
  auto process = [&](float4 (&xc)[SR][CPQ], float yl, Pos p) {
    double mine = 0.0;  // lane s < SR: this wave's part of row s's margin
#pragma unroll
    for (int s = 0; s < SR; ++s) {
      float d = 0.f;
#pragma unroll
      for (int q = 0; q < CPQ; ++q) d += dot4(w[q], xc[s][q]);
      const double t = wave_total(double(d));
      mine = lane == s ? t : mine;
    }
    if (lane < SR) red[par][wave][lane] = mine;
    lds_barrier();
    double cf = 0.0;
    if (lane < SR && lane < p.hi - p.sb) {
      double m = 0.0;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) m += red[par][v][lane];
      cf = loss_coef(m, double(yl), a.loss);
    }
    par ^= 1;
#pragma unroll
    for (int s = 0; s < SR; ++s) {
      const double c = lane_value(cf, s);
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        g[q][0] = fma(c, double(xc[s][q].x), g[q][0]);
        g[q][1] = fma(c, double(xc[s][q].y), g[q][1]);
        g[q][2] = fma(c, double(xc[s][q].z), g[q][2]);
        g[q][3] = fma(c, double(xc[s][q].w), g[q][3]);
      }
    }
  };

  // end of step t: exchange (K > 1) and update; false when the rendezvous
  // timed out
  auto finish_step = [&](int t) -> bool {
    const int Bp = min(B, S - t * B);
    if (K > 1) {
      double* mine = ds.part + ((int64_t(i) * K + k) * 2 + (t & 1)) * ds.ldp;
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
        *reinterpret_cast<double2*>(mine + c) = make_double2(g[q][0], g[q][1]);
        *reinterpret_cast<double2*>(mine + c + 2) = make_double2(g[q][2], g[q][3]);
      }
      __threadfence();
      __syncthreads();
      if (tid == 0) {
        __hip_atomic_fetch_add(ds.count + i, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t target = uint32_t(K) * uint32_t(t + 1);
        uint32_t spins = 0;
        while (__hip_atomic_load(ds.count + i, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
          if (++spins > ds.spin_limit) {
            abort_flag = 1;
            __hip_atomic_fetch_add(ds.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      }
      __syncthreads();
      if (abort_flag) return false;
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
      for (int q = 0; q < CPQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) g[q][e] = 0.0;
      for (int m = 0; m < K; ++m) {
        const double* pm = ds.part + ((int64_t(i) * K + m) * 2 + (t & 1)) * ds.ldp;
#pragma unroll
        for (int q = 0; q < CPQ; ++q) {
          const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
          const double2 u = *reinterpret_cast<const double2*>(pm + c);
          const double2 v = *reinterpret_cast<const double2*>(pm + c + 2);
          g[q][0] += u.x; g[q][1] += u.y; g[q][2] += v.x; g[q][3] += v.y;
        }
      }
    }
    const double eta = step_size(a.lr_kind, a.lr0, a.round * KS + t + 1);
    const double inv = 1.0 / double(Bp), l2 = double(a.l2);
#pragma unroll
    for (int q = 0; q < CPQ; ++q) {
      w[q].x = float(double(w[q].x) - eta * fma(g[q][0], inv, l2 * double(w[q].x)));
      w[q].y = float(double(w[q].y) - eta * fma(g[q][1], inv, l2 * double(w[q].y)));
      w[q].z = float(double(w[q].z) - eta * fma(g[q][2], inv, l2 * double(w[q].z)));
      w[q].w = float(double(w[q].w) - eta * fma(g[q][3], inv, l2 * double(w[q].w)));
#pragma unroll
      for (int e = 0; e < 4; ++e) g[q][e] = 0.0;
    }
    // every wave has passed a barrier since its last read of slot t & 1
    stage(t + 2);
    fetch(t + 3);
    return true;
  };

  // Rows of the next sub-batch load into xb while xa is processed; the copy
  // xa = xb then waits for loads that had the whole sub-batch to land.
  // Every member finishes every step (exchange + update), also the steps in
  // which it has no samples.
  float4 xa[SR][CPQ], xb[SR][CPQ];
  float ya = 0.f, yb = 0.f;
  bool ok = true;
  int done = 0;  // steps finished
  fetch(0);
  stage(0);
  fetch(1);
  stage(1);
  fetch(2);
  __syncthreads();
  Pos cur{0, 0, 0, 0};
  share(0, cur.lo, cur.hi);
  cur.sb = cur.lo;
  cur = settle(cur);
  if (cur.t < KS) load(xa, ya, cur);
  for (;;) {
    while (ok && done < min(cur.t, KS)) ok = finish_step(done++);
    if (!ok || cur.t >= KS) break;
    const Pos nx = settle(Pos{cur.t, cur.sb + SR, cur.lo, cur.hi});
    if (nx.t < KS) load(xb, yb, nx);
    process(xa, ya, cur);
    cur = nx;
#pragma unroll
    for (int s2 = 0; s2 < SR; ++s2)
#pragma unroll
      for (int q = 0; q < CPQ; ++q) xa[s2][q] = xb[s2][q];
    ya = yb;
  }

  if (k == 0) {
#pragma unroll
    for (int q = 0; q < CPQ; ++q) {
      const int64_t c = 4 * (int64_t(tid) + int64_t(kThreads) * q);
      if (c + 4 <= a.dim) {
        *reinterpret_cast<float4*>(wrow + c) = w[q];
      } else if (c < a.dim) {
        wrow[c] = w[q].x;
        if (c + 1 < a.dim) wrow[c + 1] = w[q].y;
        if (c + 2 < a.dim) wrow[c + 2] = w[q].z;
      }
    }
    if (tid == 0) {
      a.scale[i] = 1.0f;
      a.tag[i] = a.tag_value;
    }
  }
}

template <int CPQ, int SR>
hipError_t launch_wide(const SgdArgs& a, const DenseSync& ds, hipStream_t s) {
  const dim3 grid{uint32_t(a.n * ds.K)}, block{uint32_t(kThreads)};
  if (ds.K == 1) {
    hipLaunchKernelGGL((sgd_dense_wide_kernel<CPQ, SR>), grid, block, 0, s, a, ds);
    return hipGetLastError();
  }
  SgdArgs aa = a;
  DenseSync dd = ds;
  void* args[] = {&aa, &dd};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&sgd_dense_wide_kernel<CPQ, SR>), grid, block,
                                    args, 0, s);
}

}  // namespace

int dense_wide_cpq(int64_t dim) {
  if (dim <= 1024 || dim > 8192) return 0;
  return dim <= 2048 ? 1 : dim <= 4096 ? 2 : 4;
}

int dense_wide_max_members(const SgdArgs& a, int n_cu) {
  int per = 0;
  switch (dense_wide_cpq(a.dim)) {
    case 1: hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<1, 8>, kThreads, 0); break;
    case 2: hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<2, 8>, kThreads, 0); break;
    case 4: hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<4, 2>, kThreads, 0); break;
    default: return 1;
  }
  return std::max(1, per) * n_cu;
}

hipError_t launch_sgd_dense_wide(const SgdArgs& a, const DenseSync& ds, hipStream_t s) {
  switch (dense_wide_cpq(a.dim)) {
    case 1: return launch_wide<1, 8>(a, ds, s);
    case 2: return launch_wide<2, 8>(a, ds, s);
    case 4: return launch_wide<4, 2>(a, ds, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace asap
