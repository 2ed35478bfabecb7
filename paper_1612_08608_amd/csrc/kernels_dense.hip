// kernels_dense.hip -- local SGD pass on dense shards for wide models
// (Appendix A, update (A.2), first line; Section 5: each replica trains on its
// own data partition), dim in (1024, 8192].
//
// A pass is a chain of minibatch steps, and a step reads B rows of 4*dim
// bytes: HBM-bound, no dense contraction (batched GEMV + rank-B' update), so
// MFMA is not used.  One workgroup per worker would leave most of the chip
// idle when workers are few, so K workgroups share a worker: each holds the
// whole model slice in registers, takes a contiguous K-th of every
// minibatch, and once per step every member publishes its partial gradient
// (rounded to fp32) in the workspace and sums all K of them in fp64 in
// member order, so every member gets the same sum whatever the order they
// arrive in.  Members of a worker are placed on one XCD when the grid
// allows (workgroups are dealt to the XCDs round-robin; each member checks
// the XCD it runs on), and then meet in that XCD's L2: plain 16-byte stores
// (the CU's L1 writes through to the L2) and device-scope loads (a load of
// narrower scope may be served by a line the reader's L1 kept from two
// steps earlier).  Device-scope stores, which go past the L2, made the
// exchange cost a third of the pass; integer atomics on shared lines and a
// reduce-scatter with a second meeting were slower still.
// The launch is cooperative, so every member is resident and the rendezvous
// cannot wait on a workgroup that has not started; the wait is bounded
// anyway and reports a timeout instead of spinning for ever.
//
// Inside a workgroup (512 threads), thread t owns the float4 columns
// 4(t + 512 q), q < CPQ.  Rows go SR at a time ("sub-batch"); the next sub-batch's rows are
// loaded while the current one is reduced, and one LDS barrier per sub-batch
// suffices (per-wave partial margins are double-buffered in LDS).
//
// Determinism: a thread's partial dot is an fp64 sum of its 4*CPQ products;
// partials are summed in fp64 by a fixed transposed butterfly over each
// 16-lane row, then over rows and waves in index order; the gradient is accumulated in fp64 in
// batch order and the K partials are added in member order.  Every member
// applies the same update, so the K copies of the model stay identical.
#include <cmath>

#include "asap_launch.h"
#include "rounds_device.h"

namespace asap {
namespace {

// A feature row is read once per pass: non-temporal 16-byte loads (32
// workers x 4096 features x 65536 samples: 7.62 -> 7.13 ms per pass).
typedef float stream4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld_stream(const float* p) {
  const stream4 x = __builtin_nontemporal_load(reinterpret_cast<const stream4*>(p));
  return make_float4(x.x, x.y, x.z, x.w);
}

constexpr int kThreads = 512;  // 8 waves: 256 registers per lane for the row prefetch
constexpr int kWaves = kThreads / 64;
constexpr int kMaxBatch = 512;  // minibatch limit of asap_sgd_params

// d loss(y m) / d m from an fp64 margin: the hinge decision y m < 1 is taken
// in fp64; the logistic factor 1 / (1 + e^{y m}) needs only fp32 accuracy.
__device__ __forceinline__ float loss_coef(double m, float y, int loss) {
  const double ym = double(y) * m;
  if (loss == ASAP_LOSS_HINGE) return ym < 1.0 ? -y : 0.f;
  return -y / (1.f + expf(float(ym)));  // logistic
}

__device__ __forceinline__ double step_size(int lr_kind, float lr0, int64_t t) {
  return lr_kind == 0 ? double(lr0) : double(lr0) / sqrt(double(t));
}

template <int CTRL>
__device__ __forceinline__ int dpp(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}

template <int S>
__device__ __forceinline__ double xor_lane(double v) {
  int lo = __double2loint(v), hi = __double2hiint(v);
  if constexpr (S == 1) {
    lo = dpp<0xB1>(lo); hi = dpp<0xB1>(hi);    // quad_perm [1,0,3,2]
  } else if constexpr (S == 2) {
    lo = dpp<0x4E>(lo); hi = dpp<0x4E>(hi);    // quad_perm [2,3,0,1]
  } else if constexpr (S == 4) {               // i -> i ^ 7 in 8 lanes, then i ^ 3
    lo = dpp<0x1B>(dpp<0x141>(lo)); hi = dpp<0x1B>(dpp<0x141>(hi));
  } else {
    static_assert(S == 8, "xor_lane: S in {1, 2, 4, 8}");
    lo = dpp<0x128>(lo); hi = dpp<0x128>(hi);  // row_ror:8
  }
  return __hiloint2double(hi, lo);
}

// One butterfly stage of a transposed reduction: a lane keeps the half of
// its N values whose index bit matches its lane bit S, sends the other half
// to lane ^ S, and adds what it receives.  Value j of the result is input
// value 2j + (lane & S ? 1 : 0) (counting the bits used so far).
template <int S, int N>
__device__ __forceinline__ void halve(double (&d)[16], int lane) {
  const bool hi = lane & S;
#pragma unroll
  for (int j = 0; j < N / 2; ++j) {
    const double keep = hi ? d[2 * j + 1] : d[2 * j];
    const double send = hi ? d[2 * j] : d[2 * j + 1];
    d[j] = keep + xor_lane<S>(send);
  }
}

// SR values per lane -> lane l holds the sum over its 16-lane DPP row of
// value (l mod SR); each sum is formed on fixed lanes in a fixed order.
template <int SR>
__device__ __forceinline__ double row_reduce(double (&d)[16], int lane) {
  if constexpr (SR >= 2) halve<1, SR>(d, lane); else d[0] += xor_lane<1>(d[0]);
  if constexpr (SR >= 4) halve<2, SR / 2>(d, lane); else d[0] += xor_lane<2>(d[0]);
  if constexpr (SR >= 8) halve<4, SR / 4>(d, lane); else d[0] += xor_lane<4>(d[0]);
  if constexpr (SR >= 16) halve<8, SR / 8>(d, lane); else d[0] += xor_lane<8>(d[0]);
  return d[0];
}


__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), 0x00020000);
}

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Worker i and member k of this workgroup: the members of one worker on one
// XCD when the grid allows it (blocks are dealt to the 8 XCDs round-robin),
// so the exchange stays in one L2.
__device__ __forceinline__ void wide_member(int n, int K, int& i, int& k) {
  const int bid = int(blockIdx.x), nb = int(gridDim.x);
  if (nb % 8 == 0 && n % 8 == 0) {
    const int j = bid / 8;
    i = (bid % 8) * (n / 8) + j / K;
    k = j % K;
  } else {
    i = bid / K;
    k = bid % K;
  }
}

// Member k's part of worker i's pass; false when a rendezvous timed out.
template <int CPQ, int SR>
__device__ __forceinline__ bool dense_wide_pass(const SgdArgs& a, const DenseSync& ds, int i, int k) {
  __shared__ double red[2][kWaves][4][SR];  // per-row partial margins
  __shared__ int ridx[2][kMaxBatch];  // this member's row indices of steps t, t+1 (slot t & 1)
  __shared__ int abort_flag;
  const int K = ds.K;
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
  double wd[CPQ][4];  // the model slice widened once per step for the dots
  auto widen = [&]() {
#pragma unroll
    for (int q = 0; q < CPQ; ++q) {
      wd[q][0] = w[q].x; wd[q][1] = w[q].y; wd[q][2] = w[q].z; wd[q][3] = w[q].w;
    }
  };
  widen();

  const int B = a.batch, S = int(a.S);  // S < 2^31 (checked at bind)
  const int KS = (S + B - 1) / B;
  const int K0 = int(a.k0), KE = int(a.k1);  // steps [K0, KE) of the pass run here
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
  // member offsets of a full step and of the (possibly shorter) last one,
  // computed once (Bp <= 512, so 32-bit products are exact)
  const int Blast = S - (KS - 1) * B;
  const int off0 = (B * k) / K, off1 = (B * (k + 1)) / K;
  const int last0 = (Blast * k) / K, last1 = (Blast * (k + 1)) / K;
  auto share = [&](int t, int& lo_, int& hi_) {
    const int b0 = t * B;
    const bool last = t == KS - 1;
    lo_ = b0 + (last ? last0 : off0);
    hi_ = b0 + (last ? last1 : off1);
  };
  auto settle = [&](Pos p) {  // move past steps in which this member has no samples
    while (p.t < KE && p.sb >= p.hi) {
      ++p.t;
      if (p.t < KE) {
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
    if (t >= KE) return;
    int lo_, hi_;
    share(t, lo_, hi_);
    if (tid < hi_ - lo_) pi = si[lo_ + tid];
  };
  auto stage = [&](int t) {
    if (t >= KE) return;
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
        float4 v = (ok && nv[q] > 0) ? ld_stream(row + c) : make_float4(0.f, 0.f, 0.f, 0.f);
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
  bool local = false;  // all members on this XCD (set before the first step)

  // margins, coefficients and gradient of the sub-batch held in xc
  auto process = [&](float4 (&xc)[SR][CPQ], float yl, Pos p) {
    // fp64 partial dots of the SR rows (single products of scaled columns
    // can dwarf the margin), then one transposed fp64 reduction over each
    // 16-lane DPP row; lanes 16r + s (s < SR) hold row r's share
    double d[16];
#pragma unroll
    for (int s = 0; s < SR; ++s) {
      double dd = 0.0;
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        dd = fma(wd[q][0], double(xc[s][q].x), dd);
        dd = fma(wd[q][1], double(xc[s][q].y), dd);
        dd = fma(wd[q][2], double(xc[s][q].z), dd);
        dd = fma(wd[q][3], double(xc[s][q].w), dd);
      }
      d[s] = dd;
    }
    const double part = row_reduce<SR>(d, lane);
    if ((lane & 15) < SR) red[par][wave][lane >> 4][lane & 15] = part;
    lds_barrier();
    float cf = 0.f;
    if (lane < SR && lane < p.hi - p.sb) {
      // the partials of two waves are read before they are added (in wave and
      // row order, as one chain would): one LDS round trip per 8 partials
      // instead of per 2 (32 workers x 4096: 7.01 -> 6.88 ms per pass; four
      // waves at a time gained nothing more)
      double m = 0.0;
#pragma unroll
      for (int v0 = 0; v0 < kWaves; v0 += 2) {
        double tv[2][4];
#pragma unroll
        for (int v = 0; v < 2; ++v)
#pragma unroll
          for (int r = 0; r < 4; ++r) tv[v][r] = red[par][v0 + v][r][lane];
#pragma unroll
        for (int v = 0; v < 2; ++v)
#pragma unroll
          for (int r = 0; r < 4; ++r) m += tv[v][r];
      }
      cf = loss_coef(m, yl, a.loss);
    }
    par ^= 1;
    // the sub-batch's contribution in fp32 (at most SR terms), added to the
    // step's fp64 gradient
    float4 gs[CPQ];
#pragma unroll
    for (int q = 0; q < CPQ; ++q) gs[q] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int s = 0; s < SR; ++s) {
      const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cf), s));
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        gs[q].x = fmaf(c, xc[s][q].x, gs[q].x);
        gs[q].y = fmaf(c, xc[s][q].y, gs[q].y);
        gs[q].z = fmaf(c, xc[s][q].z, gs[q].z);
        gs[q].w = fmaf(c, xc[s][q].w, gs[q].w);
      }
    }
#pragma unroll
    for (int q = 0; q < CPQ; ++q) {
      g[q][0] += double(gs[q].x);
      g[q][1] += double(gs[q].y);
      g[q][2] += double(gs[q].z);
      g[q][3] += double(gs[q].w);
    }
  };

  // Members of a worker meet here.  Everything they share is written and
  // read with relaxed device-scope atomics (coherent for the whole device
  // without cache write-back or invalidation); a wave's writes are
  // acknowledged before the barrier, and one thread counts the workgroup in
  // and waits, for a bounded time, until all K members have arrived.
  // Work issued between arrive() and gather() overlaps the wait: loads
  // issued there land while the members gather.
  auto arrive = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) __hip_atomic_fetch_add(ds.count + i, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  auto gather = [&](uint32_t target) -> bool {
    if (tid == 0) {
      uint32_t spins = 0;
      while (__hip_atomic_load(ds.count + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (++spins > ds.spin_limit) {
          abort_flag = 1;
          __hip_atomic_fetch_add(ds.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
    __syncthreads();
    return abort_flag == 0;
  };

  // end of step t: exchange (K > 1) and update; false when the rendezvous
  // timed out.  `during` issues the next sub-batch's loads (see rendezvous).
  auto finish_step = [&](int t, auto&& during) -> bool {
    const int Bp = min(B, S - t * B);
    // member partials of step t: slot t & 1 (a member writes slot t & 1
    // again at step t + 2, after every member has passed the rendezvous of
    // step t + 1, which each reaches only after reading step t's partials)
    // this worker's K partials of slot t & 1, [K][CPQ][thread][4] fp32
    const auto prs =
        buf_rsrc(ds.part + (int64_t(t & 1) * a.n + i) * K * ds.ldp, uint32_t(K * ds.ldp) * 4u);
    if (K > 1) {
      // every member publishes its partial gradient, rounded to fp32, with
      // one 16-byte store per q (one writer per word: no atomic
      // read-modify-write on shared lines), ...
#pragma unroll
      for (int q = 0; q < CPQ; ++q) {
        const v4f v = {float(g[q][0]), float(g[q][1]), float(g[q][2]), float(g[q][3])};
        const uint32_t off = uint32_t((k * ds.ldp + (q * kThreads + tid) * 4) * 4);
        if (local)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, v),
                                                 prs, off, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, v),
                                                 prs, off, 0, 16);  // sc1: device scope
      }
      arrive();
    }
    during();
    if (K > 1) {
      if (!gather(ds.base + uint32_t(K) * uint32_t(t - K0 + 2))) return false;
      // ... and every member sums all K partials in fp64 in member order,
      // so all members get the same gradient bit for bit.  The loads are
      // device-scope: they never hit a stale line of this CU's L1 (members
      // on one XCD find the partials in its L2, the others in memory).
#pragma unroll
      for (int q = 0; q < CPQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) g[q][e] = 0.0;
      // the members' partials in blocks of 8, unrolled, added in member
      // order (32 workers x 4096, 8 members: 7.14 -> 7.01 ms per pass against
      // a rolled loop over the members; the compiler still issues the loads
      // two at a time beside the adds, and holding four members' loads in
      // flight at once gained nothing)
      typedef unsigned int u4v __attribute__((ext_vector_type(4)));
      for (int m0 = 0; m0 < K; m0 += 8) {
        u4v pu[8][CPQ];
#pragma unroll
        for (int mm = 0; mm < 8; ++mm)
#pragma unroll
          for (int q = 0; q < CPQ; ++q) {
            const int m = m0 + mm < K ? m0 + mm : m0;
            const uint32_t off = uint32_t((m * ds.ldp + (q * kThreads + tid) * 4) * 4);
            pu[mm][q] = __builtin_amdgcn_raw_buffer_load_b128(prs, off, 0, 16);  // sc1: device scope
          }
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
          if (m0 + mm >= K) break;
#pragma unroll
          for (int q = 0; q < CPQ; ++q) {
            const unsigned u0 = pu[mm][q][0], u1 = pu[mm][q][1], u2 = pu[mm][q][2], u3 = pu[mm][q][3];
            g[q][0] += double(__uint_as_float(u0));
            g[q][1] += double(__uint_as_float(u1));
            g[q][2] += double(__uint_as_float(u2));
            g[q][3] += double(__uint_as_float(u3));
          }
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
    widen();
    // every wave has passed a barrier since its last read of slot t & 1;
    // the barrier after the write orders it before the first read of step
    // t + 2, which can come right after this step when steps are short
    stage(t + 2);
    lds_barrier();
    fetch(t + 3);
    return true;
  };

  // Rows of the next sub-batch of the same step load into xb while xa is
  // processed; the copy xa = xb then waits for loads that had the whole
  // sub-batch to land.  The first two sub-batches of a new step load into xa
  // and xb during the exchange that ends the step before it (their row
  // indices are staged by then), so the members' wait overlaps HBM reads and
  // a member arrives without waiting for them.  Every member finishes every step
  // (exchange + update), also the steps in which it has no samples.
  float4 xa[SR][CPQ], xb[SR][CPQ];
  float ya = 0.f, yb = 0.f;
  bool ok = true;
  int done = K0;  // steps finished
  // Whether all members of the worker run on this XCD: they publish their
  // XCD and meet once before the first step (count K; step t meets at
  // K (t - K0 + 2)).
  if (K > 1) {
    const int me = xcd_id();
    if (tid == 0) __hip_atomic_store(ds.xcd + i * K + k, me, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    arrive();
    ok = gather(ds.base + uint32_t(K));
    local = ok;
    for (int m = 0; m < K; ++m)
      local = local && __hip_atomic_load(ds.xcd + i * K + m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == me;
  }
  fetch(K0);
  stage(K0);
  fetch(K0 + 1);
  stage(K0 + 1);
  fetch(K0 + 2);
  __syncthreads();
  Pos cur{K0, 0, 0, 0};
  share(K0, cur.lo, cur.hi);
  cur.sb = cur.lo;
  cur = settle(cur);
  if (cur.t < KE) load(xa, ya, cur);
  while (ok && done < min(cur.t, KE)) ok = finish_step(done++, [] {});  // steps without samples
  bool xb_loaded = false;  // the exchange that ended the last step also loaded xb
  while (ok && cur.t < KE) {
    const Pos nx = settle(Pos{cur.t, cur.sb + SR, cur.lo, cur.hi});
    const bool same = nx.t == cur.t;
    if (same && !xb_loaded) load(xb, yb, nx);
    xb_loaded = false;
    process(xa, ya, cur);
    if (same) {
#pragma unroll
      for (int s2 = 0; s2 < SR; ++s2)
#pragma unroll
        for (int q = 0; q < CPQ; ++q) xa[s2][q] = xb[s2][q];
      ya = yb;
    } else {
      while (ok && done < min(nx.t, KE)) {
        const int t = done++;
        ok = finish_step(t, [&]() {
          // both buffers are free during the exchange: the first two
          // sub-batches of the next step load while the members gather
          if (t + 1 == nx.t && nx.t < KE) {
            load(xa, ya, nx);
            const Pos n2 = settle(Pos{nx.t, nx.sb + SR, nx.lo, nx.hi});
            if (n2.t == nx.t) {
              load(xb, yb, n2);
              xb_loaded = true;
            }
          }
        });
      }
    }
    cur = nx;
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
      if (a.tag) a.tag[i] = a.tag_value;
    }
  }
  return ok;
}

template <int CPQ, int SR>
__global__ __launch_bounds__(kThreads) void sgd_dense_wide_kernel(SgdArgs a, DenseSync ds) {
  int i, k;
  wide_member(a.n, ds.K, i, k);
  (void)dense_wide_pass<CPQ, SR>(a, ds, i, k);
}

// Several rounds in one launch (rounds_device.h): the K members of a worker
// run each pass together; member 0 publishes the row, waits for the
// neighbours and reduces it, and the others wait for the reduced row.  The
// members' arrival counter keeps counting across rounds (ds.base).
template <int CPQ, int SR>
__global__ __launch_bounds__(kThreads) void rounds_dense_wide_kernel(SgdArgs a, DenseSync ds, RoundsArgs ra) {
  int i, k;
  wide_member(a.n, ds.K, i, k);
  rounds::drive(
      a, ra, i, k, ds.K, [&](int64_t pass) { rounds::fill_schedule(ra.seed, i, pass, a.S, ra.sched + int64_t(i) * a.S); },
      [&](const SgdArgs& ar) {
        const bool ok = dense_wide_pass<CPQ, SR>(ar, ds, i, k);
        // arrivals of this pass: the opening meeting and one per step
        if (ds.K > 1) ds.base += uint32_t(ds.K) * uint32_t(ar.k1 - ar.k0 + 1);
        return ok;
      });
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

template <int CPQ, int SR>
hipError_t launch_rounds_wide(const SgdArgs& a, const DenseSync& ds, const RoundsArgs& ra, hipStream_t s) {
  SgdArgs aa = a;
  DenseSync dd = ds;
  RoundsArgs rr = ra;
  void* args[] = {&aa, &dd, &rr};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&rounds_dense_wide_kernel<CPQ, SR>),
                                    dim3(uint32_t(a.n * ds.K)), dim3(kThreads), args, 0, s);
}

// Bind-time scan of dense shards: xmax[i] = max |x| over worker i's shard
// (columns < dim); out[0] += labels outside {-1, +1}, out[1] += entries that
// are not finite.  Grid: n x blocks_per_worker blocks of 256 threads.
__global__ __launch_bounds__(256) void dense_scan_kernel(const float* X, const float* y, int64_t S, int64_t dim,
                                                        int64_t ldx, uint32_t bpw, float* xmax,
                                                        unsigned long long* out) {
  const int i = int(blockIdx.x / bpw);
  const int64_t part = blockIdx.x % bpw;
  const int64_t r0 = S * part / bpw, r1 = S * (part + 1) / bpw;
  float m = 0.f;
  unsigned long long nonfinite = 0, bady = 0;
  for (int64_t r = r0; r < r1; ++r) {
    const float* row = X + (int64_t(i) * S + r) * ldx;
    for (int64_t c = threadIdx.x; c < dim; c += 256) {
      const float v = row[c];
      nonfinite += !isfinite(v);
      m = fmaxf(m, fabsf(v));
    }
    if (threadIdx.x == 0) {
      const float yy = y[int64_t(i) * S + r];
      bady += (yy != 1.0f && yy != -1.0f);
    }
  }
  __shared__ float sm[256];
  sm[threadIdx.x] = m;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) sm[threadIdx.x] = fmaxf(sm[threadIdx.x], sm[threadIdx.x + o]);
    __syncthreads();
  }
  // non-negative floats order like their bit patterns
  if (threadIdx.x == 0) atomicMax(reinterpret_cast<unsigned int*>(xmax + i), __float_as_uint(sm[0]));
  if (bady) atomicAdd(out, bady);
  if (nonfinite) atomicAdd(out + 1, nonfinite);
}

}  // namespace

hipError_t launch_dense_scan(const float* X, const float* y, int32_t n, int64_t S, int64_t dim, int64_t ldx,
                             float* xmax, unsigned long long* out, hipStream_t s) {
  const uint32_t bpw = uint32_t(std::max<int64_t>(1, std::min<int64_t>(64, S / 16)));
  hipLaunchKernelGGL(dense_scan_kernel, dim3(uint32_t(n) * bpw), dim3(256), 0, s, X, y, S, dim, ldx, bpw, xmax, out);
  return hipGetLastError();
}

int dense_wide_cpq(int64_t dim) {
  if (dim <= 1024 || dim > 8192) return 0;
  return dim <= 2048 ? 1 : dim <= 4096 ? 2 : 4;
}

int dense_wide_max_members(const SgdArgs& a, int n_cu) {
  int per = 0;
  switch (dense_wide_cpq(a.dim)) {
    case 1: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<1, 8>, kThreads, 0); break;
    case 2: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<2, 8>, kThreads, 0); break;
    case 4: (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, sgd_dense_wide_kernel<4, 1>, kThreads, 0); break;
    default: return 1;
  }
  return std::max(1, per) * n_cu;
}

hipError_t launch_rounds_dense_wide(const SgdArgs& a, const DenseSync& ds, const RoundsArgs& ra, hipStream_t s) {
  switch (dense_wide_cpq(a.dim)) {
    case 1: return launch_rounds_wide<1, 8>(a, ds, ra, s);
    case 2: return launch_rounds_wide<2, 8>(a, ds, ra, s);
    case 4: return launch_rounds_wide<4, 1>(a, ds, ra, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_sgd_dense_wide(const SgdArgs& a, const DenseSync& ds, hipStream_t s) {
  switch (dense_wide_cpq(a.dim)) {
    case 1: return launch_wide<1, 8>(a, ds, s);
    case 2: return launch_wide<2, 8>(a, ds, s);
    case 4: return launch_wide<4, 1>(a, ds, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace asap
