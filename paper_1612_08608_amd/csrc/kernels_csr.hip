// kernels_csr.hip -- local SGD pass on CSR shards (Appendix A, update (A.2),
// first line; Section 5: each replica trains on its own data partition).
//
// One workgroup (1024 threads) runs one worker's whole pass: the steps form
// a dependency chain through the model, and a workgroup barrier is the
// cheapest way to order them.  A step is bound by latency, so the kernel is
// organised around taking global round trips off that chain:
//
//  * Hot columns in LDS.  The most frequent columns of the data (chosen once
//    at bind time) keep their model entries in LDS for the whole pass and are
//    written back at the end.  A bind-time array gives every nonzero its
//    "code": -(slot + 2) for a hot column, the column itself for a cold one.
//  * Software pipeline.  While step k computes, the row descriptors of step
//    k+3, the nonzeros (code, val) of step k+2 and the cold model entries of
//    step k+1 are loaded.  Nothing computes on a loaded value before the next
//    step, so no load is waited for inside the step that issues it.  The cold
//    entries of step k+1 are read before step k writes its updates; step k+1
//    patches them from step k's cold table, which keeps the post-update value
//    of every column it changed.
//  * Cold tables are bucketed (four keys read with one 128-bit LDS load).
//  * The barrier between gradient and update orders LDS only, so loads stay
//    in flight across it; the end-of-step barrier is a full fence.
//
// Determinism: a row's margin is summed over a fixed 16-lane tree in fp64;
// each column's gradient is accumulated as an exact 64-bit fixed-point
// integer (integer LDS atomics commute).
//
// A step whose minibatch has more than 64 rows, a row with more than 16*E
// nonzeros, or more than 3/4 of the cold table in cold nonzeros takes the
// general path: margins first, then contributions in row chunks, applied
// chunk by chunk (the update is linear in the contributions).
#include <cmath>

#include "asap_launch.h"
#include "rounds_device.h"
#include "csr_device.h"
#include "csr_fast.h"

namespace asap {
namespace {

using namespace csr;
constexpr int kCold = 2048;                          // cold table slots
constexpr int kBucket = 4;
constexpr int kBucketBits = 9;
constexpr int kBuckets = kCold / kBucket;
constexpr int kEmpty = -1;
constexpr int kBMax = 512;
constexpr int kChunkPairs = kCold / 2;               // general path: nonzeros per chunk
constexpr int kColdFast = kCold * 3 / 4;             // fast path: cold nonzeros per step
static_assert(kBuckets == 1 << kBucketBits, "bucket count");

struct ColdTable {
  int key[kCold];  // bucket b is key[4b .. 4b+3], filled in slot order
  unsigned long long acc[kCold];
  float val[kCold];  // pre-update value until applied, then the post-update value
};

struct Shared {
  float vhot[kHotMax];
  unsigned long long acch[kHotMax];
  ColdTable cold[2];
  int stats[3][2];  // per step (mod 3): cold nonzeros, rows over the fast length
};
static_assert(sizeof(Shared) <= 160 * 1024, "LDS budget of one workgroup");
static_assert(kBMax <= kCold, "general-path coefficients fit a cold table's accumulators");

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int cold_bucket(int col) {
  return int((uint32_t(col) * 2654435761u) >> (32 - kBucketBits));
}

typedef int int4v __attribute__((ext_vector_type(4)));

// The four keys of bucket b in one 128-bit LDS read, for a table that no
// lane is writing.
__device__ __forceinline__ int4v bucket_keys(const ColdTable& t, int b) {
  return *reinterpret_cast<const int4v*>(&t.key[b * kBucket]);
}

// The same keys while other lanes may be claiming slots: each key is read
// with a relaxed workgroup-scope atomic load, so a retry sees new claims.
__device__ __forceinline__ int4v bucket_keys_live(ColdTable& t, int b) {
  int* k = &t.key[b * kBucket];
  int4v r;
  r.x = __hip_atomic_load(k + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  r.y = __hip_atomic_load(k + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  r.z = __hip_atomic_load(k + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  r.w = __hip_atomic_load(k + 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  return r;
}

// Slot of `col` in a table nobody is writing, or -1.  Buckets fill in slot
// order and are probed in order, so a bucket with a free slot ends the search.
__device__ __forceinline__ int cold_find(const ColdTable& t, int col) {
  int b = cold_bucket(col);
  for (int n = 0; n < kBuckets; ++n) {
    const int4v k = bucket_keys(t, b);
    if (k.x == col) return b * kBucket;
    if (k.y == col) return b * kBucket + 1;
    if (k.z == col) return b * kBucket + 2;
    if (k.w == col) return b * kBucket + 3;
    if (k.w == kEmpty) return -1;
    b = (b + 1) & (kBuckets - 1);
  }
  return -1;
}

// Value of `col` after the step that filled table t, or `fallback`.
__device__ __forceinline__ float cold_patch(const ColdTable& t, int col, float fallback) {
  const int sl = cold_find(t, col);
  return sl < 0 ? fallback : t.val[sl];
}

// Add q into col's slot, claiming the first free slot of its bucket chain if
// the column is new; the claiming lane records the pre-update value.
__device__ __forceinline__ void cold_add(ColdTable& t, int col, long long q, float vold) {
  int b = cold_bucket(col);
  int sl = -1;
  for (int n = 0; n < 4 * kBuckets && sl < 0; ++n) {
    const int4v k = bucket_keys_live(t, b);
    const int kk[kBucket] = {k.x, k.y, k.z, k.w};
    int empty = -1;
#pragma unroll
    for (int s = 0; s < kBucket; ++s) {
      if (sl < 0 && kk[s] == col) sl = b * kBucket + s;
      if (empty < 0 && kk[s] == kEmpty) empty = s;
    }
    if (sl >= 0) break;
    if (empty < 0) {
      b = (b + 1) & (kBuckets - 1);
      continue;
    }
    const int old = atomicCAS(&t.key[b * kBucket + empty], kEmpty, col);
    if (old == kEmpty) {
      sl = b * kBucket + empty;
      t.val[sl] = vold;
    } else if (old == col) {
      sl = b * kBucket + empty;
    }  // else another column took the slot: read the bucket again
  }
  if (sl >= 0) atomicAdd(&t.acc[sl], static_cast<unsigned long long>(q));
}

// Apply a cold table: v = vold - coefA * sum for every claimed column, stored
// to the model and kept in the table; the slot is cleared when `clear`.
__device__ __forceinline__ void cold_apply(ColdTable& t, const Views& w, double coefA, double from_fx,
                                           bool clear) {
  for (int sl = threadIdx.x; sl < kCold; sl += kThreads) {
    const int col = t.key[sl];
    if (col != kEmpty) {
      const float nv =
          float(double(t.val[sl]) - coefA * double(static_cast<long long>(t.acc[sl])) * from_fx);
      st_f32(w.model, uint32_t(col) * 4u, nv);
      t.val[sl] = nv;
      t.acc[sl] = 0ull;
      if (clear) t.key[sl] = kEmpty;
    }
  }
}

__device__ __forceinline__ void hot_apply(Shared& sh, int H, double coefA, double from_fx) {
  for (int h = threadIdx.x; h < H; h += kThreads) {
    const unsigned long long a = sh.acch[h];
    if (a != 0ull) {
      sh.vhot[h] = float(double(sh.vhot[h]) - coefA * double(static_cast<long long>(a)) * from_fx);
      sh.acch[h] = 0ull;
    }
  }
}

template <int E>
__device__ __forceinline__ void gather_cold(const Views& w, const DataReg<E>& d, float (&vg)[E]) {
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const int c = code_at(d, j);
    vg[j] = ld_f32(w.model, uint32_t(c >= 0 ? c : 0) * 4u);
  }
}

// Count a step's cold nonzeros and rows too long for the fast path (one
// LDS atomic per row after a 16-lane sum).
template <int E>
__device__ __forceinline__ void count_stats(Shared& sh, int slot, const DataReg<E>& d, int sub) {
  int cold = 0;
#pragma unroll
  for (int j = 0; j < E; ++j) cold += code_at(d, j) >= 0;
  cold = row16_sum_i(cold);
  if (sub == 0) {
    if (cold) atomicAdd(&sh.stats[slot][0], cold);
    if (d.ok & kRowLong) atomicAdd(&sh.stats[slot][1], 1);
  }
}

template <int E, bool PIPE>
__device__ __forceinline__ void csr_pass(const SgdArgs& a, int i, Shared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & (kRowLanes - 1);
  const int brow = wave * (64 / kRowLanes) + (lane / kRowLanes);  // fast-path row of this lane
  float* vrow = a.models + int64_t(i) * a.ld;
  const RowInfo* ri = a.rowinfo + int64_t(i) * a.S;
  const int H = a.n_hot;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  Views w;
  w.seg = a.row_ptr[int64_t(i) * a.S];
  const uint32_t nnz_w = uint32_t(a.row_ptr[int64_t(i + 1) * a.S] - w.seg);
  w.code = rsrc(a.code + w.seg, nnz_w * 4u);
  w.val = rsrc(a.val + w.seg, nnz_w * 4u);
  w.model = rsrc(vrow, uint32_t(a.dim) * 4u);

  for (int h = tid; h < H; h += kThreads) {
    sh.vhot[h] = vrow[a.hot_cols[h]];
    sh.acch[h] = 0ull;
  }
  for (int q = tid; q < kCold; q += kThreads) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      sh.cold[t].key[q] = kEmpty;
      sh.cold[t].acc[q] = 0ull;
    }
  }
  if (tid < 6) sh.stats[tid / 2][tid % 2] = 0;
  // Fixed point: a column collects at most B contributions of size <= vmax
  // (|c_b| <= 1, labels in {-1, +1}); with B * vmax < 2^e the sum stays
  // below 2^61 at scale 2^(61 - e).
  int e2 = 0;
  frexp(double(a.batch) * double(a.vmax[i]), &e2);
  const double to_fx = ldexp(1.0, 61 - e2), from_fx = ldexp(1.0, e2 - 61);
  double s = 1.0;  // w = s * v

  // Pipeline registers; at the top of step k: d0 = nonzeros of step k,
  // vg0 = its cold model entries, d1 = nonzeros of step k+1, r2 = row of
  // step k+2.  Each step loads into d2 / vg1 / r3, which the top of the
  // next step rotates in (after the end-of-step fence, so the moves do not
  // wait).  stats[k % 3] holds step k's counts.
  RowInfo r2, r3;
  DataReg<E> d0, d1, d2;
  float vg0[E], vg1[E];
  // this launch runs steps [k0, kend) of the pass; loads past kend are
  // void like those past the pass
  const int64_t k0 = a.k0, kend = a.k1;
  if (PIPE) {
    const RowInfo ra = load_row(a, ri, k0, kend, brow), rb = load_row(a, ri, k0 + 1, kend, brow);
    r2 = load_row(a, ri, k0 + 2, kend, brow);
    __syncthreads();
    load_data<E>(w, ra, row_valid(a, k0, kend, brow), sub, d0);
    load_data<E>(w, rb, row_valid(a, k0 + 1, kend, brow), sub, d1);
    __syncthreads();
    gather_cold<E>(w, d0, vg0);
    count_stats<E>(sh, int(k0 % 3), d0, sub);
  }
  __syncthreads();

  for (int64_t k = k0; k < kend; ++k) {
    if (PIPE && k > k0) {  // rotate what the previous step loaded
      d0 = d1;
      d1 = d2;
      r2 = r3;
#pragma unroll
      for (int j = 0; j < E; ++j) vg0[j] = vg1[j];
    }
    const int64_t b0 = k * a.batch;
    const int Bp = int(min(int64_t(a.batch), a.S - b0));
    const double eta = step_size(a.lr_kind, a.lr0, a.round * K + k + 1);
    const double s_new = s * (1.0 - eta * double(a.l2));
    const double coefA = eta / (double(Bp) * s_new);
    ColdTable& cur = sh.cold[k & 1];
    ColdTable& prev = sh.cold[(k + 1) & 1];
    const int st = int(k % 3);
    const bool fast = PIPE && Bp <= kFastRows && sh.stats[st][1] == 0 && sh.stats[st][0] <= kColdFast;

    if (fast) {
      // prefetch: row descriptors of k+3, nonzeros of k+2, cold entries of k+1
      r3 = load_row(a, ri, k + 3, kend, brow);
      load_data<E>(w, r2, row_valid(a, k + 2, kend, brow), sub, d2);
      gather_cold<E>(w, d1, vg1);
      count_stats<E>(sh, int((k + 1) % 3), d1, sub);

      double part = 0.0;
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const int code = code_at(d0, j);
        float v = 0.f;
        if (is_hot(code))
          v = sh.vhot[hot_slot(code)];
        else if (code >= 0)
          v = cold_patch(prev, code, vg0[j]);
        part = fma(double(d0.val[j]), double(v), part);
      }
      const double dot = row16_sum(part);
      const double cf = (d0.ok & kRowExists) ? loss_coef(s * dot, double(d0.y), a.loss) : 0.0;
      if (cf != 0.0) {  // a zero coefficient leaves the row's columns as they are
#pragma unroll
        for (int j = 0; j < E; ++j) {
          const int code = code_at(d0, j);
          if (code == -1) continue;
          const long long q = llrint(cf * double(d0.val[j]) * to_fx);
          if (is_hot(code))
            atomicAdd(&sh.acch[hot_slot(code)], static_cast<unsigned long long>(q));
          else  // the pre-update value is looked up again rather than kept in registers
            cold_add(cur, code, q, cold_patch(prev, code, vg0[j]));
        }
      }
      lds_barrier();
      hot_apply(sh, H, coefA, from_fx);
      cold_apply(cur, w, coefA, from_fx, false);
      for (int q = tid; q < kCold; q += kThreads) prev.key[q] = kEmpty;
      if (tid == 0) sh.stats[st][0] = sh.stats[st][1] = 0;
    } else {
      // general path: margins (one wave per row), then row chunks.  The
      // accumulators of the idle previous-step table hold the minibatch's
      // coefficients (bit patterns of doubles) until the step ends.
      unsigned long long* coef = prev.acc;
      for (int b = wave; b < Bp; b += kWaves) {
        const RowInfo x = ri[b0 + b];
        double part = 0.0;
        for (int e = lane; e < x.len; e += 64) {
          const long long p = x.start + e;
          const int code = a.code[p];
          float v;
          if (is_hot(code))
            v = sh.vhot[hot_slot(code)];
          else
            v = vrow[code];
          part = fma(double(a.val[p]), double(v), part);
        }
        const double dot = wave_sum(part);
        if (lane == 0) coef[b] = __builtin_bit_cast(unsigned long long, loss_coef(s * dot, double(x.y), a.loss));
      }
      __syncthreads();
      if (tid == 0) sh.stats[st][0] = sh.stats[st][1] = 0;
      int c0 = 0;
      while (c0 < Bp) {
        int c1 = c0, cnt = 0;
        while (c1 < Bp) {
          const int len = ri[b0 + c1].len;
          if (c1 > c0 && cnt + len > kChunkPairs) break;
          cnt += len;
          ++c1;
        }
        for (int b = c0 + wave; b < c1; b += kWaves) {
          const double cf = __builtin_bit_cast(double, coef[b]);
          if (cf == 0.0) continue;
          const RowInfo x = ri[b0 + b];
          for (int e = lane; e < x.len; e += 64) {
            const long long p = x.start + e;
            const int code = a.code[p];
            const long long q = llrint(cf * double(a.val[p]) * to_fx);
            if (is_hot(code))
              atomicAdd(&sh.acch[hot_slot(code)], static_cast<unsigned long long>(q));
            else
              cold_add(cur, code, q, vrow[code]);
          }
        }
        __syncthreads();
        hot_apply(sh, H, coefA, from_fx);
        cold_apply(cur, w, coefA, from_fx, true);
        __syncthreads();
        c0 = c1;
      }
      for (int q = tid; q < kCold; q += kThreads) {
        prev.key[q] = kEmpty;
        prev.acc[q] = 0ull;
      }
      if (PIPE) {  // re-prime the pipeline for step k+1 (this step's stores are visible)
        const RowInfo ra = load_row(a, ri, k + 1, kend, brow), rb = load_row(a, ri, k + 2, kend, brow);
        r3 = load_row(a, ri, k + 3, kend, brow);
        __syncthreads();
        load_data<E>(w, ra, row_valid(a, k + 1, kend, brow), sub, d1);
        load_data<E>(w, rb, row_valid(a, k + 2, kend, brow), sub, d2);
        __syncthreads();
        gather_cold<E>(w, d1, vg1);
        count_stats<E>(sh, int((k + 1) % 3), d1, sub);
      }
    }

    s = s_new;
    if (s < 1e-6) {  // fold the scale back into v before it underflows
      const float sf = float(s);
      __syncthreads();
      for (int h = tid; h < H; h += kThreads) sh.vhot[h] *= sf;
      for (int64_t c = tid; c < a.dim; c += kThreads) vrow[c] *= sf;
      for (int q = tid; q < kCold; q += kThreads) cur.key[q] = kEmpty;  // nothing left to patch
      s = 1.0;
      __syncthreads();
      if (PIPE) gather_cold<E>(w, d1, vg1);  // the next step's cold entries, rescaled
    }
    __syncthreads();  // full fence: cold stores and LDS updates visible, loads landed
  }

  for (int h = tid; h < H; h += kThreads) vrow[a.hot_cols[h]] = sh.vhot[h];
  if (tid == 0) {
    a.scale[i] = float(s);
    if (a.tag) a.tag[i] = a.tag_value;
  }
}

template <int E, bool PIPE>
__global__ __launch_bounds__(kThreads) void sgd_csr_kernel(SgdArgs a) {
  if (a.run_if && *a.run_if == 0) return;  // the planned kernel took this round
  __shared__ Shared sh;
  csr_pass<E, PIPE>(a, int(blockIdx.x), sh);
}

// Several rounds in one launch (rounds_device.h): one workgroup per worker
// runs its passes on this kernel's code and reduces its own row.
template <int E, bool PIPE>
__global__ __launch_bounds__(kThreads) void rounds_csr_kernel(SgdArgs a, RoundsArgs ra) {
  const int i = int(blockIdx.x);
  __shared__ Shared sh;
  rounds::drive(
      a, ra, i, 0, 1,
      [&](int64_t pass) {
        rounds::fill_rowinfo(ra.seed, i, pass, a.S, a.row_ptr, a.y, ra.rowinfo + int64_t(i) * a.S);
      },
      [&](const SgdArgs& ar) {
        csr_pass<E, PIPE>(ar, i, sh);
        return true;
      });
}

// The plan of pass u of a planned launch (area u of the plan ring).
__device__ __forceinline__ PlanArgs ring_area(const RoundsPlan& rp, int64_t u) {
  PlanArgs p = rp.area0;
  const int64_t d = u * rp.stride;
  p.rowinfo = reinterpret_cast<const RowInfo*>(reinterpret_cast<const char*>(p.rowinfo) + d);
  p.rows_real = reinterpret_cast<const RowInfo*>(reinterpret_cast<const char*>(p.rows_real) + d);
  p.step_off = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.step_off) + d);
  p.pack = reinterpret_cast<int2*>(reinterpret_cast<char*>(p.pack) + d);
  p.clist = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.clist) + d);
  p.clink = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.clink) + d);
  p.hlist = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.hlist) + d);
  p.cnt = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.cnt) + d);
  p.flag = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(p.flag) + d);
  return p;
}

// One thread: wait until pass u's plan is published (ready[u] carries this
// launch's token for it) or the wall clock passes `deadline`.
__device__ inline bool wait_plan(const RoundsPlan& rp, int64_t u, long long deadline) {
  while (rounds::tag_peek(rp.ready + u) != rp.token0 + u) {
    if (wall_clock64() > deadline) return false;
    __builtin_amdgcn_s_sleep(4);
  }
  return true;
}

// Several rounds in one launch on planned passes: every pass the launch
// covers has its plan in its own area of the ring (planned before the
// launch, or beside it on the library's look-ahead stream: a worker waits,
// bounded, until its pass's plan is published).  A pass whose plan
// overflowed runs the general pass code, as the stream-ordered path does,
// so both give the same bits.  With helpers, block n + i prefetches for
// worker i, pass after pass.
// EG: entries per lane of the general pass (the stream-ordered general
// kernel's, so that both give the same bits); EF: of the planned pass, sized
// for the members' slices (its bits do not depend on it).
template <int EG, int EF, bool MEM>
__global__ __launch_bounds__(kThreads) void rounds_csr_planned_kernel(SgdArgs a, RoundsArgs ra, RoundsPlan rp) {
  union LdsUnion {
    Shared g;
    FastShared f;
  };
  __shared__ LdsUnion sh;
  __shared__ int plan_ok;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  const int M = MEM ? rp.area0.members : 1;
  if (int(blockIdx.x) >= ra.n * M) {
    // prefetch workgroup of the slice of block blockIdx.x - n M: the steps
    // of each pass that this launch runs
    int i, m;
    member_of(int(blockIdx.x) - ra.n * M, ra.n, M, i, m);
    for (int64_t u = 0; u < rp.npass; ++u) {
      if (threadIdx.x == 0) plan_ok = wait_plan(rp, u, wall_clock64() + ra.wait_ticks);
      __syncthreads();
      if (!plan_ok) return;  // only costs time: the worker reports it
      rounds::acquire_fence();
      const PlanArgs p = ring_area(rp, u);
      if (__hip_atomic_load(p.flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) continue;
      const int64_t pass = rp.first_pass + u;
      int64_t q0, k0, k1, q1, j0, j1;
      rounds::steps_of(ra.r0, ra.local_steps, K, q0, k0, k1);
      rounds::steps_of(ra.r0 + ra.R - 1, ra.local_steps, K, q1, j0, j1);
      // the model buffer of the pass's first round in this launch (later
      // rounds of a pass split by local steps alternate: only a prefetch)
      int64_t rfirst = ra.local_steps == 0 ? pass : (pass * K + ra.local_steps - 1) / ra.local_steps;
      if (rfirst < ra.r0) rfirst = ra.r0;
      SgdArgs ah = a;
      ah.round = pass;
      ah.k0 = pass == q0 ? k0 : 0;
      ah.k1 = pass == q1 ? j1 : K;
      ah.rowinfo = p.rowinfo;
      ah.models = ra.buf[ra.cur ^ int((rfirst - ra.r0) & 1)];
      prefetch_pass<EF>(ah, p, i * M + m, i);
      __syncthreads();
    }
    return;
  }
  int i, m;
  member_of(int(blockIdx.x), ra.n, M, i, m);
  PlanArgs pu = ring_area(rp, 0);
  rounds::drive(
      a, ra, i, m, M,
      [&](int64_t pass) {
        const int64_t u = pass - rp.first_pass;
        if (threadIdx.x == 0) {
          plan_ok = wait_plan(rp, u, wall_clock64() + ra.wait_ticks);
          if (!plan_ok && m == 0) rounds::report_stale(ra.err, i);
        }
        __syncthreads();
        rounds::acquire_fence();  // the plan was written by other kernels
        pu = ring_area(rp, u);
      },
      [&](const SgdArgs& ar) {
        if (!plan_ok) return false;
        SgdArgs ap = ar;
        if (__hip_atomic_load(pu.flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
          // the general pass is one workgroup's: member 0 runs it alone
          ap.rowinfo = pu.rows_real;
          if (m == 0) csr_pass<EG, true>(ap, i, sh.g);
          return true;
        }
        fast_pass<EF, MEM>(ap, pu, i, m, sh.f);
        if constexpr (!MEM) return true;
        // members: member 0 publishes the worker's half-step only after
        // every member's model stores are complete and released
        const uint32_t last = ap.xtag + uint32_t(ap.round * K + ap.k1 - 1 - ap.xg0);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0) {
          if (m != 0) {
            __hip_atomic_store(pu.done + i * M + m, static_cast<unsigned long long>(last), __ATOMIC_RELEASE,
                               __HIP_MEMORY_SCOPE_AGENT);
          } else {
            const long long deadline = wall_clock64() + ra.wait_ticks;
            for (int q = 1; q < M && plan_ok; ++q)
              while (__hip_atomic_load(pu.done + i * M + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) !=
                     static_cast<unsigned long long>(last)) {
                if (wall_clock64() > deadline) {
                  plan_ok = 0;
                  atomicAdd(pu.xerr, 1);
                  break;
                }
                __builtin_amdgcn_s_sleep(2);
              }
            rounds::acquire_fence();
          }
        }
        __syncthreads();
        return plan_ok != 0 && sh.f.xabort == 0;
      });
}

template <int E, bool PIPE>
hipError_t launch_rounds_e(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s) {
  int per = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, rounds_csr_kernel<E, PIPE>, kThreads, 0);
  if (e != hipSuccess) return e;
  if (int64_t(per) * n_cu < a.n) return hipErrorCooperativeLaunchTooLarge;
  SgdArgs aa = a;
  RoundsArgs rr = ra;
  aa.rowinfo = ra.rowinfo;
  void* args[] = {&aa, &rr};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&rounds_csr_kernel<E, PIPE>), dim3(uint32_t(a.n)),
                                    dim3(kThreads), args, 0, s);
}

template <int E>
hipError_t launch_rounds_pipe(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s, bool pipe) {
  return pipe ? launch_rounds_e<E, true>(a, ra, n_cu, s) : launch_rounds_e<E, false>(a, ra, n_cu, s);
}

template <int EG, int EF, bool MEM>
hipError_t launch_rounds_planned_em(const SgdArgs& a, const RoundsArgs& ra, const RoundsPlan& rp, int n_cu,
                                    hipStream_t s) {
  int per = 0;
  hipError_t e =
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, rounds_csr_planned_kernel<EG, EF, MEM>, kThreads, 0);
  if (e != hipSuccess) return e;
  const int64_t grid = int64_t(a.n) * rp.area0.members * (rp.area0.helpers ? 2 : 1);
  if (int64_t(per) * n_cu < grid) return hipErrorCooperativeLaunchTooLarge;
  SgdArgs aa = a;
  RoundsArgs rr = ra;
  RoundsPlan pp = rp;
  void* args[] = {&aa, &rr, &pp};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&rounds_csr_planned_kernel<EG, EF, MEM>),
                                    dim3(uint32_t(grid)), dim3(kThreads), args, 0, s);
}

// One member: EF = EG.  Members: the smallest of 3, 5 and EG entries per
// lane that covers the slices' rows.
template <int EG>
hipError_t launch_rounds_planned_e(const SgdArgs& a, const RoundsArgs& ra, const RoundsPlan& rp, int n_cu,
                                   hipStream_t s) {
  if (rp.area0.members == 1) return launch_rounds_planned_em<EG, EG, false>(a, ra, rp, n_cu, s);
  const int need = rp.area0.max_slice;
  if constexpr (EG > 3)
    if (need <= kRowLanes * 3) return launch_rounds_planned_em<EG, 3, true>(a, ra, rp, n_cu, s);
  if constexpr (EG > 5)
    if (need <= kRowLanes * 5) return launch_rounds_planned_em<EG, 5, true>(a, ra, rp, n_cu, s);
  return launch_rounds_planned_em<EG, EG, true>(a, ra, rp, n_cu, s);
}

// ----------------------------------------------------------------------------
// per-round row descriptors in schedule order
// ----------------------------------------------------------------------------
// With members > 1, position q = (v, pos) of slice v = worker * members + m
// describes the slice's part of the row the worker's schedule puts there
// (row_ptr then holds the slices' offsets, [n * members * S + 1]).
__global__ __launch_bounds__(256) void rowinfo_kernel(const int32_t* sched, const int64_t* row_ptr,
                                                      const float* y, int64_t S, int64_t total,
                                                      int32_t members, RowInfo* out) {
  const int64_t q = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (q >= total) return;
  const int64_t v = q / S, pos = q - v * S, worker = v / members;
  const int64_t r = sched[worker * S + pos];
  const int64_t g = v * S + r;
  const int64_t p0 = row_ptr[g], p1 = row_ptr[g + 1];
  RowInfo ri;
  ri.start = p0;
  ri.len = int(p1 - p0);
  ri.y = y[worker * S + r];
  out[q] = ri;
}

// ----------------------------------------------------------------------------
// bind time, members > 1: the rows of each worker split by member (column
// c belongs to member c mod members), one thread per row
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void member_count_kernel(const int64_t* row_ptr, const int32_t* col, int64_t rows,
                                                           int64_t S, int32_t members, int32_t* cnt,
                                                           int32_t* maxlen) {
  const int64_t g = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (g >= rows) return;
  const int64_t i = g / S, r = g - i * S;
  int c[kMaxMembers] = {0, 0, 0, 0};
  for (int64_t p = row_ptr[g]; p < row_ptr[g + 1]; ++p) ++c[col[p] % members];
  int most = 0;
  for (int m = 0; m < members; ++m) {
    cnt[(i * members + m) * S + r] = c[m];
    most = max(most, c[m]);
  }
  atomicMax(maxlen, most);
}

__global__ __launch_bounds__(256) void member_scatter_kernel(const int64_t* row_ptr, const int32_t* col,
                                                             const float* val, const int16_t* mlut, int64_t rows,
                                                             int64_t S, int32_t members, const int64_t* vrow_ptr,
                                                             int32_t* vcode, int2* pack) {
  const int64_t g = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (g >= rows) return;
  const int64_t i = g / S, r = g - i * S;
  int64_t pos[kMaxMembers];
  for (int m = 0; m < members; ++m) pos[m] = vrow_ptr[(i * members + m) * S + r];
  for (int64_t p = row_ptr[g]; p < row_ptr[g + 1]; ++p) {
    const int c = col[p];
    const int h = mlut[c];
    const int code = h >= 0 ? -h - 2 : c;
    const int64_t q = pos[c % members]++;
    if (vcode) vcode[q] = code;
    if (pack) pack[q] = make_int2(code, __float_as_int(val[p]));
  }
}

// ----------------------------------------------------------------------------
// bind time: column frequencies (sampled) and per-nonzero codes
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void col_hist_kernel(const int32_t* col, int64_t nnz, int64_t stride,
                                                       int32_t* counts) {
  for (int64_t k = int64_t(blockIdx.x) * 256 + threadIdx.x; k * stride < nnz;
       k += int64_t(gridDim.x) * 256)
    atomicAdd(&counts[col[k * stride]], 1);
}

__global__ __launch_bounds__(256) void code_kernel(const int32_t* col, int64_t nnz, const int16_t* lut,
                                                   int32_t* code) {
  for (int64_t p = int64_t(blockIdx.x) * 256 + threadIdx.x; p < nnz; p += int64_t(gridDim.x) * 256) {
    const int c = col[p];
    const int h = lut[c];
    code[p] = h >= 0 ? -h - 2 : c;
  }
}

template <int E>
hipError_t launch_e(const SgdArgs& a, hipStream_t s, bool pipe) {
  if (pipe)
    hipLaunchKernelGGL((sgd_csr_kernel<E, true>), dim3(uint32_t(a.n)), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((sgd_csr_kernel<E, false>), dim3(uint32_t(a.n)), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rowinfo(const int32_t* sched, const int64_t* row_ptr, const float* y, int32_t n, int64_t S,
                          RowInfo* out, hipStream_t s, int32_t members) {
  const int64_t total = int64_t(n) * members * S;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(rowinfo_kernel, dim3(uint32_t((total + 255) / 256)), dim3(256), 0, s, sched, row_ptr, y, S,
                     total, members, out);
  return hipGetLastError();
}

hipError_t launch_member_count(const int64_t* row_ptr, const int32_t* col, int32_t n, int64_t S, int32_t members,
                               int32_t* cnt, int32_t* maxlen, hipStream_t s) {
  const int64_t rows = int64_t(n) * S;
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(member_count_kernel, dim3(uint32_t((rows + 255) / 256)), dim3(256), 0, s, row_ptr, col, rows, S,
                     members, cnt, maxlen);
  return hipGetLastError();
}

hipError_t launch_member_scatter(const int64_t* row_ptr, const int32_t* col, const float* val, const int16_t* mlut,
                                 int32_t n, int64_t S, int32_t members, const int64_t* vrow_ptr, int32_t* vcode,
                                 int2* pack, hipStream_t s) {
  const int64_t rows = int64_t(n) * S;
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(member_scatter_kernel, dim3(uint32_t((rows + 255) / 256)), dim3(256), 0, s, row_ptr, col, val,
                     mlut, rows, S, members, vrow_ptr, vcode, pack);
  return hipGetLastError();
}

hipError_t launch_sgd_csr(const SgdArgs& a, hipStream_t s) {
  if (a.batch > kBMax || a.n_hot > kHotMax) return hipErrorInvalidValue;
  const bool pipe = a.batch <= kFastRows;
  // entries per lane: enough for the longest row, up to 8 (longer rows take the general path)
  if (a.max_row <= kRowLanes * 2) return launch_e<2>(a, s, pipe);
  if (a.max_row <= kRowLanes * 3) return launch_e<3>(a, s, pipe);
  if (a.max_row <= kRowLanes * 4) return launch_e<4>(a, s, pipe);
  if (a.max_row <= kRowLanes * 6) return launch_e<6>(a, s, pipe);
  return launch_e<8>(a, s, pipe);
}

// the same kernel choice as launch_sgd_csr, so that both paths run the same code
hipError_t launch_rounds_csr(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s) {
  if (a.batch > kBMax || a.n_hot > kHotMax) return hipErrorInvalidValue;
  const bool pipe = a.batch <= kFastRows;
  if (a.max_row <= kRowLanes * 2) return launch_rounds_pipe<2>(a, ra, n_cu, s, pipe);
  if (a.max_row <= kRowLanes * 3) return launch_rounds_pipe<3>(a, ra, n_cu, s, pipe);
  if (a.max_row <= kRowLanes * 4) return launch_rounds_pipe<4>(a, ra, n_cu, s, pipe);
  if (a.max_row <= kRowLanes * 6) return launch_rounds_pipe<6>(a, ra, n_cu, s, pipe);
  return launch_rounds_pipe<8>(a, ra, n_cu, s, pipe);
}

// the same entry count per lane as launch_sgd_csr_fast and launch_sgd_csr
hipError_t launch_rounds_csr_planned(const SgdArgs& a, const RoundsArgs& ra, const RoundsPlan& rp, int n_cu,
                                     hipStream_t s) {
  if (a.batch > kFastRows || a.n_hot > kHotMax) return hipErrorInvalidValue;
  if (a.max_row <= kRowLanes * 2) return launch_rounds_planned_e<2>(a, ra, rp, n_cu, s);
  if (a.max_row <= kRowLanes * 3) return launch_rounds_planned_e<3>(a, ra, rp, n_cu, s);
  if (a.max_row <= kRowLanes * 4) return launch_rounds_planned_e<4>(a, ra, rp, n_cu, s);
  if (a.max_row <= kRowLanes * 6) return launch_rounds_planned_e<6>(a, ra, rp, n_cu, s);
  return launch_rounds_planned_e<8>(a, ra, rp, n_cu, s);
}

hipError_t launch_col_hist(const int32_t* col, int64_t nnz, int64_t stride, int32_t* counts, hipStream_t s) {
  if (nnz <= 0) return hipSuccess;
  const int64_t samples = (nnz + stride - 1) / stride;
  const int64_t blocks = std::min<int64_t>((samples + 255) / 256, 8192);
  hipLaunchKernelGGL(col_hist_kernel, dim3(uint32_t(blocks)), dim3(256), 0, s, col, nnz, stride, counts);
  return hipGetLastError();
}

hipError_t launch_codes(const int32_t* col, int64_t nnz, const int16_t* lut, int32_t* code, hipStream_t s) {
  if (nnz <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((nnz + 255) / 256, 65536);
  hipLaunchKernelGGL(code_kernel, dim3(uint32_t(blocks)), dim3(256), 0, s, col, nnz, lut, code);
  return hipGetLastError();
}

}  // namespace asap
