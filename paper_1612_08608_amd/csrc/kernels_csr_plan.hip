// kernels_csr_plan.hip -- the CSR SGD pass with its column bookkeeping done
// ahead of time (Appendix A, update (A.2), first line; Section 5: each
// replica trains on its own data partition).
//
// The steps of a worker's pass form a dependency chain, but which columns a
// step touches is known once the round's schedule is: it does not depend on
// the model.  So the bookkeeping that a step would otherwise do on the chain
// -- finding the distinct columns of its minibatch, giving each a slot, and
// finding which of them the previous step also changed -- runs before the
// pass, for all workers and all steps at once:
//
//  * step_scan: per worker, where each step's nonzeros start in schedule
//    order (its region in the per-nonzero plan arrays);
//  * csr_plan: per (worker, step), the distinct cold columns (slots 0..Uc-1,
//    in `clist`), the distinct hot slots (`hlist`), and for every nonzero
//    its "code" for this round, -(hot slot + 2) or its cold slot: the first
//    half of a (code, value) pair, so that the pass loads both at once (the
//    values and the hot entries' codes do not change from round to round and
//    are written at bind, which keeps that traffic away from the pass the
//    planning runs beside);
//  * csr_link: per (worker, step), the slot each cold column had in the
//    previous step, or -1.
//
// The pass (sgd_csr_fast_kernel) then keeps the step's cold values in LDS
// slots: they are gathered from the model a step ahead, and a value the
// previous step changed is taken from that step's slot through the link.
// Margins read LDS, gradients are added to slot accumulators with integer
// atomics (no hashing, no CAS), and the update walks the step's slot lists.
//
// If any step has more distinct cold columns than the LDS slots, more hot
// slots than the list registers, or a hash table overflowed, the plan raises
// a flag: the fast kernel then does nothing and the general kernel runs.
#include <cmath>

#include "asap_launch.h"
#include "csr_device.h"

namespace asap {
namespace {

using namespace csr;

constexpr int kCMax = 2048;                  // cold slots per step held in LDS
constexpr int kHList = 2048;                 // hot slots per step applied from registers
constexpr int kColdPer = kCMax / kThreads;   // 2
constexpr int kHotPer = kHList / kThreads;   // 2
constexpr int kHotWords = (kHotMax + 31) / 32;

constexpr int kPlanThreads = 512;
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kLinkBits = 12;
constexpr int kLinkTab = 1 << kLinkBits;     // link hash positions (>= 2 kCMax)

__device__ __forceinline__ uint32_t mult_hash(int c, int bits) {
  return (uint32_t(c) * 2654435761u) >> (32 - bits);
}

// Open-addressed tables of 2^bits ints (linear probing).  Insert returns
// the key's position, or -1 when the table is full.
__device__ __forceinline__ int table_insert(int* keys, int bits, int c) {
  const uint32_t mask = (1u << bits) - 1;
  uint32_t h = mult_hash(c, bits);
  for (uint32_t n = 0; n <= mask; ++n) {
    const int old = atomicCAS(&keys[h], -1, c);
    if (old == -1 || old == c) return int(h);
    h = (h + 1) & mask;
  }
  return -1;
}

__device__ __forceinline__ int table_find(const int* keys, int bits, int c) {
  const uint32_t mask = (1u << bits) - 1;
  uint32_t h = mult_hash(c, bits);
  for (uint32_t n = 0; n <= mask; ++n) {
    const int k = keys[h];
    if (k == c) return int(h);
    if (k == -1) return -1;
    h = (h + 1) & mask;
  }
  return -1;
}

// exclusive prefix sum over the NW waves of a block (wave scans, then the
// wave totals); *total gets the sum
template <int NW>
__device__ __forceinline__ int block_scan(int v, int* sc, int* total) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sc[wave] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    base += w < wave ? sc[w] : 0;
    tot += sc[w];
  }
  *total = tot;
  __syncthreads();  // sc is reused by the next scan
  return base + x - v;
}

// ----------------------------------------------------------------------------
// step offsets: step_off[i][k] = nonzeros of worker i's steps before k, in
// schedule order (stride S + 1 per worker); one 256-thread block per worker
// (small enough to run beside an SGD pass that still holds the CUs)
// ----------------------------------------------------------------------------
constexpr int kScanThreads = 256;

__global__ __launch_bounds__(kScanThreads) void step_scan_kernel(PlanArgs p) {
  __shared__ int sc[kScanThreads];
  __shared__ int carry;
  const int i = blockIdx.x, t = threadIdx.x;
  const int64_t S = p.S;
  const int B = p.batch, K = p.K;
  const RowInfo* ri = p.rowinfo + int64_t(i) * S;
  int32_t* so = p.step_off + int64_t(i) * (S + 1);
  if (t == 0) carry = 0;
  __syncthreads();
  for (int base = 0; base < K; base += kScanThreads) {
    const int k = base + t;
    int tot = 0;
    if (k < K) {
      const int64_t b0 = int64_t(k) * B;
      const int Bp = int(min<int64_t>(B, S - b0));
      for (int b = 0; b < Bp; ++b) tot += ri[b0 + b].len;
    }
    sc[t] = tot;
    __syncthreads();
    for (int o = 1; o < kScanThreads; o <<= 1) {
      const int add = t >= o ? sc[t - o] : 0;
      __syncthreads();
      sc[t] += add;
      __syncthreads();
    }
    if (k < K) so[k] = carry + sc[t] - tot;
    __syncthreads();
    if (t == 0) carry += sc[kScanThreads - 1];
    __syncthreads();
  }
  if (t == 0) so[K] = carry;
}

// ----------------------------------------------------------------------------
// plan of one (worker, step): distinct columns, slots, per-nonzero codes
// ----------------------------------------------------------------------------
// TB: table positions 2^TB >= 2 * (the step's nonzeros), LDS sized to
// match; NT threads; H nonzeros per lane and row (rows of at most 64 H).
template <int TB, int NT, int H>
__global__ __launch_bounds__(NT) void csr_plan_kernel(PlanArgs p) {
  constexpr int NW = NT / 64;
  static_assert(NT >= kHotWords, "one hot-bitmap word per thread");
  __shared__ int keys[1 << TB];
  __shared__ uint16_t ids[1 << TB];  // slots < 2^TB <= 2^13
  __shared__ uint32_t hot[kHotWords];
  __shared__ int sc[NW];
  __shared__ long long rstart[kFastRows];
  __shared__ int rlen[kFastRows];
  __shared__ int overflow;
  constexpr int kRowsPerWave = kFastRows / NW;
  const int K = p.K, B = p.batch;
  const int i = int(blockIdx.x) / K, k = int(blockIdx.x) % K;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t S = p.S;
  const int64_t seg = p.row_ptr[int64_t(i) * S];
  const int64_t b0 = int64_t(k) * B;
  const int Bp = int(min<int64_t>(B, S - b0));  // <= kFastRows
  const int32_t* so = p.step_off + int64_t(i) * (S + 1);
  const int64_t lbase = seg + so[k];
  // a table of at least twice the step's nonzeros (at most 2^TB)
  const int T = so[k + 1] - so[k];
  int bits = 8;
  while (bits < TB && (1 << bits) < 2 * T) ++bits;
  const int tab = 1 << bits;
  if (t < Bp) {
    const RowInfo r = p.rowinfo[int64_t(i) * S + b0 + t];
    rstart[t] = r.start;
    rlen[t] = r.len;
  }
  for (int q = t; q < tab; q += NT) keys[q] = -1;
  for (int q = t; q < kHotWords; q += NT) hot[q] = 0u;
  if (t == 0) overflow = 0;
  __syncthreads();
  // every code of the step in registers (rows of at most 64 H nonzeros: H
  // per lane), all loads issued before any is used; -1 marks no entry
  int cc[kRowsPerWave][H];
#pragma unroll
  for (int j = 0; j < kRowsPerWave; ++j) {
    const int b = wave + j * NW;
    const int len = b < Bp ? rlen[b] : 0;
    const long long st = b < Bp ? rstart[b] : 0;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int e = lane + 64 * h;
      cc[j][h] = e < len ? p.code[st + e] : -1;
    }
  }
#pragma unroll
  for (int j = 0; j < kRowsPerWave; ++j)
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int c = cc[j][h];
      if (c == -1) continue;
      if (is_hot(c)) {
        const int hs = hot_slot(c);
        atomicOr(&hot[hs >> 5], 1u << (hs & 31));
      } else if (table_insert(keys, bits, c) < 0) {
        overflow = 1;
      }
    }
  __syncthreads();
  // cold slots in table order: thread t numbers a contiguous run of positions
  const int per = tab / NT > 0 ? tab / NT : 1;
  const int q0 = t * per, q1 = min(q0 + per, tab);
  int cnt = 0;
  for (int q = q0; q < q1; ++q) cnt += keys[q] >= 0;
  int Uc = 0;
  int id = block_scan<NW>(cnt, sc, &Uc);
  for (int q = q0; q < q1; ++q) {
    const int key = keys[q];
    if (key >= 0) {
      ids[q] = uint16_t(id);
      p.clist[lbase + id] = key;
      ++id;
    }
  }
  // hot slots in slot order
  const uint32_t word = t < kHotWords ? hot[t] : 0u;
  int Uh = 0;
  int hid = block_scan<NW>(__popc(word), sc, &Uh);
  for (uint32_t w = word; w; w &= w - 1) p.hlist[lbase + hid++] = t * 32 + __ffs(w) - 1;
  __syncthreads();  // ids complete
#pragma unroll
  for (int j = 0; j < kRowsPerWave; ++j) {
    const int b = wave + j * NW;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int c = cc[j][h];
      if (c == -1) continue;
      int out = c;
      if (!is_hot(c)) {
        const int pos = table_find(keys, bits, c);
        out = pos >= 0 ? int(ids[pos]) : 0;
      }
      // the code half of a cold entry's (code, value) pair: a hot entry's
      // code and every value do not change from round to round and are
      // written once, at bind
      if (!is_hot(c)) reinterpret_cast<int*>(p.pack + rstart[b] + lane + 64 * h)[0] = out;
    }
  }
  if (t == 0) {
    p.cnt[(int64_t(i) * K + k) * 2 + 0] = Uc;
    p.cnt[(int64_t(i) * K + k) * 2 + 1] = Uh;
    if (overflow || Uc > kCMax || Uh > kHList) atomicOr(p.flag, 1);
  }
}

// ----------------------------------------------------------------------------
// links: slot of each cold column of step k in step k-1, or -1
// ----------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(NT) void csr_link_kernel(PlanArgs p) {
  __shared__ int keys[kLinkTab];
  __shared__ int vals[kLinkTab];
  const int K = p.K;
  const int i = int(blockIdx.x) / K, k = int(blockIdx.x) % K;
  const int t = threadIdx.x;
  const int64_t S = p.S;
  const int64_t seg = p.row_ptr[int64_t(i) * S];
  const int32_t* so = p.step_off + int64_t(i) * (S + 1);
  const int Uc = min(p.cnt[(int64_t(i) * K + k) * 2], kCMax);
  const int64_t lbase = seg + so[k];
  const int Up = k > 0 ? min(p.cnt[(int64_t(i) * K + k - 1) * 2], kCMax) : 0;
  if (Uc == 0) return;
  // a table of at least four times the previous step's columns (at most
  // 2^kLinkBits, twice kCMax)
  int bits = 6;
  while (bits < kLinkBits && (1 << bits) < 4 * Up) ++bits;
  for (int q = t; q < (1 << bits); q += NT) keys[q] = -1;
  __syncthreads();
  if (k > 0) {
    const int64_t pbase = seg + so[k - 1];
    for (int u = t; u < Up; u += NT) {
      const int pos = table_insert(keys, bits, p.clist[pbase + u]);
      if (pos >= 0) vals[pos] = u;  // columns are distinct within a step
    }
  }
  __syncthreads();
  for (int u = t; u < Uc; u += NT) {
    const int pos = k > 0 ? table_find(keys, bits, p.clist[lbase + u]) : -1;
    p.clink[lbase + u] = pos >= 0 ? vals[pos] : -1;
  }
}

// ----------------------------------------------------------------------------
// the pass on the plan
// ----------------------------------------------------------------------------
struct FastShared {
  float vhot[kHotMax];
  unsigned long long acch[kHotMax];
  float cval[2][kCMax];  // cold values of steps k (slot k & 1) and k - 1
  unsigned long long cacc[kCMax];
};
static_assert(sizeof(FastShared) <= 160 * 1024, "LDS budget of one workgroup");

// per-step constants: region start (within the worker), cold and hot counts
struct Meta {
  int soff, uc, uh;
};

// Loaded with vector (buffer) loads: a scalar load would be waited for by
// the next LDS wait (both count in lgkmcnt).  Offsets past the end read 0.
// Only lane 0 loads (the value is the same for every lane; uniform() reads
// lane 0 once the loads have landed).
__device__ __forceinline__ Meta load_meta(__amdgpu_buffer_rsrc_t so, __amdgpu_buffer_rsrc_t cn, int64_t k, int lane) {
  Meta m{0, 0, 0};
  if (lane == 0) {
    m.soff = ld_i32(so, uint32_t(k) * 4u);
    m.uc = ld_i32(cn, uint32_t(k) * 8u);
    m.uh = ld_i32(cn, uint32_t(k) * 8u + 4u);
  }
  return m;
}

__device__ __forceinline__ Meta uniform(const Meta& m) {
  return Meta{__builtin_amdgcn_readfirstlane(m.soff), __builtin_amdgcn_readfirstlane(m.uc),
              __builtin_amdgcn_readfirstlane(m.uh)};
}

// One lane's share of a fast-path row from the packed (code, value) plan:
// entries sub, sub+16, ...; an entry that no row of the wave reaches is not
// loaded at all (wmax = longest row of the wave).
template <int E>
__device__ __forceinline__ void load_packed(__amdgpu_buffer_rsrc_t pk, long long seg, const RowInfo& r, bool valid,
                                            int sub, DataReg<E>& d) {
  const int len = valid ? r.len : 0;
  int wmax = max(max(__builtin_amdgcn_readlane(len, 0), __builtin_amdgcn_readlane(len, 16)),
                 max(__builtin_amdgcn_readlane(len, 32), __builtin_amdgcn_readlane(len, 48)));
  const uint32_t st = uint32_t(r.start - seg);
  d.ok = len > 0 ? kRowExists : 0u;
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const int e = sub + kRowLanes * j;
    d.code[j] = -1;
    d.val[j] = 0.f;
    if (kRowLanes * j < wmax) {
      const uint32_t q = e < len ? st + uint32_t(e) : 0u;
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(pk, q * 8u, 0, 0);
      // element values are copied out before any reinterpretation: a
      // __builtin_bit_cast of a vector element reads element 0's bytes
      const unsigned int c0 = v[0], v1 = v[1];
      d.code[j] = int(c0);
      d.val[j] = __uint_as_float(v1);
    }
    d.ok |= uint32_t(e < len) << j;
  }
  d.y = r.y;
}

// Empty asm that takes every element: the loads that produce them are all
// issued before it, and their results are waited for once.
template <int N>
__device__ __forceinline__ void hold(float (&v)[N]) {
  static_assert(N >= 1 && N <= 8, "hold: 1..8 values");
  if constexpr (N == 1) asm volatile("" : "+v"(v[0]));
  if constexpr (N == 2) asm volatile("" : "+v"(v[0]), "+v"(v[1]));
  if constexpr (N == 3) asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]));
  if constexpr (N == 4) asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
  if constexpr (N == 5) asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]));
  if constexpr (N == 6) asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]));
  if constexpr (N == 7)
    asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]));
  if constexpr (N == 8)
    asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]));
}

constexpr uint32_t kPrefetchSpin = 1u << 16;  // polls of the pass's progress per step (bounded)
constexpr int kPrefetchLead = 3;              // steps ahead of the pass

// Prefetch workgroup of worker i (on the pass's XCD): what step k of the
// pass reads -- its rows' (code, value) pairs, its lists and the model
// entries of its cold columns -- is loaded into the XCD's L2 while the pass
// is at step k - 2, one step before the pass loads it itself.  A random
// 4-byte model read costs a whole line from memory, and one compute unit
// only has so many in flight: the pass's step time was bound by them.  This
// workgroup only loads (the values are discarded) and waits for the pass
// with a bounded spin, so it cannot change any result.
template <int E>
__device__ void prefetch_pass(const SgdArgs& a, const PlanArgs& p, int i) {
  const int tid = threadIdx.x, sub = tid & (kRowLanes - 1), b = tid / kRowLanes;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  const RowInfo* ri = a.rowinfo + int64_t(i) * a.S;
  const long long seg = a.row_ptr[int64_t(i) * a.S];
  const uint32_t nnz_w = uint32_t(a.row_ptr[int64_t(i + 1) * a.S] - seg);
  const auto pk = rsrc(p.pack + seg, nnz_w * 8u);
  const auto model = rsrc(a.models + int64_t(i) * a.ld, uint32_t(a.dim) * 4u);
  const auto clist = rsrc(p.clist + seg, nnz_w * 4u);
  const auto clink = rsrc(p.clink + seg, nnz_w * 4u);
  const auto hlist = rsrc(p.hlist + seg, nnz_w * 4u);
  const auto so_v = rsrc(p.step_off + int64_t(i) * (a.S + 1), uint32_t(a.k1) * 4u);
  const auto cn_v = rsrc(p.cnt + int64_t(i) * K * 2, uint32_t(a.k1) * 8u);
  const int64_t base = a.round * K;
  float sink = 0.f;
  for (int64_t k = a.k0 + 2; k < a.k1; ++k) {
    if (tid == 0) {
      uint32_t spins = 0;
      while (__hip_atomic_load(p.progress + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < base + k - kPrefetchLead &&
             ++spins < kPrefetchSpin)
        __builtin_amdgcn_s_sleep(4);
    }
    __syncthreads();
    const int soff = ld_i32(so_v, uint32_t(k) * 4u);
    const int uc = ld_i32(cn_v, uint32_t(k) * 8u), uh = ld_i32(cn_v, uint32_t(k) * 8u + 4u);
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < kColdPer; ++j) {
      const int u = tid + j * kThreads;
      if (u < uc) {
        const int col = ld_i32(clist, uint32_t(soff + u) * 4u);
        acc += ld_f32(model, uint32_t(col) * 4u) + float(ld_i32(clink, uint32_t(soff + u) * 4u));
      }
    }
#pragma unroll
    for (int j = 0; j < kHotPer; ++j) {
      const int u = tid + j * kThreads;
      if (u < uh) acc += float(ld_i32(hlist, uint32_t(soff + u) * 4u));
    }
    if (b < a.batch && k * a.batch + b < a.S) {
      const RowInfo r = ri[k * a.batch + b];
      const uint32_t st = uint32_t(r.start - seg);
      for (int e = sub; e < r.len; e += kRowLanes) acc += __int_as_float(ld_i32(pk, (st + uint32_t(e)) * 8u));
    }
    sink += acc;
  }
  asm volatile("" ::"v"(sink));
}

template <int E>
__global__ __launch_bounds__(kThreads) void sgd_csr_fast_kernel(SgdArgs a, PlanArgs p) {
  if (*p.flag) return;  // the general kernel takes this round
  if (int(blockIdx.x) >= a.n) {
    prefetch_pass<E>(a, p, int(blockIdx.x) - a.n);
    return;
  }
  __shared__ FastShared sh;
  const int i = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & (kRowLanes - 1);
  const int brow = wave * (64 / kRowLanes) + (lane / kRowLanes);
  float* vrow = a.models + int64_t(i) * a.ld;
  const RowInfo* ri = a.rowinfo + int64_t(i) * a.S;
  const int H = a.n_hot;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  const int64_t k0 = a.k0, kend = a.k1;  // steps [k0, kend) of the pass run here
  Views w;
  w.seg = a.row_ptr[int64_t(i) * a.S];
  const uint32_t nnz_w = uint32_t(a.row_ptr[int64_t(i + 1) * a.S] - w.seg);
  const auto pk = rsrc(p.pack + w.seg, nnz_w * 8u);
  w.model = rsrc(vrow, uint32_t(a.dim) * 4u);
  const auto clist = rsrc(p.clist + w.seg, nnz_w * 4u);
  const auto clink = rsrc(p.clink + w.seg, nnz_w * 4u);
  const auto hlist = rsrc(p.hlist + w.seg, nnz_w * 4u);
  const auto so_v = rsrc(p.step_off + int64_t(i) * (a.S + 1), uint32_t(a.k1) * 4u);  // steps past the launch read 0
  const auto cn_v = rsrc(p.cnt + int64_t(i) * K * 2, uint32_t(a.k1) * 8u);

  for (int h = tid; h < H; h += kThreads) {
    sh.vhot[h] = vrow[a.hot_cols[h]];
    sh.acch[h] = 0ull;
  }
  for (int q = tid; q < kCMax; q += kThreads) sh.cacc[q] = 0ull;
  // fixed point as in the general kernel: |column sum| <= B vmax < 2^e
  int e2 = 0;
  frexp(double(a.batch) * double(a.vmax[i]), &e2);
  const double to_fx = ldexp(1.0, 61 - e2), from_fx = ldexp(1.0, e2 - 61);
  double s = 1.0;  // w = s * v

  // Pipeline at the top of step k: d0 = nonzeros of step k, r1 = row of
  // step k+1; m0..m2 = constants of steps k..k+2; cl0/lk0/g0/hl0 = cold
  // columns, links, gathered values and hot slots of step k, cl1 = cold
  // columns of step k+1.  Step k loads d1, r2, m3, g1 (from cl1), cl2, lk1
  // and hl1, rotated in after the end-of-step fence.  Nothing a step loads
  // is used in the same step: vector loads complete in order, so waiting
  // for any of them would also wait for that step's model gathers.
  RowInfo r1, r2;
  DataReg<E> d0, d1;
  Meta m0, m1, m2, m3;
  int cl0[kColdPer], lk0[kColdPer], cl1[kColdPer], lk1[kColdPer], cl2[kColdPer];
  float g0[kColdPer], g1[kColdPer];
  int hl0[kHotPer], hl1[kHotPer];
  // list loads: a wave whose first slot is past the count issues nothing
  const int wave0 = __builtin_amdgcn_readfirstlane(wave * 64);
  auto load_cols = [&](const Meta& m, int (&cl)[kColdPer]) {
#pragma unroll
    for (int j = 0; j < kColdPer; ++j) {
      const int u = tid + j * kThreads;
      cl[j] = 0;
      if (wave0 + j * kThreads < m.uc) cl[j] = ld_i32(clist, uint32_t(m.soff + (u < m.uc ? u : 0)) * 4u);
    }
  };
  auto load_links = [&](const Meta& m, int (&lk)[kColdPer]) {
#pragma unroll
    for (int j = 0; j < kColdPer; ++j) {
      const int u = tid + j * kThreads;
      lk[j] = -1;
      if (wave0 + j * kThreads < m.uc) lk[j] = ld_i32(clink, uint32_t(m.soff + (u < m.uc ? u : 0)) * 4u);
    }
  };
  auto load_hot = [&](const Meta& m, int (&hl)[kHotPer]) {
#pragma unroll
    for (int j = 0; j < kHotPer; ++j) {
      const int u = tid + j * kThreads;
      hl[j] = 0;
      if (wave0 + j * kThreads < m.uh) hl[j] = ld_i32(hlist, uint32_t(m.soff + (u < m.uh ? u : 0)) * 4u);
    }
  };
  auto gather = [&](const Meta& m, const int (&cl)[kColdPer], float (&g)[kColdPer]) {
#pragma unroll
    for (int j = 0; j < kColdPer; ++j) {
      const int u = tid + j * kThreads;
      g[j] = 0.f;
      if (wave0 + j * kThreads < m.uc) g[j] = ld_f32(w.model, uint32_t(u < m.uc ? cl[j] : 0) * 4u);
    }
  };
  {
    const RowInfo ra = load_row(a, ri, k0, kend, brow);
    r1 = load_row(a, ri, k0 + 1, kend, brow);
    m0 = load_meta(so_v, cn_v, k0, lane);
    m1 = load_meta(so_v, cn_v, k0 + 1, lane);
    m2 = load_meta(so_v, cn_v, k0 + 2, lane);
    m0 = uniform(m0);
    m1 = uniform(m1);
    m2 = uniform(m2);
    __syncthreads();
    load_packed<E>(pk, w.seg, ra, row_valid(a, k0, kend, brow), sub, d0);
    load_cols(m0, cl0);
    load_links(m0, lk0);
    load_cols(m1, cl1);
    load_hot(m0, hl0);
    __syncthreads();
    gather(m0, cl0, g0);
  }
  __syncthreads();

  for (int64_t k = k0; k < kend; ++k) {
    if (p.helpers && tid == 0)
      __hip_atomic_store(p.progress + i, a.round * K + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (k > k0) {  // rotate what the previous step loaded
      d0 = d1;
      r1 = r2;
      m0 = m1;
      m1 = m2;
      m2 = uniform(m3);  // loaded by the previous step, landed at its fence
#pragma unroll
      for (int j = 0; j < kColdPer; ++j) {
        cl0[j] = cl1[j];
        lk0[j] = lk1[j];
        g0[j] = g1[j];
        cl1[j] = cl2[j];
      }
#pragma unroll
      for (int j = 0; j < kHotPer; ++j) hl0[j] = hl1[j];
    }
    const int64_t b0 = k * a.batch;
    const int Bp = int(min(int64_t(a.batch), a.S - b0));
    const double eta = step_size(a.lr_kind, a.lr0, a.round * K + k + 1);
    const double s_new = s * (1.0 - eta * double(a.l2));
    const double coefA = eta / (double(Bp) * s_new);
    float* cv = sh.cval[k & 1];
    const float* cvp = sh.cval[(k + 1) & 1];

    // cold values of this step: changed by the previous step of this
    // launch -> its slot, else the value gathered a step ago (the first step
    // of a launch gathers them all: the launch before wrote them back)
#pragma unroll
    for (int j = 0; j < kColdPer; ++j) {
      const int u = tid + j * kThreads;
      if (u < m0.uc) cv[u] = (k > k0 && lk0[j] >= 0) ? cvp[lk0[j]] : g0[j];
    }
    lds_barrier();
    // prefetch, issued after the barrier so that the address work of some
    // waves overlaps the LDS work of others: nonzeros, links, hot slots and
    // values of k+1, row and columns of k+2
    load_hot(m1, hl1);
    load_packed<E>(pk, w.seg, r1, row_valid(a, k + 1, kend, brow), sub, d1);
    r2 = load_row(a, ri, k + 2, kend, brow);
    m3 = load_meta(so_v, cn_v, k + 3, lane);
    gather(m1, cl1, g1);
    load_links(m1, lk1);
    load_cols(m2, cl2);
    asm volatile("" ::: "memory");  // keep the prefetch issued here, ahead of the LDS work

    // one LDS read per entry, its address chosen by the code (a read per
    // branch would serialise on the shared destination register); all reads
    // are issued before the first is used.  An absent entry reads cold slot 0,
    // which may hold anything, and its value is replaced by zero.
    float v[E];
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int code = code_at(d0, j);
      v[j] = is_hot(code) ? sh.vhot[hot_slot(code)] : cv[code < 0 ? 0 : code];
    }
    hold(v);
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < E; ++j) part = fma(double(d0.val[j]), double(code_at(d0, j) == -1 ? 0.f : v[j]), part);
    const double dot = row16_sum(part);
    const double cf = (d0.ok & kRowExists) ? loss_coef(s * dot, double(d0.y), a.loss) : 0.0;
    if (cf != 0.0) {
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const int code = code_at(d0, j);
        if (code == -1) continue;
        const long long q = llrint(cf * double(d0.val[j]) * to_fx);
        unsigned long long* dst = is_hot(code) ? &sh.acch[hot_slot(code)] : &sh.cacc[code];
        atomicAdd(dst, static_cast<unsigned long long>(q));
      }
    }
    lds_barrier();

    // update: all accumulator and value reads of a thread first, then the
    // writes (a wave whose first slot is past the count skips a slot)
    {
      unsigned long long acc[kHotPer + kColdPer];
      float old[kHotPer + kColdPer];
#pragma unroll
      for (int j = 0; j < kHotPer; ++j) {
        acc[j] = 0ull;
        old[j] = 0.f;
        if (wave0 + j * kThreads < m0.uh) {
          acc[j] = sh.acch[hl0[j]];
          old[j] = sh.vhot[hl0[j]];
        }
      }
#pragma unroll
      for (int j = 0; j < kColdPer; ++j) {
        const int u = tid + j * kThreads;
        acc[kHotPer + j] = 0ull;
        old[kHotPer + j] = 0.f;
        if (wave0 + j * kThreads < m0.uc) {
          acc[kHotPer + j] = sh.cacc[u];
          old[kHotPer + j] = cv[u];
        }
      }
      static_assert(kHotPer + kColdPer == 4, "update batch holds four slots");
      asm volatile("" : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(old[0]), "+v"(old[1]),
                   "+v"(old[2]), "+v"(old[3]));
#pragma unroll
      for (int j = 0; j < kHotPer; ++j) {
        const int u = tid + j * kThreads;
        if (u < m0.uh && acc[j] != 0ull) {
          const int h = hl0[j];
          sh.vhot[h] = float(double(old[j]) - coefA * double(static_cast<long long>(acc[j])) * from_fx);
          sh.acch[h] = 0ull;
        }
      }
#pragma unroll
      for (int j = 0; j < kColdPer; ++j) {
        const int u = tid + j * kThreads;
        if (u < m0.uc && acc[kHotPer + j] != 0ull) {
          const float nv =
              float(double(old[kHotPer + j]) - coefA * double(static_cast<long long>(acc[kHotPer + j])) * from_fx);
          cv[u] = nv;
          sh.cacc[u] = 0ull;
          st_f32(w.model, uint32_t(cl0[j]) * 4u, nv);
        }
      }
    }

    s = s_new;
    if (s < 1e-6) {  // fold the scale back into v before it underflows
      const float sf = float(s);
      __syncthreads();
      for (int h = tid; h < H; h += kThreads) sh.vhot[h] *= sf;
      for (int64_t c = tid; c < a.dim; c += kThreads) vrow[c] *= sf;
#pragma unroll
      for (int j = 0; j < kColdPer; ++j) {
        const int u = tid + j * kThreads;
        if (u < m0.uc) cv[u] *= sf;  // the next step links to these
        g1[j] *= sf;                 // gathered before the fold
      }
      s = 1.0;
    }
    __syncthreads();  // full fence: model stores complete, LDS updates visible
  }

  for (int h = tid; h < H; h += kThreads) vrow[a.hot_cols[h]] = sh.vhot[h];
  if (tid == 0) {
    a.scale[i] = float(s);
    a.tag[i] = a.tag_value;
    if (p.helpers)
      __hip_atomic_store(p.progress + i, a.round * K + kend, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__global__ void pack_values_kernel(const int32_t* __restrict__ code, const float* __restrict__ val, int64_t nnz,
                                   int2* __restrict__ pack) {
  for (int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; q < nnz; q += int64_t(gridDim.x) * blockDim.x)
    pack[q] = make_int2(code[q], __float_as_int(val[q]));
}

template <int E>
hipError_t launch_fast_e(const SgdArgs& a, const PlanArgs& p, hipStream_t s) {
  // with helpers, block n + i prefetches for block i: the same XCD when n is
  // a multiple of the 8 XCDs (blocks are dealt to them round-robin)
  const uint32_t grid = uint32_t(a.n) * (p.helpers ? 2u : 1u);
  hipLaunchKernelGGL((sgd_csr_fast_kernel<E>), dim3(grid), dim3(kThreads), 0, s, a, p);
  return hipGetLastError();
}

}  // namespace

bool csr_plan_fits(const SgdArgs& a) {
  return a.batch <= kFastRows && a.max_row <= kRowLanes * 8 && a.n_hot <= kHotMax;
}

hipError_t launch_csr_plan(const PlanArgs& p, int max_row, hipStream_t s) {
  const uint32_t blocks = uint32_t(int64_t(p.n) * p.K);
  hipLaunchKernelGGL(step_scan_kernel, dim3(uint32_t(p.n)), dim3(kScanThreads), 0, s, p);
  // the largest step holds at most batch * max_row nonzeros
  const int64_t most = 2 * int64_t(std::min(p.batch, kFastRows)) * max_row;
  // rows of at most 64 nonzeros: one per lane and 256 threads (a small
  // step leaves most of a larger block idle); else two and 512
  if (max_row <= 64) {
    if (most <= (1 << 10))
      hipLaunchKernelGGL((csr_plan_kernel<10, 256, 1>), dim3(blocks), dim3(256), 0, s, p);
    else if (most <= (1 << 11))
      hipLaunchKernelGGL((csr_plan_kernel<11, 256, 1>), dim3(blocks), dim3(256), 0, s, p);
    else if (most <= (1 << 12))
      hipLaunchKernelGGL((csr_plan_kernel<12, 256, 1>), dim3(blocks), dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((csr_plan_kernel<13, 256, 1>), dim3(blocks), dim3(256), 0, s, p);
  } else {
    if (most <= (1 << 10))
      hipLaunchKernelGGL((csr_plan_kernel<10, kPlanThreads, 2>), dim3(blocks), dim3(kPlanThreads), 0, s, p);
    else if (most <= (1 << 11))
      hipLaunchKernelGGL((csr_plan_kernel<11, kPlanThreads, 2>), dim3(blocks), dim3(kPlanThreads), 0, s, p);
    else if (most <= (1 << 12))
      hipLaunchKernelGGL((csr_plan_kernel<12, kPlanThreads, 2>), dim3(blocks), dim3(kPlanThreads), 0, s, p);
    else
      hipLaunchKernelGGL((csr_plan_kernel<13, kPlanThreads, 2>), dim3(blocks), dim3(kPlanThreads), 0, s, p);
  }
  if (max_row <= 64)
    hipLaunchKernelGGL(csr_link_kernel<256>, dim3(blocks), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(csr_link_kernel<kPlanThreads>, dim3(blocks), dim3(kPlanThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_pack_values(const int32_t* code, const float* val, int64_t nnz, int2* pack, hipStream_t s) {
  if (nnz <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((nnz + 255) / 256, 65536);
  hipLaunchKernelGGL(pack_values_kernel, dim3(uint32_t(blocks)), dim3(256), 0, s, code, val, nnz, pack);
  return hipGetLastError();
}

hipError_t launch_sgd_csr_fast(const SgdArgs& a, const PlanArgs& p, hipStream_t s) {
  if (a.max_row <= kRowLanes * 2) return launch_fast_e<2>(a, p, s);
  if (a.max_row <= kRowLanes * 3) return launch_fast_e<3>(a, p, s);
  if (a.max_row <= kRowLanes * 4) return launch_fast_e<4>(a, p, s);
  if (a.max_row <= kRowLanes * 6) return launch_fast_e<6>(a, p, s);
  return launch_fast_e<8>(a, p, s);
}

}  // namespace asap
