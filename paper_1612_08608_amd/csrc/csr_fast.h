// csr_fast.h -- the CSR SGD pass on a column plan (Appendix A, update (A.2),
// first line), as a device function: the stream-ordered planned kernel and
// the multi-round launch both run it.  The plan (kernels_csr_plan.hip) gives,
// for every step of a worker's pass, its distinct cold columns and hot
// slots, each nonzero's slot code, and each cold column's slot in the
// previous step.  The pass keeps the step's cold values in LDS slots: they
// are gathered from the model a step ahead, and a value the previous step
// changed is taken from that step's slot through the link.  Margins read
// LDS, gradients are added to slot accumulators with integer atomics (no
// hashing, no CAS), and the update walks the step's slot lists.
#pragma once

#include <cmath>

#include "asap_launch.h"
#include "csr_device.h"

namespace asap {
namespace csr {

constexpr int kCMax = 2048;                  // cold slots per step held in LDS
constexpr int kHList = 2048;                 // hot slots per step applied from registers
constexpr int kColdPer = kCMax / kThreads;   // 2
constexpr int kHotPer = kHList / kThreads;   // 2

struct FastShared {
  float vhot[kHotMax];
  unsigned long long acch[kHotMax];
  float cval[2][kCMax];  // cold values of steps k (slot k & 1) and k - 1
  unsigned long long cacc[kCMax];
  int xabort;            // members: a partner's partial margin did not arrive in time
  int xlocal;            // members: all of this worker's members run on this XCD
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

// Worker i and member m of workgroup b (grid n * members): a worker's
// members on one XCD when the grid allows (workgroups are dealt to the 8
// XCDs round-robin), so that their exchange stays in one L2.
__device__ __forceinline__ void member_of(int b, int n, int M, int& i, int& m) {
  if (M == 1) {
    i = b;
    m = 0;
  } else if (n % 8 == 0) {
    const int j = b / 8;
    i = (b % 8) * (n / 8) + j / M;
    m = j % M;
  } else {
    i = b / M;
    m = b % M;
  }
}

// hold() for 64-bit values
template <int N>
__device__ __forceinline__ void hold_u64(unsigned long long (&v)[N]) {
  static_assert(N == 4 || N == 8, "hold_u64: 4 or 8 values");
  if constexpr (N == 4) asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
  if constexpr (N == 8)
    asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                 "+v"(v[7]));
}

constexpr uint32_t kPrefetchSpin = 1u << 16;  // polls of the pass's progress per step (bounded)
constexpr int kPrefetchLead = 3;              // steps ahead of the pass

// Prefetch workgroup of slice v of worker i (on the XCD of the slice's
// pass): what step k of the pass reads -- its rows' (code, value) pairs, its
// lists and the model entries of its cold columns -- is loaded into the
// XCD's L2 while the pass is at step k - 2, one step before the pass loads
// it itself.  A random
// 4-byte model read costs a whole line from memory, and one compute unit
// only has so many in flight: the pass's step time was bound by them.  This
// workgroup only loads (the values are discarded) and waits for the pass
// with a bounded spin, so it cannot change any result.
template <int E>
__device__ void prefetch_pass(const SgdArgs& a, const PlanArgs& p, int v, int i) {
  const int tid = threadIdx.x, sub = tid & (kRowLanes - 1), b = tid / kRowLanes;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  const RowInfo* ri = p.rowinfo + int64_t(v) * a.S;
  const long long seg = p.row_ptr[int64_t(v) * a.S];
  const uint32_t nnz_w = uint32_t(p.row_ptr[int64_t(v + 1) * a.S] - seg);
  const auto pk = rsrc(p.pack + seg, nnz_w * 8u);
  const auto model = rsrc(a.models + int64_t(i) * a.ld, uint32_t(a.dim) * 4u);
  const auto clist = rsrc(p.clist + seg, nnz_w * 4u);
  const auto clink = rsrc(p.clink + seg, nnz_w * 4u);
  const auto hlist = rsrc(p.hlist + seg, nnz_w * 4u);
  const auto so_v = rsrc(p.step_off + int64_t(v) * (a.S + 1), uint32_t(a.k1) * 4u);
  const auto cn_v = rsrc(p.cnt + int64_t(v) * K * 2, uint32_t(a.k1) * 8u);
  const int64_t base = a.round * K;
  float sink = 0.f;
  for (int64_t k = a.k0 + 2; k < a.k1; ++k) {
    if (tid == 0) {
      uint32_t spins = 0;
      while (__hip_atomic_load(p.progress + v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < base + k - kPrefetchLead &&
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

// Members (p.members > 1): the partial margins of one step are exchanged
// through p.xch, two tagged 64-bit words per (member, row): the low and
// the high half of the fp64 partial, each beside the step's 32-bit tag, so
// a word is whole or stale, never torn, and no fence or counter is needed.
// Lanes 0, 1 of each 16-lane row publish; lanes 2 m', 2 m' + 1 read member
// m''s halves (a bounded wait), and every lane of the row adds the members'
// partials in member order, so all members get the same margin bit for bit.
// Reads are device-scope (a narrower load may be served by a stale line of
// the reader's L1).  Members on one XCD write with plain stores, which the
// L1 writes through to the XCD's shared L2 where the readers find them;
// members on several XCDs write device-scope, past the L2.
__device__ __forceinline__ double member_exchange(const PlanArgs& p, __amdgpu_buffer_rsrc_t xr, int m, int brow,
                                                  int lane, uint32_t tag, double part, bool live, bool local,
                                                  FastShared& sh) {
  typedef unsigned int v2u __attribute__((ext_vector_type(2)));
  const int M = p.members, sub = lane & (kRowLanes - 1), mm = sub >> 1;
  const uint32_t slot = (tag & 1u) * uint32_t(M) * 128u;  // words
  const uint32_t lo = uint32_t(__double2loint(part)), hi = uint32_t(__double2hiint(part));
  if (live && sub < 2) {
    const v2u word = {sub ? hi : lo, tag};
    const uint32_t off = (slot + uint32_t((m * 64 + brow) * 2 + sub)) * 8u;
    if (local)
      __builtin_amdgcn_raw_buffer_store_b64(word, xr, off, 0, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b64(word, xr, off, 0, 16);  // sc1: device scope
  }
  uint32_t half = 0;
  if (live && mm < M) {
    if (mm == m) {
      half = (sub & 1) ? hi : lo;
    } else {
      const uint32_t off = (slot + uint32_t((mm * 64 + brow) * 2 + (sub & 1))) * 8u;
      auto load = [&]() {
        asm volatile("" ::: "memory");  // a fresh load every poll
        return __builtin_amdgcn_raw_buffer_load_b64(xr, off, 0, 16);  // sc1: device scope
      };
      v2u w = load();
      if (uint32_t(w[1]) != tag) {
        const long long deadline = wall_clock64() + p.xwait;
        do {
          __builtin_amdgcn_s_sleep(1);
          w = load();
        } while (uint32_t(w[1]) != tag && wall_clock64() < deadline);
        if (uint32_t(w[1]) != tag) {
          sh.xabort = 1;
          atomicAdd(p.xerr, 1);
        }
      }
      half = uint32_t(w[0]);
    }
  }
  const int base = lane & ~(kRowLanes - 1);
  double dot = 0.0;
  for (int q = 0; q < M; ++q) {
    const int l = __shfl(int(half), base + 2 * q, 64);
    const int h = __shfl(int(half), base + 2 * q + 1, 64);
    dot += __hiloint2double(h, l);
  }
  return dot;
}

// Member m of worker i: its slice's planned pass (steps [a.k0, a.k1) of
// pass a.round on the plan p); `sh` is the workgroup's LDS for it.  Member 0
// writes the final L2 scale, and the epoch tag when a.tag is set.  MEM:
// p.members > 1 (with one member the slice is the whole worker and nothing
// is exchanged).
template <int E, bool MEM, int NT = kThreads>
__device__ void fast_pass(const SgdArgs& a, const PlanArgs& p, int i, int m, FastShared& sh) {
  constexpr int CP = kCMax / NT, HP = kHList / NT;  // cold and hot list slots per thread
  static_assert(NT % 64 == 0 && kCMax % NT == 0 && kHList % NT == 0, "fast_pass: thread count");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane & (kRowLanes - 1);
  const int brow = wave * (64 / kRowLanes) + (lane / kRowLanes);
  const int M = MEM ? p.members : 1, v = i * M + m;
  float* vrow = a.models + int64_t(i) * a.ld;
  const RowInfo* ri = p.rowinfo + int64_t(v) * a.S;
  const int H = p.n_mhot[m];
  const int32_t* hot_cols = p.mhot + m * kHotMax;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  const int64_t k0 = a.k0, kend = a.k1;  // steps [k0, kend) of the pass run here
  Views w;
  w.seg = p.row_ptr[int64_t(v) * a.S];
  const uint32_t nnz_w = uint32_t(p.row_ptr[int64_t(v + 1) * a.S] - w.seg);
  const auto pk = rsrc(p.pack + w.seg, nnz_w * 8u);
  w.model = rsrc(vrow, uint32_t(a.dim) * 4u);
  const auto clist = rsrc(p.clist + w.seg, nnz_w * 4u);
  const auto clink = rsrc(p.clink + w.seg, nnz_w * 4u);
  const auto hlist = rsrc(p.hlist + w.seg, nnz_w * 4u);
  const auto so_v = rsrc(p.step_off + int64_t(v) * (a.S + 1), uint32_t(a.k1) * 4u);  // steps past the launch read 0
  const auto cn_v = rsrc(p.cnt + int64_t(v) * K * 2, uint32_t(a.k1) * 8u);
  // members: this worker's exchange words, [2][M][64][2] (unused with one member)
  const auto xr = rsrc(MEM ? p.xch + size_t(i) * size_t(M) * 256u : nullptr, MEM ? uint32_t(M) * 2048u : 0u);

  for (int h = tid; h < H; h += NT) {
    sh.vhot[h] = vrow[hot_cols[h]];
    sh.acch[h] = 0ull;
  }
  for (int q = tid; q < kCMax; q += NT) sh.cacc[q] = 0ull;
  bool local = false;
  if (tid == 0) {
    sh.xabort = 0;
    sh.xlocal = 0;
    if constexpr (MEM) {
      // the members publish their XCD, tagged with the pass's first step,
      // and see whether all of them share one
      const uint32_t tag0 = a.xtag + uint32_t(a.round * K + k0 - a.xg0);
      const uint32_t me = uint32_t(xcd_id());
      unsigned long long* xid = p.xid + size_t(i) * size_t(M);
      __hip_atomic_store(xid + m, (static_cast<unsigned long long>(tag0) << 32) | me, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      const long long deadline = wall_clock64() + p.xwait;
      int same = 1;
      for (int q = 0; q < M; ++q) {
        unsigned long long w;
        while (uint32_t((w = __hip_atomic_load(xid + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) >> 32) != tag0) {
          if (wall_clock64() > deadline) break;
          __builtin_amdgcn_s_sleep(2);
        }
        if (uint32_t(w >> 32) != tag0) {
          sh.xabort = 1;
          atomicAdd(p.xerr, 1);
        }
        same &= uint32_t(w) == me;
      }
      sh.xlocal = same;
    }
  }
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
  int cl0[CP], lk0[CP], cl1[CP], lk1[CP], cl2[CP];
  float g0[CP], g1[CP];
  int hl0[HP], hl1[HP];
  // list loads: a wave whose first slot is past the count issues nothing
  const int wave0 = __builtin_amdgcn_readfirstlane(wave * 64);
  auto load_cols = [&](const Meta& m, int (&cl)[CP]) {
#pragma unroll
    for (int j = 0; j < CP; ++j) {
      const int u = tid + j * NT;
      cl[j] = 0;
      if (wave0 + j * NT < m.uc) cl[j] = ld_i32(clist, uint32_t(m.soff + (u < m.uc ? u : 0)) * 4u);
    }
  };
  auto load_links = [&](const Meta& m, int (&lk)[CP]) {
#pragma unroll
    for (int j = 0; j < CP; ++j) {
      const int u = tid + j * NT;
      lk[j] = -1;
      if (wave0 + j * NT < m.uc) lk[j] = ld_i32(clink, uint32_t(m.soff + (u < m.uc ? u : 0)) * 4u);
    }
  };
  auto load_hot = [&](const Meta& m, int (&hl)[HP]) {
#pragma unroll
    for (int j = 0; j < HP; ++j) {
      const int u = tid + j * NT;
      hl[j] = 0;
      if (wave0 + j * NT < m.uh) hl[j] = ld_i32(hlist, uint32_t(m.soff + (u < m.uh ? u : 0)) * 4u);
    }
  };
  auto gather = [&](const Meta& m, const int (&cl)[CP], float (&g)[CP]) {
#pragma unroll
    for (int j = 0; j < CP; ++j) {
      const int u = tid + j * NT;
      g[j] = 0.f;
      if (wave0 + j * NT < m.uc) g[j] = ld_f32(w.model, uint32_t(u < m.uc ? cl[j] : 0) * 4u);
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
    local = sh.xlocal != 0;
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
      __hip_atomic_store(p.progress + v, a.round * K + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (k > k0) {  // rotate what the previous step loaded
      d0 = d1;
      r1 = r2;
      m0 = m1;
      m1 = m2;
      m2 = uniform(m3);  // loaded by the previous step, landed at its fence
#pragma unroll
      for (int j = 0; j < CP; ++j) {
        cl0[j] = cl1[j];
        lk0[j] = lk1[j];
        g0[j] = g1[j];
        cl1[j] = cl2[j];
      }
#pragma unroll
      for (int j = 0; j < HP; ++j) hl0[j] = hl1[j];
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
    for (int j = 0; j < CP; ++j) {
      const int u = tid + j * NT;
      if (u < m0.uc) cv[u] = (k > k0 && lk0[j] >= 0) ? cvp[lk0[j]] : g0[j];
    }
    lds_barrier();
    // prefetch: nonzeros, links, hot slots and values of k+1, row and
    // columns of k+2, issued here, after the barrier, so that the address
    // work of some waves overlaps the LDS work of others.  The loads whose
    // results the next step's prefetch needs (metadata, rows, columns) go
    // first and the random model gathers last, so that waiting for the
    // former (loads complete in order) does not wait for the gathers (256
    // workers: pass 0.96 -> 0.94 ms with this order).  Members issue the
    // gathers after their exchange, whose polls (vector loads) would
    // otherwise wait for them (64 workers x 2 members: pass 2.30 -> 2.12 ms).
    m3 = load_meta(so_v, cn_v, k + 3, lane);
    r2 = load_row(a, ri, k + 2, kend, brow);
    load_cols(m2, cl2);
    load_packed<E>(pk, w.seg, r1, row_valid(a, k + 1, kend, brow), sub, d1);
    load_links(m1, lk1);
    load_hot(m1, hl1);
    auto gather_next = [&]() {
      gather(m1, cl1, g1);
      asm volatile("" ::: "memory");  // keep the gathers issued here, ahead of the LDS work
    };
    if constexpr (!MEM) gather_next();

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
    double dot = row16_sum(part);
    if constexpr (MEM)
      dot = member_exchange(p, xr, m, brow, lane, a.xtag + uint32_t(a.round * K + k - a.xg0), dot,
                            row_valid(a, k, kend, brow), local, sh);
    if constexpr (MEM) gather_next();
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
      unsigned long long acc[HP + CP];
      float old[HP + CP];
#pragma unroll
      for (int j = 0; j < HP; ++j) {
        acc[j] = 0ull;
        old[j] = 0.f;
        if (wave0 + j * NT < m0.uh) {
          acc[j] = sh.acch[hl0[j]];
          old[j] = sh.vhot[hl0[j]];
        }
      }
#pragma unroll
      for (int j = 0; j < CP; ++j) {
        const int u = tid + j * NT;
        acc[HP + j] = 0ull;
        old[HP + j] = 0.f;
        if (wave0 + j * NT < m0.uc) {
          acc[HP + j] = sh.cacc[u];
          old[HP + j] = cv[u];
        }
      }
      hold_u64(acc);
      hold(old);
#pragma unroll
      for (int j = 0; j < HP; ++j) {
        const int u = tid + j * NT;
        if (u < m0.uh && acc[j] != 0ull) {
          const int h = hl0[j];
          sh.vhot[h] = float(double(old[j]) - coefA * double(static_cast<long long>(acc[j])) * from_fx);
          sh.acch[h] = 0ull;
        }
      }
#pragma unroll
      for (int j = 0; j < CP; ++j) {
        const int u = tid + j * NT;
        if (u < m0.uc && acc[HP + j] != 0ull) {
          const float nv =
              float(double(old[HP + j]) - coefA * double(static_cast<long long>(acc[HP + j])) * from_fx);
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
      for (int h = tid; h < H; h += NT) sh.vhot[h] *= sf;
      for (int64_t c = m + int64_t(tid) * M; c < a.dim; c += int64_t(NT) * M) vrow[c] *= sf;  // own columns
#pragma unroll
      for (int j = 0; j < CP; ++j) {
        const int u = tid + j * NT;
        if (u < m0.uc) cv[u] *= sf;  // the next step links to these
        g1[j] *= sf;                 // gathered before the fold
      }
      s = 1.0;
    }
    __syncthreads();  // full fence: model stores complete, LDS updates visible
    if constexpr (MEM)
      if (sh.xabort) break;  // reported through p.xerr; the partners time out too
  }

  for (int h = tid; h < H; h += NT) vrow[hot_cols[h]] = sh.vhot[h];
  if (tid == 0) {
    if (m == 0) {
      a.scale[i] = float(s);
      if (a.tag) a.tag[i] = a.tag_value;
    }
    if (p.helpers)
      __hip_atomic_store(p.progress + v, a.round * K + kend, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

}  // namespace csr
}  // namespace asap
