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
#include "csr_fast.h"

namespace asap {
namespace {

using namespace csr;

constexpr int kHotWords = (kHotMax + 31) / 32;

constexpr int kPlanThreads = 256;
static_assert(kPlanStepRows == kFastRows, "the host bounds steps of the planned pass's rows");

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
// The step's T nonzeros are numbered in row order and dealt to the threads
// flat (thread t takes e = t, t + NT, ...: every lane busy whatever the row
// lengths); an LDS byte per nonzero names its row.  TB: LDS for 2^TB table
// positions (a step uses the smallest power of two >= twice its cold
// nonzeros, from 2^6 up to 2^TB).
// G: nonzeros per thread, G NT >= the step's most (rows x longest row).
template <int TB, int NT, int G>
__global__ __launch_bounds__(NT) void csr_plan_kernel(PlanArgs p) {
  constexpr int NW = NT / 64;
  constexpr int PMAX = (1 << TB) / NT;  // table positions per thread, at most
  static_assert(NT >= kHotWords && NT >= kFastRows, "one hot-bitmap word and one row per thread");
  __shared__ int keys[1 << TB];      // a column, then its slot
  __shared__ uint32_t hot[kHotWords];
  __shared__ int sc[NW];
  __shared__ int roff[kFastRows];    // a row's first nonzero in the step's numbering
  __shared__ int rlen[kFastRows];
  __shared__ int rdelta[kFastRows];  // row start - worker start - roff
  __shared__ uint8_t rowof[G * NT];
  __shared__ int overflow;
  __shared__ int ncold;  // the step's cold nonzeros
  const int K = p.K, B = p.batch;
  const int i = int(blockIdx.x) / K, k = int(blockIdx.x) % K;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t S = p.S;
  const int64_t seg = p.row_ptr[int64_t(i) * S];
  const int64_t b0 = int64_t(k) * B;
  const int Bp = int(min<int64_t>(B, S - b0));  // <= kFastRows
  const int32_t* so = p.step_off + int64_t(i) * (S + 1);
  const int64_t lbase = seg + so[k];
  const int T = so[k + 1] - so[k];
  if (T > G * NT) {  // never with the host's choice of G; the general kernel would run
    if (t == 0) {
      p.cnt[(int64_t(i) * K + k) * 2 + 0] = 0;
      p.cnt[(int64_t(i) * K + k) * 2 + 1] = 0;
      atomicOr(p.flag, 1);
    }
    return;
  }
  if (wave == 0) {
    // rows' offsets in the step's numbering: an inclusive scan over lanes
    int len = 0;
    long long st = 0;
    if (lane < Bp) {
      const RowInfo r = p.rowinfo[int64_t(i) * S + b0 + lane];
      st = r.start;
      len = r.len;
    }
    int x = len;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    roff[lane] = x - len;
    rlen[lane] = len;
    rdelta[lane] = int(st - seg) - (x - len);
  }
  for (int q = t; q < kHotWords; q += NT) hot[q] = 0u;
  if (t == 0) {
    overflow = 0;
    ncold = 0;
  }
  __syncthreads();
  for (int b = wave; b < Bp; b += NW)
    for (int x = lane; x < rlen[b]; x += 64) rowof[roff[b] + x] = uint8_t(b);
  __syncthreads();
  // the thread's codes in registers, all loads issued before any is used
  int cc[G], pos[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    cc[g] = -1;  // no entry
    pos[g] = -1;
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g * NT >= T) break;
    const int e = t + g * NT;
    if (e < T) cc[g] = p.code[seg + rdelta[rowof[e]] + e];
  }
  // a table of at least twice the step's cold nonzeros (at most 2^TB
  // positions; a step's distinct cold columns are usually far fewer than its
  // nonzeros, most of which have hot slots)
  int mine = 0;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g * NT >= T) break;
    mine += cc[g] != -1 && !is_hot(cc[g]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mine += __shfl_xor(mine, o, 64);
  if (lane == 0) atomicAdd(&ncold, mine);
  __syncthreads();
  int bits = 6;
  while (bits < TB && (1 << bits) < 2 * ncold) ++bits;
  const int tab = 1 << bits;
  for (int q = t; q < tab; q += NT) keys[q] = -1;
  __syncthreads();
  // hot slots into the bitmap, cold columns into the table (their positions
  // kept for the codes; a hot entry keeps -2, no entry -1)
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g * NT >= T) break;
    const int c = cc[g];
    if (c == -1) continue;
    pos[g] = -2;
    if (is_hot(c)) {
      const int hs = hot_slot(c);
      const uint32_t bit = 1u << (hs & 31);
      if (!(hot[hs >> 5] & bit)) atomicOr(&hot[hs >> 5], bit);
    } else {
      pos[g] = table_insert(keys, bits, c);
      if (pos[g] == -1) overflow = 1;
    }
  }
  __syncthreads();
  // cold slots: thread t numbers the positions t + j NT (a wave reads 64
  // consecutive words, no bank conflicts), read once and overwritten by the
  // slot (by the same thread, so no other reads them in between)
  int kv[PMAX];
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < PMAX; ++j) {
    kv[j] = t + j * NT < tab ? keys[t + j * NT] : -1;
    cnt += kv[j] >= 0;
  }
  int Uc = 0;
  int id = block_scan<NW>(cnt, sc, &Uc);
#pragma unroll
  for (int j = 0; j < PMAX; ++j) {
    if (kv[j] >= 0) {
      keys[t + j * NT] = id;
      p.clist[lbase + id] = kv[j];
      ++id;
    }
  }
  // hot slots in slot order
  const uint32_t word = t < kHotWords ? hot[t] : 0u;
  int Uh = 0;
  int hid = block_scan<NW>(__popc(word), sc, &Uh);
  for (uint32_t w = word; w; w &= w - 1) p.hlist[lbase + hid++] = t * 32 + __ffs(w) - 1;
  __syncthreads();  // slots complete
  // the code half of each cold entry's (code, value) pair: a hot entry's code
  // and every value do not change from round to round and are written once,
  // at bind
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g * NT >= T) break;
    const int e = t + g * NT;
    if (e >= T || pos[g] == -2) continue;  // no entry, or a hot one
    reinterpret_cast<int*>(p.pack + seg + rdelta[rowof[e]] + e)[0] = pos[g] >= 0 ? keys[pos[g]] : 0;
  }
  if (t == 0) {
    p.cnt[(int64_t(i) * K + k) * 2 + 0] = Uc;
    p.cnt[(int64_t(i) * K + k) * 2 + 1] = Uh;
    if (overflow || Uc > kCMax || Uh > kHList) atomicOr(p.flag, 1);
  }
}

// ----------------------------------------------------------------------------
// links: slot of each cold column of step k in step k-1, or -1; a block
// takes R consecutive steps of one worker and loads the first PER NT entries
// of the R + 1 lists it needs at once (any further ones where they are used).
// TB: tables of up to 2^TB positions (2^11 hold every slot; 2^12 keep the
// probes of the fullest lists short; with 2^10, a list that does not fit
// raises the flag, and the general kernel runs the round)
// ----------------------------------------------------------------------------
template <int NT, int R, int PER, int TB>
__global__ __launch_bounds__(NT) void csr_link_kernel(PlanArgs p) {
  __shared__ int keys[1 << TB];
  __shared__ uint16_t vals[1 << TB];  // slots < kCMax
  const int K = p.K, KB = (K + R - 1) / R;
  const int i = int(blockIdx.x) / KB, k0 = (int(blockIdx.x) % KB) * R;
  const int t = threadIdx.x;
  const int64_t S = p.S;
  const int64_t seg = p.row_ptr[int64_t(i) * S];
  const int32_t* so = p.step_off + int64_t(i) * (S + 1);
  // entry r is step k0 + r - 1
  int U[R + 1];
  int64_t base[R + 1];
  int col[R + 1][PER];
#pragma unroll
  for (int r = 0; r <= R; ++r) {
    const int k = k0 + r - 1;
    U[r] = k >= 0 && k < K ? min(p.cnt[(int64_t(i) * K + k) * 2], kCMax) : 0;
    base[r] = seg + (U[r] ? so[k] : 0);
  }
#pragma unroll
  for (int r = 0; r <= R; ++r)
#pragma unroll
    for (int j = 0; j < PER; ++j) col[r][j] = t + j * NT < U[r] ? p.clist[base[r] + t + j * NT] : -1;
#pragma unroll
  for (int r = 1; r <= R; ++r) {
    const int Uc = U[r], Up = U[r - 1];
    if (Uc == 0) continue;  // uniform: every thread skips the step
    if (Up == 0) {  // no previous step, or one without cold columns
      for (int u = t; u < Uc; u += NT) p.clink[base[r] + u] = -1;
      continue;
    }
    if (Up > (1 << TB)) {  // uniform; never when 2^TB >= kCMax
      if (t == 0) atomicOr(p.flag, 1);
      continue;
    }
    // a table of at least twice the previous step's columns, at most 2^TB
    // positions (linear probing holds up to that many)
    int bits = 6;
    while (bits < TB && (1 << bits) < 2 * Up) ++bits;
    __syncthreads();  // the previous step's lookups are done
    for (int q = t; q < (1 << bits); q += NT) keys[q] = -1;
    __syncthreads();
    // columns are distinct within a step
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (col[r - 1][j] < 0) continue;
      const int pos = table_insert(keys, bits, col[r - 1][j]);
      if (pos >= 0) vals[pos] = uint16_t(t + j * NT);
    }
    for (int u = t + PER * NT; u < Up; u += NT) {
      const int pos = table_insert(keys, bits, p.clist[base[r - 1] + u]);
      if (pos >= 0) vals[pos] = uint16_t(u);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (col[r][j] < 0) continue;
      const int pos = table_find(keys, bits, col[r][j]);
      p.clink[base[r] + t + j * NT] = pos >= 0 ? int(vals[pos]) : -1;
    }
    for (int u = t + PER * NT; u < Uc; u += NT) {
      const int pos = table_find(keys, bits, p.clist[base[r] + u]);
      p.clink[base[r] + u] = pos >= 0 ? int(vals[pos]) : -1;
    }
  }
}

// ----------------------------------------------------------------------------
// the pass on the plan (csr_fast.h); block n + i prefetches for worker i
// ----------------------------------------------------------------------------
// NT threads: 1024 (64 rows of 16 lanes), or 512 for minibatches of at most
// 32 rows when the pass fills the device, so that planning blocks fit beside
// it on every compute unit (the results do not depend on NT).
template <int E, bool MEM, int NT = kThreads>
__global__ __launch_bounds__(NT) void sgd_csr_fast_kernel(SgdArgs a, PlanArgs p) {
  if (*p.flag) return;  // the general kernel takes this round
  const int M = MEM ? p.members : 1;
  int i, m;
  if (int(blockIdx.x) >= a.n * M) {
    // block n M + b prefetches for the slice of block b (same XCD when n M
    // is a multiple of 8)
    member_of(int(blockIdx.x) - a.n * M, a.n, M, i, m);
    prefetch_pass<E>(a, p, i * M + m, i);
    return;
  }
  __shared__ FastShared sh;
  member_of(int(blockIdx.x), a.n, M, i, m);
  fast_pass<E, MEM, NT>(a, p, i, m, sh);
}

__global__ void pack_values_kernel(const int32_t* __restrict__ code, const float* __restrict__ val, int64_t nnz,
                                   int2* __restrict__ pack) {
  for (int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; q < nnz; q += int64_t(gridDim.x) * blockDim.x)
    pack[q] = make_int2(code[q], __float_as_int(val[q]));
}

template <int E>
hipError_t launch_fast_e(const SgdArgs& a, const PlanArgs& p, hipStream_t s) {
  if (p.members > 1) {
    // members wait for each other every step: cooperative, so that all are
    // resident at once
    const uint32_t grid = uint32_t(a.n) * uint32_t(p.members) * (p.helpers ? 2u : 1u);
    SgdArgs aa = a;
    PlanArgs pp = p;
    void* args[] = {&aa, &pp};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&sgd_csr_fast_kernel<E, true>), dim3(grid),
                                      dim3(kThreads), args, 0, s);
  }
  if (p.helpers == 0 && a.batch <= kFastRows / 2 && int64_t(a.n) * 2 > p.n_cu) {
    hipLaunchKernelGGL((sgd_csr_fast_kernel<E, false, kThreads / 2>), dim3(uint32_t(a.n)), dim3(kThreads / 2), 0, s,
                       a, p);
    return hipGetLastError();
  }
  // with helpers, block n + i prefetches for block i: the same XCD when n is
  // a multiple of the 8 XCDs (blocks are dealt to them round-robin)
  const uint32_t grid = uint32_t(a.n) * (p.helpers ? 2u : 1u);
  hipLaunchKernelGGL((sgd_csr_fast_kernel<E, false>), dim3(grid), dim3(kThreads), 0, s, a, p);
  return hipGetLastError();
}

}  // namespace

bool csr_plan_fits(const SgdArgs& a) {
  return a.batch <= kFastRows && a.max_row <= kRowLanes * 8 && a.n_hot <= kHotMax;
}

hipError_t launch_csr_plan(const PlanArgs& p, int64_t most, hipStream_t s) {
  const uint32_t blocks = uint32_t(int64_t(p.n) * p.K);
  hipLaunchKernelGGL(step_scan_kernel, dim3(uint32_t(p.n)), dim3(kScanThreads), 0, s, p);
  // `most` bounds a step's nonzeros (the longest rows of the fullest slice,
  // found at bind; never more than batch * longest row).  A step's table
  // holds its distinct cold columns, of which a plan that the pass can take
  // has at most kCMax: 2^11 positions hold them all (linear probing fills a
  // table completely; a fuller step overflows into the general kernel, as
  // does a step over kCMax), and a step uses twice its cold nonzeros, so
  // that the probes stay short in all but the fullest steps.  Small tables
  // keep more blocks resident, also beside a pass that fills the device:
  // where steps have few cold nonzeros (estimated at bind), 2^10 positions,
  // five times the estimate (a step with more distinct cold columns than
  // that overflows into the general kernel).
  static_assert((1 << 11) >= kCMax, "a 2^11-position table holds every cold slot");
  constexpr int NT = kPlanThreads;
  // the pass of several members per worker takes at most half the compute
  // units: planning then runs beside it on the others
  const bool beside = p.members > 1 && int64_t(p.workers) * p.members * 2 <= p.n_cu;
  if (most <= 2 * NT)
    hipLaunchKernelGGL((csr_plan_kernel<10, NT, 2>), dim3(blocks), dim3(NT), 0, s, p);
  else if (most <= 4 * NT)
    hipLaunchKernelGGL((csr_plan_kernel<11, NT, 4>), dim3(blocks), dim3(NT), 0, s, p);
  else if (most <= 8 * NT && p.cold_step <= 192)  // small tables: more blocks fit beside a 512-thread pass
    hipLaunchKernelGGL((csr_plan_kernel<10, NT, 8>), dim3(blocks), dim3(NT), 0, s, p);
  else if (most <= 8 * NT)
    hipLaunchKernelGGL((csr_plan_kernel<11, NT, 8>), dim3(blocks), dim3(NT), 0, s, p);
  else if (most <= 16 * NT && p.cold_step <= 192)
    hipLaunchKernelGGL((csr_plan_kernel<10, NT, 16>), dim3(blocks), dim3(NT), 0, s, p);
  else if (most <= 16 * NT && !beside)
    hipLaunchKernelGGL((csr_plan_kernel<11, NT, 16>), dim3(blocks), dim3(NT), 0, s, p);
  // beyond 16 nonzeros per thread, or beside a pass on compute units of its
  // own, twice the threads (planning beside 64 workers x 2 members in
  // 512-thread blocks: the pass 2.34 -> 2.30 ms; alone, 256-thread blocks
  // plan faster)
  else if (p.cold_step <= 768)
    hipLaunchKernelGGL((csr_plan_kernel<11, 2 * NT, 16>), dim3(blocks), dim3(2 * NT), 0, s, p);
  else  // and a table of 2^12 positions for steps with many cold columns
    hipLaunchKernelGGL((csr_plan_kernel<12, 2 * NT, 16>), dim3(blocks), dim3(2 * NT), 0, s, p);
  static_assert(kFastRows * kRowLanes * 8 <= 32 * kPlanThreads, "16 nonzeros per thread of 2 NT cover the longest plannable step");
  // steps whose lists (at most their cold nonzeros, estimated) fit one
  // entry per thread with some margin: 8 steps per block, the lists' heads
  // loaded at once, tables of 2^10 positions; else 4 steps, whole lists, in
  // tables of 2^12 positions for lists of more than 768 entries
  static_assert(kCMax % 256 == 0, "whole lists in registers");
  if (p.cold_step <= 192) {
    const uint32_t lb = uint32_t(int64_t(p.n) * ((p.K + 7) / 8));
    hipLaunchKernelGGL((csr_link_kernel<256, 8, 1, 10>), dim3(lb), dim3(256), 0, s, p);
  } else {
    const uint32_t lb = uint32_t(int64_t(p.n) * ((p.K + 3) / 4));
    if (p.cold_step <= 768)
      hipLaunchKernelGGL((csr_link_kernel<256, 4, kCMax / 256, 11>), dim3(lb), dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((csr_link_kernel<256, 4, kCMax / 256, 12>), dim3(lb), dim3(256), 0, s, p);
  }
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
  if (a.max_row <= kRowLanes * 5) return launch_fast_e<5>(a, p, s);
  if (a.max_row <= kRowLanes * 6) return launch_fast_e<6>(a, p, s);
  return launch_fast_e<8>(a, p, s);
}

}  // namespace asap
