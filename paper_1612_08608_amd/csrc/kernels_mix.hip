// kernels_mix.hip -- the stochastic reduce (Appendix A, update equation
// (A.2), second line): W'[i] = sum_{j in N_in(i)} P_ij W[j].
//
// The reduce is a low fan-in streaming product: every output element is
// deg+1 fused multiply-adds over rows that are each read by deg+1 outputs.
// It is bound by HBM bandwidth (arithmetic intensity < 1 flop/byte), so MFMA
// has no role here.  What matters is that every model byte crosses HBM once.
//
// slab kernel (n a power of two in [8, 1024], rows of at most 17 entries):
// each workgroup owns a contiguous range of column chunks; a chunk holds all
// n rows of a column range, sized so that it holds a whole 128-byte line of
// every row (128 KiB above 512 rows, 64 KiB above 256, else 32 KiB), and is
// staged in LDS, so each neighbour re-read is an LDS read.  The loads of the
// next chunk (two below 1024 rows) are in flight while one is computed.  A
// thread keeps the neighbour lists of its output rows in registers (two
// weights per row when all of a row's entries but its own share one weight).
// LDS slots of a row are XOR-swizzled by the row's low bits so that lanes
// reading random rows spread over the banks.  Results are transposed across
// groups of 8 lanes (DPP) so that each store writes a whole 128-byte line of
// a row rather than 16 bytes in each of 64 rows.
//
// tile kernel (any n): a tile is one 1 KiB segment of 16 consecutive output
// rows, one wave per row segment with 16-byte loads; the tiles of one column
// range go to one XCD so that re-reads of a neighbour's segment hit its L2.
//
// Precision: the slab kernel accumulates its at most 17 terms with fp32
// fused multiply-adds (error below 17 ulp of sum_j |P_ij w_j|); the tile and
// mean kernels take rows of any length (a hub, the complete graph) and
// accumulate in fp64, rounding once.
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

// Non-temporal 16-byte accesses, for data a reduce reads or writes exactly
// once (the slab kernel's staging loads and result stores): 4-5% faster
// than plain accesses for 1024 x 2^20 models.
typedef float nt4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld_nt(const float4* p) {
  const nt4 x = __builtin_nontemporal_load(reinterpret_cast<const nt4*>(p));
  return make_float4(x.x, x.y, x.z, x.w);
}
__device__ __forceinline__ void st_nt(float4* p, const float4& v) {
  const nt4 x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<nt4*>(p));
}

__device__ __forceinline__ void fma4(float4& acc, float w, const float4& x) {
  acc.x = fmaf(w, x.x, acc.x);
  acc.y = fmaf(w, x.y, acc.y);
  acc.z = fmaf(w, x.z, acc.z);
  acc.w = fmaf(w, x.w, acc.w);
}

// fp64 accumulator of one float4 slot: rows of any length (the tile and mean
// kernels) sum without fp32 error growth; the result is rounded once
struct Acc4 {
  double x = 0.0, y = 0.0, z = 0.0, w = 0.0;
  __device__ void fma(double wt, const float4& v) {
    x = ::fma(wt, double(v.x), x);
    y = ::fma(wt, double(v.y), y);
    z = ::fma(wt, double(v.z), z);
    w = ::fma(wt, double(v.w), w);
  }
  __device__ float4 round() const { return make_float4(float(x), float(y), float(z), float(w)); }
};

__device__ __forceinline__ void store_tail(float* d, const float4& v, int64_t c, int64_t dim) {
  if (c + 4 <= dim) {
    *reinterpret_cast<float4*>(d) = v;
  } else {
    d[0] = v.x;
    if (c + 1 < dim) d[1] = v.y;
    if (c + 2 < dim) d[2] = v.z;
  }
}

// One wave per row: its lanes check the row's in-neighbours' tags together
// (a thread per row walking 255 neighbours took 0.2 ms on the complete
// graph of 256 workers).
__global__ __launch_bounds__(64) void epoch_check_kernel(MixArgs a) {
  const int r = int(blockIdx.x), lane = int(threadIdx.x);
  const int p0 = a.nbr_ptr[r], p1 = a.nbr_ptr[r + 1];
  int ok = 1;
  for (int p = p0 + lane; p < p1; p += 64) ok &= (a.tag_src[a.nbr_idx[p]] == a.expect);
  ok = __all(ok);
  if (lane == 0) {
    a.row_ok[r] = ok;
    if (!ok) {
      atomicAdd(&a.err[kErrEpochCount], 1);
      atomicMin(&a.err[kErrEpochWorker], r);
    }
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
      Acc4 acc;
      const int p0 = a.nbr_ptr[r], p1 = a.nbr_ptr[r + 1];
      for (int p = p0; p < p1; ++p) {
        const int j = a.nbr_idx[p];
        double wt = a.nbr_w[p];
        if (a.scale) wt *= double(a.scale[j]);
        acc.fma(wt, *reinterpret_cast<const float4*>(a.src + int64_t(j) * a.ld + c));
      }
      store_tail(a.dst + int64_t(r) * a.ld + c, acc.round(), c, a.dim);
    }
    if (seg == 0 && lane == 0) a.tag_dst[r] = a.next;
  }
}

// Complete graph with uniform weights (all-reduce, Figure 2a): every output
// row is the same weighted column sum, so compute it once per column and
// broadcast it: n reads and n writes per column instead of n^2 reads.  The
// sum runs over j ascending with the same fp64 fused multiply-adds as
// mix_kernel, so both kernels produce identical bits on this graph.  On the
// complete graph one stale worker makes every row stale.
__global__ __launch_bounds__(64) void mean_kernel(MixArgs a, uint32_t nseg) {
  const uint32_t seg = xcd_tile(blockIdx.x, nseg);
  const int lane = threadIdx.x;
  int stale = 0;
  for (int j = lane; j < a.n; j += 64) stale |= !a.row_ok[j];
  if (__ballot(stale) != 0ull) return;
  const int64_t c = int64_t(seg) * kSegFloats + lane * 4;
  if (c < a.dim) {
    const double w0 = a.nbr_w[0];
    Acc4 acc;
    // 32 rows' loads in flight per wave (one wave per segment leaves few
    // waves on a CU): 256 workers x 2^18 beside the next round's planning,
    // 0.32 -> 0.24 ms; the order of the sum is unchanged
#pragma unroll 32
    for (int j = 0; j < a.n; ++j) {
      double wt = w0;
      if (a.scale) wt *= double(a.scale[j]);
      acc.fma(wt, *reinterpret_cast<const float4*>(a.src + int64_t(j) * a.ld + c));
    }
    const float4 out = acc.round();
#pragma unroll 4
    for (int j = 0; j < a.n; ++j) store_tail(a.dst + int64_t(j) * a.ld + c, out, c, a.dim);
  }
  if (seg == 0)
    for (int j = lane; j < a.n; j += 64) a.tag_dst[j] = a.next;
}

// Barrier that orders LDS only: global loads stay in flight across it, and
// global stores need not have landed.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

constexpr int kOut = 8;                             // outputs transposed and stored together

// x of lane i ^ S (S = 1, 2, 4) by DPP moves: quad_perm [1,0,3,2] and
// [2,3,0,1] are the xor-1 and xor-2 exchanges; xor 4 is the mirror inside
// each 8-lane half-row (i -> i ^ 7) followed by quad_perm [3,2,1,0]
// (i -> i ^ 3).
template <int S>
__device__ __forceinline__ float xor_lane(float x) {
  int v = __builtin_bit_cast(int, x);
  if constexpr (S == 1) {
    v = __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  } else if constexpr (S == 2) {
    v = __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  } else {
    static_assert(S == 4, "xor_lane: S in {1, 2, 4}");
    v = __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
    v = __builtin_amdgcn_update_dpp(0, v, 0x1B, 0xF, 0xF, false);
  }
  return __builtin_bit_cast(float, v);
}

template <int S>
__device__ __forceinline__ float4 xor_lane4(const float4& x) {
  return make_float4(xor_lane<S>(x.x), xor_lane<S>(x.y), xor_lane<S>(x.z), xor_lane<S>(x.w));
}

__device__ __forceinline__ float4 sel4(bool c, const float4& a, const float4& b) {
  return make_float4(c ? a.x : b.x, c ? a.y : b.y, c ? a.z : b.z, c ? a.w : b.w);
}

// v[k] of lane i <- v[i] of lane k, within aligned groups of 8 lanes:
// butterfly exchanges with the lanes i ^ s, s = 4, 2, 1.
template <int S>
__device__ __forceinline__ void transpose_stage(float4 (&v)[kOut], int lane_in) {
  const bool hi = lane_in & S;
#pragma unroll
  for (int k = 0; k < kOut; ++k) {
    if (k & S) continue;
    // a lane keeps the slot whose bit S matches its own and sends the other
    // (value selects only: a select of the slot to write would put v in
    // scratch memory)
    const float4 lo_v = v[k], hi_v = v[k | S];
    const float4 recv = xor_lane4<S>(sel4(hi, lo_v, hi_v));
    v[k] = sel4(hi, recv, lo_v);
    v[k | S] = sel4(hi, hi_v, recv);
  }
}

__device__ __forceinline__ void transpose8(float4 (&v)[kOut], int lane_in) {
  transpose_stage<4>(v, lane_in);
  transpose_stage<2>(v, lane_in);
  transpose_stage<1>(v, lane_in);
}

// 1 to 3 leading components of v (a row's ragged last float4)
__device__ __forceinline__ void store_partial(float* d, float4 v, int k) {
  d[0] = v.x;
  if (k > 1) d[1] = v.y;
  if (k > 2) d[2] = v.z;
}

// LDS reads in flight per thread
template <int DEG, int R> constexpr int slab_group() { return DEG <= 5 ? DEG : (R == 2 && DEG > 9 ? 1 : 4); }

// Slab kernel.  A THREADS-thread workgroup walks a contiguous
// range of column chunks; a chunk is all n rows of 4 VEC / n columns (VEC
// float4), staged in LDS.  Thread t stages float4 slots t + THREADS m of the
// chunk (m < VEC / THREADS); NBUF register buffers keep the loads of the
// next NBUF chunks in flight while one is computed.  Outputs: with R = 2
// (n = 2 THREADS) thread t computes rows t and t + THREADS, the whole chunk
// of each; with R = 1 row t mod n, VEC / THREADS float4 of it from
// (t div n) VEC / THREADS on.  Groups of 8 outputs of 8 consecutive lanes (8
// consecutive rows) are transposed across the lanes, so that each store
// instruction writes whole 128-byte lines: 8 lanes fill 128 contiguous
// bytes of one row.  With UNI every entry of a row but its own carries one
// weight, so a row keeps two weights instead of DEG.
template <int DEG, int R, int THREADS, int NBUF, int VEC, bool UNI>
__global__ __launch_bounds__(THREADS) void mix_slab_kernel(MixArgs a, int nchunks) {
  constexpr int kSlabThreads = THREADS;
  constexpr int kSlabVec = VEC;
  constexpr int kSlabPF = kSlabVec / THREADS;      // float4 staged per thread per chunk
  __shared__ float4 slab[kSlabVec];
  const int n = a.n;
  const int Q = kSlabVec / n;                // float4 per row per chunk (>= 8)
  const int C = 4 * Q;                       // columns per chunk
  const int X = min(Q, 8) - 1;               // swizzle mask
  const int tid = threadIdx.x;
  constexpr int OPR = kSlabPF / R;           // outputs per row per thread per chunk
  static_assert(OPR >= kOut && OPR % kOut == 0, "mix_slab_kernel: whole groups of transposed outputs");
  constexpr int G = slab_group<DEG, R>();
  // this thread's output rows and first float4
  int orow[R];
  int oq0;
  if constexpr (R == 2) {
    orow[0] = tid;
    orow[1] = tid + kSlabThreads;
    oq0 = 0;
  } else {
    orow[0] = tid % n;
    oq0 = (tid / n) * OPR;
  }
  // jq = j*Q | (j & X): the slot of float4 q of row j is jq ^ q, because
  // X < Q and Q is a power of two (see the staging writes below).
  // jq < n*Q = 8192, so two of them share a register.
  // Weights: with UNI every entry of a row but its own has one weight (the
  // launcher checked it bit for bit, and no scale applies), so a row keeps
  // (own weight, other weight, own position, length) and weight p is picked
  // by selects, the same value as the general table would give.
  uint32_t jq2[R][(DEG + 1) / 2];
  float nw[R][UNI ? 1 : DEG];
  float uw_self[R], uw_off[R];
  int upos[R], ulen[R];
  bool ok[R];
#pragma unroll
  for (int rr = 0; rr < R; ++rr) {
    const int row = orow[rr];
#pragma unroll
    for (int u = 0; u < (DEG + 1) / 2; ++u) jq2[rr][u] = 0u;
    const int p0 = a.nbr_ptr[row], deg = a.nbr_ptr[row + 1] - p0;
    uw_self[rr] = 0.f;
    uw_off[rr] = 0.f;
    upos[rr] = -1;
    ulen[rr] = deg;
#pragma unroll
    for (int u = 0; u < DEG; ++u) {
      const bool has = u < deg;  // padding: own row, weight 0
      const int j = has ? a.nbr_idx[p0 + u] : row;
      float wt = has ? a.nbr_w[p0 + u] : 0.f;
      if (a.scale && has) wt *= a.scale[j];
      jq2[rr][u / 2] |= uint32_t(j * Q | (j & X)) << (16 * (u & 1));
      if constexpr (UNI) {
        if (has && j == row) {
          uw_self[rr] = wt;
          upos[rr] = u;
        } else if (has) {
          uw_off[rr] = wt;
        }
      } else {
        nw[rr][u] = wt;
      }
    }
    ok[rr] = a.row_ok[row] != 0;
  }
  const int per = (nchunks + int(gridDim.x) - 1) / int(gridDim.x);
  const int ch0 = int(blockIdx.x) * per, ch1 = min(nchunks, ch0 + per);

  // Staging: slot s = tid + THREADS m of a chunk is float4 s mod Q of row s div
  // Q.  The per-thread part of the address is a 32-bit byte offset below
  // 2^31 (the launcher checks it); the rest is wave-uniform.
  const int lq = __builtin_ctz(Q);
  const bool wideq = Q > kSlabThreads;       // n == 8: Q = 1024
  const int q0 = wideq ? tid : (tid & (Q - 1));
  const int r0 = wideq ? 0 : (tid >> lq);
  const uint32_t voff = (uint32_t(r0) * uint32_t(a.ld) + 4u * uint32_t(q0)) * 4u;
  auto srow = [&](int m) {                   // uniform row offset of slot m
    return wideq ? (m >> 1) : m * (kSlabThreads >> lq);
  };
  auto sq = [&](int m) {                     // uniform float4 offset of slot m
    return wideq ? (m & 1) * kSlabThreads : 0;
  };
  auto load = [&](float4 (&buf)[kSlabPF], int ch) {
    const bool live = ch < ch1;
    const int64_t off = int64_t(live ? ch : ch0) * C;
    // an empty asm makes voff opaque per chunk, so the compiler does not
    // hoist 16 64-bit row addresses out of the chunk loop
    uint32_t vo = voff;
    asm volatile("" : "+v"(vo));
#pragma unroll
    for (int m = 0; m < kSlabPF; ++m) {
      const bool in = live && off + 4 * (q0 + sq(m)) < a.dim;
      const char* base = reinterpret_cast<const char*>(a.src + off + int64_t(srow(m)) * a.ld + 4 * sq(m));
      buf[m] = in ? ld_nt(reinterpret_cast<const float4*>(base + vo)) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto stage = [&](const float4 (&buf)[kSlabPF]) {
#pragma unroll
    for (int m = 0; m < kSlabPF; ++m) {
      const int r = r0 + srow(m), q = q0 + sq(m);
      slab[(r * Q | (r & X)) ^ q] = buf[m];
    }
  };
  // Output float4 q of row rr of this thread from the staged chunk.  Padding
  // entries read the own row with weight 0, which adds an exact zero, so the
  // reads of a group issue back to back with no branches.
  // the state of the row being computed, copied out of the per-row arrays
  // by selects (a runtime row index into those arrays would put them in
  // scratch memory)
  uint32_t jl[(DEG + 1) / 2];
  float nl[UNI ? 1 : DEG];
  float ls_self = 0.f, ls_off = 0.f;
  int lpos = 0, llen = 0;
  auto select_row = [&](int rr) {
    const bool second = R == 2 && rr == 1;
#pragma unroll
    for (int k = 0; k < (DEG + 1) / 2; ++k) jl[k] = second ? jq2[R - 1][k] : jq2[0][k];
    if constexpr (UNI) {
      ls_self = second ? uw_self[R - 1] : uw_self[0];
      ls_off = second ? uw_off[R - 1] : uw_off[0];
      lpos = second ? upos[R - 1] : upos[0];
      llen = second ? ulen[R - 1] : ulen[0];
    } else {
#pragma unroll
      for (int k = 0; k < DEG; ++k) nl[k] = second ? nw[R - 1][k] : nw[0][k];
    }
  };
  auto lweight = [&](int p) -> float {
    if constexpr (UNI) {
      const float w_in = p == lpos ? ls_self : ls_off;
      return p < llen ? w_in : 0.f;
    } else {
      return nl[p];
    }
  };
  auto slab_row = [&](int q) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    // Empty asm statements pin the register plan: the packed slots stay
    // packed and the weights stay in registers (not reloaded from memory),
    // and the reads of one group are not hoisted above the previous group.
#pragma unroll
    for (int k = 0; k < (DEG + 1) / 2; ++k) asm volatile("" : "+v"(jl[k]));
    if constexpr (UNI) {
      asm volatile("" : "+v"(ls_self), "+v"(ls_off), "+v"(lpos), "+v"(llen));
    } else {
#pragma unroll
      for (int k = 0; k < DEG; ++k) asm volatile("" : "+v"(nl[k]));
    }
#pragma unroll
    for (int p0 = 0; p0 < DEG; p0 += G) {
      if (p0 > 0) asm volatile("" ::: "memory");
      float4 x[G];
#pragma unroll
      for (int p = p0; p < p0 + G && p < DEG; ++p)
        x[p - p0] = slab[((jl[p / 2] >> (16 * (p & 1))) & 0xffffu) ^ q];
#pragma unroll
      for (int p = p0; p < p0 + G && p < DEG; ++p) fma4(acc, lweight(p), x[p - p0]);
    }
    // all four components here, or the compiler splits 16-byte LDS reads
    asm volatile("" : "+v"(acc.x), "+v"(acc.y), "+v"(acc.z), "+v"(acc.w));
    return acc;
  };
  const int lane = int(threadIdx.x) & 63;
  const int lane_in = lane & (kOut - 1);
  uint64_t okmask[R];
#pragma unroll
  for (int rr = 0; rr < R; ++rr) okmask[rr] = __ballot(ok[rr]);
  // one transposed group of 8 outputs: rows row_base + k, columns from c
  auto store_group = [&](const float4 (&res)[kOut], int64_t c, int row_base, uint64_t okm) {
    if (c < a.dim) {
      const bool full = c + 4 <= a.dim;
      const int k_tail = int(min<int64_t>(a.dim - c, 4));
#pragma unroll
      for (int k = 0; k < kOut; ++k) {
        if ((okm >> (lane - lane_in + k)) & 1) {
          float* d = a.dst + int64_t(row_base + k) * a.ld + c;
          if (full) {
            st_nt(reinterpret_cast<float4*>(d), res[k]);
          } else {
            store_partial(d, res[k], k_tail);
          }
        }
      }
    }
  };
  // With two output rows per thread and up to 5 entries per row, the second
  // row's group is held back and stored after the next chunk's loads are
  // issued, so that the wait for those loads at the next staging does not
  // also wait for these stores to drain (1024 x 2^20: d = 2 1.745 -> 1.714
  // ms, d = 4 1.772 -> 1.755 ms; with 9 entries, holding the whole group or
  // half of it made d = 8 slower: its longer neighbour sums let the stores
  // drain anyway).
  constexpr bool kDefer = R == 2 && DEG <= 5 && OPR == kOut;
  float4 pend[kDefer ? kOut : 1];
  int64_t pend_c = -1;
  auto compute = [&](int ch) {
    // one row at a time (R = 2: the second row's state is selected in, not
    // kept beside the first's while its outputs are computed)
#pragma unroll 1
    for (int rr = 0; rr < R; ++rr) {
      select_row(rr);
      const int row_base = (R == 2 && rr == 1 ? orow[R - 1] : orow[0]) & ~(kOut - 1);
      const uint64_t okm = R == 2 && rr == 1 ? okmask[R - 1] : okmask[0];
#pragma unroll 1
      for (int h = 0; h < OPR / kOut; ++h) {
        float4 res[kOut];
#pragma unroll
        for (int u = 0; u < kOut; ++u) res[u] = slab_row(oq0 + h * kOut + u);
        transpose8(res, lane_in);
        const int64_t c = int64_t(ch) * C + 4 * (oq0 + h * kOut + lane_in);
        if (kDefer && rr == R - 1) {
#pragma unroll
          for (int u = 0; u < (kDefer ? kOut : 1); ++u) pend[u] = res[u];
          pend_c = c;
        } else {
          store_group(res, c, row_base, okm);
        }
      }
    }
  };
  auto flush = [&]() {
    if constexpr (kDefer) {
      if (pend_c >= 0) store_group(pend, pend_c, orow[R - 1] & ~(kOut - 1), okmask[R - 1]);
      pend_c = -1;
    }
  };
  if constexpr (NBUF == 2) {
    float4 bufA[kSlabPF], bufB[kSlabPF];
    load(bufA, ch0);
    load(bufB, ch0 + 1);
    for (int ch = ch0; ch < ch1; ch += 2) {
      lds_barrier();  // the previous chunk is no longer read
      stage(bufA);
      lds_barrier();
      load(bufA, ch + 2);
      compute(ch);
      if (ch + 1 < ch1) {
        lds_barrier();
        stage(bufB);
        lds_barrier();
        load(bufB, ch + 3);
        compute(ch + 1);
      }
    }
  } else {
    float4 bufA[kSlabPF];
    load(bufA, ch0);
    for (int ch = ch0; ch < ch1; ++ch) {
      lds_barrier();  // the previous chunk is no longer read
      stage(bufA);
      lds_barrier();
      load(bufA, ch + 1);
      flush();
      compute(ch);
    }
    flush();
  }
  if (blockIdx.x == 0) {
    const bool head = R == 2 || tid < n;
#pragma unroll
    for (int rr = 0; rr < R; ++rr)
      if (head && ok[rr]) a.tag_dst[orow[rr]] = a.next;
  }
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
  hipLaunchKernelGGL(epoch_check_kernel, dim3(uint32_t(a.n)), dim3(64), 0, s, a);
  return hipGetLastError();
}

namespace {
// whether the slab kernel takes this graph: n a power of two in [8, 1024]
// and rows of at most 17 entries
bool slab_graph(int n, int max_deg) { return n >= 8 && n <= 1024 && !(n & (n - 1)) && max_deg <= 17; }

// Shapes: above 256 rows one 512-thread workgroup per CU with a 128 KiB
// (above 512 rows) or 64 KiB chunk; up to 256 rows 256-thread workgroups
// with 32 KiB chunks, up to four per CU.  Every chunk holds a whole 128-byte
// line of every row (Q >= 8 float4).  Small workgroups leave room on a CU for
// the kernels that plan the next round beside the reduce: 256 workers x
// 2^18, random 8-regular: reduce 0.32 -> 0.29 ms, round 1.36 -> 1.32 ms.
int slab_threads(int n) { return n > 256 ? 512 : 256; }
int slab_vec(int n) { return n > 512 ? 8192 : n > 256 ? 4096 : 2048; }
int slab_per_cu(int n) { return n > 256 ? 1 : 4; }

// per-thread staging offset (rows below THREADS/Q, float4 slots below Q) and
// chunk count within 31 bits
bool slab_fits(const MixArgs& a) {
  const int T = slab_threads(a.n);
  const int Q = slab_vec(a.n) / a.n, C = 4 * Q;
  const int rows = Q > T ? 1 : T / Q;
  if ((int64_t(rows - 1) * a.ld + 4 * int64_t(std::min(Q, T))) * 4 >= (int64_t(1) << 31)) return false;
  return (a.dim + C - 1) / C < (int64_t(1) << 31);
}
}  // namespace

bool mix_slab_applies(const MixArgs& a, int max_deg) { return slab_graph(a.n, max_deg) && slab_fits(a); }

// Slab kernel when n is a power of two in [8, 1024] and every row has at most
// 17 entries (returns hipErrorNotSupported otherwise).
template <int DEG>
hipError_t launch_slab(const MixArgs& a, int n_cu, hipStream_t s) {
  if (!slab_fits(a)) return hipErrorNotSupported;
  const int C = 4 * (slab_vec(a.n) / a.n);
  const int nchunks = int((a.dim + C - 1) / C);
  const int grid = std::max(1, std::min(nchunks, slab_per_cu(a.n) * n_cu));
  const dim3 g(grid), b(slab_threads(a.n));
  if (a.n > 512) {
    if (a.uniform_rows)
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 2, 512, 1, 8192, true>), g, b, 0, s, a, nchunks);
    else
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 2, 512, 1, 8192, false>), g, b, 0, s, a, nchunks);
  } else if (a.n > 256) {
    if (a.uniform_rows)
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 1, 512, 2, 4096, true>), g, b, 0, s, a, nchunks);
    else
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 1, 512, 2, 4096, false>), g, b, 0, s, a, nchunks);
  } else {
    if (a.uniform_rows)
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 1, 256, 2, 2048, true>), g, b, 0, s, a, nchunks);
    else
      hipLaunchKernelGGL((mix_slab_kernel<DEG, 1, 256, 2, 2048, false>), g, b, 0, s, a, nchunks);
  }
  return hipGetLastError();
}

hipError_t launch_mix_slab(const MixArgs& a, int max_deg, int n_cu, hipStream_t s) {
  if (!slab_graph(a.n, max_deg)) return hipErrorNotSupported;
  if (max_deg <= 3) return launch_slab<3>(a, n_cu, s);
  if (max_deg <= 5) return launch_slab<5>(a, n_cu, s);
  if (max_deg <= 9) return launch_slab<9>(a, n_cu, s);
  return launch_slab<17>(a, n_cu, s);
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
