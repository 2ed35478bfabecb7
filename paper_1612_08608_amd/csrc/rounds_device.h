// rounds_device.h -- device side of the multi-round launch: many rounds of
// (A.2) (Appendix A) in one persistent launch, synchronised per worker by
// the fine-grained NOTIFY-ACK protocol of Section 4 instead of a device-wide
// kernel boundary between the half-step and the reduce.
//
// Worker i in round r (buffer e = the buffer of round r):
//   1. local pass on W[e][i] in place (the same device code as the
//      stream-ordered kernels);
//   2. NOTIFY: release-store tag[e][i] = 2r + 1;
//   3. WAIT: every in-neighbour j has tag[e][j] >= 2r + 1 (its half-step of
//      round r is published), and every out-neighbour k has
//      tag[e][k] >= 2r (it has finished its reduce of round r - 1, the last
//      read of W[e^1][i] before this round overwrites it: the ACK);
//   4. reduce row i into W[e^1][i] with the arithmetic of the reduce kernel
//      the stream-ordered path would launch for this graph;
//   5. release-store tag[e^1][i] = 2(r + 1): the ACK of round r and the
//      "round r + 1 starts from this row" tag.
// A worker then goes straight on to round r + 1, overlapping other workers'
// reduces, which is the point of the protocol.  The tags only grow, so a
// wait on ">=" can never miss a value that has already been overwritten.
// Every wait is bounded by a wall-clock deadline; a wait that runs out
// stops the worker and is reported like a stale neighbour of the stream
// path (epoch error words).  All workgroups are resident (cooperative
// launch), so a worker never waits on one that cannot run.
#pragma once

#include "asap_common.h"
#include "asap_launch.h"

namespace asap {
namespace rounds {

__device__ __forceinline__ int64_t tag_peek(const int64_t* p) {
  // relaxed device-scope load: reaches the coherent level without
  // invalidating this XCD's L2 on every poll
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void tag_release(int64_t* p, int64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void acquire_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

// Device-coherent 16-byte load (cache policy sc1): served from memory or a
// coherent level, never from a stale line of this XCD's L2.  The reduce
// reads neighbours' rows this way instead of invalidating the whole L2 after
// each wait, which would also evict the worker's shard.
__device__ __forceinline__ float4 load_coherent(const float* row, uint32_t bytes, uint32_t off) {
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), 0, int(bytes), 0x00020000);
  const auto u = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 16);
  const unsigned u0 = u[0], u1 = u[1], u2 = u[2], u3 = u[3];
  return make_float4(__uint_as_float(u0), __uint_as_float(u1), __uint_as_float(u2), __uint_as_float(u3));
}

// One thread: wait until *tag >= want or until the wall clock passes
// `deadline`; false when the deadline passed first.
__device__ inline bool wait_tag(const int64_t* tag, int64_t want, long long deadline) {
  while (tag_peek(tag) < want) {
    if (wall_clock64() > deadline) return false;
    __builtin_amdgcn_s_sleep(4);
  }
  return true;
}

// One thread: wait until tags[list[u]] >= want for every u < cnt.  Returns
// -1 when all have arrived, else the first worker still missing at the
// deadline.  The caller issues one acquire fence after the wait.
__device__ inline int wait_tags(const int64_t* tags, const int32_t* list, int cnt, int64_t want,
                                long long deadline) {
  for (int u = 0; u < cnt; ++u)
    if (!wait_tag(tags + list[u], want, deadline)) return list[u];
  return -1;
}

__device__ inline void report_stale(int32_t* err, int worker) {
  atomicAdd(&err[kErrEpochCount], 1);
  atomicMin(&err[kErrEpochWorker], worker);
}

// Steps of round r: a whole pass (L = 0), else L steps of the sequence of
// passes (round r covers steps k0 .. k0 + L - 1 of pass (r L) div K).
__device__ __forceinline__ void steps_of(int64_t r, int32_t L, int64_t K, int64_t& pass, int64_t& k0, int64_t& k1) {
  if (L == 0) {
    pass = r;
    k0 = 0;
    k1 = K;
  } else {
    const int64_t g = r * L;
    pass = g / K;
    k0 = g % K;
    k1 = k0 + L;
  }
}

// Whole workgroup: worker i's schedule row of `pass` (the values the
// schedule kernel writes).
__device__ inline void fill_schedule(uint64_t seed, int i, int64_t pass, int64_t S, int32_t* row) {
  const Perm p = perm_make(seed, i, pass, uint32_t(S));
  for (int64_t pos = threadIdx.x; pos < S; pos += blockDim.x) row[pos] = int32_t(perm_at(p, uint32_t(pos)));
}

// Whole workgroup: worker i's row descriptors of `pass` in schedule order
// (the values the row-descriptor kernel writes).
__device__ inline void fill_rowinfo(uint64_t seed, int i, int64_t pass, int64_t S, const int64_t* row_ptr,
                                    const float* y, RowInfo* out) {
  const Perm p = perm_make(seed, i, pass, uint32_t(S));
  for (int64_t pos = threadIdx.x; pos < S; pos += blockDim.x) {
    const int64_t g = int64_t(i) * S + int64_t(perm_at(p, uint32_t(pos)));
    const int64_t p0 = row_ptr[g], p1 = row_ptr[g + 1];
    RowInfo r;
    r.start = p0;
    r.len = int(p1 - p0);
    r.y = y[g];
    out[pos] = r;
  }
}

// Whole workgroup: row i of the reduce, W[e^1][i] = sum_j P_ij s_j W[e][j]
// over the in-neighbours in row order.  F64: every term and the sum in fp64,
// rounded once (the tile and mean kernels); else fp32 weights w_ij * s_j and
// fp32 fused multiply-adds from +0 (the slab kernel).  Columns go in blocks
// of kMixVec float4 per thread so that each neighbour's index and weight are
// read once per block; no LDS (the CSR pass leaves almost none).  Rows and
// scales written by other workgroups are read device-coherently (their
// writers released them before the tags this workgroup waited for).
constexpr int kMixVec = 4;

// Member `part` of `parts` reduces the part-th of the row's float4 columns
// (the whole row with one part); every output element has the same
// arithmetic whatever the split.
template <bool F64>
__device__ void mix_row(const RoundsArgs& ra, int i, int e, int64_t ld, int64_t dim, int part, int parts) {
  const int p0 = ra.in_ptr[i], deg = ra.in_ptr[i + 1] - p0;
  const float* scale = ra.scaled ? ra.scale2 + int64_t(e) * ra.n : nullptr;
  const float* src = ra.buf[e];
  float* dst = ra.buf[e ^ 1] + int64_t(i) * ld;
  const int64_t nq_all = (dim + 3) / 4, T = blockDim.x;
  const int64_t per = (nq_all + parts - 1) / parts;
  const int64_t qb = min(nq_all, per * part), nq = min(nq_all, qb + per);
  for (int64_t q0 = qb + threadIdx.x; q0 < nq; q0 += kMixVec * T) {
    double ad[kMixVec][4];
    float4 af[kMixVec];
#pragma unroll
    for (int v = 0; v < kMixVec; ++v) {
      ad[v][0] = ad[v][1] = ad[v][2] = ad[v][3] = 0.0;
      af[v] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int u = 0; u < deg; ++u) {
      const int j = ra.in_idx[p0 + u];
      float wf = ra.in_w[p0 + u];
      double wd = ra.in_w[p0 + u];
      if (scale) {
        const float sj = __hip_atomic_load(scale + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        wf *= sj;
        wd *= double(sj);
      }
      const float* row = src + int64_t(j) * ld;
#pragma unroll
      for (int v = 0; v < kMixVec; ++v) {
        const int64_t q = q0 + v * T;
        if (q < nq) {
          const float4 x = load_coherent(row, uint32_t(ld) * 4u, uint32_t(q) * 16u);
          if constexpr (F64) {
            ad[v][0] = fma(wd, double(x.x), ad[v][0]);
            ad[v][1] = fma(wd, double(x.y), ad[v][1]);
            ad[v][2] = fma(wd, double(x.z), ad[v][2]);
            ad[v][3] = fma(wd, double(x.w), ad[v][3]);
          } else {
            af[v].x = fmaf(wf, x.x, af[v].x);
            af[v].y = fmaf(wf, x.y, af[v].y);
            af[v].z = fmaf(wf, x.z, af[v].z);
            af[v].w = fmaf(wf, x.w, af[v].w);
          }
        }
      }
    }
#pragma unroll
    for (int v = 0; v < kMixVec; ++v) {
      const int64_t q = q0 + v * T, c = 4 * q;
      if (q >= nq) continue;
      const float4 out =
          F64 ? make_float4(float(ad[v][0]), float(ad[v][1]), float(ad[v][2]), float(ad[v][3])) : af[v];
      if (c + 4 <= dim) {
        *reinterpret_cast<float4*>(dst + c) = out;
      } else {
        dst[c] = out.x;
        if (c + 1 < dim) dst[c + 1] = out.y;
        if (c + 2 < dim) dst[c + 2] = out.z;
      }
    }
  }
}

// The round loop of one workgroup: member `member` of the `members`
// workgroups of worker i.  Member 0 publishes the half-step (NOTIFY) once
// pass_fn has returned on every member, waits for the neighbours, and lets
// the other members go (ra.msync[i][0]); each member reduces its part of
// the row's columns and reports it (ra.msync[i][1 + member]); member 0 then
// publishes the reduced row (ACK), which the others wait for before their
// next pass.  `prepare(pass)` writes the pass's schedule inputs (whole
// workgroup); `pass_fn(a)` runs the half-step and returns false when the
// members' own rendezvous timed out.
template <class Prepare, class Pass>
__device__ void drive(SgdArgs a, const RoundsArgs& ra, int i, int member, int members, Prepare&& prepare,
                      Pass&& pass_fn) {
  __shared__ int stop;
  const int tid = threadIdx.x, n = ra.n;
  const int64_t K = (a.S + a.batch - 1) / a.batch;
  if (tid == 0) {
    // the launch starts from the state a reduce (or asap_set_round) leaves:
    // every row of the current buffer tagged "round r0 starts here"; only
    // worker i writes its own tags, so this read is not racy
    stop = tag_peek(ra.tag + int64_t(ra.cur) * n + i) != tag_start(ra.r0);
    if (stop && member == 0) report_stale(ra.err, i);
  }
  __syncthreads();
  if (stop) return;
  int64_t have = -1;
  for (int64_t u = 0; u < ra.R; ++u) {
    const int64_t r = ra.r0 + u;
    const int e = ra.cur ^ int(u & 1);
    int64_t pass, k0, k1;
    steps_of(r, ra.local_steps, K, pass, k0, k1);
    if (pass != have) {
      prepare(pass);
      have = pass;
      __syncthreads();
    }
    a.models = ra.buf[e];
    a.round = pass;
    a.k0 = k0;
    a.k1 = k1;
    a.scale = ra.scale2 + int64_t(e) * n;
    a.tag = nullptr;  // published below, after the whole workgroup's stores
    const bool ok = pass_fn(a);
    __syncthreads();
    if (!ok) return;
    int64_t* te = ra.tag + int64_t(e) * n;
    int64_t* tn = ra.tag + int64_t(e ^ 1) * n;
    int64_t* ms = ra.msync + int64_t(i) * kMemberSync;
    if (tid == 0) {
      const long long deadline = wall_clock64() + ra.wait_ticks;
      if (member == 0) {
        tag_release(te + i, tag_half(r));  // NOTIFY
        const int pi = ra.in_ptr[i], po = ra.out_ptr[i];
        int miss = wait_tags(te, ra.in_idx + pi, ra.in_ptr[i + 1] - pi, tag_half(r), deadline);
        if (miss < 0) miss = wait_tags(te, ra.out_idx + po, ra.out_ptr[i + 1] - po, tag_start(r), deadline);
        // no acquire fence: the reduce reads what the neighbours released
        // with device-coherent loads (the workgroup barrier below keeps
        // them after this wait)
        stop = miss >= 0;
        if (stop) report_stale(ra.err, i);
        else if (members > 1) tag_release(ms, tag_half(r));  // the other members may reduce
      } else {
        stop = !wait_tag(ms, tag_half(r), deadline);
      }
    }
    __syncthreads();
    if (stop) return;
    if (ra.fp64_mix)
      mix_row<true>(ra, i, e, a.ld, a.dim, member, members);
    else
      mix_row<false>(ra, i, e, a.ld, a.dim, member, members);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's part of the row is written
    __syncthreads();
    if (tid == 0) {
      const long long deadline = wall_clock64() + ra.wait_ticks;
      if (member == 0) {
        for (int q = 1; q < members && !stop; ++q) stop = !wait_tag(ms + 1 + q, tag_half(r), deadline);
        if (stop) report_stale(ra.err, i);
        else tag_release(tn + i, tag_start(r + 1));  // ACK, and round r + 1 starts from this row
      } else {
        tag_release(ms + 1 + member, tag_half(r));  // this part is reduced
        stop = !wait_tag(tn + i, tag_start(r + 1), deadline);
        acquire_fence();
      }
    }
    __syncthreads();
    if (stop) return;
  }
}

}  // namespace rounds
}  // namespace asap
