// asap_launch.h -- kernel launchers shared by the host library and the .hip
// translation units.  Internal; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asap.h"

namespace asap {

// Epoch tags: 2r = "models of round r at the start of the round",
// 2r + 1 = "round r half-step published" (the NOTIFY of Section 4).
__host__ __device__ inline int64_t tag_start(int64_t r) { return 2 * r; }
__host__ __device__ inline int64_t tag_half(int64_t r) { return 2 * r + 1; }

// The XCD (accelerator complex die) the calling wave runs on: hardware
// register XCC_ID, bits [3:0].  Workgroups of a launch are dealt to the
// XCDs round-robin.
__device__ __forceinline__ int xcd_id() {
  return int(__builtin_amdgcn_s_getreg(20 | (0 << 6) | ((16 - 1) << 11)) & 0xfu);
}

// Device error words (int32 each).
enum { kErrEpochCount = 0, kErrEpochWorker = 1, kErrRendezvous = 2, kErrWords = 16 };

struct MixArgs {
  const float* src;  // [n][ld] models being read (buffer e)
  float* dst;        // [n][ld] models being written (buffer e^1)
  int64_t ld, dim;
  int32_t n;
  const int32_t* nbr_ptr;
  const int32_t* nbr_idx;
  const float* nbr_w;
  const float* scale;  // per-worker L2 scale of the half-step, or null
  const int64_t* tag_src;
  int64_t* tag_dst;
  int64_t expect;  // tag every in-neighbour must carry in buffer e
  int64_t next;    // tag written for every reduced row in buffer e^1
  int32_t* err;
  int32_t* row_ok;  // [n] verdict of the epoch check (1 = every in-neighbour published)
  int32_t uniform_rows;  // 1: in every row all entries but the own one have one weight (bitwise)
};

hipError_t launch_epoch_check(const MixArgs& a, hipStream_t s);
hipError_t launch_mix(const MixArgs& a, hipStream_t s);
hipError_t launch_mix_slab(const MixArgs& a, int max_deg, int n_cu, hipStream_t s);
hipError_t launch_mean(const MixArgs& a, hipStream_t s);

// Row descriptor of one minibatch position, in schedule order.
struct RowInfo {
  long long start;  // offset of the row's first nonzero
  int len;          // nonzeros in the row
  float y;          // label
};

// Columns whose model entries the CSR kernel keeps in LDS for a whole pass.
constexpr int kHotMax = 8128;

struct SgdArgs {
  float* models;  // current buffer [n][ld]
  int64_t ld, dim;
  int32_t n;
  int64_t S;        // samples per worker
  const float* y;   // [n*S]
  // dense shards
  const float* X;   // [n][S][ldx]
  int64_t ldx;
  // CSR shards
  const int64_t* row_ptr;  // [n*S+1]
  const int32_t* col;
  const float* val;
  const float* vmax;       // [n] max |val| per worker
  const RowInfo* rowinfo;  // [n][S] this round's rows in schedule order
  const int32_t* code;     // [nnz] -(hot slot + 2) for a hot column, else the column
  const int32_t* hot_cols; // [n_hot] column of each hot slot
  int32_t n_hot;
  int32_t max_row;         // longest row (nonzeros)
  // schedule of this round, [n][S]
  const int32_t* sched;
  uint64_t seed;    // schedule seed (the dense pass evaluates the order itself)
  int32_t loss, lr_kind;
  float lr0, l2;
  int32_t batch;
  int64_t round;    // the pass the steps belong to: step k has t = round * K + k + 1
  int64_t k0, k1;   // steps [k0, k1) of that pass run in this launch (K = ceil(S / batch))
  float* scale;     // [n] out: final L2 scale (CSR)
  int64_t* tag;     // [n] tags of the current buffer
  int64_t tag_value;
  const int32_t* run_if;  // CSR general kernel: when set, run only if *run_if != 0
  // planned CSR pass with members (PlanArgs::members > 1): the exchange tag
  // of global step g = round * K + k is xtag + (g - xg0); the library keeps
  // tags unique for the life of a context
  uint32_t xtag;
  int64_t xg0;
};

// Per-round plan of a CSR pass (see kernels_csr_plan.hip).  The per-step
// lists live in the region of the worker's nonzeros where that step's
// nonzeros start in schedule order (step_off), so each list array has one
// entry per nonzero.
struct PlanArgs {
  const RowInfo* rowinfo;   // [n][S] this round's rows in schedule order
  const RowInfo* rows_real; // [workers][S] the same for whole workers (the general pass; = rowinfo with one member)
  const int32_t* code;      // [nnz] static codes: -(hot slot + 2) or column
  const int64_t* row_ptr;   // [n*S+1]
  int32_t n;
  int64_t S;
  int32_t batch;
  int32_t K;                // steps per pass
  int32_t* step_off;        // [n][S+1]
  const float* val;         // [nnz] values
  int2* pack;               // [nnz] this round: (-(hot slot + 2) or cold slot, value bits)
  int32_t* clist;           // [nnz] cold columns of each step, by slot
  int32_t* clink;           // [nnz] slot of the same column in the previous step, or -1
  int32_t* hlist;           // [nnz] distinct hot slots of each step
  int32_t* cnt;             // [n][S][2] distinct cold, hot per step
  int32_t* flag;            // [1] set when some step does not fit the fast kernel
  int64_t* progress;        // [n] global step the pass of each worker is on (round * K + k)
  int32_t helpers;          // 1: one prefetch workgroup per worker beside the pass
  // Members: `members` workgroups share a worker, member m owning the
  // columns c with c mod members == m.  The plan arrays above then describe
  // n * members "slices" (slice v = worker * members + member: the worker's
  // rows restricted to the member's columns, laid out like a worker of their
  // own), and n counts slices.  With one member a slice is the worker.
  int32_t members;
  int32_t workers;          // real workers
  int32_t max_slice;        // longest row of one member's columns
  int32_t n_cu;             // compute units of the device
  int32_t cold_step;        // cold nonzeros of a slice's step, on average (a sampled estimate)
  const int32_t* mhot;      // [members][kHotMax] column of each member's hot slot
  int32_t n_mhot[4];        // hot slots of each member
  unsigned long long* xch;  // [workers][2][members][64][2] tagged halves of partial margins (step parity 2nd)
  unsigned long long* done; // [workers][members] multi-round launch: tag of a member's last step
  unsigned long long* xid;  // [workers][members] (tag of a pass's first step, XCD) of each member
  int32_t* xerr;            // error word: a member waited too long for a partner
  long long xwait;          // wall-clock ticks a member waits for a partner
};
constexpr int kMaxMembers = 4;
bool csr_plan_fits(const SgdArgs& a);
// Rows of a planned CSR step, at most (the planned pass's minibatch limit).
constexpr int kPlanStepRows = 64;
// most: the most nonzeros one step of a slice can hold
hipError_t launch_csr_plan(const PlanArgs& p, int64_t most, hipStream_t s);
// pack[q] = (code[q], bits of val[q]) for every nonzero: the round-invariant
// part of the plan (the planning kernel rewrites the cold entries' codes)
hipError_t launch_pack_values(const int32_t* code, const float* val, int64_t nnz, int2* pack, hipStream_t s);
hipError_t launch_sgd_csr_fast(const SgdArgs& a, const PlanArgs& p, hipStream_t s);

hipError_t launch_schedule(uint64_t seed, int64_t round, int32_t n, int64_t S, int32_t* out,
                           hipStream_t s);
hipError_t launch_sgd_dense(const SgdArgs& a, hipStream_t s);

// Dense SGD for dim in (1024, 8192]: K workgroups per worker sum their
// partial gradients once per step as 64-bit fixed point in `acc`
// ([3][n][ldp], zero at launch), scaled from xmax ([n], max |x| of each
// shard); `count` ([n], zero at launch) counts arrivals.  A rendezvous that
// waits longer than spin_limit polls adds 1 to *err and ends the pass.
struct DenseSync {
  float* part;  // [2][n][K][ldp]: fp32 member partial gradients of step t (slot t & 1)
  int32_t* xcd;  // [n][K]: the XCD each member runs on
  uint32_t* count;
  int64_t ldp;
  int32_t K;
  uint32_t spin_limit;
  int32_t* err;
  uint32_t base;  // arrivals already counted when the pass starts
};
// Several rounds in one persistent launch with per-worker NOTIFY-ACK
// (Section 4; device side in rounds_device.h).  Workgroups of worker i run
// the same half-step code as the stream-ordered kernels, then reduce row i
// themselves.
struct RoundsArgs {
  float* buf[2];       // the two model buffers [n][ld]
  int32_t cur;         // buffer of round r0
  int32_t n;
  int64_t r0, R;       // rounds r0 .. r0 + R - 1
  int32_t local_steps; // as asap_sgd_params.local_steps
  uint64_t seed;       // schedule seed
  const int32_t* in_ptr;   // [n+1] graph rows: in-neighbours (self included)
  const int32_t* in_idx;
  const float* in_w;
  const int32_t* out_ptr;  // [n+1] the transpose: workers that read row i
  const int32_t* out_idx;
  int64_t* tag;        // [2][n] epoch tags, as the stream-ordered path keeps them
  float* scale2;       // [2][n] L2 scale of each worker's half-step, per buffer
  int32_t scaled;      // fold the scales into the weights (CSR with l2 > 0)
  int32_t fp64_mix;    // 1: reduce in fp64 (tile / mean kernels); 0: fp32 (slab kernel)
  long long wait_ticks;  // wall-clock ticks a worker waits for its neighbours
  int32_t* err;        // device error words
  int32_t* sched;      // [n][S] dense: this pass's schedule rows
  RowInfo* rowinfo;    // [n][S] CSR: this pass's row descriptors
  int64_t* msync;      // [n][kMemberSync] members of a worker: reduce go, parts done (-1 at launch)
};
constexpr int kMemberSync = 9;  // the go word and one word per member (up to 8)
// Plans of the passes of a multi-round launch on planned CSR passes: pass
// first_pass + u has its plan in area u (the pointers of area0 advanced by
// u * stride bytes); the area is published when ready[u] == token0 + u.
struct RoundsPlan {
  PlanArgs area0;
  int64_t stride;
  int64_t first_pass, npass;
  const int64_t* ready;
  int64_t token0;
};
constexpr int kRoundsMaxDeg = 64;  // in- and out-neighbours of a worker in a multi-round launch
hipError_t launch_rounds_dense(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s);
hipError_t launch_rounds_dense_wide(const SgdArgs& a, const DenseSync& ds, const RoundsArgs& ra, hipStream_t s);
hipError_t launch_rounds_csr(const SgdArgs& a, const RoundsArgs& ra, int n_cu, hipStream_t s);
hipError_t launch_rounds_csr_planned(const SgdArgs& a, const RoundsArgs& ra, const RoundsPlan& rp, int n_cu,
                                     hipStream_t s);
// whether the stream-ordered reduce of this graph runs the slab kernel
bool mix_slab_applies(const MixArgs& a, int max_deg);

hipError_t launch_dense_scan(const float* X, const float* y, int32_t n, int64_t S, int64_t dim, int64_t ldx,
                             float* xmax, unsigned long long* out, hipStream_t s);
int dense_wide_cpq(int64_t dim);                               // 0: not handled
int dense_wide_max_members(const SgdArgs& a, int n_cu);        // co-resident workgroups
hipError_t launch_sgd_dense_wide(const SgdArgs& a, const DenseSync& ds, hipStream_t s);
hipError_t launch_sgd_csr(const SgdArgs& a, hipStream_t s);
hipError_t launch_rowinfo(const int32_t* sched, const int64_t* row_ptr, const float* y, int32_t n, int64_t S,
                          RowInfo* out, hipStream_t s, int32_t members = 1);
// Bind time, members > 1: cnt[(i * members + m) * S + r] = nonzeros of row r
// of worker i in member m's columns; *maxlen (zeroed before) = the largest.
hipError_t launch_member_count(const int64_t* row_ptr, const int32_t* col, int32_t n, int64_t S, int32_t members,
                               int32_t* cnt, int32_t* maxlen, hipStream_t s);
// Bind time, members > 1: each nonzero to its slice position (vrow_ptr, rows
// keep their entries' order): vcode (if not null) gets its code from mlut
// (member-local hot slot or -1), pack (if not null) its (code, value) pair.
hipError_t launch_member_scatter(const int64_t* row_ptr, const int32_t* col, const float* val, const int16_t* mlut,
                                 int32_t n, int64_t S, int32_t members, const int64_t* vrow_ptr, int32_t* vcode,
                                 int2* pack, hipStream_t s);
hipError_t launch_col_hist(const int32_t* col, int64_t nnz, int64_t stride, int32_t* counts, hipStream_t s);
hipError_t launch_codes(const int32_t* col, int64_t nnz, const int16_t* lut, int32_t* code, hipStream_t s);

// Bind-time scan of CSR shards: vmax[i] = max |val| of worker i; out[0] =
// max row length, out[1] = count of columns outside [0, dim), out[2] =
// count of labels outside {-1, +1}, out[3] = count of rows with unsorted or
// repeated columns, out[4] = count of rows whose offsets decrease or are
// negative (plus one if row_ptr[0] != 0), out[5] = most nonzeros of one
// worker.  out must be zeroed before.
hipError_t launch_csr_scan(const int64_t* row_ptr, const int32_t* col, const float* val,
                           const float* y, int32_t n, int64_t S, int64_t dim, float* vmax,
                           int64_t* out, hipStream_t s);
hipError_t launch_fill_i64(int64_t* p, int64_t count, int64_t value, hipStream_t s);
hipError_t launch_fill_f32(float* p, int64_t count, float value, hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int64_t count, int32_t value, hipStream_t s);

struct MetricArgs {
  const float* W;  // current buffer [n][ld]
  int64_t ld, dim;
  int32_t n;
  const float* scale;  // or null
  int64_t S;
  const float* y;
  const float* X;
  int64_t ldx;
  const int64_t* row_ptr;
  const int32_t* col;
  const float* val;
  int32_t loss;
  float l2;
  double* wbar;     // [dim]
  double* part;     // partial sums: metric_part_doubles(n, S)
  double* out;      // [4] device
};

// The loss pass splits each worker's samples (and model entries) over
// metric_chunks(n, S) workgroups, so that about 2048 workgroups share the
// data however few workers there are.
constexpr int kMetricColBlocks = 4096;
inline int metric_chunks(int64_t n, int64_t S) {
  int64_t c = n >= 2048 ? 1 : 2048 / n;
  if (c > 64) c = 64;
  if (S > 0 && c > S) c = S;
  return int(c < 1 ? 1 : c);
}
inline size_t metric_part_doubles(int64_t n, int64_t S) {
  return size_t(2 * kMetricColBlocks) + 3 * size_t(n) * size_t(metric_chunks(n, S));
}
hipError_t launch_metrics(const MetricArgs& a, hipStream_t s);

// asap_metrics with its scratch (w_bar, partial sums, the four results) in
// the library's static device array instead of the context's workspace.
// Fills a.wbar / a.part / a.out itself, runs the same kernels, copies the
// results to out_host and synchronises `s`.  Returns hipErrorInvalidValue
// when dim or n exceeds the array's limits (kStaticMetricMaxDim,
// kStaticMetricMaxWorkers).
constexpr int64_t kStaticMetricMaxDim = int64_t(1) << 20;
constexpr int64_t kStaticMetricMaxWorkers = 16384;
hipError_t metrics_static_scratch(MetricArgs a, hipStream_t s, double* out_host);

}  // namespace asap
