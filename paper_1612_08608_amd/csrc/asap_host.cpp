// asap_host.cpp -- the C ABI: graph builders, validation, the round state
// machine (double buffer + epoch tags) and kernel dispatch.
//
// The library owns no device memory.  Device state (graph copy, epoch tags,
// per-worker L2 scales, error words, the round's sample schedule and metric
// partials) lives in the caller's workspace at fixed offsets.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <string>
#include <vector>

#include "asap.h"
#include "asap_common.h"
#include "asap_launch.h"

using namespace asap;

namespace {

thread_local std::string g_free_error;  // message of the last context-free failure

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

enum DataKind { kNoData = 0, kDense = 1, kCsr = 2 };

// dense workspace: up to 8 workgroups per worker, sized for a 256-CU device
// (the launch takes fewer when fewer are co-resident)
constexpr int kDenseMaxMembers = 8;
constexpr int kDenseCus = 256;
constexpr uint32_t kDenseSpinLimit = 1u << 20;
constexpr int32_t kRoundsWaitMs = 10000;  // default bound on one neighbour wait of the multi-round launch

// Per-round buffers of the CSR pass: the sample schedule, row descriptors
// and the column plan.  CSR workspaces hold two, so that the next round can
// be planned while this one runs.
struct RoundPlan {
  size_t sched = 0, rowinfo = 0, vrowinfo = 0, soff = 0, pack = 0, clist = 0, clink = 0, hlist = 0, cnt = 0,
         flag = 0;
};

constexpr long long kMemberWaitMs = 2000;  // bound on one wait of a planned-pass member for a partner

}  // namespace

struct asap_ctx {
  int32_t n = 0;
  int64_t dim = 0;
  std::vector<int32_t> ptr, idx;
  std::vector<float> w;
  std::vector<int32_t> optr, oidx;  // the transpose: the workers that read row i
  bool complete_uniform = false;
  bool uniform_rows = false;  // every row: the entries other than its own share one weight (bitwise)
  int32_t max_deg = 0;  // longest row of the graph (entries, self included)
  int32_t max_out = 0;  // most workers that read one row
  int32_t n_cu = 256;   // compute units of the device the workspace is on
  long long clock_khz = 100000;  // its wall clock (s_memrealtime) rate

  // caller-owned device memory
  char* ws = nullptr;
  size_t ws_bytes = 0;
  float* buf[2] = {nullptr, nullptr};
  int64_t ld = 0;

  int kind = kNoData;
  const float* X = nullptr;
  int64_t ldx = 0;
  const float* y = nullptr;
  int64_t S = 0;
  const int64_t* row_ptr = nullptr;
  const int32_t* col = nullptr;
  const float* val = nullptr;
  int64_t nnz = 0;

  // CSR: columns kept in LDS by the SGD kernel (chosen at workspace bind)
  std::vector<int32_t> hot_cols;
  std::vector<int16_t> hot_lut;
  int32_t max_row = 0;
  int64_t max_wnnz = 0;  // most nonzeros of one worker's shard
  // members of the planned CSR pass: workgroups per worker, member m owning
  // the columns c mod members == m (1: the worker's pass is one workgroup)
  int32_t members = 1;
  int32_t members_req = 0;   // asap_set_csr_members (0: chosen from the worker and compute-unit counts)
  int32_t max_slice = 0;     // longest row of one member's columns
  // step_most[b]: the most nonzeros b rows of one slice hold (the b longest
  // rows of the fullest slice), b <= kPlanStepRows: what one planned step holds
  std::vector<int32_t> step_most;
  int32_t n_mhot[kMaxMembers] = {0, 0, 0, 0};
  double cold_share = 1.0;   // of the nonzeros, those without a hot slot (sampled at bind)
  uint64_t xseq = 1;         // exchange tag of the next planned step (never reused by a context)

  // workspace layout (byte offsets)
  size_t off_ptr = 0, off_idx = 0, off_w = 0, off_optr = 0, off_oidx = 0, off_tag = 0, off_scale = 0, off_err = 0,
         off_vmax = 0, off_scan = 0, off_wbar = 0, off_part = 0, off_out = 0, off_rowok = 0,
         off_code = 0, off_lut = 0, off_hot = 0, off_dacc = 0, off_dxcd = 0, off_dcount = 0, off_progress = 0,
         off_vrp = 0, off_vcode = 0, off_mlut = 0, off_mhot = 0, off_xch = 0, off_done = 0, off_xid = 0,
         off_msync = 0, total = 0;
  RoundPlan plan[2];
  int32_t dense_k = 1;  // workgroups per worker the dense workspace is sized for

  // plan ring of the multi-round launch (asap_bind_rounds_plan): epoch
  // tokens [areas] int64 at the start, then `areas` plan areas of
  // ring_stride bytes laid out as ring_lay
  char* ring = nullptr;
  int64_t ring_areas = 0;
  size_t ring_stride = 0;
  RoundPlan ring_lay;
  int64_t ring_epoch = 0;
  bool ring_valid = false;
  hipEvent_t ev_ring_free = nullptr;  // after the last launch that read the ring

  // round state
  int32_t cur = 0;
  int64_t round = 0;
  bool half_done = false;
  bool half_scaled = false;  // the half-step left per-worker L2 scales to fold
  bool tags_ready = false;

  // look-ahead planning of the CSR pass: after launching the last steps of
  // pass q, the plan of pass q + 1 (same seed and batch) is built on a
  // stream of the library's own into the other RoundPlan; a later call uses
  // it when its pass, seed and batch match
  hipStream_t ahead = nullptr;
  hipEvent_t ev_start = nullptr, ev_ready[2] = {nullptr, nullptr}, ev_used[2] = {nullptr, nullptr};
  bool ahead_valid = false;
  int ahead_slot = 0;
  uint64_t ahead_seed = 0;
  int64_t ahead_pass = -1;
  int32_t ahead_batch = 0;

  // the half-step inputs enqueued by asap_prepare_sgd (or by asap_local_sgd
  // itself): which RoundPlan holds them and for which pass, seed and batch
  // (they serve every round whose steps lie in that pass)
  bool prep_valid = false;
  int prep_slot = 0;
  uint64_t prep_seed = 0;
  int64_t prep_pass = -1;
  int32_t prep_batch = 0;

  std::string err;
};

namespace {

asap_status fail(asap_ctx* c, asap_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c)
    c->err = buf;
  else
    g_free_error = buf;
  return s;
}

asap_status hip_fail(asap_ctx* c, hipError_t e, const char* what) {
  return fail(c, ASAP_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

template <class T>
T* at(asap_ctx* c, size_t off) {
  return reinterpret_cast<T*>(c->ws + off);
}

// Members of the planned CSR pass: the caller's choice, else 4 or 2
// workgroups per worker while they take at most half the compute units
// (the other half plans the next pass beside it), else 1.
int32_t csr_members(asap_ctx* c) {
  if (c->members_req > 0) return c->members_req;
  int cus = c->n_cu;
  {
    int dev_id = 0, q = 0;
    if (hipGetDevice(&dev_id) == hipSuccess &&
        hipDeviceGetAttribute(&q, hipDeviceAttributeMultiprocessorCount, dev_id) == hipSuccess && q > 0)
      cus = q;
  }
  for (int32_t m = kMaxMembers; m > 1; m /= 2)
    if (int64_t(c->n) * m <= cus / 2) return m;
  return 1;
}

void layout(asap_ctx* c) {
  const size_t n = size_t(c->n), nnz = c->idx.size();
  size_t o = 0;
  c->off_ptr = o;   o = align_up(o + (n + 1) * 4);
  c->off_idx = o;   o = align_up(o + nnz * 4);
  c->off_w = o;     o = align_up(o + nnz * 4);
  c->off_optr = o;  o = align_up(o + (n + 1) * 4);
  c->off_oidx = o;  o = align_up(o + nnz * 4);
  c->off_tag = o;   o = align_up(o + 2 * n * 8);
  c->off_scale = o; o = align_up(o + 2 * n * 4);  // [2][n]: the multi-round launch keeps one per buffer
  c->off_err = o;   o = align_up(o + kErrWords * 4);
  c->off_vmax = o;  o = align_up(o + n * 4);
  c->off_scan = o;  o = align_up(o + 8 * 8);
  c->off_rowok = o; o = align_up(o + n * 4);
  c->off_msync = o; o = align_up(o + n * kMemberSync * 8);
  c->plan[0].sched = o; o = align_up(o + n * size_t(c->S) * 4);
  c->off_wbar = o;  o = align_up(o + size_t(c->dim) * 8);
  c->off_part = o;  o = align_up(o + metric_part_doubles(int64_t(n), c->S) * 8);
  c->off_out = o;   o = align_up(o + 8 * 8);
  const bool csr = c->kind == kCsr;
  c->off_code = o;    o = align_up(o + (csr ? size_t(c->nnz) * 4 : 0));
  c->off_lut = o;     o = align_up(o + (csr ? size_t(c->dim) * 2 : 0));
  c->off_hot = o;     o = align_up(o + (csr ? size_t(kHotMax) * 4 : 0));
  c->off_progress = o; o = align_up(o + (csr ? n * kMaxMembers * 8 : 0));  // one word per slice
  c->members = csr ? csr_members(c) : 1;
  const size_t M = size_t(c->members), split = csr && M > 1 ? 1 : 0;
  c->off_vrp = o;   o = align_up(o + split * (n * M * size_t(c->S) + 1) * 8);
  c->off_vcode = o; o = align_up(o + split * size_t(c->nnz) * 4);
  c->off_mlut = o;  o = align_up(o + split * size_t(c->dim) * 2);
  c->off_mhot = o;  o = align_up(o + split * M * kHotMax * 4);
  c->off_xch = o;   o = align_up(o + split * 2 * n * M * 128 * 8);
  c->off_done = o;  o = align_up(o + split * n * M * 8);
  c->off_xid = o;   o = align_up(o + split * n * M * 8);
  // per-round buffers of the CSR pass, twice: one entry per nonzero per list
  const size_t nz = csr ? size_t(c->nnz) : 0, nS = csr ? n * size_t(c->S) : 0;
  for (int k = 0; k < 2; ++k) {
    RoundPlan& r = c->plan[k];
    if (k == 1) { r.sched = o; o = align_up(o + (csr ? nS * 4 : 0)); }
    r.rowinfo = o; o = align_up(o + nS * sizeof(RowInfo));
    r.vrowinfo = r.rowinfo;
    if (split) { r.vrowinfo = o; o = align_up(o + M * nS * sizeof(RowInfo)); }
    r.soff = o;    o = align_up(o + (csr ? M * n * (size_t(c->S) + 1) * 4 : 0));
    r.pack = o;    o = align_up(o + nz * 8);
    r.clist = o;   o = align_up(o + nz * 4);
    r.clink = o;   o = align_up(o + nz * 4);
    r.hlist = o;   o = align_up(o + nz * 4);
    r.cnt = o;     o = align_up(o + M * nS * 2 * 4);
    r.flag = o;    o = align_up(o + (csr ? 4 : 0));
  }
  const int cpq = c->kind == kDense ? dense_wide_cpq(c->dim) : 0;
  c->dense_k = cpq ? std::max(1, std::min(kDenseMaxMembers, kDenseCus / std::max(1, c->n))) : 1;
  const size_t ldp = size_t(cpq) * 2048;
  c->off_dacc = o;    o = align_up(o + (c->dense_k > 1 ? 2 * n * size_t(c->dense_k) * ldp * 4 : 0));
  c->off_dxcd = o;    o = align_up(o + (c->dense_k > 1 ? n * size_t(c->dense_k) * 4 : 0));
  c->off_dcount = o;  o = align_up(o + (cpq ? n * 4 : 0));
  c->total = o;
}

// Waits for look-ahead planning still in flight and forgets it.  Every call
// that may precede a release or rebinding of memory the planning reads or
// writes comes here first.
void drain_ahead(asap_ctx* c) {
  if (c->ahead) (void)hipStreamSynchronize(c->ahead);
  c->ahead_valid = false;
  c->prep_valid = false;
}

void release_ahead(asap_ctx* c) {
  drain_ahead(c);
  if (c->ahead) (void)hipStreamDestroy(c->ahead);
  for (hipEvent_t* ev : {&c->ev_start, &c->ev_ready[0], &c->ev_ready[1], &c->ev_used[0], &c->ev_used[1],
                         &c->ev_ring_free})
    if (*ev) {
      (void)hipEventDestroy(*ev);
      *ev = nullptr;
    }
  c->ahead = nullptr;
  c->ring_valid = false;
}

void unbind_workspace(asap_ctx* c) {
  drain_ahead(c);
  c->ring_valid = false;  // its bind-time halves depend on the data and the workspace's codes
  c->ws = nullptr;
  c->ws_bytes = 0;
  c->tags_ready = false;
}

// --------------------------------------------------------------------------
// graph validation
// --------------------------------------------------------------------------
asap_status check_graph(asap_ctx* c, int32_t n, const int32_t* ptr, const int32_t* idx,
                        const float* w, uint32_t flags) {
  if (ptr[0] != 0) return fail(c, ASAP_E_GRAPH, "nbr_ptr[0] must be 0");
  for (int32_t i = 0; i < n; ++i)
    if (ptr[i + 1] < ptr[i]) return fail(c, ASAP_E_GRAPH, "nbr_ptr decreases at row %d", i);
  const int64_t nnz = ptr[n];
  if (nnz > int64_t(n) * n) return fail(c, ASAP_E_GRAPH, "more than n*n entries");
  std::vector<double> colsum(n, 0.0);
  for (int32_t i = 0; i < n; ++i) {
    bool self = false;
    double rs = 0.0;
    for (int32_t p = ptr[i]; p < ptr[i + 1]; ++p) {
      const int32_t j = idx[p];
      if (j < 0 || j >= n) return fail(c, ASAP_E_GRAPH, "row %d: neighbour %d out of range", i, j);
      if (p > ptr[i] && idx[p - 1] >= j)
        return fail(c, ASAP_E_GRAPH, "row %d: neighbours not strictly ascending", i);
      if (j == i) self = true;
      const float wt = w[p];
      if (!std::isfinite(wt) || wt < 0.0f)
        return fail(c, ASAP_E_GRAPH, "row %d: weight %g is negative or not finite", i, double(wt));
      rs += wt;
      colsum[j] += wt;
    }
    if (!self) return fail(c, ASAP_E_GRAPH, "row %d lacks its self entry", i);
    const double tol = 1e-6 + double(ptr[i + 1] - ptr[i]) * std::ldexp(1.0, -24);
    if (!(flags & ASAP_ALLOW_NON_DS) && std::fabs(rs - 1.0) > tol)
      return fail(c, ASAP_E_GRAPH, "row %d sums to %.9g, not 1 (P must be doubly stochastic)", i, rs);
  }
  if (!(flags & ASAP_ALLOW_NON_DS)) {
    for (int32_t j = 0; j < n; ++j) {
      // column j collects at most n weights
      const double tol = 1e-6 + double(n) * std::ldexp(1.0, -24);
      if (std::fabs(colsum[j] - 1.0) > tol)
        return fail(c, ASAP_E_GRAPH, "column %d sums to %.9g, not 1 (P must be doubly stochastic)", j,
                    colsum[j]);
    }
  }
  return ASAP_OK;
}

bool is_complete_uniform(int32_t n, const int32_t* ptr, const float* w) {
  if (int64_t(ptr[n]) != int64_t(n) * n) return false;
  uint32_t w0;
  std::memcpy(&w0, &w[0], 4);
  for (int64_t p = 0; p < int64_t(n) * n; ++p) {
    uint32_t b;
    std::memcpy(&b, &w[p], 4);
    if (b != w0) return false;
  }
  return true;  // n*n strictly ascending in-range entries = every j in every row
}

asap_status need_device(asap_ctx* c) {
  if (!c->buf[0] || !c->buf[1]) return fail(c, ASAP_E_STATE, "models are not bound");
  if (!c->ws) return fail(c, ASAP_E_STATE, "workspace is not bound");
  if (!c->tags_ready) return fail(c, ASAP_E_STATE, "workspace is not initialised");
  return ASAP_OK;
}

asap_status check_params(asap_ctx* c, const asap_sgd_params* p) {
  if (!p) return fail(c, ASAP_E_INVALID_ARG, "params is NULL");
  if (p->loss != ASAP_LOSS_LOGISTIC && p->loss != ASAP_LOSS_HINGE)
    return fail(c, ASAP_E_INVALID_ARG, "unknown loss %d", p->loss);
  if (p->lr_kind != ASAP_LR_CONST && p->lr_kind != ASAP_LR_INV_SQRT)
    return fail(c, ASAP_E_INVALID_ARG, "unknown lr_kind %d", p->lr_kind);
  if (!(std::isfinite(p->lr0) && p->lr0 > 0.0f)) return fail(c, ASAP_E_INVALID_ARG, "lr0 must be > 0");
  if (!(std::isfinite(p->l2) && p->l2 >= 0.0f)) return fail(c, ASAP_E_INVALID_ARG, "l2 must be >= 0");
  if (p->batch < 1) return fail(c, ASAP_E_INVALID_ARG, "batch must be >= 1");
  if (c->kind == kCsr && p->batch > 512)
    return fail(c, ASAP_E_INVALID_ARG, "CSR minibatch is limited to 512 rows");
  if (p->local_steps < 0) return fail(c, ASAP_E_INVALID_ARG, "local_steps must be >= 0");
  if (p->local_steps > 0) {
    const int64_t K = (c->S + p->batch - 1) / p->batch;
    if (K % p->local_steps)
      return fail(c, ASAP_E_INVALID_ARG, "local_steps %d does not divide the %lld steps of a pass", p->local_steps,
                  (long long)K);
  }
  return ASAP_OK;
}

// The CSR kernel keeps the model entries of the most frequent columns in LDS
// for a whole pass.  Frequencies come from every 2^k-th nonzero (a sample
// large enough to rank the heavy columns); ties break by column index so the
// choice is deterministic.  Every nonzero then gets its code: -(slot + 2)
// for a hot column, the column itself otherwise.
asap_status choose_hot_columns(asap_ctx* c, hipStream_t s) {
  hipError_t e;
  const int64_t D = c->dim;
  int32_t* counts = at<int32_t>(c, c->off_wbar);  // the metric buffer is free at bind time
  int64_t stride = 1;
  while (c->nnz / stride > (int64_t(1) << 24)) stride *= 2;
  std::vector<int32_t> h(size_t(D), 0);
  if ((e = launch_fill_i32(counts, D, 0, s)) || (e = launch_col_hist(c->col, c->nnz, stride, counts, s)) ||
      (e = hipMemcpyAsync(h.data(), counts, size_t(D) * 4, hipMemcpyDeviceToHost, s)) ||
      (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "column histogram");
  std::vector<int32_t> cols;
  for (int64_t j = 0; j < D; ++j)
    if (h[j] > 0) cols.push_back(int32_t(j));
  const size_t H = std::min<size_t>(cols.size(), kHotMax);
  std::partial_sort(cols.begin(), cols.begin() + H, cols.end(), [&](int32_t x, int32_t y) {
    return h[x] != h[y] ? h[x] > h[y] : x < y;
  });
  c->hot_cols.assign(cols.begin(), cols.begin() + H);
  c->hot_lut.assign(size_t(D), int16_t(-1));
  for (size_t k = 0; k < H; ++k) c->hot_lut[c->hot_cols[k]] = int16_t(k);
  int16_t* lut = at<int16_t>(c, c->off_lut);
  if ((H && (e = hipMemcpyAsync(at<int32_t>(c, c->off_hot), c->hot_cols.data(), H * 4, hipMemcpyHostToDevice, s))) ||
      (e = hipMemcpyAsync(lut, c->hot_lut.data(), size_t(D) * 2, hipMemcpyHostToDevice, s)) ||
      (e = launch_codes(c->col, c->nnz, lut, at<int32_t>(c, c->off_code), s)) ||
      (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "hot column tables");
  c->n_mhot[0] = int32_t(H);
  // the share of the sampled nonzeros without a hot slot (of their member's
  // set when there are several): planning sizes its link kernel by it
  double all = 0.0, cold = 0.0;
  for (int32_t j : cols) all += h[j];
  if (c->members == 1)
    for (size_t k = H; k < cols.size(); ++k) cold += h[cols[k]];
  if (c->members > 1) {
    // each member keeps the most frequent of its own columns, by the same
    // order
    const int32_t M = c->members;
    std::vector<int32_t> mhot(size_t(M) * kHotMax, 0);
    std::vector<int16_t> mlut(size_t(D), int16_t(-1));
    for (int32_t m = 0; m < M; ++m) {
      std::vector<int32_t> own;
      for (int32_t j : cols)
        if (j % M == m) own.push_back(j);
      const size_t Hm = std::min<size_t>(own.size(), kHotMax);
      std::partial_sort(own.begin(), own.begin() + Hm, own.end(), [&](int32_t x, int32_t y) {
        return h[x] != h[y] ? h[x] > h[y] : x < y;
      });
      for (size_t k = 0; k < Hm; ++k) {
        mhot[size_t(m) * kHotMax + k] = own[k];
        mlut[own[k]] = int16_t(k);
      }
      for (size_t k = Hm; k < own.size(); ++k) cold += h[own[k]];
      c->n_mhot[m] = int32_t(Hm);
    }
    if ((e = hipMemcpyAsync(at<int32_t>(c, c->off_mhot), mhot.data(), mhot.size() * 4, hipMemcpyHostToDevice, s)) ||
        (e = hipMemcpyAsync(at<int16_t>(c, c->off_mlut), mlut.data(), size_t(D) * 2, hipMemcpyHostToDevice, s)) ||
        (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "member hot column tables");
  }
  c->cold_share = all > 0.0 ? cold / all : 0.0;
  return ASAP_OK;
}

// Members > 1: the slices' row offsets (each worker's rows restricted to
// each member's columns, slice v = worker * members + member, laid out one
// after another) and every nonzero's code in slice order.  One member: the
// slices are the workers.
// step_most from the row lengths of every slice ([slices][S], in slice order).
void set_step_most(asap_ctx* c, const std::vector<int32_t>& len, int64_t slices) {
  c->step_most.assign(kPlanStepRows + 1, 0);
  std::vector<int32_t> top;
  for (int64_t v = 0; v < slices; ++v) {
    top.assign(len.begin() + v * c->S, len.begin() + (v + 1) * c->S);
    const int64_t b = std::min<int64_t>(kPlanStepRows, c->S);
    std::partial_sort(top.begin(), top.begin() + b, top.end(), std::greater<int32_t>());
    int32_t acc = 0;
    for (int64_t q = 0; q < b; ++q) {
      acc += top[size_t(q)];
      c->step_most[size_t(q + 1)] = std::max(c->step_most[size_t(q + 1)], acc);
    }
  }
  for (int q = 1; q <= kPlanStepRows; ++q) c->step_most[q] = std::max(c->step_most[q], c->step_most[q - 1]);
}

// The most nonzeros one planned step of `batch` rows can hold.
int64_t step_bound(const asap_ctx* c, int32_t batch) {
  const int32_t b = std::min<int32_t>(batch, kPlanStepRows);
  if (size_t(b) < c->step_most.size()) return c->step_most[size_t(b)];
  return int64_t(b) * c->max_slice;  // not measured: rows times the longest row
}

asap_status split_members(asap_ctx* c, hipStream_t s) {
  c->max_slice = c->max_row;
  hipError_t e;
  if (c->members == 1) {
    // the rows' lengths, for the bound on a step's nonzeros
    const size_t rows = size_t(c->n) * size_t(c->S);
    std::vector<int64_t> rp(rows + 1);
    if ((e = hipMemcpyAsync(rp.data(), c->row_ptr, (rows + 1) * 8, hipMemcpyDeviceToHost, s)) ||
        (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "row offsets readback");
    std::vector<int32_t> len(rows);
    for (size_t q = 0; q < rows; ++q) len[q] = int32_t(rp[q + 1] - rp[q]);
    set_step_most(c, len, c->n);
    return ASAP_OK;
  }
  const int32_t M = c->members;
  const size_t rows = size_t(c->n) * size_t(M) * size_t(c->S);
  // the counts (int32) go to the slice-offset array first, which the
  // offsets (int64, summed on the host) then replace
  int32_t* cnt = at<int32_t>(c, c->off_vrp);
  int32_t* mx = at<int32_t>(c, c->off_scan);
  std::vector<int32_t> h(rows);
  if ((e = launch_fill_i32(mx, 1, 0, s)) ||
      (e = launch_member_count(c->row_ptr, c->col, c->n, c->S, M, cnt, mx, s)) ||
      (e = hipMemcpyAsync(h.data(), cnt, rows * 4, hipMemcpyDeviceToHost, s)) ||
      (e = hipMemcpyAsync(&c->max_slice, mx, 4, hipMemcpyDeviceToHost, s)) || (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "member split counts");
  std::vector<int64_t> vrp(rows + 1);
  int64_t acc = 0;
  for (size_t q = 0; q < rows; ++q) {
    vrp[q] = acc;
    acc += h[q];
  }
  vrp[rows] = acc;
  if (acc != c->nnz) return fail(c, ASAP_E_INVALID_ARG, "member split counted %lld of %lld nonzeros",
                                 (long long)acc, (long long)c->nnz);
  set_step_most(c, h, int64_t(c->n) * M);
  int64_t* d_vrp = at<int64_t>(c, c->off_vrp);
  if ((e = hipMemcpyAsync(d_vrp, vrp.data(), (rows + 1) * 8, hipMemcpyHostToDevice, s)) ||
      (e = launch_member_scatter(c->row_ptr, c->col, c->val, at<int16_t>(c, c->off_mlut), c->n, c->S, M, d_vrp,
                                 at<int32_t>(c, c->off_vcode), nullptr, s)) ||
      (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "member split");
  return ASAP_OK;
}

// The bind-time halves of a plan's (code, value) pairs, in slice order.
hipError_t write_pack(asap_ctx* c, int2* pack, hipStream_t s) {
  if (c->members == 1) return launch_pack_values(at<int32_t>(c, c->off_code), c->val, c->nnz, pack, s);
  return launch_member_scatter(c->row_ptr, c->col, c->val, at<int16_t>(c, c->off_mlut), c->n, c->S, c->members,
                               at<int64_t>(c, c->off_vrp), nullptr, pack, s);
}

}  // namespace

// ============================================================================
// host-only builders
// ============================================================================
extern "C" asap_status asap_graph_ring(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx) {
  if (n < 3 || n > (1 << 28)) return fail(nullptr, ASAP_E_INVALID_ARG, "ring needs 3 <= n <= 2^28");
  if (!nbr_ptr || !nbr_idx) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL output");
  for (int32_t i = 0; i < n; ++i) {
    int32_t a = (i + n - 1) % n, b = i, d = (i + 1) % n;
    int32_t r[3] = {a, b, d};
    std::sort(r, r + 3);
    nbr_ptr[i] = 3 * i;
    for (int k = 0; k < 3; ++k) nbr_idx[3 * i + k] = r[k];
  }
  nbr_ptr[n] = 3 * n;
  return ASAP_OK;
}

namespace {
int32_t ceil_sqrt(int32_t n) {
  int32_t s = 0;
  while (int64_t(s) * s < n) ++s;
  return s;
}
}  // namespace

extern "C" asap_status asap_graph_root_expander(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx) {
  if (n < 3 || n > (1 << 28)) return fail(nullptr, ASAP_E_INVALID_ARG, "root expander needs 3 <= n <= 2^28");
  if (!nbr_ptr || !nbr_idx) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL output");
  const int32_t r = ceil_sqrt(n);  // 2 <= r < n, so i, i-1, i-r are distinct
  for (int32_t i = 0; i < n; ++i) {
    int32_t v[3] = {i, (i + n - 1) % n, (i + n - r) % n};
    std::sort(v, v + 3);
    nbr_ptr[i] = 3 * i;
    for (int k = 0; k < 3; ++k) nbr_idx[3 * i + k] = v[k];
  }
  nbr_ptr[n] = 3 * n;
  return ASAP_OK;
}

extern "C" asap_status asap_graph_chain(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx) {
  if (n < 2 || n > (1 << 28)) return fail(nullptr, ASAP_E_INVALID_ARG, "chain needs 2 <= n <= 2^28");
  if (!nbr_ptr || !nbr_idx) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL output");
  for (int32_t i = 0; i < n; ++i) {
    const int32_t a = (i + n - 1) % n;
    nbr_ptr[i] = 2 * i;
    nbr_idx[2 * i] = std::min(a, i);
    nbr_idx[2 * i + 1] = std::max(a, i);
  }
  nbr_ptr[n] = 2 * n;
  return ASAP_OK;
}

extern "C" asap_status asap_graph_complete(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx) {
  if (n < 1 || n > 46340) return fail(nullptr, ASAP_E_INVALID_ARG, "complete needs 1 <= n <= 46340");
  if (!nbr_ptr || !nbr_idx) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL output");
  for (int32_t i = 0; i < n; ++i) {
    nbr_ptr[i] = i * n;
    for (int32_t j = 0; j < n; ++j) nbr_idx[int64_t(i) * n + j] = j;
  }
  nbr_ptr[n] = n * n;
  return ASAP_OK;
}

namespace {

struct Stream64 {
  uint64_t state;
  uint64_t next() {
    state += kGamma;
    return mix64(state);
  }
  // Uniform in [0, m): reject the top (2^64 mod m) values.
  uint64_t below(uint64_t m) {
    const uint64_t rem = (0 - m) % m;  // 2^64 mod m
    for (;;) {
      const uint64_t r = next();
      if (rem == 0 || r < 0 - rem) return r % m;
    }
  }
};

bool connected(const std::vector<std::vector<int32_t>>& adj) {
  const size_t n = adj.size();
  std::vector<char> seen(n, 0);
  std::vector<int32_t> q;
  q.reserve(n);
  q.push_back(0);
  seen[0] = 1;
  for (size_t h = 0; h < q.size(); ++h)
    for (int32_t v : adj[q[h]])
      if (!seen[v]) {
        seen[v] = 1;
        q.push_back(v);
      }
  return q.size() == n;
}

}  // namespace

extern "C" asap_status asap_graph_random_regular(int32_t n, int32_t d, uint64_t seed,
                                                 int32_t* nbr_ptr, int32_t* nbr_idx) {
  // a 1-regular graph on more than two nodes is a matching and never connected
  if (n < 2 || n > (1 << 20) || d < 1 || d >= n || (int64_t(n) * d) % 2 || (d == 1 && n > 2))
    return fail(nullptr, ASAP_E_INVALID_ARG,
                "random_regular needs 1 <= d < n <= 2^20, n*d even, d >= 2 unless n == 2");
  if (!nbr_ptr || !nbr_idx) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL output");
  Stream64 rng{derive_key(seed, kTagGraph, uint64_t(n), uint64_t(d), 0)};
  std::vector<std::vector<int32_t>> adj(n);
  std::vector<int32_t> stubs;
  for (;;) {
    stubs.clear();
    for (int32_t v = 0; v < n; ++v)
      for (int32_t k = 0; k < d; ++k) stubs.push_back(v);
    for (auto& a : adj) a.clear();
    uint64_t stalls = 0;
    bool ok = true;
    while (!stubs.empty()) {
      const uint64_t m = stubs.size();
      const uint64_t a = rng.below(m), b = rng.below(m);
      const int32_t u = stubs[a], v = stubs[b];
      const bool exists = std::find(adj[u].begin(), adj[u].end(), v) != adj[u].end();
      if (a == b || u == v || exists) {
        if (++stalls > 100 * m) {
          ok = false;
          break;
        }
        continue;
      }
      stalls = 0;
      adj[u].push_back(v);
      adj[v].push_back(u);
      for (uint64_t k : {std::max(a, b), std::min(a, b)}) {
        stubs[k] = stubs.back();
        stubs.pop_back();
      }
    }
    if (ok && connected(adj)) break;
  }
  int32_t p = 0;
  for (int32_t i = 0; i < n; ++i) {
    std::vector<int32_t> row = adj[i];
    row.push_back(i);
    std::sort(row.begin(), row.end());
    nbr_ptr[i] = p;
    for (int32_t j : row) nbr_idx[p++] = j;
  }
  nbr_ptr[n] = p;
  return ASAP_OK;
}

extern "C" asap_status asap_metropolis_weights(int32_t n, const int32_t* ptr, const int32_t* idx,
                                               float* w) {
  if (n < 1 || !ptr || !idx || !w) return fail(nullptr, ASAP_E_INVALID_ARG, "bad arguments");
  for (int32_t i = 0; i < n; ++i) {
    double off = 0.0;
    int32_t self = -1;
    const int32_t di = ptr[i + 1] - ptr[i] - 1;
    for (int32_t p = ptr[i]; p < ptr[i + 1]; ++p) {
      const int32_t j = idx[p];
      if (j < 0 || j >= n) return fail(nullptr, ASAP_E_GRAPH, "row %d: neighbour out of range", i);
      if (j == i) {
        self = p;
        continue;
      }
      const int32_t dj = ptr[j + 1] - ptr[j] - 1;
      const double pij = 1.0 / (1.0 + double(std::max(di, dj)));
      off += pij;
      w[p] = float(pij);
    }
    if (self < 0) return fail(nullptr, ASAP_E_GRAPH, "row %d lacks its self entry", i);
    w[self] = float(1.0 - off);
  }
  return ASAP_OK;
}

extern "C" asap_status asap_schedule(int64_t samples, uint64_t seed, int32_t worker, int64_t round,
                                     int32_t* out) {
  if (samples < 0 || samples >= (int64_t(1) << 31) || (samples > 0 && !out))
    return fail(nullptr, ASAP_E_INVALID_ARG, "samples must be in [0, 2^31) with a non-NULL out");
  const Perm p = perm_make(seed, worker, round, uint32_t(samples));
  for (int64_t k = 0; k < samples; ++k) out[k] = int32_t(perm_at(p, uint32_t(k)));
  return ASAP_OK;
}

// ============================================================================
// context
// ============================================================================
namespace {
// The graph of a context (host copy) and what is derived from it: its
// transpose (the workers that read each row, ascending), the longest row and
// column, and whether it is the complete graph with uniform weights.
void set_graph(asap_ctx* c, int32_t n, const int32_t* nbr_ptr, const int32_t* nbr_idx, const float* nbr_w) {
  c->n = n;
  c->ptr.assign(nbr_ptr, nbr_ptr + n + 1);
  c->idx.assign(nbr_idx, nbr_idx + nbr_ptr[n]);
  c->w.assign(nbr_w, nbr_w + nbr_ptr[n]);
  c->complete_uniform = is_complete_uniform(n, nbr_ptr, nbr_w);
  c->uniform_rows = true;
  for (int32_t i = 0; i < n && c->uniform_rows; ++i) {
    bool first = true;
    uint32_t bits = 0;
    for (int32_t p = nbr_ptr[i]; p < nbr_ptr[i + 1]; ++p) {
      if (nbr_idx[p] == i) continue;
      uint32_t b;
      std::memcpy(&b, &nbr_w[p], 4);
      if (!first && b != bits) c->uniform_rows = false;
      bits = b;
      first = false;
    }
  }
  c->max_deg = 0;
  for (int32_t i = 0; i < n; ++i) c->max_deg = std::max(c->max_deg, nbr_ptr[i + 1] - nbr_ptr[i]);
  c->optr.assign(size_t(n) + 1, 0);
  for (int32_t p = 0; p < nbr_ptr[n]; ++p) ++c->optr[size_t(nbr_idx[p]) + 1];
  c->max_out = 0;
  for (int32_t j = 0; j < n; ++j) {
    c->max_out = std::max(c->max_out, c->optr[size_t(j) + 1]);
    c->optr[size_t(j) + 1] += c->optr[size_t(j)];
  }
  c->oidx.resize(size_t(nbr_ptr[n]));
  std::vector<int32_t> fill(c->optr.begin(), c->optr.end() - 1);
  for (int32_t i = 0; i < n; ++i)
    for (int32_t p = nbr_ptr[i]; p < nbr_ptr[i + 1]; ++p) c->oidx[size_t(fill[size_t(nbr_idx[p])]++)] = i;
}
}  // namespace

extern "C" asap_status asap_create(int32_t n, int64_t dim, const int32_t* nbr_ptr,
                                   const int32_t* nbr_idx, const float* nbr_w, uint32_t flags,
                                   asap_ctx** out) {
  if (!out) return fail(nullptr, ASAP_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (n < 1 || n > (1 << 20)) return fail(nullptr, ASAP_E_INVALID_ARG, "n_workers must be in [1, 2^20]");
  if (dim < 1 || dim > (int64_t(1) << 34)) return fail(nullptr, ASAP_E_INVALID_ARG, "dim must be in [1, 2^34]");
  if (!nbr_ptr || !nbr_idx || !nbr_w) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL graph array");
  if (flags & ~uint32_t(ASAP_ALLOW_NON_DS)) return fail(nullptr, ASAP_E_INVALID_ARG, "unknown flags");
  asap_status s = check_graph(nullptr, n, nbr_ptr, nbr_idx, nbr_w, flags);
  if (s != ASAP_OK) return s;
  asap_ctx* c = new asap_ctx;
  c->dim = dim;
  set_graph(c, n, nbr_ptr, nbr_idx, nbr_w);
  layout(c);
  *out = c;
  return ASAP_OK;
}

extern "C" asap_status asap_workspace_size(const asap_ctx* c, size_t* bytes) {
  if (!c || !bytes) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL argument");
  *bytes = c->total;
  return ASAP_OK;
}

extern "C" asap_status asap_bind_models(asap_ctx* c, float* b0, float* b1, int64_t ld, void* stream) {
  (void)stream;
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!b0 || !b1 || b0 == b1) return fail(c, ASAP_E_INVALID_ARG, "need two distinct model buffers");
  if (ld < c->dim || ld % 64) return fail(c, ASAP_E_INVALID_ARG, "ld must be >= dim and a multiple of 64");
  if ((uintptr_t(b0) | uintptr_t(b1)) % 256) return fail(c, ASAP_E_INVALID_ARG, "model buffers must be 256-byte aligned");
  c->buf[0] = b0;
  c->buf[1] = b1;
  c->ld = ld;
  c->cur = 0;
  c->round = 0;
  c->half_done = false;
  c->half_scaled = false;
  unbind_workspace(c);
  return ASAP_OK;
}

extern "C" asap_status asap_bind_dense(asap_ctx* c, const float* X, const float* y, int64_t S,
                                       int64_t ldx) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!X || !y) return fail(c, ASAP_E_INVALID_ARG, "NULL data pointer");
  if (S < 1 || S >= (int64_t(1) << 31)) return fail(c, ASAP_E_INVALID_ARG, "samples must be in [1, 2^31)");
  if (ldx < c->dim || ldx % 4 || uintptr_t(X) % 16)
    return fail(c, ASAP_E_INVALID_ARG, "ldx must be >= dim, a multiple of 4, X 16-byte aligned");
  if (c->dim > 16384) return fail(c, ASAP_E_INVALID_ARG, "dense path supports dim <= 16384");
  c->kind = kDense;
  c->X = X;
  c->y = y;
  c->S = S;
  c->ldx = ldx;
  c->row_ptr = nullptr;
  c->col = nullptr;
  c->val = nullptr;
  layout(c);
  unbind_workspace(c);
  return ASAP_OK;
}

extern "C" asap_status asap_bind_csr(asap_ctx* c, const int64_t* row_ptr, const int32_t* col,
                                     const float* val, const float* y, int64_t S, int64_t nnz,
                                     void* stream) {
  (void)stream;
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!row_ptr || !y || (nnz > 0 && (!col || !val))) return fail(c, ASAP_E_INVALID_ARG, "NULL data pointer");
  if (nnz < 0) return fail(c, ASAP_E_INVALID_ARG, "nnz must be >= 0");
  if (S < 1 || S >= (int64_t(1) << 31)) return fail(c, ASAP_E_INVALID_ARG, "samples must be in [1, 2^31)");
  if (c->dim >= (int64_t(1) << 30)) return fail(c, ASAP_E_INVALID_ARG, "CSR path needs dim < 2^30");
  c->kind = kCsr;
  c->nnz = nnz;
  c->row_ptr = row_ptr;
  c->col = col;
  c->val = val;
  c->y = y;
  c->S = S;
  c->X = nullptr;
  c->ldx = 0;
  layout(c);
  unbind_workspace(c);
  return ASAP_OK;
}

extern "C" asap_status asap_set_csr_members(asap_ctx* c, int32_t members) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (members != 0 && members != 1 && members != 2 && members != 4)
    return fail(c, ASAP_E_INVALID_ARG, "members must be 0, 1, 2 or 4 (got %d)", members);
  c->members_req = members;
  if (c->kind == kCsr) {
    layout(c);
    unbind_workspace(c);
  }
  return ASAP_OK;
}

extern "C" asap_status asap_get_csr_members(const asap_ctx* c, int32_t* members) {
  if (!c || !members) return fail(const_cast<asap_ctx*>(c), ASAP_E_INVALID_ARG, "ctx or members is NULL");
  *members = c->members;
  return ASAP_OK;
}

extern "C" asap_status asap_bind_workspace(asap_ctx* c, void* dev, size_t bytes, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!dev || uintptr_t(dev) % kAlign) return fail(c, ASAP_E_INVALID_ARG, "workspace must be 256-byte aligned");
  if (bytes < c->total)
    return fail(c, ASAP_E_INVALID_ARG, "workspace too small: %zu < %zu bytes", bytes, c->total);
  if (!c->buf[0]) return fail(c, ASAP_E_STATE, "bind the models before the workspace");
  drain_ahead(c);
  c->ring_valid = false;
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    int dev_id = 0, cus = 0;
    if (hipGetDevice(&dev_id) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id) == hipSuccess && cus > 0)
      c->n_cu = cus;
    int khz = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev_id) == hipSuccess && khz > 0)
      c->clock_khz = khz;
  }
  c->ws = static_cast<char*>(dev);
  c->ws_bytes = bytes;
  c->tags_ready = false;
  hipError_t e;
  const size_t n = size_t(c->n), nnz = c->idx.size();
  if ((e = hipMemcpyAsync(at<int32_t>(c, c->off_ptr), c->ptr.data(), (n + 1) * 4, hipMemcpyHostToDevice, s)) ||
      (e = hipMemcpyAsync(at<int32_t>(c, c->off_idx), c->idx.data(), nnz * 4, hipMemcpyHostToDevice, s)) ||
      (e = hipMemcpyAsync(at<float>(c, c->off_w), c->w.data(), nnz * 4, hipMemcpyHostToDevice, s)) ||
      (e = hipMemcpyAsync(at<int32_t>(c, c->off_optr), c->optr.data(), (n + 1) * 4, hipMemcpyHostToDevice, s)) ||
      (e = hipMemcpyAsync(at<int32_t>(c, c->off_oidx), c->oidx.data(), nnz * 4, hipMemcpyHostToDevice, s)))
    return hip_fail(c, e, "graph upload");
  if ((e = launch_fill_i64(at<int64_t>(c, c->off_tag), 2 * int64_t(n), -1, s)) ||
      (e = launch_fill_i64(at<int64_t>(c, c->off_tag) + c->cur * n, int64_t(n), tag_start(c->round), s)) ||
      (e = launch_fill_f32(at<float>(c, c->off_scale), 2 * int64_t(n), 1.0f, s)) ||
      (e = launch_fill_i32(at<int32_t>(c, c->off_err), 1, 0, s)) ||
      (e = launch_fill_i32(at<int32_t>(c, c->off_err) + 1, 1, INT_MAX, s)) ||
      (e = launch_fill_i32(at<int32_t>(c, c->off_err) + kErrRendezvous, 1, 0, s)) ||
      (c->kind == kCsr && (e = launch_fill_i64(at<int64_t>(c, c->off_progress), int64_t(n) * kMaxMembers, -1, s))))
    return hip_fail(c, e, "workspace init");
  if (c->kind == kDense && dense_wide_cpq(c->dim)) {
    // max |x| per shard (the fixed-point scale of the member exchange),
    // labels and finiteness
    int64_t* scan = at<int64_t>(c, c->off_scan);
    if ((e = launch_fill_i64(scan, 8, 0, s)) || (e = launch_fill_f32(at<float>(c, c->off_vmax), c->n, 0.0f, s)) ||
        (e = launch_dense_scan(c->X, c->y, c->n, c->S, c->dim, c->ldx, at<float>(c, c->off_vmax),
                               reinterpret_cast<unsigned long long*>(scan), s)))
      return hip_fail(c, e, "dense scan");
    int64_t h[2];
    if ((e = hipMemcpyAsync(h, scan, sizeof h, hipMemcpyDeviceToHost, s)) || (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "dense scan readback");
    if (h[0]) return fail(c, ASAP_E_INVALID_ARG, "%lld labels outside {-1, +1}", (long long)h[0]);
    if (h[1]) return fail(c, ASAP_E_INVALID_ARG, "%lld feature values are not finite", (long long)h[1]);
  }
  if (c->kind == kCsr) {
    int64_t* scan = at<int64_t>(c, c->off_scan);
    if ((e = launch_fill_i64(scan, 8, 0, s)) ||
        (e = launch_csr_scan(c->row_ptr, c->col, c->val, c->y, c->n, c->S, c->dim,
                             at<float>(c, c->off_vmax), scan, s)))
      return hip_fail(c, e, "CSR scan");
    int64_t h[8];
    if ((e = hipMemcpyAsync(h, scan, sizeof h, hipMemcpyDeviceToHost, s)) || (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "CSR scan readback");
    if (h[4]) return fail(c, ASAP_E_INVALID_ARG, "row_ptr must start at 0 and not decrease (%lld bad rows)", (long long)h[4]);
    if (h[1]) return fail(c, ASAP_E_INVALID_ARG, "%lld CSR columns outside [0, dim)", (long long)h[1]);
    if (h[2]) return fail(c, ASAP_E_INVALID_ARG, "%lld labels outside {-1, +1}", (long long)h[2]);
    if (h[3]) return fail(c, ASAP_E_INVALID_ARG, "%lld CSR rows with unsorted or repeated columns", (long long)h[3]);
    if (h[0] > 4096) return fail(c, ASAP_E_INVALID_ARG, "a CSR row holds %lld > 4096 nonzeros", (long long)h[0]);
    if (h[5] >= (int64_t(1) << 30))
      return fail(c, ASAP_E_INVALID_ARG, "a worker holds %lld >= 2^30 nonzeros", (long long)h[5]);
    int64_t last = 0;
    if ((e = hipMemcpyAsync(&last, c->row_ptr + int64_t(c->n) * c->S, 8, hipMemcpyDeviceToHost, s)) ||
        (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "row_ptr readback");
    if (last != c->nnz)
      return fail(c, ASAP_E_INVALID_ARG, "row_ptr[n*S] = %lld but nnz = %lld", (long long)last, (long long)c->nnz);
    c->max_row = int32_t(h[0]);
    c->max_wnnz = h[5];
    asap_status hs = choose_hot_columns(c, s);
    if (hs != ASAP_OK) return hs;
    hs = split_members(c, s);
    if (hs != ASAP_OK) return hs;
    // the value half of every planned (code, value) pair, and the code half
    // of a hot entry, do not change from round to round: written here, once
    // per plan slot (planning rewrites the cold entries' codes)
    for (int k = 0; k < 2; ++k)
      if ((e = write_pack(c, at<int2>(c, c->plan[k].pack), s))) return hip_fail(c, e, "plan values");
    if (c->members > 1) {
      const int64_t nm = int64_t(n) * c->members;
      if ((e = launch_fill_i64(at<int64_t>(c, c->off_xch), 2 * nm * 128, 0, s)) ||
          (e = launch_fill_i64(at<int64_t>(c, c->off_done), nm, 0, s)) ||
          (e = launch_fill_i64(at<int64_t>(c, c->off_xid), nm, 0, s)))
        return hip_fail(c, e, "member exchange init");
    }
    if (!c->ahead) {
      if ((e = hipStreamCreateWithFlags(&c->ahead, hipStreamNonBlocking))) {
        c->ahead = nullptr;
        return hip_fail(c, e, "look-ahead stream");
      }
      for (hipEvent_t* ev : {&c->ev_start, &c->ev_ready[0], &c->ev_ready[1], &c->ev_used[0], &c->ev_used[1]})
        if ((e = hipEventCreateWithFlags(ev, hipEventDisableTiming))) {
          *ev = nullptr;
          release_ahead(c);
          return hip_fail(c, e, "look-ahead events");
        }
    }
  }
  c->tags_ready = true;
  return ASAP_OK;
}

namespace {

SgdArgs sgd_args(asap_ctx* c, const asap_sgd_params* p, const RoundPlan& rp) {
  SgdArgs a{};
  a.models = c->buf[c->cur];
  a.ld = c->ld;
  a.dim = c->dim;
  a.n = c->n;
  a.S = c->S;
  a.y = c->y;
  a.X = c->X;
  a.ldx = c->ldx;
  a.row_ptr = c->row_ptr;
  a.col = c->col;
  a.val = c->val;
  a.vmax = at<float>(c, c->off_vmax);
  a.sched = at<int32_t>(c, rp.sched);
  a.seed = p->seed;
  a.loss = p->loss;
  a.lr_kind = p->lr_kind;
  a.lr0 = p->lr0;
  a.l2 = p->l2;
  a.batch = p->batch;
  {
    // steps of this round: the whole pass round, or local_steps steps of
    // the sequence of passes
    const int64_t K = (c->S + p->batch - 1) / p->batch;
    if (p->local_steps == 0) {
      a.round = c->round;
      a.k0 = 0;
      a.k1 = K;
    } else {
      const int64_t g = c->round * p->local_steps;
      a.round = g / K;
      a.k0 = g % K;
      a.k1 = a.k0 + p->local_steps;
    }
  }
  a.scale = at<float>(c, c->off_scale);
  a.tag = at<int64_t>(c, c->off_tag) + size_t(c->cur) * c->n;
  a.tag_value = tag_half(c->round);
  a.rowinfo = at<RowInfo>(c, rp.rowinfo);
  a.code = at<int32_t>(c, c->off_code);
  a.hot_cols = at<int32_t>(c, c->off_hot);
  a.n_hot = int32_t(c->hot_cols.size());
  a.max_row = c->max_row;
  return a;
}

// The planned pass applies when its shape fits (csr_plan_fits, on the
// members' slices) and a worker's (code, value) pairs are addressed by
// 32-bit byte offsets.
bool planned_pass(const asap_ctx* c, const SgdArgs& a) {
  SgdArgs f = a;
  f.max_row = c->max_slice;
  return csr_plan_fits(f) && c->max_wnnz < (int64_t(1) << 29);
}

// The planned pass's arguments: the exchange tags of its `steps` steps
// (unique for the life of the context).  The pass gives the same bits for
// any entries-per-lane count that covers its rows, so the stream-ordered
// launch sizes it for the slices' rows; the multi-round launch keeps the
// general pass's (whole rows), which shares its kernel.
SgdArgs fast_args(asap_ctx* c, const SgdArgs& a, int64_t steps) {
  SgdArgs f = a;
  f.xtag = uint32_t(c->xseq);
  f.xg0 = a.round * ((c->S + a.batch - 1) / a.batch) + a.k0;
  c->xseq += uint64_t(steps);
  return f;
}

// The plan arrays of rp live at `base` + their offsets: the workspace by
// default, or an area of the multi-round launch's plan ring.
PlanArgs plan_args(asap_ctx* c, const asap_sgd_params* p, const RoundPlan& rp, char* base = nullptr) {
  if (!base) base = c->ws;
  auto at = [base](size_t off) { return base + off; };
  const bool split = c->members > 1;
  PlanArgs pa{};
  pa.rowinfo = reinterpret_cast<RowInfo*>(at(rp.vrowinfo));
  pa.rows_real = reinterpret_cast<RowInfo*>(at(rp.rowinfo));
  pa.code = split ? ::at<int32_t>(c, c->off_vcode) : ::at<int32_t>(c, c->off_code);
  pa.row_ptr = split ? ::at<int64_t>(c, c->off_vrp) : c->row_ptr;
  pa.n = c->n * c->members;  // slices
  pa.members = c->members;
  pa.workers = c->n;
  pa.max_slice = c->max_slice;
  pa.n_cu = c->n_cu;
  // cold nonzeros of a slice's step, on average
  const double rows = double(c->n) * double(c->S);
  pa.cold_step = rows > 0.0 ? int32_t(std::min(double(p->batch) * double(c->nnz) / rows * c->cold_share / c->members,
                                               double(1 << 30)))
                            : 0;
  pa.mhot = split ? ::at<int32_t>(c, c->off_mhot) : ::at<int32_t>(c, c->off_hot);
  for (int m = 0; m < kMaxMembers; ++m) pa.n_mhot[m] = m < c->members ? c->n_mhot[m] : 0;
  pa.xch = split ? ::at<unsigned long long>(c, c->off_xch) : nullptr;
  pa.done = split ? ::at<unsigned long long>(c, c->off_done) : nullptr;
  pa.xid = split ? ::at<unsigned long long>(c, c->off_xid) : nullptr;
  pa.xerr = ::at<int32_t>(c, c->off_err) + kErrRendezvous;
  pa.xwait = kMemberWaitMs * c->clock_khz;
  pa.S = c->S;
  pa.batch = p->batch;
  pa.K = int32_t((c->S + p->batch - 1) / p->batch);
  pa.step_off = reinterpret_cast<int32_t*>(at(rp.soff));
  pa.val = c->val;
  pa.pack = reinterpret_cast<int2*>(at(rp.pack));
  pa.clist = reinterpret_cast<int32_t*>(at(rp.clist));
  pa.clink = reinterpret_cast<int32_t*>(at(rp.clink));
  pa.hlist = reinterpret_cast<int32_t*>(at(rp.hlist));
  pa.cnt = reinterpret_cast<int32_t*>(at(rp.cnt));
  pa.flag = reinterpret_cast<int32_t*>(at(rp.flag));
  pa.progress = ::at<int64_t>(c, c->off_progress);
  // a prefetch workgroup per slice when each pair lands on one XCD and the
  // pairs fit on the device; with several members only while they leave half
  // of it to the next round's planning (64 workers x 2 members with helpers:
  // pass 2.30 -> 1.92 ms, but the planning then waited for the pass and the
  // round took 2.9 instead of 2.4 ms)
  const int64_t pairs = 2 * int64_t(c->n) * c->members;
  pa.helpers = (c->n % 8 == 0 && pairs <= (split ? c->n_cu / 2 : c->n_cu)) ? 1 : 0;
  return pa;
}

// Everything a CSR round needs before its SGD pass, on stream s: the sample
// schedule of (seed, round), the row descriptors and, when the planned pass
// applies, the column plan of every worker and step.
hipError_t prepare_csr_round(asap_ctx* c, const asap_sgd_params* p, int64_t round, const RoundPlan& rp, bool planned,
                             hipStream_t s, char* base = nullptr) {
  if (!base) base = c->ws;
  int32_t* sched = reinterpret_cast<int32_t*>(base + rp.sched);
  hipError_t e = launch_schedule(p->seed, round, c->n, c->S, sched, s);
  if (e == hipSuccess)
    e = launch_rowinfo(sched, c->row_ptr, c->y, c->n, c->S, reinterpret_cast<RowInfo*>(base + rp.rowinfo), s);
  if (planned) {
    const PlanArgs pa = plan_args(c, p, rp, base);
    if (e == hipSuccess && c->members > 1)
      e = launch_rowinfo(sched, pa.row_ptr, c->y, c->n, c->S, reinterpret_cast<RowInfo*>(base + rp.vrowinfo), s,
                         c->members);
    if (e == hipSuccess) e = launch_fill_i32(pa.flag, 1, 0, s);
    if (e == hipSuccess) e = launch_csr_plan(pa, step_bound(c, p->batch), s);
  }
  return e;
}

// The current round's half-step inputs on stream s (the schedule of its
// pass; for CSR also the row descriptors and the plan), unless already
// enqueued for this pass, seed and batch (they then serve every round of the
// pass).  A CSR pass planned ahead by asap_local_sgd is waited for instead
// of planned again.
hipError_t prepare_half_step(asap_ctx* c, const asap_sgd_params* p, hipStream_t s) {
  const int64_t pass = sgd_args(c, p, c->plan[0]).round;
  if (c->prep_valid && c->prep_pass == pass && c->prep_seed == p->seed && c->prep_batch == p->batch)
    return hipSuccess;
  hipError_t e = hipSuccess;
  int slot = c->prep_valid ? c->prep_slot : 0;  // a replaced plan is rewritten in place
  if (c->kind == kCsr) {
    const bool hit = c->ahead_valid && c->ahead_pass == pass && c->ahead_seed == p->seed &&
                     c->ahead_batch == p->batch;
    if (c->ahead_valid) {
      slot = c->ahead_slot;
      e = hipStreamWaitEvent(s, c->ev_ready[slot], 0);  // a miss rewrites that slot after it
    }
    c->ahead_valid = false;
    const bool planned = planned_pass(c, sgd_args(c, p, c->plan[slot]));
    if (e == hipSuccess && !hit) e = prepare_csr_round(c, p, pass, c->plan[slot], planned, s);
  } else if (dense_wide_cpq(c->dim)) {
    // the wide dense pass reads its rows' order from the schedule; the
    // narrow one evaluates the permutation itself
    e = launch_schedule(p->seed, pass, c->n, c->S, at<int32_t>(c, c->plan[0].sched), s);
  }
  c->prep_valid = e == hipSuccess;
  c->prep_slot = slot;
  c->prep_pass = pass;
  c->prep_seed = p->seed;
  c->prep_batch = p->batch;
  return e;
}

asap_status check_half_step(asap_ctx* c, const asap_sgd_params* p) {
  asap_status st = need_device(c);
  if (st != ASAP_OK) return st;
  if (c->kind == kNoData) return fail(c, ASAP_E_STATE, "no data bound");
  if (c->half_done) return fail(c, ASAP_E_STATE, "the half-step of round %lld already ran", (long long)c->round);
  return check_params(c, p);
}

}  // namespace

extern "C" asap_status asap_prepare_sgd(asap_ctx* c, const asap_sgd_params* p, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  asap_status st = check_half_step(c, p);
  if (st != ASAP_OK) return st;
  const hipError_t e = prepare_half_step(c, p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ASAP_OK : hip_fail(c, e, "half-step preparation");
}

extern "C" asap_status asap_local_sgd(asap_ctx* c, const asap_sgd_params* p, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  asap_status st = check_half_step(c, p);
  if (st != ASAP_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = prepare_half_step(c, p, s);
  if (e != hipSuccess) return hip_fail(c, e, "half-step preparation");
  const int slot = c->prep_slot;
  if (c->kind == kCsr) {
    SgdArgs a = sgd_args(c, p, c->plan[slot]);
    const bool planned = planned_pass(c, a);
    const bool pass_ends = a.k1 == (c->S + p->batch - 1) / p->batch;
    if (planned) {
      // the general kernel runs only if the plan says a step does not fit;
      // it goes first, so that when it exits at once its launch does not
      // queue behind the next round's planning (which starts at ev_start)
      const PlanArgs pa = plan_args(c, p, c->plan[slot]);
      a.run_if = pa.flag;
      if (e == hipSuccess) e = launch_sgd_csr(a, s);
      if (e == hipSuccess && c->ahead) e = hipEventRecord(c->ev_start, s);
      if (e == hipSuccess) {
        SgdArgs f = fast_args(c, a, a.k1 - a.k0);
        f.max_row = c->max_slice;
        e = launch_sgd_csr_fast(f, pa, s);
      }
    } else {
      if (e == hipSuccess && c->ahead) e = hipEventRecord(c->ev_start, s);
      if (e == hipSuccess) e = launch_sgd_csr(a, s);
    }
    if (e == hipSuccess && c->ahead) e = hipEventRecord(c->ev_used[slot], s);
    if (e != hipSuccess) return hip_fail(c, e, "SGD kernel");
    if (planned && pass_ends && c->ahead) {
      // plan the next pass into the other slot, concurrently with this
      // launch: after this call's inputs are ready (ev_start) and after the
      // slot's last reader (ev_used).  With fewer workers than compute
      // units it runs beside the launch; otherwise it fills its tail and
      // overlaps the reduce.
      const int o = slot ^ 1;
      if ((e = hipStreamWaitEvent(c->ahead, c->ev_start, 0)) || (e = hipStreamWaitEvent(c->ahead, c->ev_used[o], 0)) ||
          (e = prepare_csr_round(c, p, a.round + 1, c->plan[o], true, c->ahead)) ||
          (e = hipEventRecord(c->ev_ready[o], c->ahead)))
        return hip_fail(c, e, "look-ahead planning");
      c->ahead_valid = true;
      c->ahead_slot = o;
      c->ahead_seed = p->seed;
      c->ahead_pass = a.round + 1;
      c->ahead_batch = p->batch;
    }
  } else {
    SgdArgs a = sgd_args(c, p, c->plan[0]);
    if (dense_wide_cpq(c->dim)) {
      DenseSync ds{};
      ds.part = at<float>(c, c->off_dacc);
      ds.count = at<uint32_t>(c, c->off_dcount);
      ds.xcd = at<int32_t>(c, c->off_dxcd);
      ds.ldp = int64_t(dense_wide_cpq(c->dim)) * 2048;
      ds.K = std::max(1, std::min(c->dense_k, dense_wide_max_members(a, c->n_cu) / c->n));
      ds.spin_limit = kDenseSpinLimit;
      ds.err = at<int32_t>(c, c->off_err) + kErrRendezvous;
      e = launch_fill_i32(reinterpret_cast<int32_t*>(ds.count), c->n, 0, s);
      if (e == hipSuccess) e = launch_sgd_dense_wide(a, ds, s);
    } else {
      e = launch_sgd_dense(a, s);
    }
    if (e != hipSuccess) return hip_fail(c, e, "SGD kernel");
  }
  c->half_done = true;
  c->half_scaled = (c->kind == kCsr) && p->l2 > 0.0f;
  return ASAP_OK;
}

extern "C" asap_status asap_stochastic_reduce(asap_ctx* c, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  asap_status st = need_device(c);
  if (st != ASAP_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t n = size_t(c->n);
  MixArgs a{};
  a.src = c->buf[c->cur];
  a.dst = c->buf[c->cur ^ 1];
  a.ld = c->ld;
  a.dim = c->dim;
  a.n = c->n;
  a.nbr_ptr = at<int32_t>(c, c->off_ptr);
  a.nbr_idx = at<int32_t>(c, c->off_idx);
  a.nbr_w = at<float>(c, c->off_w);
  a.scale = c->half_scaled ? at<float>(c, c->off_scale) : nullptr;
  a.tag_src = at<int64_t>(c, c->off_tag) + size_t(c->cur) * n;
  a.tag_dst = at<int64_t>(c, c->off_tag) + size_t(c->cur ^ 1) * n;
  a.expect = c->half_done ? tag_half(c->round) : tag_start(c->round);
  a.next = tag_start(c->round + 1);
  a.err = at<int32_t>(c, c->off_err);
  a.row_ok = at<int32_t>(c, c->off_rowok);
  a.uniform_rows = c->uniform_rows && !a.scale;
  hipError_t e = launch_epoch_check(a, s);
  if (e == hipSuccess) {
    if (c->complete_uniform) {
      e = launch_mean(a, s);
    } else {
      e = launch_mix_slab(a, c->max_deg, c->n_cu, s);
      if (e == hipErrorNotSupported) e = launch_mix(a, s);
    }
  }
  if (e != hipSuccess) return hip_fail(c, e, "reduce kernel");
  c->cur ^= 1;
  c->round += 1;
  c->half_done = false;
  c->half_scaled = false;
  return ASAP_OK;
}

extern "C" asap_status asap_round(asap_ctx* c, const asap_sgd_params* p, void* stream) {
  asap_status s = asap_local_sgd(c, p, stream);
  if (s != ASAP_OK) return s;
  return asap_stochastic_reduce(c, stream);
}

namespace {

// One area of the plan ring: the arrays of one pass's plan (as a RoundPlan
// slot of the workspace); returns its size.
size_t ring_layout(const asap_ctx* c, RoundPlan* lay) {
  const size_t n = size_t(c->n), nS = n * size_t(c->S), nz = size_t(c->nnz), M = size_t(c->members);
  size_t o = 0;
  lay->sched = o;   o = align_up(o + nS * 4);
  lay->rowinfo = o; o = align_up(o + nS * sizeof(RowInfo));
  lay->vrowinfo = lay->rowinfo;
  if (M > 1) { lay->vrowinfo = o; o = align_up(o + M * nS * sizeof(RowInfo)); }
  lay->soff = o;    o = align_up(o + M * n * (size_t(c->S) + 1) * 4);
  lay->pack = o;    o = align_up(o + nz * 8);
  lay->clist = o;   o = align_up(o + nz * 4);
  lay->clink = o;   o = align_up(o + nz * 4);
  lay->hlist = o;   o = align_up(o + nz * 4);
  lay->cnt = o;     o = align_up(o + M * nS * 2 * 4);
  lay->flag = o;    o = align_up(o + 4);
  return o;
}

size_t ring_head(int64_t areas) { return align_up(size_t(areas) * 8); }

}  // namespace

extern "C" asap_status asap_rounds_plan_size(const asap_ctx* c, int64_t passes, size_t* bytes) {
  if (!c || !bytes) return fail(const_cast<asap_ctx*>(c), ASAP_E_INVALID_ARG, "ctx or bytes is NULL");
  if (passes < 1 || passes > (int64_t(1) << 20)) return fail(const_cast<asap_ctx*>(c), ASAP_E_INVALID_ARG,
                                                             "passes must be in [1, 2^20]");
  if (c->kind != kCsr) return fail(const_cast<asap_ctx*>(c), ASAP_E_STATE, "no CSR data bound");
  RoundPlan lay;
  *bytes = ring_head(passes) + size_t(passes) * ring_layout(c, &lay);
  return ASAP_OK;
}

extern "C" asap_status asap_bind_rounds_plan(asap_ctx* c, void* dev, size_t bytes, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!dev || uintptr_t(dev) % kAlign) return fail(c, ASAP_E_INVALID_ARG, "plan ring must be 256-byte aligned");
  if (c->kind != kCsr) return fail(c, ASAP_E_STATE, "no CSR data bound");
  if (!c->ws || !c->tags_ready) return fail(c, ASAP_E_STATE, "bind the workspace before the plan ring");
  RoundPlan lay;
  const size_t stride = ring_layout(c, &lay);
  int64_t areas = 0;
  while (ring_head(areas + 1) + size_t(areas + 1) * stride <= bytes) ++areas;
  if (areas < 1) return fail(c, ASAP_E_INVALID_ARG, "plan ring too small for one pass (%zu bytes)", bytes);
  drain_ahead(c);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(dev);
  hipError_t e = launch_fill_i64(reinterpret_cast<int64_t*>(base), areas, -1, s);
  // the bind-time halves of every area's (code, value) pairs, as for the
  // workspace's two plan slots
  for (int64_t u = 0; u < areas && e == hipSuccess; ++u)
    e = write_pack(c, reinterpret_cast<int2*>(base + ring_head(areas) + size_t(u) * stride + lay.pack), s);
  if (e == hipSuccess && !c->ev_ring_free) {
    if ((e = hipEventCreateWithFlags(&c->ev_ring_free, hipEventDisableTiming))) c->ev_ring_free = nullptr;
  }
  if (e == hipSuccess) e = hipEventRecord(c->ev_ring_free, s);
  if (e != hipSuccess) return hip_fail(c, e, "plan ring");
  c->ring = base;
  c->ring_areas = areas;
  c->ring_stride = stride;
  c->ring_lay = lay;
  c->ring_valid = true;
  return ASAP_OK;
}

extern "C" asap_status asap_run_rounds(asap_ctx* c, const asap_sgd_params* p, int64_t rounds, int32_t wait_ms,
                                       void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  asap_status st = check_half_step(c, p);
  if (st != ASAP_OK) return st;
  if (rounds < 1 || rounds > (int64_t(1) << 40)) return fail(c, ASAP_E_INVALID_ARG, "rounds must be in [1, 2^40]");
  if (wait_ms < 0) return fail(c, ASAP_E_INVALID_ARG, "wait_ms must be >= 0");
  if (c->max_deg > kRoundsMaxDeg || c->max_out > kRoundsMaxDeg)
    return fail(c, ASAP_E_STATE, "a worker has %d in- and %d out-neighbours; the multi-round launch takes at most %d",
                c->max_deg, c->max_out, kRoundsMaxDeg);
  if (c->ld * 4 >= (int64_t(1) << 31))
    return fail(c, ASAP_E_STATE, "the multi-round launch takes rows of under 2^31 bytes (ld = %lld)", (long long)c->ld);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the launch rewrites the schedule and row-descriptor area of plan slot 0
  drain_ahead(c);
  hipError_t e;
  int dev_id = 0, khz = 0;
  if ((e = hipGetDevice(&dev_id)) || (e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev_id)))
    return hip_fail(c, e, "wall clock rate");
  const int64_t n = c->n;
  SgdArgs a = sgd_args(c, p, c->plan[0]);
  RoundsArgs ra{};
  ra.buf[0] = c->buf[0];
  ra.buf[1] = c->buf[1];
  ra.cur = c->cur;
  ra.n = c->n;
  ra.r0 = c->round;
  ra.R = rounds;
  ra.local_steps = p->local_steps;
  ra.seed = p->seed;
  ra.in_ptr = at<int32_t>(c, c->off_ptr);
  ra.in_idx = at<int32_t>(c, c->off_idx);
  ra.in_w = at<float>(c, c->off_w);
  ra.out_ptr = at<int32_t>(c, c->off_optr);
  ra.out_idx = at<int32_t>(c, c->off_oidx);
  ra.tag = at<int64_t>(c, c->off_tag);
  ra.scale2 = at<float>(c, c->off_scale);
  ra.scaled = (c->kind == kCsr && p->l2 > 0.0f) ? 1 : 0;
  {
    // the reduce arithmetic of the kernel asap_stochastic_reduce launches
    MixArgs m{};
    m.n = c->n;
    m.ld = c->ld;
    m.dim = c->dim;
    ra.fp64_mix = (c->complete_uniform || !mix_slab_applies(m, c->max_deg)) ? 1 : 0;
  }
  ra.wait_ticks = (long long)(wait_ms ? wait_ms : kRoundsWaitMs) * (long long)std::max(khz, 1);
  ra.err = at<int32_t>(c, c->off_err);
  ra.sched = at<int32_t>(c, c->plan[0].sched);
  ra.rowinfo = at<RowInfo>(c, c->plan[0].rowinfo);
  ra.msync = at<int64_t>(c, c->off_msync);
  // the members' words carry round tags, which a launch after asap_set_round
  // may repeat: every launch starts from -1
  if ((e = launch_fill_i64(ra.msync, int64_t(n) * kMemberSync, -1, s))) return hip_fail(c, e, "launch init");
  if (c->kind == kCsr) {
    // the passes this launch covers
    const int64_t K = (c->S + p->batch - 1) / p->batch;
    auto pass_of = [&](int64_t r) { return p->local_steps == 0 ? r : r * p->local_steps / K; };
    const int64_t first = pass_of(c->round), npass = pass_of(c->round + rounds - 1) - first + 1;
    if (c->ring_valid && planned_pass(c, a) && npass <= c->ring_areas) {
      // every pass gets its plan in its own ring area: beside the launch on
      // the look-ahead stream when the launch leaves compute units free
      // (workers wait for their pass's plan), else before it on `stream`
      RoundsPlan rp{};
      rp.area0 = plan_args(c, p, c->ring_lay, c->ring + ring_head(c->ring_areas));
      rp.stride = int64_t(c->ring_stride);
      rp.first_pass = first;
      rp.npass = npass;
      rp.ready = reinterpret_cast<const int64_t*>(c->ring);
      rp.token0 = (++c->ring_epoch) << 24;
      const int64_t blocks = int64_t(c->n) * c->members * (rp.area0.helpers ? 2 : 1);
      const bool beside = c->ahead && blocks + 64 <= c->n_cu;
      hipStream_t ps = beside ? c->ahead : s;
      if (beside) e = hipStreamWaitEvent(ps, c->ev_ring_free, 0);
      else e = hipSuccess;
      for (int64_t u = 0; u < npass && e == hipSuccess; ++u) {
        char* area = c->ring + ring_head(c->ring_areas) + size_t(u) * c->ring_stride;
        e = prepare_csr_round(c, p, first + u, c->ring_lay, true, ps, area);
        if (e == hipSuccess) e = launch_fill_i64(reinterpret_cast<int64_t*>(c->ring) + u, 1, rp.token0 + u, ps);
      }
      if (e != hipSuccess) return hip_fail(c, e, "launch planning");
      // exchange tags of every step the launch runs (rounds are consecutive steps)
      const int64_t per_round = p->local_steps == 0 ? K : p->local_steps;
      e = launch_rounds_csr_planned(fast_args(c, a, rounds * per_round), ra, rp, c->n_cu, s);
      if (e == hipSuccess) e = hipEventRecord(c->ev_ring_free, s);
    } else {
      e = launch_rounds_csr(a, ra, c->n_cu, s);
    }
  } else if (dense_wide_cpq(c->dim)) {
    DenseSync ds{};
    ds.part = at<float>(c, c->off_dacc);
    ds.count = at<uint32_t>(c, c->off_dcount);
    ds.xcd = at<int32_t>(c, c->off_dxcd);
    ds.ldp = int64_t(dense_wide_cpq(c->dim)) * 2048;
    ds.K = std::max(1, std::min(c->dense_k, dense_wide_max_members(a, c->n_cu) / c->n));
    ds.spin_limit = kDenseSpinLimit;
    ds.err = at<int32_t>(c, c->off_err) + kErrRendezvous;
    ds.base = 0;
    e = launch_fill_i32(reinterpret_cast<int32_t*>(ds.count), n, 0, s);
    if (e == hipSuccess) e = launch_rounds_dense_wide(a, ds, ra, s);
  } else {
    e = launch_rounds_dense(a, ra, c->n_cu, s);
  }
  if (e == hipErrorCooperativeLaunchTooLarge)
    return fail(c, ASAP_E_STATE, "the %d workers' workgroups do not fit on the device at once", c->n);
  if (e != hipSuccess) return hip_fail(c, e, "multi-round kernel");
  c->cur ^= int32_t(rounds & 1);
  c->round += rounds;
  c->half_done = false;
  c->half_scaled = false;
  c->prep_valid = false;
  return ASAP_OK;
}

extern "C" asap_status asap_current(const asap_ctx* c, int32_t* buffer, int64_t* round,
                                    int32_t* half_step_done) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (buffer) *buffer = c->cur;
  if (round) *round = c->round;
  if (half_step_done) *half_step_done = c->half_done ? 1 : 0;
  return ASAP_OK;
}

extern "C" asap_status asap_set_round(asap_ctx* c, int64_t round, int32_t buffer, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (round < 0 || (buffer != 0 && buffer != 1)) return fail(c, ASAP_E_INVALID_ARG, "bad round or buffer");
  asap_status st = need_device(c);
  if (st != ASAP_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t n = c->n;
  hipError_t e;
  if ((e = launch_fill_i64(at<int64_t>(c, c->off_tag), 2 * n, -1, s)) ||
      (e = launch_fill_i64(at<int64_t>(c, c->off_tag) + buffer * n, n, tag_start(round), s)))
    return hip_fail(c, e, "tag reset");
  c->cur = buffer;
  c->round = round;
  c->half_done = false;
  c->half_scaled = false;
  return ASAP_OK;
}

extern "C" asap_status asap_get_graph(const asap_ctx* c, int32_t* n_workers, int64_t* n_entries, int32_t* nbr_ptr,
                                      int32_t* nbr_idx, float* nbr_w) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!n_workers || !n_entries) return fail(nullptr, ASAP_E_INVALID_ARG, "NULL count output");
  const int given = (nbr_ptr != nullptr) + (nbr_idx != nullptr) + (nbr_w != nullptr);
  if (given != 0 && given != 3) return fail(nullptr, ASAP_E_INVALID_ARG, "give all three graph arrays or none");
  *n_workers = c->n;
  *n_entries = int64_t(c->idx.size());
  if (given) {
    std::copy(c->ptr.begin(), c->ptr.end(), nbr_ptr);
    std::copy(c->idx.begin(), c->idx.end(), nbr_idx);
    std::copy(c->w.begin(), c->w.end(), nbr_w);
  }
  return ASAP_OK;
}

extern "C" asap_status asap_drop_workers(asap_ctx* c, int32_t n_drop, const int32_t* dropped,
                                         const int32_t* nbr_ptr, const int32_t* nbr_idx, const float* nbr_w,
                                         uint32_t flags, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!dropped || n_drop < 1 || n_drop >= c->n)
    return fail(c, ASAP_E_INVALID_ARG, "drop between 1 and n - 1 = %d workers", c->n - 1);
  for (int32_t q = 0; q < n_drop; ++q)
    if (dropped[q] < 0 || dropped[q] >= c->n || (q > 0 && dropped[q] <= dropped[q - 1]))
      return fail(c, ASAP_E_INVALID_ARG, "dropped workers must be ascending, distinct and in [0, %d)", c->n);
  if (!nbr_ptr || !nbr_idx || !nbr_w) return fail(c, ASAP_E_INVALID_ARG, "NULL graph array");
  if (flags & ~uint32_t(ASAP_ALLOW_NON_DS)) return fail(c, ASAP_E_INVALID_ARG, "unknown flags");
  const int32_t n2 = c->n - n_drop;
  asap_status st = check_graph(c, n2, nbr_ptr, nbr_idx, nbr_w, flags);
  if (st != ASAP_OK) return st;
  if (!c->buf[0]) return fail(c, ASAP_E_STATE, "bind the models first");
  if (c->half_done) return fail(c, ASAP_E_STATE, "the half-step of round %lld is pending", (long long)c->round);
  drain_ahead(c);
  // survivors' rows of the current buffer, in order, into the other buffer
  // (runs of consecutive survivors move in one copy)
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float* src = c->buf[c->cur];
  float* dst = c->buf[c->cur ^ 1];
  const size_t row = size_t(c->ld) * sizeof(float);
  int32_t to = 0, q = 0;
  for (int32_t i = 0; i < c->n;) {
    if (q < n_drop && dropped[q] == i) {
      ++q;
      ++i;
      continue;
    }
    int32_t j = i;
    while (j < c->n && !(q < n_drop && dropped[q] == j)) ++j;
    const hipError_t e = hipMemcpyAsync(dst + size_t(to) * c->ld, src + size_t(i) * c->ld, row * size_t(j - i),
                                        hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(c, e, "model compaction");
    to += j - i;
    i = j;
  }
  c->cur ^= 1;
  set_graph(c, n2, nbr_ptr, nbr_idx, nbr_w);
  // the shards were laid out per worker of the old numbering
  c->kind = kNoData;
  c->X = nullptr;
  c->y = nullptr;
  c->row_ptr = nullptr;
  c->col = nullptr;
  c->val = nullptr;
  c->S = 0;
  c->nnz = 0;
  c->half_scaled = false;
  layout(c);
  unbind_workspace(c);
  return ASAP_OK;
}

extern "C" asap_status asap_schedule_device(asap_ctx* c, uint64_t seed, int64_t round,
                                            int32_t* dev_out, void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (c->kind == kNoData) return fail(c, ASAP_E_STATE, "no data bound");
  if (!dev_out || round < 0) return fail(c, ASAP_E_INVALID_ARG, "bad arguments");
  hipError_t e = launch_schedule(seed, round, c->n, c->S, dev_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "schedule kernel");
  return ASAP_OK;
}

namespace {

// Checks and the kernel arguments shared by asap_metrics and
// asap_metrics_noalloc; the scratch pointers (w_bar, partials, results) are
// left for the caller.
asap_status metric_args(asap_ctx* c, int32_t loss, float l2, const double* out, MetricArgs* a) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (!out) return fail(c, ASAP_E_INVALID_ARG, "out is NULL");
  if (loss != ASAP_LOSS_LOGISTIC && loss != ASAP_LOSS_HINGE) return fail(c, ASAP_E_INVALID_ARG, "unknown loss");
  if (!(std::isfinite(l2) && l2 >= 0.0f)) return fail(c, ASAP_E_INVALID_ARG, "l2 must be >= 0");
  asap_status st = need_device(c);
  if (st != ASAP_OK) return st;
  *a = MetricArgs{};
  a->W = c->buf[c->cur];
  a->ld = c->ld;
  a->dim = c->dim;
  a->n = c->n;
  a->scale = c->half_scaled ? at<float>(c, c->off_scale) : nullptr;
  a->S = c->kind == kNoData ? 0 : c->S;
  a->y = c->y;
  a->X = c->X;
  a->ldx = c->ldx;
  a->row_ptr = c->row_ptr;
  a->col = c->col;
  a->val = c->val;
  a->loss = loss;
  a->l2 = l2;
  return ASAP_OK;
}

}  // namespace

extern "C" asap_status asap_metrics(asap_ctx* c, int32_t loss, float l2, double* out, void* stream) {
  MetricArgs a;
  asap_status st = metric_args(c, loss, l2, out, &a);
  if (st != ASAP_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  a.wbar = at<double>(c, c->off_wbar);
  a.part = at<double>(c, c->off_part);
  a.out = at<double>(c, c->off_out);
  hipError_t e = launch_metrics(a, s);
  if (e != hipSuccess) return hip_fail(c, e, "metrics kernels");
  if ((e = hipMemcpyAsync(out, a.out, 4 * sizeof(double), hipMemcpyDeviceToHost, s)) ||
      (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "metrics readback");
  return ASAP_OK;
}

extern "C" asap_status asap_metrics_noalloc(asap_ctx* c, int32_t loss, float l2, double* out, void* stream) {
  MetricArgs a;
  asap_status st = metric_args(c, loss, l2, out, &a);
  if (st != ASAP_OK) return st;
  if (c->dim > kStaticMetricMaxDim || c->n > kStaticMetricMaxWorkers)
    return fail(c, ASAP_E_INVALID_ARG,
                "asap_metrics_noalloc handles dim <= %lld and n <= %lld (got dim %lld, n %d); use asap_metrics",
                (long long)kStaticMetricMaxDim, (long long)kStaticMetricMaxWorkers, (long long)c->dim, c->n);
  hipError_t e = metrics_static_scratch(a, static_cast<hipStream_t>(stream), out);
  if (e != hipSuccess) return hip_fail(c, e, "metrics kernels (static scratch)");
  return ASAP_OK;
}

extern "C" asap_status asap_check(asap_ctx* c, void* stream, int32_t* bad_worker) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if (bad_worker) *bad_worker = -1;
  if (!c->ws) return fail(c, ASAP_E_STATE, "workspace is not bound");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t h[3];
  hipError_t e;
  if ((e = hipMemcpyAsync(h, at<int32_t>(c, c->off_err), sizeof h, hipMemcpyDeviceToHost, s)) ||
      (e = hipStreamSynchronize(s)))
    return hip_fail(c, e, "error readback");
  if (h[kErrRendezvous] != 0) {
    if ((e = launch_fill_i32(at<int32_t>(c, c->off_err) + kErrRendezvous, 1, 0, s)) ||
        (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "error reset");
    return fail(c, ASAP_E_DEVICE, "SGD: %d waits of a worker's workgroups for each other timed out; the pass was cut short",
                h[kErrRendezvous]);
  }
  if (h[0] != 0) {
    if (bad_worker) *bad_worker = h[1];
    if ((e = launch_fill_i32(at<int32_t>(c, c->off_err), 1, 0, s)) ||
        (e = launch_fill_i32(at<int32_t>(c, c->off_err) + 1, 1, INT_MAX, s)) ||
        (e = hipStreamSynchronize(s)))
      return hip_fail(c, e, "error reset");
    return fail(c, ASAP_E_EPOCH, "%d reduce rows skipped on a neighbour epoch-tag mismatch (lowest worker %d)",
                h[0], h[1]);
  }
  return ASAP_OK;
}

extern "C" asap_status asap_debug_set_tag(asap_ctx* c, int32_t buffer, int32_t worker, int64_t value,
                                          void* stream) {
  if (!c) return fail(nullptr, ASAP_E_INVALID_ARG, "ctx is NULL");
  if ((buffer != 0 && buffer != 1) || worker < 0 || worker >= c->n)
    return fail(c, ASAP_E_INVALID_ARG, "bad buffer or worker");
  if (!c->ws) return fail(c, ASAP_E_STATE, "workspace is not bound");
  hipError_t e = launch_fill_i64(at<int64_t>(c, c->off_tag) + size_t(buffer) * c->n + worker, 1, value,
                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(c, e, "tag write");
  return ASAP_OK;
}

extern "C" const char* asap_last_error(const asap_ctx* c) {
  return c ? c->err.c_str() : g_free_error.c_str();
}

extern "C" void asap_destroy(asap_ctx* c) {
  if (!c) return;
  release_ahead(c);
  delete c;
}
