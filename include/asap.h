/*
 * asap.h -- C ABI of the ASAP stochastic-reduce hot path on one MI355X.
 *
 * The problem (Appendix A): n workers minimise sum_i f_i(w) where f_i is
 * private to worker i; worker i reads only the models of its in-neighbours
 * N(i) and its own.  One round is the update equation (A.2):
 *
 *   half-step   w_i <- w_i - eta_t grad f_i(w_i)       (here: one local SGD
 *                                                       pass over i's shard)
 *   reduce      w_i <- sum_{j in N_in(i)} P_ij w_j     (the stochastic reduce)
 *
 * with P the mixing matrix of the "Network requirement" paragraph (row i holds
 * the weights of i's in-neighbours, self included; doubly stochastic so that
 * every worker has the same influence).  The NOTIFY-ACK protocol of Section 4
 * (a reader reduces only after all of its senders published the round's
 * model; a sender overwrites only after all readers acknowledged) becomes two
 * model buffers with per-worker epoch tags: the half-step writes buffer e and
 * tags it (NOTIFY), the reduce reads buffer e only after checking every
 * neighbour's tag and writes buffer e^1 (the consumed buffer is free again at
 * the end of the reduce: ACK by stream order).
 *
 * Conventions
 *  - Every call returns an asap_status; nothing throws across the ABI.
 *  - Argument and state errors are detected before anything is enqueued.
 *    Device-side errors (an epoch-tag mismatch) are reported by asap_check.
 *  - The library never allocates device memory: the caller owns the
 *    workspace, the two model buffers and the data shards (device pointers,
 *    e.g. from torch tensors) and keeps them alive until asap_destroy.  The
 *    one exception is the static array of asap_metrics_noalloc (8.4 MiB per
 *    GPU, created with the library's code object, never freed).
 *  - With CSR data bound, the library also owns one non-blocking stream
 *    (default priority) and a few events, created at asap_bind_workspace
 *    and released by asap_destroy; see asap_local_sgd.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    All device work is asynchronous on that stream, in call order.
 *  - A context is not thread-safe; use one per host thread.
 *  - Host-pointer arguments are read during the call only, unless stated.
 */
#ifndef ASAP_H
#define ASAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct asap_ctx asap_ctx;

typedef enum asap_status {
  ASAP_OK = 0,
  ASAP_E_INVALID_ARG = 1, /* bad pointer, size, alignment or value            */
  ASAP_E_GRAPH = 2,       /* graph CSR malformed or P not doubly stochastic   */
  ASAP_E_STATE = 3,       /* call out of order (e.g. no data bound, reduce    */
                          /* before models are bound, SGD twice in a round)   */
  ASAP_E_DEVICE = 4,      /* a HIP runtime call failed                        */
  ASAP_E_EPOCH = 5        /* a reduce found a neighbour model of the wrong    */
                          /* round (NOTIFY missing); reported by asap_check   */
} asap_status;

/* loss of the local objective f_i (mean loss over the shard + l2/2 ||w||^2) */
enum { ASAP_LOSS_LOGISTIC = 0, ASAP_LOSS_HINGE = 1 };
/* step size eta_t, t counted from 1 per worker across rounds               */
enum { ASAP_LR_CONST = 0, ASAP_LR_INV_SQRT = 1 };
/* asap_create flags */
enum { ASAP_ALLOW_NON_DS = 1u /* accept weights that are not doubly stochastic */ };

/* Parameters of one local pass (the half-step of (A.2)).
 *  loss     ASAP_LOSS_*; logistic: log(1 + exp(-y m)); hinge: max(0, 1 - y m)
 *  lr_kind  ASAP_LR_*;   eta_t = lr0 or lr0 / sqrt(t)
 *  lr0      > 0, finite
 *  l2       >= 0, finite; the (l2/2)||w||^2 term of every f_i
 *  batch    minibatch size B >= 1; the pass takes K = ceil(S/B) steps, the
 *           last one over the S mod B remaining samples when B does not
 *           divide S
 *  local_steps  0: a round's half-step is one full pass (K steps).  L >= 1
 *           dividing K: L steps; the steps of all rounds are the passes one
 *           after the other, so round r runs steps k0 .. k0 + L - 1 of pass
 *           q with q = (r L) div K, k0 = (r L) mod K, pass q in the order of
 *           asap_schedule(S, seed, i, q), and t = q K + k + 1.  L = 1 is
 *           (A.2) as printed: one gradient step, then the mix.
 *  seed     seed of the sample schedule (see asap_schedule)              */
typedef struct asap_sgd_params {
  int32_t loss;
  int32_t lr_kind;
  float lr0;
  float l2;
  int32_t batch;
  int32_t local_steps;
  uint64_t seed;
} asap_sgd_params;

/* ---------------------------------------------------------------------------
 * Host-only graph and schedule builders (no device, no context).
 * Figure 2 and Section 3 name the all-reduce (complete), expander and chain
 * topologies; Appendix A fixes P = A / in-degree with self-loops.
 * Row i of a graph CSR lists the in-neighbours of worker i in ascending
 * order, self included.  Output arrays are caller-allocated with the sizes
 * stated; on error their contents are unspecified.
 * ------------------------------------------------------------------------- */

/* Ring: N_in(i) = {i-1, i, i+1} mod n.  n >= 3.  nbr_ptr[n+1], nbr_idx[3n]. */
asap_status asap_graph_ring(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx);

/* Root expander (Figure 2(c); Section 3): every worker sends to its
 * neighbour i+1, which keeps the graph connected, and to worker i+r with
 * r = ceil(sqrt(n)), all mod n; so N_in(i) = {i-r, i-1, i} mod n, out- and
 * in-degree 2 (the graph the paper evaluates).  The rounding of sqrt(n) is
 * not stated; ceil is used.  n >= 3.  nbr_ptr[n+1], nbr_idx[3n]. */
asap_status asap_graph_root_expander(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx);

/* Chain (Figure 2(d)): worker i sends to i+1 only, wrapping around at the
 * end (a directed ring), so N_in(i) = {i-1, i} mod n and P = A/2 is doubly
 * stochastic; its gap 1 - cos(pi/n) is 0.0079 for 25 workers, the value
 * Section 6 quotes for its 25-process chain.  n >= 2.  nbr_ptr[n+1],
 * nbr_idx[2n]. */
asap_status asap_graph_chain(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx);

/* Complete graph (all-reduce): N_in(i) = all j.  1 <= n <= 46340.
 * nbr_ptr[n+1], nbr_idx[n*n]. */
asap_status asap_graph_complete(int32_t n, int32_t* nbr_ptr, int32_t* nbr_idx);

/* Connected simple random d-regular graph (an expander with high
 * probability), 1 <= d < n, n*d even, n <= 1<<20, d >= 2 unless n == 2
 * (a perfect matching on more nodes is never connected).  Stub pairing on a
 * SplitMix64 stream keyed by (seed, n, d): draw two stub positions a, b
 * uniformly; reject a == b, a self-pair or an existing edge; else add the
 * edge and remove position max(a,b) then min(a,b) by swap-with-last.  More
 * than 100 * (stubs left) consecutive rejections, or a disconnected result,
 * restarts with the stream continuing.  nbr_ptr[n+1], nbr_idx[n*(d+1)]. */
asap_status asap_graph_random_regular(int32_t n, int32_t d, uint64_t seed,
                                      int32_t* nbr_ptr, int32_t* nbr_idx);

/* Metropolis-Hastings weights of an in-neighbour CSR (self required):
 * P_ij = 1/(1 + max(d_i, d_j)) for j != i, P_ii = 1 - sum_{j != i} P_ij,
 * computed in double and rounded once to float; d_i = row length - 1.
 * On a d-regular graph this is the paper's A/(d+1).  nbr_w[nbr_ptr[n]]. */
asap_status asap_metropolis_weights(int32_t n, const int32_t* nbr_ptr,
                                    const int32_t* nbr_idx, float* nbr_w);

/* Sample schedule pi_{worker,round}: a permutation of [0, samples) (the
 * paper lets every replica train on its own portion of the data, Section 5;
 * the order is this library's reading).  Minibatch k of the round is
 * positions [kB, min((k+1)B, S)).  Built as a keyed 4-round Feistel
 * bijection on 2h bits (h = ceil(ceil(log2 S)/2)), with MurmurHash3's fmix32
 * as round function and cycle walking into [0, S).  0 <= samples < 2^31.
 * out[samples] (host). */
asap_status asap_schedule(int64_t samples, uint64_t seed, int32_t worker,
                          int64_t round, int32_t* out);

/* ---------------------------------------------------------------------------
 * Context
 * ------------------------------------------------------------------------- */

/* Create a context for n_workers models of `dim` floats over the graph
 * (nbr_ptr[n+1], nbr_idx[nnz], nbr_w[nnz], host, copied).  Checks: CSR
 * monotone from 0; indices in range, strictly ascending per row; self
 * present (a worker uses its own model, Appendix A); weights finite and
 * >= 0; unless ASAP_ALLOW_NON_DS, every row sum and column sum is 1 within
 * 1e-6 + (row length) * 2^-24 (doubly stochastic, Appendix A).  A complete
 * graph whose weights are all bitwise equal takes the column-mean reduce.
 * Errors: ASAP_E_INVALID_ARG (sizes, NULLs), ASAP_E_GRAPH. */
asap_status asap_create(int32_t n_workers, int64_t dim, const int32_t* nbr_ptr,
                        const int32_t* nbr_idx, const float* nbr_w,
                        uint32_t flags, asap_ctx** out);

/* Bytes of device workspace the context needs (graph copy, epoch tags,
 * per-worker L2 scales, error words, metric partials). */
asap_status asap_workspace_size(const asap_ctx* ctx, size_t* bytes);

/* Bind caller-owned device workspace (256-byte aligned, >= the size above)
 * and upload the graph on `stream`.  Must precede every device call.  Waits
 * for look-ahead work on the previous workspace (asap_local_sgd) first. */
asap_status asap_bind_workspace(asap_ctx* ctx, void* dev, size_t bytes, void* stream);

/* Bind the two model buffers, each [n][ld] fp32 row-major on the device,
 * 256-byte aligned, ld >= dim and a multiple of 64.  Buffer 0 holds the
 * round-0 models; the round counter is reset to 0 and every epoch tag of
 * buffer 0 is set to "round 0 published".  Entries in [dim, ld) are never
 * written and their values do not affect any result.  A row stride that is a multiple of 4 KiB
 * puts every row start in the same DRAM channel and bank and slows the
 * reduce, which reads all rows at one column range at a time; pad such an ld
 * (the Python binding adds 128 floats). */
asap_status asap_bind_models(asap_ctx* ctx, float* buf0, float* buf1, int64_t ld,
                             void* stream);

/* Bind dense shards: X [n][samples][ldx] fp32 (ldx >= dim, multiple of 4,
 * 16-byte aligned), y [n][samples] fp32 in {-1, +1}; worker i owns
 * X[i], y[i].  dim <= 16384 on this path.  samples >= 1.  Entries of X past
 * dim are never used.  For dim > 1024 a pass may use several workgroups per
 * worker that meet once per minibatch step (a cooperative launch); the
 * workspace holds their partial gradients. */
asap_status asap_bind_dense(asap_ctx* ctx, const float* X, const float* y,
                            int64_t samples, int64_t ldx);

/* Bind CSR shards with global offsets: worker i owns rows [i*S, (i+1)*S);
 * row_ptr [n*S+1] int64 (row_ptr[0] = 0, non-decreasing, row_ptr[n*S] =
 * nnz), col [nnz] int32 in [0, dim) strictly ascending within a row, val
 * [nnz] fp32, y [n*S] fp32 in {-1, +1}; dim < 2^30 and fewer than 2^30
 * nonzeros per worker.  The next
 * asap_bind_workspace scans the shards (synchronising its stream) and
 * rejects violations with ASAP_E_INVALID_ARG; rows may hold at most 4096
 * nonzeros.  It also ranks the columns by frequency: the most frequent
 * (up to 8128) are kept in on-chip memory during each SGD pass.  Shards of
 * 2^29 or more nonzeros per worker always take the general SGD kernel. */
asap_status asap_bind_csr(asap_ctx* ctx, const int64_t* row_ptr, const int32_t* col,
                          const float* val, const float* y, int64_t samples, int64_t nnz,
                          void* stream);

/* Members of the planned CSR pass (Appendix A, update (A.2), first line: a
 * worker's minibatch step): `members` workgroups (1, 2 or 4) share each
 * worker's pass, member m owning the model columns c with c mod members ==
 * m; once per step they exchange their partial margins (fp64) and add them
 * in member order, so every member takes the same loss derivative.  0 (the
 * default) chooses 4 or 2 while members * n_workers is at most half the
 * device's compute units, else 1.  With several members the multi-round
 * launch needs members * n_workers workgroups resident at once.  The
 * result differs from one member's only in how the margins' fp64 sums are
 * grouped.  Call before asap_workspace_size: it re-lays out the workspace
 * (a bound workspace is unbound).  Errors: ASAP_E_INVALID_ARG for any
 * other value. */
asap_status asap_set_csr_members(asap_ctx* ctx, int32_t members);
/* The members in effect (after asap_bind_csr; 1 before). */
asap_status asap_get_csr_members(const asap_ctx* ctx, int32_t* members);

/* Half-step of (A.2) for all workers: worker i runs one pass of minibatch
 * SGD over its shard, in the order of asap_schedule(S, seed, i, round), on
 * its row of the current buffer, and tags it (NOTIFY).  Margins of a step
 * use the pre-step model; the gradient is the batch mean (1/B') sum c_b x_b
 * + l2 w; t = round * ceil(S/B) + k + 1.  At most once per round, before
 * the reduce.  Errors: ASAP_E_STATE (no data/models/workspace bound or SGD
 * already done this round), ASAP_E_INVALID_ARG.
 * CSR look-ahead: the per-round sample schedule and column plan do not
 * depend on the models, so after enqueueing round r on `stream` the call
 * also plans round r + 1 (same seed and batch) on the library's own stream,
 * concurrently with round r, into a second plan area of the workspace; a
 * later call for that round, seed and batch waits for it (an event) instead
 * of planning, any other call plans afresh.  That work reads the bound
 * shards and writes only the workspace, and every asap_bind_* call and
 * asap_destroy waits for it before returning: until then the workspace and
 * the shards must stay allocated. */
asap_status asap_local_sgd(asap_ctx* ctx, const asap_sgd_params* p, void* stream);

/* Optional first half of asap_local_sgd: enqueue on `stream` the current
 * round's sample schedule (asap_schedule of Section 5's per-worker pass
 * order; for CSR data also the row descriptors and the column plan, or a
 * wait for the look-ahead plan of this round), so that the SGD kernels of
 * the following asap_local_sgd with the same round, seed and batch start at
 * once.  asap_local_sgd does this itself when it was not done (or was done
 * for other parameters).  Same errors as asap_local_sgd. */
asap_status asap_prepare_sgd(asap_ctx* ctx, const asap_sgd_params* p, void* stream);

/* Stochastic reduce of (A.2), all workers: W'[i] = sum_j P_ij W[j] from the
 * current buffer into the other one, after checking that every neighbour's
 * tag says "published this round" (a mismatch skips that worker's row and
 * is reported by asap_check as ASAP_E_EPOCH).  Then the buffers flip and the
 * round counter advances.  May run without a preceding local_sgd (pure
 * mixing).  Errors: ASAP_E_STATE. */
asap_status asap_stochastic_reduce(asap_ctx* ctx, void* stream);

/* asap_local_sgd followed by asap_stochastic_reduce. */
asap_status asap_round(asap_ctx* ctx, const asap_sgd_params* p, void* stream);

/* `rounds` consecutive rounds (half-step, then reduce) in ONE persistent
 * launch on `stream`, synchronised per worker by the fine-grained NOTIFY-ACK
 * protocol of Section 4 rather than by kernel boundaries: worker i reduces
 * as soon as its in-neighbours have published this round's half-step, and
 * starts its next half-step right after its own reduce, while slower
 * workers are still reducing.  Before overwriting its row in the other
 * buffer it waits until every worker that reads that row (its out-neighbours
 * in the graph) has acknowledged the previous round.
 *
 * Result: bit for bit the models, buffer index, round counter and epoch
 * tags that `rounds` calls of asap_round with the same parameters leave,
 * provided asap_round runs the same half-step code: dense shards always;
 * CSR shards when the stream-ordered path takes its general kernel, or
 * when it takes the planned pass and a plan ring holds every pass of the
 * launch (asap_bind_rounds_plan).  With the planned pass and no ring the
 * launch runs the general kernel, and the two paths agree to the oracle's
 * tolerance but not bitwise.
 *
 * Requirements: state as after a reduce or asap_set_round (no half-step
 * pending); every worker has at most 64 in-neighbours and at most 64
 * out-neighbours (self included); rows of under 2^31 bytes; all workgroups
 * of the launch fit on the device at once (one per worker; K per worker for
 * dense D in (1024, 8192]); else ASAP_E_STATE.  `wait_ms` bounds each wait for a neighbour (0: 10 s).
 * A wait that runs out stops that worker and, in turn, its neighbours; the
 * launch ends and asap_check reports ASAP_E_EPOCH.  The models are then
 * undefined (restore a checkpoint).  A worker whose starting tag is not the
 * round's start tag stops the same way.  Uses the schedule area of the
 * workspace; forgets any CSR plan prepared ahead.  Asynchronous. */
asap_status asap_run_rounds(asap_ctx* ctx, const asap_sgd_params* p, int64_t rounds, int32_t wait_ms,
                            void* stream);

/* Plan ring of the multi-round launch (Section 4 with the planned CSR
 * pass).  With CSR shards whose minibatch steps fit the planned pass
 * (batch <= 64, rows of at most 128 nonzeros in each member's columns, fewer than 2^29 nonzeros per
 * worker) the stream-ordered path plans every pass's column bookkeeping
 * ahead of the pass.  A launch of asap_run_rounds can do the same when the
 * caller binds device memory for the plans of the passes it covers: one
 * area per pass (a launch of R rounds covers R passes, or ceil(R L / K) + 1
 * at most with L local steps of a K-step pass).  asap_rounds_plan_size
 * gives the bytes for `passes` areas (CSR data must be bound;
 * ASAP_E_STATE otherwise); asap_bind_rounds_plan binds caller-owned memory
 * (256-byte aligned; as many areas as fit) after the workspace, writes the
 * round-invariant half of every area on `stream`, and keeps it until the
 * next asap_bind_* or asap_drop_workers call, which unbind it.  A launch
 * whose passes fit in the bound areas then runs the planned pass inside the
 * launch: the plans are made before it on `stream`, or beside it on the
 * library's own stream when the launch leaves compute units free (a worker
 * waits, within wait_ms, until its pass's plan is published), and the
 * result is bit for bit that of the stream-ordered rounds.  Otherwise the
 * launch runs the general CSR kernel. */
asap_status asap_rounds_plan_size(const asap_ctx* ctx, int64_t passes, size_t* bytes);
asap_status asap_bind_rounds_plan(asap_ctx* ctx, void* dev, size_t bytes, void* stream);

/* Where the live models are: index (0 or 1) of the buffer holding the
 * current round's models, the round number, and whether this round's
 * half-step already ran (1) or not (0).  Any out pointer may be NULL. */
asap_status asap_current(const asap_ctx* ctx, int32_t* buffer, int64_t* round,
                         int32_t* half_step_done);

/* Resume: declare that `buffer` holds the models at the start of `round`
 * (e.g. restored from a checkpoint); re-tags that buffer on `stream`.
 * The schedule and step counter continue exactly from `round`. */
asap_status asap_set_round(asap_ctx* ctx, int64_t round, int32_t buffer, void* stream);

/* Reconfiguration after a failure: the graph should be easy to generate
 * for a variable number of machines (the properties listed before
 * Section 4), so the survivors go on with a graph built for their number.
 * Workers dropped[0..n_drop) (ascending, distinct, 1 <= n_drop < n) leave;
 * the others keep their current models, renumbered 0..n-n_drop-1 in their
 * old order (the sample schedule is then keyed by the new number), and use
 * the in-neighbour CSR (nbr_ptr, nbr_idx, nbr_w) over n - n_drop workers
 * from the current round on (validated as in asap_create, `flags` alike).
 * On `stream`, the surviving rows of the current buffer are copied, in
 * order, into the other buffer, which becomes current; the round counter is
 * kept.  The data shards were laid out per old worker, so they are
 * unbound: bind the survivors' shards (asap_bind_dense / asap_bind_csr with
 * n - n_drop workers) and a workspace of the new size before the next
 * half-step.  Needs bound models and no half-step pending (ASAP_E_STATE);
 * argument errors (ASAP_E_INVALID_ARG, ASAP_E_GRAPH) leave the context as it
 * was.  The model buffers keep their size (the first n - n_drop rows are
 * used). */
asap_status asap_drop_workers(asap_ctx* ctx, int32_t n_drop, const int32_t* dropped, const int32_t* nbr_ptr,
                              const int32_t* nbr_idx, const float* nbr_w, uint32_t flags, void* stream);

/* The graph the context runs on: as given to asap_create, or to the last
 * asap_drop_workers (the survivors' graph).  Parity hook: the rows P_i. of
 * update (A.2) that the reduce applies.  Host only, no stream.  Two calls:
 * with nbr_ptr, nbr_idx and nbr_w all NULL it writes *n_workers and
 * *n_entries only; then nbr_ptr [n+1], nbr_idx [n_entries] and nbr_w
 * [n_entries] (host, caller-owned) receive the CSR bit for bit.  Either all
 * three arrays or none: ASAP_E_INVALID_ARG otherwise, or when ctx,
 * n_workers or n_entries is NULL. */
asap_status asap_get_graph(const asap_ctx* ctx, int32_t* n_workers, int64_t* n_entries, int32_t* nbr_ptr,
                           int32_t* nbr_idx, float* nbr_w);

/* The schedules of all workers for `round`, computed by the same device
 * code the SGD kernels use: dev_out [n][S] int32 (device).  Parity hook. */
asap_status asap_schedule_device(asap_ctx* ctx, uint64_t seed, int64_t round,
                                 int32_t* dev_out, void* stream);

/* Per-round metrics, off the hot path (fp64 accumulation on the device;
 * synchronises `stream`).  out[4] (host):
 *   out[0] = mean_i f_i(w_i)   (each worker on its own shard and model)
 *   out[1] = F(w_bar) = (1/n) sum_i f_i(w_bar), w_bar the mean model
 *   out[2] = ||W - 1 w_bar^T||_F (consensus distance, Appendix A bound)
 *   out[3] = mean of all model entries (preserved by the reduce)
 * out[0] and out[1] are NaN when no data is bound. */
asap_status asap_metrics(asap_ctx* ctx, int32_t loss, float l2, double* out, void* stream);

/* asap_metrics for callers that cannot allocate device memory or bring a
 * workspace for it (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and results, bit for
 * bit, but w_bar, the partial sums and the four results live in a static
 * device array of the library (8.4 MiB per GPU, held until the process
 * ends) instead of the context's workspace.  Allocates nothing.  Limits:
 * dim <= 2^20 and n_workers <= 16384, else ASAP_E_INVALID_ARG.  Every call on
 * one GPU uses that GPU's single array, so calls that overlap on one GPU
 * (other streams, other host threads, other contexts) race and must be
 * serialised by the caller; the array keeps the last call's contents.
 * Synchronises `stream`.  out[4] (host) as for asap_metrics. */
asap_status asap_metrics_noalloc(asap_ctx* ctx, int32_t loss, float l2, double* out, void* stream);

/* Synchronise `stream` and read the device error words.  Returns
 * ASAP_E_EPOCH (and clears the words) if any reduce since the last check
 * found a mismatched tag; *bad_worker (may be NULL) gets the lowest such
 * worker.  Returns ASAP_E_DEVICE (and clears the word) if a dense SGD pass
 * with several workgroups per worker found a member missing at a step's
 * rendezvous for too long; that pass stopped early and its models are not
 * valid. */
asap_status asap_check(asap_ctx* ctx, void* stream, int32_t* bad_worker);

/* Failure-injection hook for tests: overwrite the epoch tag of `worker` in
 * `buffer` with `value` on `stream`. */
asap_status asap_debug_set_tag(asap_ctx* ctx, int32_t buffer, int32_t worker,
                               int64_t value, void* stream);

/* Message of the last failed call on this context ("" if none). */
const char* asap_last_error(const asap_ctx* ctx);

/* Release the context (host memory only; no device memory is owned). */
void asap_destroy(asap_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* ASAP_H */
