/*
 * vfl.h - C ABI of the MI355X (gfx950) two-party publisher/subscriber
 * split-learning training step (PubSub-VFL, arXiv 2510.12494).
 *
 * What one step computes (paper, Section 3 "Problem Formulation", Eqs. 1-2;
 * Section 4.1 "System Design"; Algorithm 1):
 *   - the passive party B runs its bottom model f_B on its features and
 *     publishes the embedding z_B of a batch group to the embedding channel
 *     of that group, optionally clipped per row and with Gaussian noise
 *     added (Appendix "Differential Privacy Protocol");
 *   - the active party A (labels + top model g) subscribes to that channel,
 *     runs f_A, g([z_A | z_B]), the binary cross-entropy of Eq. (1), and
 *     back-propagates; it publishes the per-row gradient w.r.t. z_B to the
 *     gradient channel (optionally clipped and noised) and updates its and
 *     the top model's parameters with SGD (Eq. 2);
 *   - B fetches the gradient, back-propagates it through f_B at the
 *     parameters that produced the embedding (the delayed parameter of
 *     Assumption 4 and the Theorem's update rule) and updates its current
 *     parameters with SGD.
 * With staleness s, B may publish up to s groups ahead of the group A
 * consumes; each party's k worker replicas process k consecutive batches of
 * a group with the same parameters and their gradients are averaged with row
 * weights (parameter-server step), giving one update per party per group.
 *
 * Memory and ownership.  The caller allocates one device workspace of
 * vfl_workspace_size() bytes and every input buffer; the library never
 * allocates or frees device memory.  The context owns only HIP events and
 * host metadata.  All pointers in vfl_batch are device pointers; they must
 * stay valid until the enqueued work that reads them has completed (for B:
 * until vfl_bottom_backward of that group has completed, because the
 * backward re-reads B's inputs).
 *
 * Streams.  Party A's work (A's bottom, top model, A's update) runs on
 * stream_a, party B's on stream_b; the two are ordered only through the
 * channel events (an embedding slot's "published" event and a gradient
 * slot's "published" event).  No call blocks the host except
 * vfl_get_param, vfl_get_message, vfl_check, vfl_get_trace and vfl_destroy.
 *
 * Errors.  Every call returns a vfl_status; nothing else crosses the ABI.
 * vfl_last_error() gives a text for the last failure on a context; with a
 * NULL context, the text of the calling thread's last vfl_workspace_size or
 * vfl_create failure (empty after a success).
 */
#ifndef VFL_H
#define VFL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VFL_OK = 0,
  VFL_E_INVALID = 1,    /* bad argument, shape, alignment or option */
  VFL_E_NOMEM = 2,      /* workspace smaller than vfl_workspace_size() */
  VFL_E_HIP = 3,        /* a HIP runtime call failed (text in vfl_last_error) */
  VFL_E_NOT_READY = 4,  /* subscribing to a group not yet published */
  VFL_E_STALE = 5,      /* publishing would exceed the staleness bound s */
  VFL_E_STATE = 6       /* call out of order (wrong group for this phase) */
} vfl_status;

typedef enum { VFL_F32 = 0, VFL_BF16 = 1 } vfl_dtype;

typedef enum {
  VFL_PARTY_A = 0,      /* active party: labels + top model */
  VFL_PARTY_B = 1,      /* passive party: publishes its embeddings */
  VFL_TOP = 2           /* the top model (held by A) */
} vfl_party;

enum { VFL_PARAM_W = 0, VFL_PARAM_B = 1, VFL_PARAM_TABLE = 2 };

/* vfl_opts.flags */
enum {
  VFL_NOISE_EMB = 1,    /* add Gaussian noise to the published embedding */
  VFL_NOISE_GRAD = 2,   /* add Gaussian noise to the returned gradient */
  VFL_CLIP_EMB = 4,     /* clip each embedding row to L2 norm clip_c */
  VFL_CLIP_GRAD = 8,    /* clip each gradient row to L2 norm clip_c */
  VFL_FIFO_DISCARD = 16,/* a full channel discards its oldest group (see
                           vfl_bottom_forward) instead of VFL_E_STALE */
  VFL_LOSS_MSE = 32     /* regression: the top model's output is a prediction
                           and the loss the mean squared error over the
                           group's rows (labels are real-valued targets)
                           instead of the binary cross-entropy of Eq. (1) */
};

#define VFL_MAX_LAYERS 16
#define VFL_MAX_REPLICAS 8
#define VFL_MAX_STALENESS 4   /* channel capacity p = q = 5 slots */

/* A party's bottom model: input = [embeddings of n_cat fields | dense].
 * Field f's table occupies rows [f*vocab, (f+1)*vocab) of one table of
 * n_cat*vocab rows x emb_dim float32 columns.  Layer l maps widths[l-1]
 * (the input width for l = 0) to widths[l]; bit l of relu_mask puts a ReLU
 * after layer l. */
typedef struct {
  int32_t dense_in, n_cat, vocab, emb_dim, n_layers;
  int32_t widths[VFL_MAX_LAYERS];
  uint32_t relu_mask;
} vfl_bottom_spec;

/* The top model on [z_A | z_B]: n_layers >= 2 fully connected layers, the
 * last of width 1 (the logit, or with VFL_LOSS_MSE the prediction; linear);
 * bit j of relu_mask puts a ReLU after hidden layer j.  Party A's layers and
 * the top model's hidden layers together number at most VFL_MAX_LAYERS. */
typedef struct {
  int32_t n_layers;
  int32_t widths[VFL_MAX_LAYERS];
  uint32_t relu_mask;
} vfl_top_spec;

/* dtype: storage and matrix-product operand type of activations, messages
 * and weight copies (VFL_BF16: bf16 operands, float32 accumulation, float32
 * master parameters and updates; VFL_F32: float32 throughout).  batch: rows
 * per replica; staleness s in [0, VFL_MAX_STALENESS]; replicas k in
 * [1, VFL_MAX_REPLICAS]; lr: SGD step; clip_c: L2 bound C; sigma: noise
 * multiplier (noise std = sigma * C, C = 1 when clipping is off); seed:
 * Philox4x32-10 key (low word, high word). */
typedef struct {
  vfl_dtype dtype;
  int32_t batch, staleness, replicas;
  float lr, clip_c, sigma;
  uint64_t seed;
  uint32_t flags;
} vfl_opts;

/* One replica's batch.  dense: [rows x ld] row-major, dtype elements (NULL
 * when dense_in == 0; ld == 0 means dense_in; ld * element size must be a
 * multiple of 16 bytes and dense 16-byte aligned).  ids: int32 [rows x n_cat]
 * (per-field id in [0, vocab)).  labels: float32 [rows] in {0, 1}, party A
 * only.  row0: global sample id of row 0 (keys the noise).  The k replicas
 * of one call must lie back to back (replica r starts where r-1 ends, in
 * every array and in row0), each of `batch` rows except the last. */
typedef struct {
  const void* dense;
  int64_t ld;
  const int32_t* ids;
  const float* labels;
  int32_t rows;
  int64_t row0;
} vfl_batch;

typedef struct vfl_ctx vfl_ctx;

/* Bytes of device workspace the configuration needs (host-only call). */
vfl_status vfl_workspace_size(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                              const vfl_top_spec* top, const vfl_opts* o, size_t* bytes);

/* Create a context over a caller-owned device workspace (256-byte aligned) of
 * at least vfl_workspace_size() bytes; stream_a / stream_b are hipStream_t
 * (NULL: the null stream).  They may be the same stream: both parties' work
 * then runs in enqueue order, with no overlap.  Parameters start at zero: set them with
 * vfl_set_param before the first step. */
vfl_status vfl_create(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                      const vfl_top_spec* top, const vfl_opts* o, void* workspace,
                      size_t bytes, void* stream_a, void* stream_b, vfl_ctx** out);

/* For callers that cannot allocate device memory (code that must not call
 * hipMalloc, such as harnesses that forbid it or set-up that precedes a
 * graph capture): vfl_create with the library's own static workspace of the
 * current device instead of a caller's buffer.  The library holds one
 * array of VFL_STATIC_WORKSPACE_BYTES per device from its load on that
 * device until the process ends; this call allocates no device memory (no
 * hipMalloc, hipFree or allocating library routine) and, like vfl_create,
 * clears the part of the array the configuration uses before returning.
 * stream_a / stream_b as for vfl_create, on the current device.  Every
 * later call on the context behaves exactly as on a vfl_create context.
 * At most one context holds a device's array at a time: VFL_E_STATE while
 * another one has not been destroyed (vfl_destroy releases the array;
 * contexts that shared it would race).  VFL_E_NOMEM when the configuration's
 * vfl_workspace_size exceeds VFL_STATIC_WORKSPACE_BYTES, VFL_E_INVALID for
 * a configuration vfl_create rejects. */
#define VFL_STATIC_WORKSPACE_BYTES (64u << 20)
vfl_status vfl_create_static(const vfl_bottom_spec* a, const vfl_bottom_spec* b,
                             const vfl_top_spec* top, const vfl_opts* o, void* stream_a,
                             void* stream_b, vfl_ctx** out);

/* Copy one parameter tensor in or out (float32 master copy).  party
 * VFL_PARTY_A / VFL_PARTY_B / VFL_TOP; kind VFL_PARAM_W ([out x in]
 * row-major), VFL_PARAM_B ([out]) or VFL_PARAM_TABLE (layer ignored).
 * bytes must equal the tensor size.  *_on_device selects a device or host
 * pointer.  Both calls complete (synchronise both streams) before returning. */
vfl_status vfl_set_param(vfl_ctx* c, vfl_party party, int32_t layer, int32_t kind,
                         const void* src, size_t bytes, int32_t src_on_device);
vfl_status vfl_get_param(vfl_ctx* c, vfl_party party, int32_t layer, int32_t kind,
                         void* dst, size_t bytes, int32_t dst_on_device);

/* Bottom forward of batch group `group` for one party (enqueue only).
 * Party B: uses B's current parameters (the version is recorded), stashes
 * the weights and activations in the group's slot (group mod (s+1)); at most
 * s+1 groups may be in flight (published and not yet back-propagated), else
 * VFL_E_STALE.  With VFL_FIFO_DISCARD the channel instead discards its
 * oldest group (the buffer mechanism of Section 4.1 "System Design"): its embedding when A
 * has not taken it yet (A then skips that group), else its gradient; either
 * way B drops the group without an update and reuses its slot
 * (VFL_E_STALE remains when A is inside that group's step).  Party A: group
 * must be the next group A consumes.  per_replica: n_replicas (1..k)
 * back-to-back batches. */
vfl_status vfl_bottom_forward(vfl_ctx* c, vfl_party party, int64_t group,
                              const vfl_batch* per_replica, int32_t n_replicas);

/* Party B: clip + noise (when enabled) of the group's embedding into the
 * embedding channel slot, write the slot header {group, tick, version} and
 * record the slot's event.  Must follow vfl_bottom_forward(B, group). */
vfl_status vfl_publish(vfl_ctx* c, int64_t group);

/* Party A, after vfl_bottom_forward(A, group): wait for the group's
 * embedding (VFL_E_NOT_READY if vfl_publish(group) was not enqueued), run the
 * top model, the loss (mean BCE of the group's rows written to *loss_dev when
 * loss_dev is not NULL, a device float), the top backward and the top SGD
 * step; publish the gradient message to the group's gradient slot and
 * record its event. */
vfl_status vfl_top_step(vfl_ctx* c, int64_t group, float* loss_dev);

/* Backward + SGD of one party for `group` (after vfl_top_step(group)).
 * Party B waits for the gradient slot's event and back-propagates with the
 * weights and activations stashed by its forward of that group; the update
 * goes to B's current parameters and increments B's version. */
vfl_status vfl_bottom_backward(vfl_ctx* c, vfl_party party, int64_t group);

/* Waiting deadline (Section 4.1 "System Design"): party A gives up on `group`, the next
 * group it would consume, before its forward (host-decided, for instance
 * after a deadline on the embedding's event).  A moves on to group + 1; B's
 * backward of the group (vfl_bottom_backward or the tick's vfl_step) then
 * releases its slot without an update and without waiting for a gradient.
 * Retraining the group's rows is the caller's: feed them again under a
 * later group id.  VFL_E_STATE if group is not A's next group or A is inside
 * a step.  vfl_run refuses to start while a discarded group awaits B's
 * backward; vfl_get_state likewise. */
vfl_status vfl_discard(vfl_ctx* c, int64_t group);

/* One tick t of the deterministic schedule: when n_b > 0, B's forward and
 * publish of group t; when n_a > 0, A's forward, top step and backward of
 * group u = t - s, then B's backward of u.  (b: group t's batches, a: group
 * u's batches with labels.)  With this schedule B's forward of group g uses
 * version max(0, g - s) and the update from group u is delayed by min(u, s).
 * A group u discarded by vfl_discard skips A's phases; B releases it. */
vfl_status vfl_step(vfl_ctx* c, int64_t t, const vfl_batch* a, int32_t n_a,
                    const vfl_batch* b, int32_t n_b, float* loss_dev);

/* A party's resident dataset for vfl_run: row r of every array belongs to
 * sample r.  dense [n_rows x ld] (alignment as for vfl_batch), ids [n_rows x
 * n_cat], labels [n_rows] (party A).  Device pointers, owned by the caller,
 * valid while the binding is used. */
typedef struct {
  const void* dense;
  int64_t ld;
  const int32_t* ids;
  const float* labels;
} vfl_dataset;

/* Bind both parties' resident datasets of n_rows rows for vfl_run. */
vfl_status vfl_bind_dataset(vfl_ctx* c, const vfl_dataset* a, const vfl_dataset* b, int64_t n_rows);

/* Run ticks t0 .. t0+n-1 of vfl_step's schedule over the bound dataset.
 * Group g covers rows [(g mod E) * R, ...) with E = ceil(n_rows / R) groups
 * per epoch (the last group of an epoch is short; its rows are split into
 * replicas of `batch` rows like any group), which are exactly the batches a
 * caller of vfl_step would pass.  The ticks replay captured HIP graphs: one
 * of VFL_GRAPH_CYCLES * (s+1) ticks per phase t mod (s+1), launched n / that
 * many times, and one of the remaining ticks (captured per phase and
 * length).  Every launch derives its tick's rows, noise step and channel
 * headers from a device-side tick record that the graph's last node
 * advances, so the host launches whole graphs only.  Steady state only: t0
 * >= s+1, ticks 0 .. t0-1 already run, no discarded group awaiting B's
 * backward and, after a discard, s+1 further ticks run with vfl_step (the
 * groups in flight then carry the versions the replays derive);
 * VFL_E_STATE otherwise.  loss_ring (device float [loss_len], nullable)
 * receives group u's mean loss at index u mod loss_len. */
#define VFL_GRAPH_CYCLES 4
vfl_status vfl_run(vfl_ctx* c, int64_t t0, int64_t n, float* loss_ring, int64_t loss_len);

/* Copy a channel slot to host memory after synchronising: which 0 = the
 * embedding of `group`, 1 = its gradient message; [rows x width] of the
 * context dtype (float32 or bf16 bits).  header (may be NULL) receives the
 * slot header {group, tick, version}.  VFL_E_STATE if the slot no longer
 * holds that group. */
vfl_status vfl_get_message(vfl_ctx* c, int32_t which, int64_t group, void* dst,
                           size_t bytes, int32_t header[3]);

/* Integer schedule trace, one row of 7 int64 per enqueued tick/phase:
 * {tick, group published or -1, its slot or -1, B version used by that
 * forward or -1, group consumed or -1, its slot or -1, B version after the
 * update or -1}.  Writes min(cap_rows, rows) rows; *rows = total. */
vfl_status vfl_get_trace(vfl_ctx* c, int64_t* buf, size_t cap_rows, size_t* rows);

/* Pure host function: the trace row of tick t of vfl_step's schedule for
 * staleness s and n_groups groups (no context, no GPU). */
vfl_status vfl_schedule_tick(int64_t t, int32_t s, int64_t n_groups, int64_t out[7]);

/* Semi-asynchronous replicas (Section 4.1 "Intra-party Semi-asynchronous
 * Mechanism", Eq. 5; the aggregation step of Algorithm 1).  Each of a
 * party's n workers is its own context (k = 1, the worker's batch of
 * `batch` rows per group, its own parameters and local SGD); every
 * Delta T_t units the party's parameter server averages the workers'
 * parameters and broadcasts the result.  A unit is an epoch in Algorithm 1
 * (or any fixed number of ticks); after unit t (t = 1, 2, ...) the caller
 * averages when t mod vfl_sync_interval(dt0, t) == 0.  With one unit per
 * tick and Delta T = 1 the replicas stay equal to one context of k = n
 * replicas (gradient averaging), up to float32 rounding.
 *
 * vfl_sync_interval (pure host): *dt = Delta T_t of Eq. 5, the ceiling of
 * dt0/2 * tanh(2t/dt0 - 2) + dt0/2, in [1, dt0] (dt0 >= 1, t >= 0).
 *
 * vfl_replica_average: enqueue the average of the float32 master
 * parameters of `parties` (bit VFL_PARTY_A: A's bottom layers, its table
 * and the top model; bit VFL_PARTY_B: B's bottom layers and table) over the
 * n contexts ctxs[0 .. n-1] (1 <= n <= 16, distinct, one configuration, on
 * the current device), weighted by the rows each context's party applied
 * since its previous average (the weights sum to 1; a context that applied
 * none gets weight 0), and write it to every context.  Ordered after the
 * work already enqueued on each context's stream of that party (A: stream_a,
 * B: stream_b) and before their later work; it then rewrites the operand
 * copies of the averaged weights (A's current copies; B's copies in the
 * slot of its next forward, while the slots of groups in flight keep the
 * weights their forward used, as B's delayed backward needs).  Versions and
 * the schedule do not change.  VFL_E_STATE when party A of a context is
 * inside a group's step or no context applied rows since the last average;
 * VFL_E_INVALID for bad arguments. */
vfl_status vfl_sync_interval(int32_t dt0, int64_t t, int32_t* dt);
vfl_status vfl_replica_average(vfl_ctx* const* ctxs, int32_t n, uint32_t parties);

/* Checkpoint and resume.  The state of a context is what the next tick
 * depends on: both parties' parameters (float32 masters, tables, B's
 * per-slot stashed weight copies), the contents and headers of the
 * publisher/subscriber channel slots (Section 4.1: the embedding ring, the
 * gradient ring and B's stashed activations, masks and clip factors of the
 * groups in flight), the versions and next groups of both parties, and the
 * integer schedule trace.  The image is a host buffer of vfl_state_size()
 * bytes (the size grows with the trace: ask again right before
 * vfl_get_state).  vfl_get_state synchronises both streams and copies the
 * whole workspace to the image; VFL_E_STATE while party A is inside a
 * group's step (after vfl_bottom_forward(A) and before its
 * vfl_bottom_backward), VFL_E_INVALID if bytes is too small.
 * vfl_set_state synchronises both streams, restores the image into this
 * context (the same one, or a fresh one created with the same specs,
 * dtype, batch, staleness and replicas on any workspace; the hyper-
 * parameters lr, clip, sigma, seed and flags are this context's), and
 * leaves every channel event complete; VFL_E_INVALID for a foreign,
 * truncated or mismatched image (the context is then unchanged).  A
 * restored run continues exactly as the original from the tick after the
 * image: its results are bitwise those of the uninterrupted run.  Batch
 * pointers of the slots are not part of the image (only the forward that
 * filled a slot reads them). */
vfl_status vfl_state_size(const vfl_ctx* c, size_t* bytes);
vfl_status vfl_get_state(vfl_ctx* c, void* host_buf, size_t bytes);
vfl_status vfl_set_state(vfl_ctx* c, const void* host_buf, size_t bytes);

/* Planner of the system-planning phase (Section 4.3 "System Planning Phase", Algorithm 2; host
 * only, no context).  A party's profile: per-iteration forward and backward
 * delays T = coef * B^exp * w / C of its bottom (Eqs. 7-8) and, for party A,
 * of the top model (Eq. 9; zero coefficients for party B), its total cores
 * C, its candidate worker counts [w_min, w_max] and its memory model
 * M(B) = mem_base + mem_coef * B^chi per worker against mem_cap
 * (mem_coef <= 0: no memory bound). */
typedef struct {
  double lambda, gamma, phi, beta;
  double lambda_top, gamma_top, phi_top, beta_top;
  double cores;
  int32_t w_min, w_max;
  double mem_base, mem_coef, mem_cap;
} vfl_plan_party;

/* The exchange: embedding and gradient bytes per batch row (E and G of a
 * batch of B rows are B times these), the bandwidth B_b in bytes per
 * second, and the memory exponent chi. */
typedef struct {
  double emb_bytes_per_row, grad_bytes_per_row, bandwidth, chi;
} vfl_plan_link;

/* The (w_a, w_p, B) that minimises max(T_A, T_P) + (E + G) / B_b over the
 * candidate batch sizes batches[0 .. n_batches) that both memory models
 * allow and every worker count in the two ranges (Algorithm 2's
 * enumeration; ties keep the first in batch, w_a, w_p order).  out =
 * {w_a, w_p, B}; *cost (may be NULL) the minimum.  VFL_E_INVALID for bad
 * profiles or when no candidate is feasible. */
vfl_status vfl_plan(const vfl_plan_party* a, const vfl_plan_party* p, const vfl_plan_link* link,
                    const int32_t* batches, int32_t n_batches, int32_t out[3], double* cost);

/* Fit one delay term T = coef * B^exp of Eqs. 7-9 to n measured pairs
 * (batch[i], seconds[i]) of a batch-size sweep (host only): exp and
 * log(coef) minimise sum_i (log T_i - log coef - exp * log B_i)^2, the way
 * the constants of the Appendix's Table 7 come from measured delays.
 * VFL_E_INVALID for n < 2, a non-positive or non-finite value, or fewer than
 * two distinct batch sizes. */
vfl_status vfl_fit_delay(const double* batch, const double* seconds, int32_t n, double* coef,
                         double* expo);

/* Synchronise both streams and report the device-side checks since the
 * context was created: the number of times a consumer found a slot header
 * whose group differs from the one it expected (0 when the channel is
 * race-free), and (bad_ids, may be NULL) the number of categorical ids
 * outside [0, vocab) that the forwards read.  Such an id is used as the
 * nearest valid one (0 or vocab - 1), so no access leaves its field's
 * table; it is counted once per forward that takes its row. */
vfl_status vfl_check(vfl_ctx* c, uint32_t* header_mismatches, uint32_t* bad_ids);

/* Raw Philox4x32-10 words of the noise generator (enqueued on `stream`,
 * a hipStream_t): out_dev[(r * groups + q) * 4 + i] = word i for counter
 * (step, row0 + r, q, tag) and key (seed low word, seed high word), for
 * r < rows, q < groups.  out_dev: device uint32 [rows * groups * 4]. */
vfl_status vfl_philox(uint64_t seed, uint32_t step, uint32_t tag, uint32_t row0, int32_t rows,
                      int32_t groups, uint32_t* out_dev, void* stream);

/* Kernel classes for vfl_timing_* (bit i of a mask selects class i). */
typedef enum {
  VFL_K_FWD = 0,        /* party B: bottom forward + published embedding */
  VFL_K_ACTIVE = 1,     /* party A: bottom + top forward, loss, input-gradient
                           chains, gradient message */
  VFL_K_BWD = 2,        /* party B: cut-layer backward + input-gradient chain */
  VFL_K_DW = 3,         /* weight-gradient products (SGD fused when unsplit) */
  VFL_K_REDUCE = 4,     /* split-partial and logit reductions + SGD */
  VFL_K_CAST = 5,       /* weight operand copies */
  VFL_K_EMB_SGD = 6,    /* sorted sparse SGD of the tables */
  VFL_K_GEMM = 7,       /* layer products of party B's wide layers (input gradient) */
  VFL_K_DWT = 8,        /* large-tile bf16 weight-gradient products (partials + SGD) */
  VFL_K_AVG = 9,        /* replica parameter averaging (vfl_replica_average) */
  VFL_K_COUNT = 10
} vfl_kernel_class;

/* Measurement hook: while class_mask is non-zero, every launch of a
 * selected class is bracketed by two HIP events on its own stream (this adds
 * two event records per launch and nothing else); in vfl_run's replayed
 * graphs, the launches of every fourth tick of the captured cycle, and
 * vfl_timing_read then reports those of the last replay.  vfl_timing_read
 * synchronises both streams and returns, for one class, the summed kernel
 * durations in milliseconds, the number of launches and the summed
 * algorithmic work (matrix-product FLOPs for VFL_K_FWD .. VFL_K_DW, VFL_K_GEMM
 * and VFL_K_DWT, bytes
 * that the kernel must move at minimum for the others); then it resets that class.
 * Enabling with mask 0 stops recording. */
vfl_status vfl_timing_enable(vfl_ctx* c, uint32_t class_mask);
vfl_status vfl_timing_read(vfl_ctx* c, int32_t kernel_class, double* ms, int64_t* launches,
                           double* work);

/* Text of the last failure on c (owned by the context, valid until its next
 * call); c == NULL: the calling thread's last vfl_workspace_size/vfl_create
 * failure (thread-local storage, valid until that thread's next such call). */
const char* vfl_last_error(const vfl_ctx* c);

/* Synchronise both streams and release the context's events and host state.
 * The workspace stays the caller's. */
vfl_status vfl_destroy(vfl_ctx* c);

#ifdef __cplusplus
}
#endif
#endif /* VFL_H */
