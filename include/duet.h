/*
 * duet.h -- C ABI of the mixed-batch paged-attention library for MI355X (gfx950).
 *
 * One serving iteration's attention over a paged KV cache, split the way the paper
 * splits a mixed prefill/decode iteration (Section 4 overview, Algorithm 1):
 *   - prefill requests (chunked prefill, possibly with a cached prefix) run a causal,
 *     compute-bound attention on MFMA;
 *   - decode requests (one new token each) run a bandwidth-bound split-K paged attention
 *     followed by a small reduce kernel;
 *   - the two halves either share the whole GPU on one stream (temporal sharing), or run
 *     concurrently on two streams bound to disjoint CU sets (spatial sharing, Section 4.3).
 * A host-side roofline latency model (Section 4.1) and the split optimiser of Section 4.2 /
 * Algorithm 1 choose between the two.
 *
 * Conventions
 *   - Every function returns DUET_OK (0) or a negative DUET_E* code; the message of the last
 *     failure on the calling thread is returned by duet_last_error().  Argument checks run
 *     before any GPU work is enqueued: a call that fails launches nothing.
 *   - No C++ exception crosses this boundary.
 *   - Device pointers are plain HIP device addresses.  The caller owns every tensor (q, caches,
 *     page table, workspace, out); the library never allocates or frees caller memory.  It owns
 *     its streams, events, pinned staging buffers and latency-model tables.
 *   - GPU work is asynchronous to the host: it starts after the work already queued on the
 *     caller's `stream` and completes before work queued there later.
 *   - Give spatially shared calls a created stream, not the legacy default stream (NULL): HIP
 *     synchronises every launch on a blocking stream, the CU-masked ones included, with work
 *     pending on the default stream, and back-to-back calls always leave some there (the next
 *     call's fork and the previous call's join).  Measured on a 32-layer iteration: 4878 vs
 *     4385 us per step.  Results do not depend on the stream.
 *
 * Tensor layouts (one layer)
 *   q, out    [T, h_q, d]                 tokens of all requests, packed in seq_meta order
 *   k_cache   [P, h_kv, page_size, d]     token-major pages
 *   v_cache   [P, h_kv, d, page_size]     dim-major pages (each dim's page_size tokens contiguous)
 *   page_table[R, max_pages] int32        logical page j of request r is physical page
 *                                         page_table[r * max_pages + j]; token t of request r is
 *                                         slot t % page_size of logical page t / page_size.
 *   Element type is bf16 or fp32 (shape.dtype) for q, caches and out.  Accumulation is fp32.
 *
 * Attention semantics (Section 2 and Section 4.1): request r with q_len scheduled tokens and
 * cached_len cached tokens has kv_len = cached_len + q_len keys, the new tokens' keys and values
 * already written to the cache.  Query i sits at absolute position cached_len + i and attends
 * keys 0 .. cached_len + i with weights softmax(q.k / sqrt(d)).  Query head h reads kv head
 * h / (h_q / h_kv).
 */
#ifndef DUET_H
#define DUET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------------------------ */
#define DUET_OK 0
#define DUET_EINVAL (-1)       /* bad argument: null pointer, size out of range, bad split */
#define DUET_EUNSUPPORTED (-2) /* valid but unsupported: head_dim, page size, dtype, group size */
#define DUET_EWORKSPACE (-3)   /* workspace smaller than duet_workspace_bytes() */
#define DUET_EHIP (-4)         /* a HIP runtime call failed */
#define DUET_ENOMEM (-5)       /* host or pinned allocation failed */
#define DUET_EPAGE (-6)        /* a kernel met a page id outside [0, num_phys_pages) */
#define DUET_EIO (-7)          /* latency-model file could not be read or written */

/* ---- enums --------------------------------------------------------------------------------- */
#define DUET_BF16 0
#define DUET_F32 1

#define DUET_KIND_PREFILL 0
#define DUET_KIND_DECODE 1

#define DUET_AGG 0   /* temporal sharing: both halves on the caller's stream, all CUs */
#define DUET_SPLIT 1 /* spatial sharing: decode on cus_decode CUs, prefill on cus_prefill CUs */
#define DUET_CONCURRENT 2 /* control for measurements: both halves at once on two streams that may
                             each use every CU (concurrency without partitioning); accepted by the
                             attention calls only, not by the latency model */

/* status_flags of duet_choose_cu_split (bit set) */
#define DUET_STATUS_SLO_INFEASIBLE 1 /* no decode share meets the TBT bound; aggregated returned */
#define DUET_STATUS_UNCALIBRATED 2   /* the model still holds the nominal MI355X peaks */

#define DUET_TOTAL_CUS 256
#define DUET_CU_STEP 8 /* CU shares are multiples of 8: one CU per XCD */
/* The S_d grid of duet_choose_cu_split: multiples of 32 CUs.  CU-mask bit b selects a CU on XCD
 * b mod 8 and shader engine (b / 8) mod 4; the dispatcher deals a kernel's workgroups evenly to
 * the shader engines of each XCD, so only multiples of 32 give every shader engine the same
 * number of CUs.  Other multiples of 8 are accepted by every call but run 25-35% slower than the
 * multiple of 32 below them (measured on the decode kernel). */
#define DUET_SPLIT_STEP 32

/* ---- plain structs (same bytes on host and device) ------------------------------------------ */
typedef struct {
  int32_t num_q_heads;  /* h_q */
  int32_t num_kv_heads; /* h_kv, divides h_q */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t page_size;    /* 16 */
  int32_t dtype;        /* DUET_BF16 or DUET_F32 */
  int32_t num_layers;   /* L: t_total = L * t_attn in the latency model; layers run by duet_attn_iteration */
} duet_shape;

typedef struct {
  int32_t kind;       /* DUET_KIND_PREFILL or DUET_KIND_DECODE (decode requires q_len == 1) */
  int32_t q_start;    /* first row of this request in q / out */
  int32_t q_len;      /* scheduled (new) tokens, >= 1 */
  int32_t cached_len; /* tokens already in the cache before this iteration, >= 0 */
} duet_seq_meta;

typedef struct {
  const duet_seq_meta* reqs; /* host array, num_reqs entries; row r uses page_table row r */
  int32_t num_reqs;
} duet_batch;

typedef struct {
  int32_t mode;           /* DUET_AGG, DUET_SPLIT or (attention calls only) DUET_CONCURRENT */
  int32_t cus_prefill;    /* S_p, multiple of 8 (SPLIT) */
  int32_t cus_decode;     /* S_d, multiple of 8 (SPLIT), S_p + S_d <= 256 */
  int32_t k_decode_steps; /* k of Section 4.2: decode steps planned per prefill step (>= 1) */
} duet_cu_split;

typedef struct {
  /* Filled by duet_last_kernel_times() when profiling is on, for the last duet_attn_mixed_batch
   * or duet_attn_iteration call, from HIP events on each kernel's own stream.  Per-kernel
   * durations are means over the call's layers. */
  double decode_partial_us; /* split-K paged decode kernel, per launch (with bf16 it includes the
                               merge of the layer before, except in the first layer) */
  double decode_reduce_us;  /* partial merge kernel, per launch (a bf16 call launches one, after
                               its last layer) */
  double prefill_us;        /* prefill attention kernel, per launch */
  double decode_total_us;   /* decode half: first partial start to last reduce end (with AGG the
                               halves interleave on one stream, so the two spans overlap) */
  double iteration_us;      /* fork to join on the caller's stream */
  double decode_start_us;   /* fork to the start of the first decode partial kernel */
  double prefill_start_us;  /* fork to the start of the first prefill kernel */
  double prefill_total_us;  /* prefill half: first prefill start to last prefill end */
  double layers;            /* number of layers of the call */
  /* duet_attn_lookahead calls only (0 otherwise; the decode_partial/reduce fields are then 0,
   * since the decode kernels run inside graphs): */
  double decode_steps;         /* k */
  double decode_step_us;       /* decode half span / k (with AGG the span includes the prefill) */
  double decode_first_step_us; /* start of decode step 0 to its end: when step 0's tokens are ready */
} duet_kernel_times;

typedef struct duet_ctx duet_ctx;
typedef struct duet_model duet_model;

/* ---- latency model (host only; Section 4.1, 4.2, Algorithm 1) ----------------------------- */

/* New model holding nominal MI355X tables: Pi(S) = 2.5 PFLOP/s * S/256 (dense bf16 MFMA),
 * B(S) = 8 TB/s * S/256, for S = 8, 16, ..., 256.  The caller frees it with duet_model_destroy. */
int duet_model_create(duet_model** out);
int duet_model_destroy(duet_model* m);

/* The model's work accounting (Section 4.1): sums over the requests of `kind` (-1 = all) of
 * F = 4 h_q q (q + c) d + 2 h_q q (q + c) and B = 2 h_q q d b + 2 h_kv (q + c) d b, times
 * shape->num_layers.  Host only; used to turn measured kernel times into achieved rates. */
int duet_batch_work(const duet_shape* shape, const duet_batch* batch, int32_t kind, double* flops, double* bytes);

/* Replace the achievable-throughput tables (Section 4.2: profiled once per partition size).
 * cus[i] must be the 32 values 8, 16, ..., 256 in order; flops_per_s and bytes_per_s > 0.
 * Marks the model calibrated and clears any sharing tables. */
int duet_model_set_tables(duet_model* m, int32_t n, const int32_t* cus, const double* flops_per_s,
                          const double* bytes_per_s);
int duet_model_get_tables(const duet_model* m, int32_t n, int32_t* cus, double* flops_per_s,
                          double* bytes_per_s);
/* Sharing tables: Pi(S) and B(S) of each share measured while the other half runs on the other
 * CUs.  When set, the halves of a SPLIT batch holding both kinds use them instead of the
 * standalone tables (an extension of Section 4.2: the two partitions of a spatially shared GPU
 * slow each other down through HBM, L2 and power).  Same layout and checks as
 * duet_model_set_tables.  get returns the standalone tables and *is_set = 0 when none are set. */
int duet_model_set_sharing_tables(duet_model* m, int32_t n, const int32_t* cus, const double* flops_per_s,
                                  const double* bytes_per_s);
int duet_model_get_sharing_tables(const duet_model* m, int32_t n, int32_t* cus, double* flops_per_s,
                                  double* bytes_per_s, int32_t* is_set);

/* Spatial-sharing efficiencies in (0, 1]: when a SPLIT batch holds both kinds, the two halves
 * run at the same time and slow each other down (shared HBM, L2 and power); the prefill half's
 * Pi (from the sharing tables if set) is then multiplied by prefill_eff and the decode half's B
 * by decode_eff.  Aggregated
 * predictions and single-kind batches use the tables as they are.  Calibrate decode_eff so that
 * decode latency is never under-predicted (appendix: under-prediction is the harmful
 * direction). */
int duet_model_set_efficiency(duet_model* m, double prefill_eff, double decode_eff);
/* Fixed latency tables, seconds per layer: when the requests a prediction covers include
 * prefill (decode) requests, each layer adds prefill_s[i] (decode_s[i]) of the share cus[i] =
 * 8 (i + 1).  An extension of the Section 4.1 roofline for what a roofline leaves out (kernel
 * launches, the decode kernel's tail when its last work items finish); all zero by default,
 * which is the paper's model.  Entries >= 0 and finite; not cleared by duet_model_set_tables. */
int duet_model_set_launch_tables(duet_model* m, int32_t n, const int32_t* cus, const double* prefill_s,
                                 const double* decode_s);
int duet_model_get_launch_tables(const duet_model* m, int32_t n, int32_t* cus, double* prefill_s, double* decode_s);
int duet_model_save(const duet_model* m, const char* path); /* small JSON file */
int duet_model_load(duet_model* m, const char* path);

/* Predicted latency (microseconds) of one iteration of shape->num_layers layers.
 * AGG: L * (sum_r max(F_r / Pi(256), B_r / B(256)) + the launch terms of the kinds present).
 * SPLIT: max(k * t_d(S_d), t_p(S_p)) with t_X(S) = L * (sum_{r in X} max(F_r / Pi(S), B_r / B(S))
 * + launch_X(S) if X holds a request).
 * F_r = 4 h_q q (q + c) d + 2 h_q q (q + c); B_r = 2 h_q q d b + 2 h_kv (q + c) d b.
 * m may be NULL (nominal tables). */
int duet_predict_iter_latency(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                              duet_cu_split split, double* us);

/* One partition's predicted time (microseconds) for shape->num_layers layers: t_X(S) of the
 * requests of `kind` on `cus` CUs, the quantity Algorithm 1 compares (t_d(S_d), t_p(S_p)).
 * shared != 0 prices a half that runs beside the other (the sharing tables and efficiencies)
 * when the batch holds both kinds.  m may be NULL (nominal tables). */
int duet_predict_partition_latency(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                                   int32_t kind, int32_t cus, int32_t shared, double* us);

/* Algorithm 1: aggregated if the whole-GPU prediction meets tbt_slo_us, else the (S_p, S_d, k)
 * maximising (k T_decode + T_prefill) / max(k t_d, t_p) subject to t_d <= tbt_slo_us, with S_d in
 * 32, 64, ..., 224 (DUET_SPLIT_STEP) and k in {floor(t_p/t_d), floor(t_p/t_d) + 1} minus 0.  Ties keep the first
 * (smallest S_d, then smaller k).  max_decode_steps > 0 caps k at the number of decode steps the
 * caller can launch ahead (Section 4.3, look-ahead decode): both candidates are clamped to the
 * cap, which keeps the best allowed k because rho rises in k up to floor(t_p/t_d) and falls after
 * it; <= 0 leaves k uncapped.  predicted_us,
 * rho and status_flags may be NULL; rho is 0 for aggregated.  m may be NULL (nominal tables). */
int duet_choose_cu_split(const duet_model* m, const duet_shape* shape, const duet_batch* batch,
                         double tbt_slo_us, int32_t max_decode_steps, duet_cu_split* out,
                         double* predicted_us, double* rho, int32_t* status_flags);

/* ---- full-model estimate (Section 4.1: token-level operators, overall estimation) --------- */

/* Dense dimensions of the transformer block around the attention layers. */
typedef struct {
  int32_t ffn_dim;     /* m: width of the gate-up output and of the down projection's input, >= 1 */
  int32_t vocab_size;  /* classifier output width, >= 0 (0 leaves the classifier out) */
  int32_t flags;       /* DUET_BLOCK_* bits */
} duet_block_shape;
#define DUET_BLOCK_GQA_QKV 1        /* QKV projection d -> (h_q + 2 h_kv) head_dim; the paper states d -> d */
#define DUET_BLOCK_FUSED_GATE_UP 2  /* gate-up projection d -> 2 m; the paper states d -> m */

/* Full-model iteration latency (Section 4.1, "Token-Level Operators" and "Overall Estimation"):
 * t = num_layers (t_tok + t_attn) + t_cls.  t_attn is duet_predict_iter_latency's per-layer term.
 * t_tok sums, over the token-level operators of one layer on the n tokens the requests process
 * (n = sum of q_len), max(F / Pi(S), B / B(S)):
 *   RMSNorm, QKV (d -> d), output (d -> d), residual add, RMSNorm, gate-up (d -> m), SwiGLU,
 *   down (m -> d), residual add; d = num_q_heads * head_dim, b = element bytes;
 *   linear d_i -> d_o: F = 2 n d_i d_o, B = (n d_i + d_i d_o + n d_o) b (Section 4.1);
 *   the paper leaves the others open; read here as RMSNorm F = 4 n d, B = 2 n d b + d b;
 *   SwiGLU F = 5 n m, B = 3 n m b; residual add F = n d, B = 3 n d b.
 * t_cls is a linear operator d -> vocab_size on one row per request.  SPLIT: each partition runs
 * every layer and the classifier for its own requests (reading the weights itself), with the
 * same tables as duet_predict_iter_latency, and t = max(k t_decode(S_d), t_prefill(S_p)).  One
 * GPU: no all-reduce term.  Host only; m may be NULL (nominal tables). */
int duet_predict_model_latency(const duet_model* m, const duet_shape* shape, const duet_block_shape* block,
                               const duet_batch* batch, duet_cu_split split, double* us);

/* Algorithm 1 on the full-model estimate.  Arguments, results and flags as duet_choose_cu_split;
 * T_decode and T_prefill, the tokens of rho, are unchanged. */
int duet_choose_cu_split_model(const duet_model* m, const duet_shape* shape, const duet_block_shape* block,
                               const duet_batch* batch, double tbt_slo_us, int32_t max_decode_steps,
                               duet_cu_split* out, double* predicted_us, double* rho, int32_t* status_flags);

/* ---- token-level operators (Section 4.1: the operators that act on each token independently).
 * The block forward chains them around the attention kernels; they are exported one by one so
 * each can be checked against its definition on its own inputs.  All tensors are caller-owned
 * contiguous bf16 device arrays, row-major; work is enqueued on `stream` (asynchronous). ---- */

/* y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * weight for rows r of x [rows, d] (d a multiple of 8):
 * fp32 arithmetic, one rounding to bf16.  DUET_EINVAL for null pointers, bad sizes or eps <= 0. */
int duet_rmsnorm(duet_ctx* ctx, const void* x, const void* weight, void* y, int32_t rows, int32_t d, float eps,
                 void* stream);
/* act[r] = silu(g[r]) * u[r] with g, u the two halves of gate_up [rows, 2 m] (gate columns first),
 * silu(g) = g / (1 + exp(-g)): fp32 arithmetic, one rounding to bf16; m a multiple of 8. */
int duet_swiglu(duet_ctx* ctx, const void* gate_up, void* act, int32_t rows, int32_t m, void* stream);
/* The QKV split of one layer (Section 2: the new tokens' keys and values enter the cache before
 * attention): qkv [T, (h_q + 2 h_kv) d] rows in seq_meta order; each row's first h_q d columns go
 * to q [T, h_q, d]; its key and value columns go to slot pos % 16 of physical page
 * page_table[r][pos / 16] of k_cache [P, h_kv, 16, d] and v_cache [P, h_kv, d, 16], pos =
 * cached_len + the row's index in its request.  A pure copy.  workspace of at least
 * duet_workspace_bytes(); page ids outside the pool are not written and set its error word. */
int duet_qkv_split(duet_ctx* ctx, const duet_shape* shape, const void* qkv, void* q, void* k_cache, void* v_cache,
                   int64_t num_phys_pages, const int32_t* page_table, int32_t max_pages_per_req,
                   const duet_batch* batch, void* workspace, size_t workspace_bytes, void* stream);

/* ---- GPU context ----------------------------------------------------------------------------- */

/* Infrastructure (no passage of its own): the device state every call below uses.
 * Context on HIP device `device`: checks for gfx950 and 256 CUs, creates the CU-masked stream
 * pool lazily (one stream per distinct CU set, kept for the context's lifetime), events and
 * pinned staging buffers, and a latency model with nominal tables.  *out is owned by the caller
 * and released with duet_destroy. */
int duet_init(int device, duet_ctx** out);
/* duet_init, then the context's latency model loaded from `model_path`, a file written by
 * duet_model_save after calibration (Section 4.2: the per-partition throughput tables are
 * profiled once, ahead of serving, and reused).  DUET_EIO if the file cannot be read or parsed;
 * then nothing is created. */
int duet_init_with_model(int device, const char* model_path, duet_ctx** out);
int duet_destroy(duet_ctx* ctx);
/* The context's own latency model (owned by the context; valid until duet_destroy). */
duet_model* duet_ctx_model(duet_ctx* ctx);

/* Infrastructure (memory sizing for the iteration of Section 4.3).
 * Bytes of device workspace duet_attn_mixed_batch and duet_attn_iteration need for this shape
 * and batch: an error word, the decode work-queue counters, metadata, work lists, two buffers
 * of decode split-K partials (consecutive layers alternate between them) and the partial states
 * of prefill pieces (bf16: a prefill unit whose causal key range is long against the batch's
 * total runs as several pieces over runs of its keys, merged by the last one to finish, and when
 * a batch has at least 512 whole units its 256 shortest run as 4 pieces each; at most 512 + 1024
 * pieces write a partial, 128 KiB each at head_dim 128).  The layers of a call share all of
 * it, so the size does not depend on shape->num_layers.  Host only. */
int duet_workspace_bytes(const duet_shape* shape, const duet_batch* batch, size_t* bytes);

/* One layer's attention over a mixed batch (Section 4.3: prefill and decode of one iteration
 * multiplexed in space).  q [T, h_q, d] (T = sum of q_len, requests' rows contiguous from
 * q_start), k_cache [num_phys_pages, h_kv, 16, d] (token-major pages), v_cache
 * [num_phys_pages, h_kv, d, 16] (dim-major pages), page_table [num_reqs, max_pages_per_req]
 * int32, workspace and out [T, h_q, d] are device pointers owned by the caller; batch lives in
 * host memory.  Prefill requests go to the MFMA prefill kernel, decode requests to the split-K
 * decode kernel and its reduce kernel.  AGG runs decode then prefill on `stream` (all CUs).
 * SPLIT forks onto two CU-masked streams (decode on the first cus_decode CUs, prefill on the last
 * cus_prefill CUs) and joins back onto `stream`; work enqueued on `stream` before the call is complete before
 * either half starts, and work enqueued after it sees the whole output.  The result is
 * bit-identical for every split and every placement of the pages: all reduction orders depend
 * on logical token positions and on the batch only.  Page ids read by a kernel outside [0, num_phys_pages) are
 * not dereferenced; they set an error word that duet_check_device_error() reports.  Invalid
 * arguments return DUET_EINVAL / DUET_EUNSUPPORTED / DUET_EWORKSPACE before anything is enqueued.
 * Calls on one context are serialised by the host (a mutex); the caller must not reuse a
 * workspace before the call that uses it has finished on `stream`.  k_decode_steps is not used
 * here (one step). */
int duet_attn_mixed_batch(duet_ctx* ctx, const duet_shape* shape, const void* q, const void* k_cache,
                          const void* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                          int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split,
                          void* workspace, size_t workspace_bytes, void* out, void* stream);

/* For callers that cannot allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): duet_attn_mixed_batch without the workspace argument.  The call's
 * workspace is a file-scope device array of DUET_NOALLOC_SCRATCH_BYTES held by each device the
 * library runs on until the process ends; the call allocates nothing (no device or pinned memory,
 * no streams, no events).  Batches whose work lists and partials need more return
 * DUET_EWORKSPACE, as do work lists beyond the 1 MiB of pinned staging duet_init preallocates.
 * Under DUET_SPLIT or DUET_CONCURRENT the CU-masked streams must already exist: one earlier call
 * of duet_attn_mixed_batch or duet_attn_iteration with the same split creates them (the context
 * keeps the streams of its most recently used split or mode); otherwise DUET_EINVAL.  Profiling
 * is ignored.  The output is bit-identical to duet_attn_mixed_batch's.  Every call on a device shares that device's array,
 * which keeps the last call's contents (each call's upload clears the parts that must start at
 * zero): calls that overlap on one device, from any context or thread, race.  Page ids outside
 * the pool are never dereferenced; the error word they set lives in the scratch and is not
 * reported. */
#define DUET_NOALLOC_SCRATCH_BYTES (64u << 20)
int duet_attn_mixed_batch_noalloc(duet_ctx* ctx, const duet_shape* shape, const void* q, const void* k_cache,
                                  const void* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                                  int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* out,
                                  void* stream);

/* The attention of a whole serving iteration: shape->num_layers layers (at most 1024) over the
 * same batch and page table (Section 4.3: each partition runs its phase's layers as one stream of
 * work; Section 4.1: t_total = L * t_attn).  q, k_cache, v_cache and out are host arrays of
 * num_layers device pointers, each laid out as in duet_attn_mixed_batch.  The work lists are
 * built and uploaded once; with SPLIT each half runs its kernels for every layer back to back on
 * its CU-masked stream (the host enqueues the halves layer by layer, alternating), with one fork
 * and one join per call; AGG runs layer by layer, decode then prefill, on `stream`.  With bf16,
 * layer l's decode split merge runs inside layer l + 1's decode kernel (one reduce kernel per call,
 * after the last layer), so no layer's output is complete before the call returns.  Layer l's
 * output is bit-identical to duet_attn_mixed_batch on layer l's pointers. */
int duet_attn_iteration(duet_ctx* ctx, const duet_shape* shape, const void* const* q,
                        const void* const* k_cache, const void* const* v_cache, int64_t num_phys_pages,
                        const int32_t* page_table, int32_t max_pages_per_req, const duet_batch* batch,
                        duet_cu_split split, void* workspace, size_t workspace_bytes, void* const* out,
                        void* stream);

/* ---- the whole block (Section 4.1, token-level operators) --------------------------------------
 *
 * L transformer blocks over a mixed batch, each partition running its own tokens through every
 * operator on its CUs (Section 4.3: the decode and prefill partitions each run the model for
 * their requests).  Per layer: h = RMSNorm(x) g_attn; qkv = h W_qkv; the query columns go to
 * attention and the new tokens' key and value columns are written into the paged cache (token t
 * of a request with c cached tokens at position c + t); a = attention (the kernels above);
 * x += a W_o; h = RMSNorm(x) g_ffn; [g | u] = h W_gate_up; x += (silu(g) * u) W_down.  RMSNorm
 * is x / sqrt(mean(x^2) + eps); silu(g) = g / (1 + exp(-g)).  bf16 tensors, fp32 arithmetic
 * inside each operator, bf16 between operators; the projections run on hipBLASLt. */
typedef struct {
  const void* attn_norm; /* [d] (d = h_q * head_dim) */
  const void* w_qkv;     /* [d, (h_q + 2 h_kv) head_dim] row-major: query, key, value columns */
  const void* w_o;       /* [d, d] */
  const void* ffn_norm;  /* [d] */
  const void* w_gate_up; /* [d, 2 ffn_dim]: gate columns 0 .. ffn_dim - 1, then up */
  const void* w_down;    /* [ffn_dim, d] */
} duet_block_weights;

/* Byte offsets in the duet_block_forward workspace of its activation buffers, in this order:
 * RMSNorm output [T, d], QKV projection [T, d_qkv], queries [T, h_q, d_h], attention output
 * [T, h_q, d_h], gate-up projection [T, 2 m], SwiGLU output [T, m] (bf16, T = scheduled tokens).
 * After a call they hold the last layer's activations (the RMSNorm buffer: the one before the
 * feed-forward part; with look-ahead, the decode rows of the last step).  Host only. */
int duet_block_buffers(const duet_shape* shape, const duet_block_shape* block, const duet_batch* batch,
                       int32_t k_decode_steps, size_t* offsets);
/* Workspace of duet_block_forward with k_decode_steps decode steps: duet_workspace_bytes' layout
 * (with the work lists of look-ahead steps 1 .. k - 1), the activations of every scheduled token
 * ([T, d] x4, [T, (h_q + 2 h_kv) head_dim], [T, 2 ffn_dim], [T, ffn_dim], bf16) and two hipBLASLt
 * workspaces.  Host only. */
int duet_block_workspace_bytes(const duet_shape* shape, const duet_block_shape* block, const duet_batch* batch,
                               int32_t k_decode_steps, size_t* bytes);

/* Runs shape->num_layers blocks in place on the residual stream x [T, d] (bf16, rows packed per
 * request in batch order).  weights, k_cache and v_cache are host arrays of num_layers entries
 * (device pointers; caches laid out as in duet_attn_mixed_batch); every scheduled token's key and
 * value rows are written to its layer's cache.  block->flags must be DUET_BLOCK_GQA_QKV |
 * DUET_BLOCK_FUSED_GATE_UP (the layout above); ffn_dim and d are multiples of 8; bf16 only;
 * norm_eps > 0.  AGG runs everything on `stream`; SPLIT runs the decode requests' rows on the
 * decode CUs and the prefill requests' rows on the prefill CUs, each partition all layers back
 * to back, and needs each kind's rows to be one contiguous range (DUET_EUNSUPPORTED otherwise).
 * Requests must not share cache pages.  A page id outside [0, num_phys_pages) met while writing
 * or reading the cache is not dereferenced and sets the error word.  Stream, ownership and
 * validation rules as for duet_attn_iteration.  Look-ahead (Section 4.3): with
 * split.k_decode_steps = k > 1 the decode requests run k steps in the call; step s = 1 .. k - 1
 * takes their next residual rows from x_ahead[s - 1] ([R_d, d] bf16 device memory, decode requests
 * in batch order, updated in place), writes those tokens' keys and values at position
 * cached_len + s (the page table must cover cached_len + k tokens) and attends over them; under
 * SPLIT the steps run back to back on the decode CUs while the prefill partition runs once.  With
 * profiling on, duet_last_kernel_times() reports iteration_us (fork to join) and, under a split,
 * decode_total_us / decode_start_us / decode_first_step_us (the decode partition; step s's tokens
 * are ready at its end) and prefill_total_us / prefill_start_us. */
int duet_block_forward(duet_ctx* ctx, const duet_shape* shape, const duet_block_shape* block,
                       const duet_block_weights* weights, float norm_eps, void* x, void* const* x_ahead,
                       void* const* k_cache, void* const* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                       int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                       size_t workspace_bytes, void* stream);

/* ---- serving engine: continuous batching with chunked prefill (Sections 2-4) ------------------
 *
 * The batch former of the serving loop and its paged KV-cache allocator (host only).  Requests
 * wait in arrival order.  Each step schedules, under a token budget, first one token for every
 * running request whose prompt is fully prefilled (in admission order), then prompt tokens of
 * the partly prefilled requests and then of the waiting ones, chunking the last prompt taken.
 * The pages the step's tokens need are reserved from a free list; a request keeps its pages
 * until it has produced its output tokens.  The caller runs the step on the GPU (e.g.
 * duet_block_forward, which writes the scheduled tokens' keys and values into those pages), then
 * calls duet_engine_complete. */
typedef struct duet_engine duet_engine;

/* token_budget >= 1 tokens per step; page_size 16; num_pages cache pages (ids 0 .. num_pages - 1,
 * handed out in order, or in a splitmix64 Fisher-Yates permutation when shuffle_seed != 0);
 * page-table rows of max_pages_per_req entries. */
int duet_engine_create(int32_t token_budget, int32_t page_size, int64_t num_pages, int32_t max_pages_per_req,
                       uint64_t shuffle_seed, duet_engine** out);
int duet_engine_destroy(duet_engine* engine);
/* Queues a request; *id (may be NULL) receives its id (0, 1, ... in call order).  DUET_EINVAL if a
 * length is < 1 or prompt + output tokens need more than max_pages_per_req pages. */
int duet_engine_add_request(duet_engine* engine, int32_t prompt_len, int32_t output_len, int64_t* id);
/* Forms the next step into host arrays of max_reqs rows: meta (rows packed, decodes first, q_start
 * running), page_table [max_reqs, max_pages_per_req] (-1 padded) and req_ids (may be NULL);
 * *num_reqs may be 0.  DUET_ENOMEM when the free pages do not cover the step (nothing changes;
 * there is no preemption, so the pool must hold the pages of every running request), DUET_EINVAL
 * when max_reqs is too small or the previous step is not completed. */
int duet_engine_step(duet_engine* engine, duet_seq_meta* meta, int32_t* page_table, int64_t* req_ids,
                     int32_t max_reqs, int32_t* num_reqs);
/* Section 4.3: the same step with decode_steps = k >= 1 look-ahead decode steps (for
 * duet_attn_lookahead with k_decode_steps = k): each decode's page-table row covers
 * cached_len + k tokens (the rows of meta are as for one step).  DUET_EINVAL also when a decode's
 * k tokens would need more than max_pages_per_req pages. */
int duet_engine_step_lookahead(duet_engine* engine, int32_t decode_steps, duet_seq_meta* meta, int32_t* page_table,
                               int64_t* req_ids, int32_t max_reqs, int32_t* num_reqs);
/* Marks the last step done: chunks advance, each decode gains its token (after a look-ahead step,
 * min(k, its remaining output) tokens), finished requests release their pages. */
int duet_engine_complete(duet_engine* engine);
/* The same when only the first decode_steps_run (1 .. the step's k) look-ahead steps ran, e.g. a step
 * formed with pages for the largest k allowed before Algorithm 1 chose a smaller one; the pages
 * reserved for the other steps stay with their requests. */
int duet_engine_complete_lookahead(duet_engine* engine, int32_t decode_steps_run);
int duet_engine_stats(const duet_engine* engine, int64_t* waiting, int64_t* running, int64_t* free_pages);

/* ---- look-ahead decode (Section 4.3, interruption-free dispatch) -------------------------------
 *
 * Decode requests get KV slots for k future steps ahead of time, and the k decode steps run back
 * to back with no host synchronisation between them; the decode kernels of a step are replayed
 * from a graph recorded once, while the prefill kernels are launched one by one.  Here one call
 * is one prefill step plus k = split.k_decode_steps decode steps (Algorithm 1 sizes k so that k
 * decode steps fit in one prefill step: t = max(k t_d, t_p)). */

/* Workspace for duet_attn_lookahead with k_decode_steps steps (shape->num_layers layers):
 * duet_workspace_bytes' layout plus the metadata and work lists of steps 1 .. k - 1.  Host
 * only. */
int duet_lookahead_workspace_bytes(const duet_shape* shape, const duet_batch* batch, int32_t k_decode_steps,
                                   size_t* bytes);

/* One prefill step and k = split.k_decode_steps (1 .. 64) decode steps over shape->num_layers
 * layers (num_layers * k <= 16384).
 *   Step 0 is duet_attn_iteration on (q, k_cache, v_cache, out): every request of the batch,
 *   the decode tokens at position cached_len already in the cache.
 *   Decode step s = 1 .. k - 1, layer l, uses index x = (s - 1) * num_layers + l of the
 *   look-ahead arrays.  Decode request i (the i-th kind-DECODE row of batch, in order) first
 *   writes its new token's key row k_ahead[x][i] and value row v_ahead[x][i] (each [h_kv, d])
 *   at position p = cached_len + s: slot p % 16 of physical page page_table[r][p / 16]; keys
 *   into the token-major k_cache[l], values into the dim-major v_cache[l] column.  It then
 *   attends over the p + 1 keys 0 .. p with query q_ahead[x][i] ([h_q, d]) into out_ahead[x][i].
 *   q_ahead, k_ahead, v_ahead and out_ahead are host arrays of (k - 1) * num_layers device
 *   pointers to [R_d, h_q or h_kv, d] tensors (R_d = number of decode requests), caller-owned;
 *   they may be NULL when k == 1 or R_d == 0.
 * Steps run in order, so step s reads the tokens steps 1 .. s - 1 wrote.  Every decode request's
 * page_table row must hold pages for cached_len + k tokens; the slots written must not be read
 * by any other request of the batch (the prefill half runs at the same time).
 * SPLIT / CONCURRENT: the first prefill layer is enqueued on the prefill stream, then every decode
 * step on the decode stream, then the other prefill layers; one fork and one join on `stream`.
 * AGG: decode step 0,
 * then the prefill layers, then decode steps 1 .. k - 1, on `stream`.
 * Decode steps run from graphs by default: the kernels of the steps that run back to back (all k
 * steps with SPLIT / CONCURRENT; step 0, then steps 1 .. k - 1, with AGG and while profiling is
 * on, so that an event can mark when step 0's tokens are ready) are captured on first use, and the
 * graph is replayed on later calls whose launch arguments (pointers, work-list sizes, CU share)
 * are the same; at most 128 graphs are kept per context (least recently used evicted, after a
 * device synchronisation).  Outputs and cache writes are bit-identical with graphs on or off,
 * and step 0 is bit-identical to duet_attn_iteration.  Errors as duet_attn_iteration; a page id
 * outside [0, num_phys_pages) at a written slot skips the write and sets the error word. */
int duet_attn_lookahead(duet_ctx* ctx, const duet_shape* shape, const void* const* q, const void* const* q_ahead,
                        const void* const* k_ahead, const void* const* v_ahead, void* const* k_cache,
                        void* const* v_cache, int64_t num_phys_pages, const int32_t* page_table,
                        int32_t max_pages_per_req, const duet_batch* batch, duet_cu_split split, void* workspace,
                        size_t workspace_bytes, void* const* out, void* const* out_ahead, void* stream);

/* Decode steps of duet_attn_lookahead from graphs (enable != 0, the default) or launched one
 * kernel at a time (enable == 0). */
int duet_set_decode_graphs(duet_ctx* ctx, int32_t enable);

/* Graphs held by the context, and how many decode-step graphs were captured / replayed so far. */
int duet_decode_graph_stats(duet_ctx* ctx, int64_t* cached, int64_t* captured, int64_t* replayed);

/* Infrastructure (the page-table contract of the paged cache, Section 2): the kernels never
 * dereference a page id outside [0, num_phys_pages) and record one in the workspace's error word.
 * Synchronises `stream`, reads the error word and clears it: DUET_OK or DUET_EPAGE. */
int duet_check_device_error(duet_ctx* ctx, void* workspace, void* stream);

/* Section 2: attention reads each request's cached keys and values through its page table.
 * Copy request `req`'s logical keys (which == 0, from a token-major cache) or values (which == 1,
 * from a dim-major cache) into out_contig [kv_len, h_kv, d] -- the page gather the attention
 * kernels perform, exported so it can be checked bit for bit.  Device pointers are the
 * caller's; page ids outside the pool set the error word of duet_check_device_error. */
int duet_gather_kv(duet_ctx* ctx, const duet_shape* shape, int32_t which, const void* cache,
                   int64_t num_phys_pages, const int32_t* page_table, int32_t max_pages_per_req,
                   int32_t req, int32_t kv_len, void* out_contig, void* stream);

/* Profiling level: 0 off; 1 records HIP events at the fork and the join of every
 * duet_attn_mixed_batch / duet_attn_iteration call on the caller's stream (iteration latency
 * only); 2 also records events around each kernel on the stream it runs on (these add small
 * gaps between kernels).
 * duet_last_kernel_times() waits for the last call's events and returns the durations (kernel
 * fields are 0 at level 1). */
int duet_set_profiling(duet_ctx* ctx, int32_t level);
int duet_last_kernel_times(duet_ctx* ctx, duet_kernel_times* out);

/* ---- calibration probes (Section 3 "Opportunity", Section 4.2 profiling) -------------------- */

/* Streaming HBM read over `bytes` of device memory at `buf` on a stream restricted to `cus` CUs
 * (256 = the unrestricted stream); repeated `iters` times.  Returns achieved bytes/s. */
int duet_probe_read_bw(duet_ctx* ctx, int32_t cus, const void* buf, size_t bytes, int32_t iters,
                       double* bytes_per_s);
/* Register-resident bf16 MFMA loop (16x16x32, four independent chains, two waves per SIMD) on
 * `cus` CUs; `iters` trips of 32 MFMAs per wave (8192 keeps a full-chip launch long enough that
 * dispatch and ramp stay out of the figure).  Returns achieved FLOP/s. */
int duet_probe_mfma(duet_ctx* ctx, int32_t cus, int32_t iters, double* flops_per_s);
/* Record the hardware placement of `blocks` workgroups launched on the stream restricted to
 * `cus` CUs taken from the low end (high_end == 0, the decode side) or the high end (1, the
 * prefill side) of the CU bit order.  hw_ids_dev receives 2 uint32 per workgroup:
 * (XCC_ID register, HW_ID register).  Synchronous. */
int duet_probe_placement(duet_ctx* ctx, int32_t cus, int32_t high_end, int32_t blocks, uint32_t* hw_ids_dev);
/* Fill `m` with Pi(S) and B(S) measured by the two probes for S = 8, 16, ..., 256, using
 * scratch device memory of `scratch_bytes` at `scratch` for the read probe. */
int duet_calibrate(duet_ctx* ctx, duet_model* m, const void* scratch, size_t scratch_bytes);

/* Thread-local message of the last failure ("" if none). */
const char* duet_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DUET_H */
