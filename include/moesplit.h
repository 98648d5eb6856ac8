/*
 * moesplit.h -- C ABI of libmoesplit, the per-layer MoE forward over split
 * experts for one AMD Instinct MI355X (gfx950).
 *
 * Method: arXiv 2509.08342 ("MoEpic").  Each expert's SwiGLU FFN is cut into
 * a top and a bottom segment (Sec. 2.3, split ratio theta = share of the top
 * segment).  Top segments of some experts are cached in a budgeted VRAM pool
 * (Sec. 3.1, 3.4.1: per-layer budget V_i, cache size C_i = V_i / theta_i);
 * bottom segments and uncached experts stay in host RAM and are copied into a
 * VRAM buffer on demand or by speculative prefetch (Sec. 3.2).  After routing,
 * resident segments are computed while missing ones are copied (Sec. 3.2,
 * Eq. (5)-(6)).
 *
 * The cut runs along the FFN intermediate axis: the top segment holds units
 * [0, F_top) of W_gate/W_up columns and W_down rows, the bottom [F_top, F).
 * Each segment's contribution is a partial down-projection and the partials
 * sum to the unsplit expert, so the layer output does not depend on r, on
 * residency or on prediction.
 *
 * Conventions for every entry point:
 *  - Return value: ms_status.  No exceptions cross the ABI.  On MS_E_INVALID,
 *    MS_E_BUDGET, MS_E_STATE and MS_E_UNSUPPORTED the context state is
 *    unchanged.  MS_E_HIP means a HIP runtime call failed; the context is then
 *    poisoned and every later call except ms_last_error/ms_destroy returns
 *    MS_E_HIP.  ms_last_error() gives a human-readable message.
 *  - A context is used by one host thread at a time.
 *  - Streams are passed as void* (a hipStream_t); NULL means the null stream.
 *    The library creates two more streams of its own (default priority): a
 *    copy stream for host-to-device segment transfers and a side stream for
 *    computing streamed segments.
 *  - "h_dev", "y_dev", ... are device pointers owned by the caller.
 *    Host arrays passed to ms_set_* are copied before the call returns.
 *  - Element type of weights and activations is the model's dtype (MS_F32 or
 *    MS_BF16, bf16 passed as raw 16-bit patterns); accumulation is fp32.
 */
#ifndef MOESPLIT_H
#define MOESPLIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MS_OK = 0,
  MS_E_INVALID = 1,     /* bad argument (pointer, index, size, range)        */
  MS_E_BUDGET = 2,      /* device pool or top-segment cache too small         */
  MS_E_STATE = 3,       /* call not valid in the current state                */
  MS_E_HIP = 4,         /* HIP runtime error; context poisoned                */
  MS_E_NOMEM = 5,       /* host allocation (pinned store) failed              */
  MS_E_UNSUPPORTED = 6  /* shape outside what the kernels support             */
} ms_status;

typedef enum { MS_F32 = 0, MS_BF16 = 1 } ms_dtype;

/* Model shape.  Sec. 2.1: L layers, N (= n_experts) experts per layer, K
 * (= top_k) activated per token, hidden width d.  d_ff is each expert's
 * intermediate width F.  n_shared always-active experts of width d_ff_shared
 * (weight 1) extend the paper's module for models that have them; they are
 * always VRAM-resident and count as non-expert parameters U_n (Sec. 3.4.1).
 * renormalize = 1 divides the selected scores by their sum as in Eq. (2).
 * max_tokens bounds T of every forward; n_buffer_slots is the number of
 * full-expert slots of the VRAM staging buffer U_b (0 -> 2*top_k: one set for
 * the running layer, one for the next layer's prefetch).  ffn_splits is the
 * number of work-groups that share one 64-unit chunk of the FFN kernel (1, 2
 * or 4, and at most 2 when d_model > 4096: MS_E_UNSUPPORTED beyond; 0 ->
 * chosen from the shape so that a decode step fills the GPU).  It
 * changes the summation grouping, not what is computed.  expert_bits = 2 or
 * 4 stores the routed experts as affine b-bit codes (the HQQ format of the
 * paper's 2-bit Mixtral setting, Sec. 4.1; see ms_set_expert_q); 0 keeps
 * them in the model dtype.  b-bit experts need dtype MS_BF16, no shared
 * experts, d_ff a multiple of 64, d_model a multiple of 64 in [256, 8192] and
 * ffn_splits 0 or 1 (MS_E_UNSUPPORTED otherwise).  Every shape needs
 * d_ff and d_ff_shared at most 65535 * 64 and n_shared at most 32767
 * (MS_E_UNSUPPORTED otherwise). */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t d_ff;
  int32_t n_experts;
  int32_t top_k;
  int32_t n_shared;
  int32_t d_ff_shared;
  int32_t dtype;
  int32_t renormalize;
  int32_t max_tokens;
  int32_t n_buffer_slots;
  int32_t ffn_splits;
  int32_t expert_bits;
} ms_model_desc;

/* Sizes the library derives from a model shape (pure host arithmetic). */
typedef struct {
  uint64_t chunk_bytes;       /* bytes of one 64-unit chunk: 3 * 64 * d * elem,
                                 b-bit experts 24 * b * d + 12 * d             */
  int32_t n_chunks;           /* ceil(F / 64)                                  */
  uint64_t expert_bytes;      /* n_chunks * chunk_bytes (U_e, zero-padded)     */
  uint64_t fixed_pool_bytes;  /* device pool bytes needed besides top caches:
                                 routers, shared experts, work buffers and the
                                 staging buffer                                */
  uint64_t buffer_bytes;      /* of which: staging buffer (U_b)                */
} ms_sizes;

/* Per-layer statistics (counts since the last ms_reset_stats). */
typedef struct {
  uint64_t forwards;
  uint64_t tokens;
  uint64_t selected;          /* (token, expert) selections                   */
  uint64_t experts_active;    /* distinct experts summed over forwards         */
  uint64_t alpha;             /* active experts fully in VRAM at routing time  */
  uint64_t beta;              /* active experts with only the top cached       */
  uint64_t gamma;             /* active experts with nothing in VRAM           */
  uint64_t buffer_hits;       /* active experts whose missing part had already
                                 been (at least partly) prefetched             */
  uint64_t bytes_miss;        /* H2D bytes issued after routing                */
  uint64_t bytes_prefetch;    /* H2D bytes issued by prefetch                  */
  uint64_t bytes_prefetch_used;  /* prefetched bytes a forward then consumed  */
  uint64_t bytes_prefetch_dropped; /* prefetch bytes dropped before issue     */
  uint64_t predicted_hits;    /* selected experts among the top-K predicted    */
  uint64_t predictions;       /* forwards that had a prediction to check       */
  uint64_t cache_inserts;     /* top segments cached by the online policy      */
} ms_layer_stats;

/* Timeline record (see ms_timeline_begin). */
typedef enum {
  MS_IV_ROUTER = 0,        /* router + top-K (+ prediction) kernel              */
  MS_IV_GROUP = 1,         /* token grouping kernel                              */
  MS_IV_FFN_RESIDENT = 2,  /* SwiGLU over resident chunks (compute stream)       */
  MS_IV_FFN_STREAMED = 3,  /* SwiGLU over streamed chunks (side stream)          */
  MS_IV_COMBINE = 4,       /* weighted combine kernel                            */
  MS_IV_COPY_MISS = 5,     /* H2D copy issued after routing                      */
  MS_IV_COPY_PREFETCH = 6, /* H2D copy issued by prefetch                        */
  MS_IV_COPY_TOP = 7,      /* H2D copy of a top segment (ms_load_top)            */
  MS_IV_PREDICT = 8,       /* prediction ranking kernel                          */
  MS_IV_FFN_DOWN = 9       /* matrix-core down-projection (prefill path)         */
} ms_interval_kind;

typedef struct {
  int32_t kind;       /* ms_interval_kind                                        */
  int32_t layer;
  double t0_ms;       /* start, ms since the timeline origin event               */
  double t1_ms;       /* end                                                     */
  uint64_t bytes;     /* kernels: weight bytes read (algorithmic);
                         copies: bytes transferred                               */
} ms_interval;

typedef struct ms_ctx ms_ctx;

/* ---- sizing (no GPU needed) ------------------------------------------------ */

/* Derived sizes of a model shape.  MS_E_INVALID if a field is out of range
 * (non-positive sizes, top_k > n_experts, unknown dtype); MS_E_UNSUPPORTED if
 * the kernels do not cover the shape: d_model must be a multiple of 64 in
 * [256, 8192], n_experts at most 512, top_k at most 64, and max_tokens * top_k
 * at most 2^24. */
ms_status ms_query_sizes(const ms_model_desc* desc, ms_sizes* out);

/* The split point and cache size of Sec. 3.4 for one layer, without a
 * context: F_top = 64 * floor(r * F / 64 + 1/2) clamped to [0, F] (whole
 * chunks), top_bytes = chunks(F_top) * chunk_bytes, and C_i =
 * floor(budget_bytes / top_bytes) capped at n_experts (0 if top_bytes = 0).
 * r must lie in [0, 1]. */
ms_status ms_split_plan(const ms_model_desc* desc, uint64_t budget_bytes, float r,
                        int32_t* top_units_out, uint64_t* top_bytes_out,
                        int32_t* top_slots_out);

/* ---- context --------------------------------------------------------------- */

/* Create a context on the current HIP device.  dev_pool/pool_bytes is a
 * caller-owned device allocation that emulates the VRAM budget V of Eq. (8):
 * every device byte the library uses (routers, shared experts, work buffers,
 * the staging buffer U_b and the top-segment caches sum_i V_i) is carved from
 * it.  pool_bytes must cover ms_sizes.fixed_pool_bytes (else MS_E_BUDGET).
 * The pinned host expert store (hipHostMalloc) is allocated here:
 * n_layers * n_experts * expert_bytes (MS_E_NOMEM on failure), unless
 * host_store_experts > 0 limits it to that many distinct expert blobs, in
 * which case experts must be provided with ms_alias_expert beyond that. */
ms_status ms_create(const ms_model_desc* desc, void* dev_pool, uint64_t pool_bytes,
                    int32_t host_store_experts, ms_ctx** out);
void ms_destroy(ms_ctx* ctx);
const char* ms_last_error(const ms_ctx* ctx);

/* Router R^i of layer i (Sec. 2.1): w_r host [d][E] in the model dtype
 * (logits = h . w_r); bias host [E] fp32 or NULL, added to the logits. */
ms_status ms_set_router(ms_ctx* ctx, int32_t layer, const void* w_r, const float* bias);

/* Expert e of layer i: host w_gate [d][F], w_up [d][F], w_down [F][d] in the
 * model dtype, E(h) = (silu(h.w_gate) * (h.w_up)) . w_down.  Copied into the
 * pinned host store in chunk-packed order: per 64-unit chunk, the 64 gate
 * columns, the 64 up columns and the 64 down rows, each as d-contiguous rows,
 * so that a top segment is a contiguous prefix of the blob and a bottom
 * segment a contiguous suffix (gate and up rows k-tiled: 64 consecutive
 * elements of one row, then the next row's).  The store is pinned, coherent
 * host memory, read by the device over PCIe.  Setting an expert again waits
 * for work in flight, rewrites its blob in place (also for every expert
 * aliasing it), drops staged copies of it and re-copies its cached top
 * segments, so later forwards use only the new weights. */
ms_status ms_set_expert(ms_ctx* ctx, int32_t layer, int32_t e, const void* w_gate,
                        const void* w_up, const void* w_down);

/* Expert e of layer i of a b-bit model (expert_bits = b): affine codes with
 * one fp16 scale s and zero z per group of 64 consecutive elements along each
 * matrix's input axis, w = (q - z) * s.  Matrices are [out][in]: gate and up
 * [F][d] (W_gate = gate^T), down [d][F] (W_down = down^T).  gate_q, up_q:
 * host [F][d * b / 8] bytes, down_q: host [d][F * b / 8] bytes, codes packed
 * 8 / b per byte, element i of a row at bits (i % (8 / b)) * b of byte
 * i / (8 / b); gate_m, up_m: host [F][d / 64][2], down_m: host [d][F / 64][2]
 * uint16 fp16 bit patterns (scale, zero).  Repacked into the chunk order of
 * the b-bit kernel in the pinned store (a top segment is still a prefix of
 * the blob); rewrite semantics as ms_set_expert.  MS_E_STATE on a model
 * whose experts are not b-bit (and ms_set_expert returns MS_E_STATE on one
 * whose experts are). */
ms_status ms_set_expert_q(ms_ctx* ctx, int32_t layer, int32_t e, const void* gate_q, const void* gate_m,
                          const void* up_q, const void* up_m, const void* down_q, const void* down_m);

/* Make expert (layer, e) use the host blob of (src_layer, src_e), which must
 * already be set.  Lets a deep stack reuse a few distinct weight sets. */
ms_status ms_alias_expert(ms_ctx* ctx, int32_t layer, int32_t e, int32_t src_layer,
                          int32_t src_e);

/* Shared expert s of layer i (same layout, width d_ff_shared), copied to the
 * device pool and always resident. */
ms_status ms_set_shared_expert(ms_ctx* ctx, int32_t layer, int32_t s, const void* w_gate,
                               const void* w_up, const void* w_down);

/* Cache configuration of Sec. 3.4 (the output of Algorithm 1, or any other
 * plan): per-layer budget V_i in bytes and split ratio theta_i = r[i] in
 * [0, 1].  Derives F_top, top_bytes and C_i per layer as in ms_split_plan,
 * carves sum_i C_i * top_bytes_i from the pool (MS_E_BUDGET if it does not
 * fit), writes C_i to top_slots_out[i] (nullable), and resets residency: no
 * top cached, staging buffer empty.  Synchronises the library's streams. */
ms_status ms_configure(ms_ctx* ctx, const uint64_t* budget_bytes, const float* r,
                       int32_t* top_slots_out);

/* Cache the top segment of expert e in layer i: asynchronous H2D copy of the
 * blob prefix into a free cache slot on the copy stream; later forwards wait
 * for it.  MS_E_BUDGET if all C_i slots are taken, MS_E_STATE if already
 * cached or if the layer's split has no top (F_top = 0). */
ms_status ms_load_top(ms_ctx* ctx, int32_t layer, int32_t e);

/* Drop expert e's top segment from layer i's cache (MS_E_STATE if not
 * cached).  The slot is reused only after forwards that read it finished. */
ms_status ms_evict_top(ms_ctx* ctx, int32_t layer, int32_t e);

/* Residency of layer i's experts: state_out[E] = 0 nothing, 1 top segment
 * cached, 2 whole expert in VRAM (top cached with F_top = F). */
ms_status ms_residency(ms_ctx* ctx, int32_t layer, uint8_t* state_out);

/* Speculative prediction of Eq. (3): apply layer i's router to h (usually the
 * previous layer's activation h^{i-1}) and rank layer i's experts by the
 * token-summed softmax score, descending, lower index first on equal scores.
 * h_dev [T][d] (model dtype) on `stream`.  Blocks until the result is on the
 * host: order_out[E] (int32), score_out[E] (fp32, nullable). */
ms_status ms_predict(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T,
                     void* stream, int32_t* order_out, float* score_out);

/* Prefetch of Sec. 3.2: copy the missing part of experts[0..n) of layer i
 * into the staging buffer, one expert after the other in the given order --
 * the bottom segment if the top is cached, the whole expert otherwise --
 * while free buffer slots last.  Copies are issued a few chunks ahead;
 * whatever is not yet issued when layer i's routing result is known
 * (ms_forward of layer i) is dropped. */
ms_status ms_prefetch(ms_ctx* ctx, int32_t layer, const int32_t* experts, int32_t n);

/* Flags of ms_forward. */
#define MS_FWD_PREDICT_NEXT 1  /* after issuing the misses, predict the next
                                  layer (layer+1, or layer 0 of the next token
                                  after the last layer) from this layer's h and
                                  prefetch its experts (Sec. 3.2)            */
#define MS_FWD_MATRIX_CORES 2  /* force the prefill path: gate/up and down
                                  projections on the matrix cores (bf16 only) */
#define MS_FWD_NO_MATRIX_CORES 4 /* force the decode path (chunk kernel)    */
/* Without either flag a bf16 forward takes the prefill path when
 * T * top_k >= 8 * n_experts (on average >= 8 tokens per expert). */

/* MoE module of layer i (Eq. (2) without residual and Norm) on T tokens,
 * 0 <= T <= max_tokens:
 *   idx_dev[T][K] (int32): experts with the K largest router logits, in
 *     descending order, lower index first on equal logits (a NaN logit
 *     counts as -inf, in the ranking and in the softmax scores);
 *   w_dev[T][K] (fp32): softmax scores of the selected experts, divided by
 *     their sum if renormalize;
 *   y_dev[T][d] (fp32): sum_k w[t][k] * E_{idx[t][k]}(h_t) + shared experts.
 * Enqueued on `stream`; returns after the missing segments have been
 * issued (the host waits for the routing result).  Outputs are valid once
 * `stream` has completed.  h_dev, y_dev, idx_dev, w_dev must not be reused
 * by the caller before that.  The library marks the end of the forward on
 * `stream` only when something waits for it (ms_sync, ms_load_top, a
 * forward on another stream, ms_destroy), so `stream` must stay valid until
 * then. */
ms_status ms_forward(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T,
                     float* y_dev, int32_t* idx_dev, float* w_dev, int32_t flags,
                     void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture elsewhere in their stream, tight serving loops, harnesses that
 * forbid hipMalloc): ms_forward with its per-forward work buffers (router
 * logits, grouping, FFN partials, combine sums, activations, routing
 * workspace) in a fixed array of 64 MiB in device memory that the library
 * holds on every GPU it runs on until the process ends, instead of in the
 * context's pool.  Same arguments, semantics and outputs as ms_forward; the
 * call allocates no device or pinned memory and creates no HIP objects.
 * MS_E_UNSUPPORTED if the context's work buffers (they grow with
 * max_tokens) exceed 64 MiB.  Every call on a GPU, from any context, uses
 * that GPU's one array: calls of one context are ordered like its
 * ms_forward calls, but calls of two contexts on the same GPU that overlap
 * in time race on the array and give undefined outputs. */
ms_status ms_forward_noalloc(ms_ctx* ctx, int32_t layer, const void* h_dev, int32_t T,
                             float* y_dev, int32_t* idx_dev, float* w_dev, int32_t flags,
                             void* stream);

/* Wait until every copy and kernel the library issued has finished. */
ms_status ms_sync(ms_ctx* ctx);

/* Drop the staging buffer's contents (prefetched or streamed segments). */
ms_status ms_drop_buffer(ms_ctx* ctx);

ms_status ms_stats(ms_ctx* ctx, int32_t layer, ms_layer_stats* out);
ms_status ms_reset_stats(ms_ctx* ctx);

/* ---- Cache configurator (Sec. 3.3-3.4, Eq. (4)-(11), Algorithm 1) ---- */

/* Statistics of layer i gathered by ms_forward since ms_create or
 * ms_reset_plan_stats (Sec. 3.4.2), normalised: hit[C] = H_i(C), the share of
 * activations whose expert was among the C highest cache priorities (Eq. (4))
 * at that forward, C = 0..N; pred[y-1] = P_i(y), the tokens per token that
 * activated the expert the prediction ranked y-th; pred_hit[(y-1)*(N+1)+C] =
 * PH_i(y, C), the share of tokens for which that expert was among the C
 * highest priorities.  P and PH count the forwards that had a prediction for
 * layer i (MS_FWD_PREDICT_NEXT of the previous layer or ms_predict); a batch
 * of T tokens shares its prediction.  Host arrays of N+1, N and N*(N+1)
 * doubles (any may be NULL).  tokens_out (may be NULL): [q, q_pred]. */
ms_status ms_plan_stats(ms_ctx* ctx, int32_t layer, double* hit, double* pred, double* pred_hit,
                        uint64_t* tokens_out);
ms_status ms_reset_plan_stats(ms_ctx* ctx);

/* Cache priority of every expert of layer i (Eq. (4)): mu * rho^(nu/omega),
 * mu = activations so far, nu = forwards since the last activation (a batch
 * counts as one forward).  rho, omega from ms_set_cache_policy (default
 * 0.25, 128).  prio_out: host [N] doubles. */
ms_status ms_lcp_priority(ms_ctx* ctx, int32_t layer, double* prio_out);

/* Inputs of the configurator: model shape, profiled latencies in
 * microseconds (Sec. 3.4.1: attention, MoE layer, head, one whole expert's
 * load), and per-layer statistics laid out as ms_plan_stats returns them
 * ([L] consecutive blocks). */
typedef struct {
  int32_t n_layers, n_experts, top_k;
  uint64_t expert_bytes;
  double t_att_us, t_moe_us, t_head_us, t_load_us;
  const double* hit;       /* [L][N+1]   */
  const double* pred;      /* [L][N]     */
  const double* pred_hit;  /* [L][N][N+1] */
} ms_plan_problem;

/* Algorithm 1's VramAllocation over a total expert budget v_e_bytes (V_e):
 * starting from start_budgets ([L] bytes, each > 0; NULL: V_e / L each),
 * repeatedly move floor(zeta * V_e) bytes from the layer whose exposed
 * loading latency grows least to the one whose latency falls most, while the
 * summed exposed latency decreases (at most max_iter moves).  Each layer's
 * split ratio solves the sub-problem of Eq. (11) under the window its
 * predecessor leaves (Eq. (7)).  Outputs (host arrays of L; any but
 * budgets_out may be NULL): budgets, split ratios theta_i, cache sizes C_i
 * (the planner's count of experts), exposed latencies (us) and the moves
 * taken.  Pure host arithmetic; needs no context.  MS_E_INVALID for bad
 * sizes, zeta outside (0, 1), or a start budget <= 0. */
ms_status ms_plan_solve(const ms_plan_problem* p, uint64_t v_e_bytes, double zeta, const uint64_t* start_budgets,
                        int32_t max_iter, uint64_t* budgets_out, double* theta_out, int32_t* cache_out,
                        double* exposed_us_out, int32_t* iters_out);

/* Apply a plan (Algorithm 1, "update the expert cache"): ms_configure with
 * these budgets and ratios, then per layer cache the top segments of the C_i
 * experts of highest priority (Eq. (4); ties to the lower index).  Waits for
 * work in flight; clears the staging buffer. */
ms_status ms_cache_update(ms_ctx* ctx, const uint64_t* budgets, const float* r);

/* Online replacement (Sec. 3.3): after a forward in which a selected expert
 * had no cached top, cache its top segment (copied from the staging slot
 * that holds the whole expert) in place of the cached expert the policy
 * ranks lowest: MS_CACHE_LCP by Eq. (4), MS_CACHE_LRU by last activation,
 * MS_CACHE_LFU by activation count, MS_CACHE_RND uniformly (seeded), each
 * with ties to the lower index.  Missed experts are taken in descending
 * order of the policy's rank, at most one per cache slot and forward; each
 * takes the lowest-numbered free slot if there is one, and an expert cached
 * in this forward is not evicted in it.  MS_CACHE_STATIC (the
 * default) never changes the cache on its own.  rho in (0, 1) and omega > 0
 * parameterise Eq. (4) for the statistics and LCP.  MS_CACHE_RND's ranks:
 * every forward of a layer with a cache draws one key per expert, in index
 * order, from a SplitMix64 generator (Steele, Lea and Flood, OOPSLA 2014)
 * whose state this call sets to seed XOR 0x9e3779b97f4a7c15; a key is the
 * output's top 53 bits.  The generator is shared by the context's layers. */
typedef enum {
  MS_CACHE_STATIC = 0,
  MS_CACHE_LCP = 1,
  MS_CACHE_LRU = 2,
  MS_CACHE_LFU = 3,
  MS_CACHE_RND = 4
} ms_cache_policy;
ms_status ms_set_cache_policy(ms_ctx* ctx, int32_t policy, double rho, double omega, uint64_t seed);

/* Engine of the host-to-device segment copies on the copy stream.
 * MS_COPY_KERNEL (the default): a streaming kernel of a few work-groups that
 * reads the pinned store over PCIe.  MS_COPY_DMA: the DMA engines
 * (hipMemcpyAsync), which leave the compute units and their caches to the
 * kernels that run beside the copy, except while the copy stream waits for
 * unfinished work of another stream (a staging slot's previous reader, a
 * layer's last forward): those copies still run as the kernel, ordered on
 * the GPU (a DMA transfer queued behind such a wait can stall for
 * milliseconds).  Switching to MS_COPY_DMA first makes one 1 MiB DMA
 * transfer into the library's workspace and waits for it (the first DMA
 * transfer of a process is slow); MS_E_NOMEM if its pinned source cannot be
 * allocated.  Results do not depend on the engine. */
typedef enum {
  MS_COPY_KERNEL = 0,
  MS_COPY_DMA = 1
} ms_copy_engine;
ms_status ms_set_copy_engine(ms_ctx* ctx, int32_t engine);

/* Glue between stacked MoE layers (outside the layer; the residual stream
 * of a stack whose layers are MoE only, with a weightless RMSNorm):
 * out[t] = x / sqrt(mean(x^2) + 1e-6) with x = h[t] + y[t] in fp32.
 * h_dev [T][d] in the model dtype, y_dev [T][d] fp32 (an ms_forward output),
 * out_dev [T][d] in the model dtype (bf16 rounded to nearest even); out_dev
 * may equal h_dev.  Device pointers, 16-byte aligned; enqueued on `stream`
 * after the context's previous work there.  MS_E_INVALID for T outside
 * [0, max_tokens] or a NULL/misaligned pointer. */
ms_status ms_residual_norm(ms_ctx* ctx, const void* h_dev, const float* y_dev, int32_t T, void* out_dev,
                           void* stream);

/* Timeline instrumentation.  ms_timeline_begin records an origin event on
 * `stream` and from then on brackets every kernel and copy the library
 * issues with HIP events on the stream it runs on (at most `capacity`
 * records; their events are created here, up front).  ms_timeline_end
 * synchronises, writes up to `cap` records to
 * out[] (in issue order) and their count to n_out, and stops recording. */
ms_status ms_timeline_begin(ms_ctx* ctx, void* stream, int32_t capacity);
ms_status ms_timeline_end(ms_ctx* ctx, ms_interval* out, int32_t cap, int32_t* n_out);

/* ---- the decoder loop around the MoE layer ---------------------------------
 *
 * Sec. 2.1: each layer is an attention module, h = Norm(x + Att(x))
 * (Eq. (1)), then the MoE module (Eq. (2), ms_forward); a head follows the
 * last layer.  The paper defers attention to the designs it cites; these
 * stateless calls implement causal grouped-query attention with rotary
 * position embeddings (Mixtral's convention) so that a whole decoder loop
 * runs on the GPU and the prefetch of Sec. 3.2 overlaps real attention.
 * Every buffer is a caller-owned device pointer (bf16 as raw 16-bit
 * patterns, 16-byte aligned where marked), every call is enqueued on
 * `stream` and returns MS_OK, MS_E_INVALID (bad sizes or pointers; nothing
 * enqueued), MS_E_UNSUPPORTED (shape beyond the kernels) or MS_E_HIP (the
 * launch failed).  Norm between modules is ms_residual_norm. */

/* y[t][o] = sum_i x[t][i] w[o][i] (+ add[t][o] if add is not NULL), fp32
 * accumulation: x [T][n_in] bf16 (16-byte aligned), w [n_out][n_in] bf16
 * (the nn.Linear layout, 16-byte aligned), y and add [T][n_out] fp32 (add
 * may alias y).  n_in a multiple of 8, at most 8192. */
ms_status ms_dense(const void* x, const void* w, int32_t T, int32_t n_in, int32_t n_out, float* y, const float* add,
                   void* stream);

/* Rotary embedding and key/value append for T tokens at positions
 * pos0 .. pos0 + T - 1 (pos0 + T <= max_ctx).  qkv [T][(Hq + 2 Hkv) D] fp32:
 * per token the Hq query heads, then the Hkv key heads, then the Hkv value
 * heads, D wide each (D even, Hq a multiple of Hkv).  Pair (i, i + D/2) of
 * a query or key head turns by p * base^(-2 i / D) (angle in double
 * precision); results are rounded to bf16: q_out [T][Hq][D], keys into
 * k_cache [Hkv][max_ctx][D] and values (not rotated) into v_cache
 * [Hkv][max_ctx][D] at row p. */
ms_status ms_rope_kv(const float* qkv, int32_t T, int32_t Hq, int32_t Hkv, int32_t D, int32_t pos0, double base,
                     void* q_out, void* k_cache, void* v_cache, int32_t max_ctx, void* stream);

/* Causal grouped-query attention: token t (at position pos0 + t) attends to
 * cache rows 0 .. pos0 + t; query head h uses key/value head h / (Hq / Hkv);
 * scores q.k / sqrt(D), softmax with the maximum subtracted, fp32.  q
 * [T][Hq][D] bf16 (from ms_rope_kv), caches as in ms_rope_kv (16-byte
 * aligned), out [T][Hq][D] bf16.  MS_E_UNSUPPORTED unless D is a power
 * of two in [8, 512], Hq / Hkv is 1, 2, 4 or 8 and
 * (Hq / Hkv) (5 D + pos0 + T) <= 16000 (queries, scores and partial sums of
 * a work-group in LDS; Mixtral's 4 x 128 heads: contexts up to 3360). */
ms_status ms_attention(const void* q, const void* k_cache, const void* v_cache, int32_t T, int32_t Hq, int32_t Hkv,
                       int32_t D, int32_t pos0, int32_t max_ctx, void* out, void* stream);

/* Greedy token choice: idx_out[t] = arg max over x[t][0 .. n) (fp32 [T][n]),
 * the lowest index on ties. */
ms_status ms_argmax(const float* x, int32_t T, int32_t n, int32_t* idx_out, void* stream);

/* Embedding gather: out[t] = table[ids[t]] (bf16 rows of d, d a multiple of
 * 8; table and out 16-byte aligned); ids outside [0, n_vocab) are clamped. */
ms_status ms_embed(const int32_t* ids, const void* table, int32_t n_vocab, int32_t T, int32_t d, void* out,
                   void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOESPLIT_H */
