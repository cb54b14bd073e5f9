/*
 * moe.h - C ABI of the mixed-precision MoE layer library for AMD MI355X
 * (gfx950).
 *
 * The library runs one sparse MoE layer (HOBBIT, arXiv 2411.01433):
 *
 *   y = sum_{i<K} G(x)_{e_i} * E_{e_i}(x)                        (Eq. 1)
 *
 * where G is a linear gate followed by top-k and a softmax over the K
 * selected logits (Section 2.1; "normalised" gate values, Section 3.2),
 * and E is a SwiGLU expert  E(x) = W2 (silu(W1 x) * (W3 x)).  Each expert
 * carries a precision tag standing for its state in the expert cache.  A
 * resident expert runs at the precision it is held in; for a cache-miss
 * expert the token-level rule of Section 3.2 (Eq. 2) chooses per token:
 * rank the K gate values in descending order, score s_i = sum of the gate
 * values ranked above slot i (s_0 = 0), then
 *   s <= t1       -> full precision (fp16)
 *   t1 < s <= t2  -> low-precision copy (int4 or int2, from the tag)
 *   s > t2        -> skipped (the term is dropped, no renormalisation)
 * and the top-ranked expert always runs at full precision.
 *
 * Low-precision copies (Section 2.2, Section 4.1 "Configurations") are
 * symmetric, group-wise along the input dimension, group = 32, one fp16
 * scale per group:  s = fp16_rne(max|w| / qmax),  q = clamp(rne(w / s),
 * -2^(b-1), qmax),  qmax = 2^(b-1) - 1;  stored offset-binary u = q + 2^(b-1),
 * element j of a row at bit b*(j mod 8/b) of byte j*b/8.
 *
 * Conventions for every entry point
 *  - Pointers documented "device" are HIP device pointers on the current
 *    device; "host" pointers are ordinary process memory.
 *  - Matrices are row-major.  Expert weights use the [out, in] layout:
 *    W1, W3: [d_ff, d_model]; W2: [d_model, d_ff]; the gate Wg: [E, d_model].
 *  - fp16 = IEEE binary16; fp32 = IEEE binary32.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued asynchronously on it; no entry point synchronises the
 *    host except moe_layer_init, moe_layer_destroy and moe_set_expert_
 *    precision when it has to allocate a low-precision copy.
 *  - Argument errors are detected before any work is enqueued and return
 *    MOE_EINVAL with nothing enqueued.  A failing HIP call returns MOE_EHIP;
 *    a device fault of earlier work surfaces as MOE_EHIP at a later call.
 *  - moe_last_error() returns a thread-local description of the last
 *    failure on the calling thread.
 *  - No C++ exception crosses this interface.
 *  - One handle must not be used from two streams concurrently (it owns a
 *    single workspace, which moe_layer_share_workspace may share with
 *    other handles).
 */
#ifndef MOE_H
#define MOE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct moe_layer* moe_layer_t;

typedef enum {
    MOE_OK = 0,
    MOE_EINVAL = -1,       /* bad argument; nothing was enqueued */
    MOE_ENOMEM = -2,       /* device or host allocation failed */
    MOE_EHIP = -3,         /* a HIP runtime call failed */
    MOE_ESTATE = -4,       /* handle destroyed / not usable */
    MOE_EUNSUPPORTED = -5  /* shape or option outside what the kernels take */
} moe_status;

/* Per-expert precision tag: the expert's state in the expert cache. */
typedef enum {
    MOE_TAG_FP16 = 0,       /* resident at full precision (cache hit) */
    MOE_TAG_INT4 = 1,       /* resident as its int4 copy: always int4 */
    MOE_TAG_INT2 = 2,       /* resident as its int2 copy: always int2 */
    MOE_TAG_MISS_INT4 = 3,  /* cache miss, low copy int4: Eq. 2 rule decides */
    MOE_TAG_MISS_INT2 = 4,  /* cache miss, low copy int2: Eq. 2 rule decides */
    /* int8 models (Section 4.1: int2 copies replace int8 experts): the high
     * copy is the expert's int8 quantisation (same quantiser, b = 8) */
    MOE_TAG_INT8 = 5,           /* resident as its int8 copy: always int8 */
    MOE_TAG_MISS_INT8_INT2 = 6  /* cache miss, int8 high / int2 low copy:
                                   Eq. 2 rule decides */
} moe_tag;

/* Precision class used for one (token, slot), as reported in prec_used. */
enum { MOE_PREC_HIGH = 0, MOE_PREC_LOW = 1, MOE_PREC_SKIP = 2 };

/* Layer shape and rule parameters.
 *  d_model, d_ff  multiples of 64 (two quantisation groups: one 16-byte int2
 *                 load spans 64 weights), d_model <= 16384, d_ff <= 65536
 *  n_experts      1..64;  top_k 1..min(8, n_experts)
 *  group_size     must be 32
 *  max_tokens     largest n_tokens any call will pass (sizes the workspace);
 *                 1..8192
 *  t1, t2         Eq. 2 thresholds (Section 3.2); t2 >= 1 disables skipping
 *  rms_eps        epsilon of the RMSNorm used by the *_residual entry points
 *  flags          reserved, must be 0 */
typedef struct {
    int32_t d_model;
    int32_t d_ff;
    int32_t n_experts;
    int32_t top_k;
    int32_t group_size;
    int32_t max_tokens;
    float t1;
    float t2;
    float rms_eps;
    uint32_t flags;
} moe_layer_desc;

/* Create a layer.  Eq. 1 gating and experts.
 *  w_router  device, fp16 [n_experts, d_model], borrowed
 *  w1, w3    host arrays of n_experts device pointers, fp16 [d_ff, d_model]
 *  w2        host array of n_experts device pointers, fp16 [d_model, d_ff]
 * The fp16 weights are borrowed: they must stay valid and unchanged for the
 * life of the handle.  The pointer arrays themselves are copied.  Every
 * expert starts tagged MOE_TAG_FP16.  Allocates the workspace and the
 * device expert table; synchronises `stream`.  *out receives the handle. */
moe_status moe_layer_init(const moe_layer_desc* desc, const void* w_router,
                          const void* const* w1, const void* const* w3,
                          const void* const* w2, void* stream,
                          moe_layer_t* out);

/* Set an expert's precision tag (Section 3.2 / 3.4: its cache state).  A tag
 * that needs a quantised copy (int4 / int2 low copies; the int8 high copy of
 * MOE_TAG_INT8 and MOE_TAG_MISS_INT8_INT2) builds it from the fp16 weights
 * with the quantiser below the first time (allocating it: library-owned,
 * freed by moe_layer_destroy); the table entry is updated in stream order,
 * so calls enqueued later on `stream` see the new tag. */
moe_status moe_set_expert_precision(moe_layer_t layer, int32_t expert,
                                    int32_t tag, void* stream);

/* One decode step of the layer (Eq. 1 with the Section 3.2 rule), for
 * 1 <= n_tokens <= min(max_tokens, 64) tokens.
 *  x          device, fp16 [n_tokens, d_model] (input hidden states)
 *  y          device, fp32 [n_tokens, d_model] (output, overwritten)
 *  topk_idx   device int32 [n_tokens, top_k] or NULL: selected experts,
 *             slot 0 = largest logit (exact ties: lower index first)
 *  topk_w     device fp32 [n_tokens, top_k] or NULL: normalised gate values
 *  prec_used  device int8 [n_tokens, top_k] or NULL: MOE_PREC_* per slot */
moe_status moe_decode_step(moe_layer_t layer, int32_t n_tokens, const void* x,
                           float* y, int32_t* topk_idx, float* topk_w,
                           int8_t* prec_used, void* stream);

/* Allocation-free variant of moe_decode_step, for callers that cannot
 * allocate device memory around a step: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same kernels and the same
 * results as moe_decode_step; the call allocates nothing (no hipMalloc, no
 * hipFree, no allocating library routine).  Its workspace (work list, pair
 * permutation, routing outputs, SwiGLU activations h and, from 3 tokens on,
 * the per-pair expert outputs) lives in a static device array of 8 MiB that
 * each GPU the library runs on holds until the process ends, instead of the
 * handle's workspace.  A step needs about
 *   n_tokens * top_k * (2 d_ff + (n_tokens >= 3 ? 4 d_model : 0) + 17) + 2 KiB
 * bytes of it (each region rounded up to 256 bytes); a larger step returns
 * MOE_EINVAL with nothing enqueued (a Mixtral-shaped layer, d_model 4096,
 * d_ff 14336, top-2, fits up to 64 tokens).  Every call on one GPU shares that
 * GPU's array, which keeps the last call's contents: calls that overlap on one
 * GPU (other streams, threads or handles) race and must be ordered by the
 * caller.  Nothing in it needs to start at zero (each call writes what it
 * reads).  Arguments as moe_decode_step. */
moe_status moe_decode_step_noalloc(moe_layer_t layer, int32_t n_tokens, const void* x,
                                   float* y, int32_t* topk_idx, float* topk_w,
                                   int8_t* prec_used, void* stream);

/* Decode step with the residual glue used between stacked layers:
 *  h       device fp32 [n_tokens, d_model], in/out: h += MoE(x)
 *  x_next  device fp16 [n_tokens, d_model], out: fp16(rmsnorm(h)) with
 *          rmsnorm(v) = v / sqrt(mean(v^2) + rms_eps) (no gain)
 * Other arguments as moe_decode_step. */
moe_status moe_decode_step_residual(moe_layer_t layer, int32_t n_tokens,
                                    const void* x, float* h, void* x_next,
                                    int32_t* topk_idx, float* topk_w,
                                    int8_t* prec_used, void* stream);

/* Decode step of a stacked layer that takes the residual stream itself
 * (Eq. 1 with the Section 3.2 rule inside the pre-norm residual glue):
 *  h  device fp32 [n_tokens, d_model], in/out: on entry the residual
 *     stream before this layer; the step forms x = fp16(rmsnorm(h)) (as
 *     moe_rmsnorm), then h += MoE(x)
 *  x  device fp16 [n_tokens, d_model], out: that x (the layer's input)
 * A stack of layers is one call per layer on the same h; the results equal
 * moe_rmsnorm followed by moe_decode_step_residual per layer, bit for bit,
 * with one launch fewer per layer (the router forms the norm when the
 * step's activations fit in its LDS: n_tokens * d_model <= 32768 and
 * d_model <= 4096).  Other arguments, limits and errors as
 * moe_decode_step. */
moe_status moe_decode_step_prenorm(moe_layer_t layer, int32_t n_tokens, float* h,
                                   void* x, int32_t* topk_idx, float* topk_w,
                                   int8_t* prec_used, void* stream);

/* Prefill: the same layer for 1 <= n_tokens <= max_tokens tokens, with the
 * experts run as an MFMA grouped GEMM.  Arguments as moe_decode_step. */
moe_status moe_prefill(moe_layer_t layer, int32_t n_tokens, const void* x,
                       float* y, int32_t* topk_idx, float* topk_w,
                       int8_t* prec_used, void* stream);

/* Prefill with the residual glue (see moe_decode_step_residual). */
moe_status moe_prefill_residual(moe_layer_t layer, int32_t n_tokens,
                                const void* x, float* h, void* x_next,
                                int32_t* topk_idx, float* topk_w,
                                int8_t* prec_used, void* stream);

/* The RMSNorm of the residual glue on its own, to form the first layer's
 * input of a stack:  x[t] = fp16(h[t] / sqrt(mean_j h[t,j]^2 + eps)), no gain.
 *  h  device fp32 [n_tokens, d_model];  x  device fp16 [n_tokens, d_model]
 *  n_tokens >= 1; d_model a positive multiple of 64, <= 16384; eps >= 0.
 *  Needs no handle; pointers 16-byte aligned. */
moe_status moe_rmsnorm(const float* h, void* x, int32_t n_tokens, int32_t d_model,
                       float eps, void* stream);

/* Copy an expert's quantised copy out (for inspection and parity).
 *  matrix  0 = W1, 1 = W3, 2 = W2;  bits 8, 4 or 2 (the copy must exist)
 *  codes   device u8 [rows, cols*bits/8];  scales device fp16 [rows, cols/32]
 * where [rows, cols] is the matrix's shape. */
moe_status moe_export_packed(moe_layer_t layer, int32_t expert, int32_t matrix,
                             int32_t bits, void* codes, void* scales,
                             void* stream);

/* Quantise any fp16 matrix with the layer's quantiser (the format above).
 *  w       device fp16 [rows, cols]; cols a multiple of 32
 *  codes   device u8 [rows, cols*bits/8];  scales device fp16 [rows, cols/32]
 *  bits    8, 4 or 2.  Needs no handle. */
moe_status moe_quantize(const void* w, int64_t rows, int64_t cols, int32_t bits,
                        void* codes, void* scales, void* stream);

/* Stage timing, for measurement.  While enabled, every decode / prefill call
 * records HIP events on its stream between its kernels: stage 0 = routing
 * and work list, 1 = expert up-projection with SwiGLU, 2 = expert
 * down-projection with the weighted combine, 3 = the residual RMSNorm of
 * the *_residual entry points (0 otherwise).  moe_layer_stage_times
 * synchronises on the recorded events, returns in ms[0..3] the summed
 * milliseconds per stage and in *n_calls the number of calls since timing
 * was (re-)enabled, and restarts the sums.  Events cost a few microseconds
 * per call: leave timing off outside measurement runs.  enable = 0 turns
 * it off. */
moe_status moe_layer_enable_timing(moe_layer_t layer, int32_t enable);
moe_status moe_layer_stage_times(moe_layer_t layer, double* ms,
                                 int32_t* n_calls);

/* Run `layer` on the per-call workspace of `owner` and free its own.  The
 * workspace (work list, pair permutation and positions, routing buffers,
 * h [max_tokens*top_k, d_ff] fp16 and the per-pair outputs [max_tokens*top_k,
 * d_model] fp32) holds nothing between calls, so the layers of a stack
 * (Eq. 1 applied layer after layer), which run one after another, can all
 * use one: about 46 MB per Mixtral-shaped layer at 512 prefill tokens.
 * The layer keeps its own expert table, copies and tags.
 *  - Both must have equal d_model, d_ff, top_k and max_tokens and live on
 *    the same device (else MOE_EINVAL).  If `owner` itself runs on another
 *    layer's workspace, `layer` joins that one.
 *  - Calls on layers that share a workspace must not overlap: enqueue them
 *    on one stream, or order the streams.  moe_decode_step_noalloc is not
 *    affected (it uses the static scratch).
 *  - Sharing twice with the same workspace is a no-op.  A layer that
 *    already runs on another workspace, or whose workspace others share,
 *    cannot be re-shared (MOE_ESTATE).
 *  - The workspace's owner must be destroyed last: moe_layer_destroy on it
 *    fails with MOE_ESTATE while other layers share it.
 * Synchronises the device (the freed workspace may be in use by earlier
 * work); `stream` orders the copy of the expert table to its new place. */
moe_status moe_layer_share_workspace(moe_layer_t layer, moe_layer_t owner, void* stream);

/* Free the handle, its workspace and its low-precision copies (synchronises
 * the device first).  The borrowed fp16 weights are not touched.  Fails
 * with MOE_ESTATE, freeing nothing, while other layers run on its
 * workspace (moe_layer_share_workspace). */
moe_status moe_layer_destroy(moe_layer_t layer);

/* ---- Expert storage and loading (Dynamic Expert Loader) ---------------
 * Section 3.2 and Fig. 6: expert copies live in host Expert Storage and a
 * cache miss loads the copy of the precision the Eq. 2 rule chose into the
 * GPU expert cache; Section 2.2: an int4 copy moves about a quarter of the
 * fp16 bytes, so it loads about four times faster.  A store keeps one layer's experts in pinned host memory
 * (hipHostMalloc): fp16 W1, W3 [d_ff, d_model], W2 [d_model, d_ff] and
 * their low_bits copy (codes + fp16 group scales, the same quantiser and
 * layout as moe_quantize).  Loads are hipMemcpyAsync transfers on the
 * caller's stream into caller-owned device buffers ("cache slots");
 * moe_layer_bind_expert points a layer's expert at such slots. */
typedef struct moe_store* moe_store_t;

/* d_model, d_ff: positive multiples of 64 (<= 16384 / 65536); n_experts
 * 1..64; low_bits 4 or 2.  Allocates the pinned storage on the current
 * device (MOE_ENOMEM if it cannot). */
moe_status moe_store_create(int32_t d_model, int32_t d_ff, int32_t n_experts,
                            int32_t low_bits, moe_store_t* out);

/* Bytes of one matrix's fp16 weights, low-precision codes and scales (the
 * three matrices of an expert have equal sizes). */
moe_status moe_store_sizes(moe_store_t store, int64_t* fp16_bytes, int64_t* code_bytes,
                           int64_t* scale_bytes);

/* Fill expert `expert` from device fp16 weights (16-byte aligned): copies
 * them to the host and quantises them on the device into the host low
 * copy.  Synchronises `stream`. */
moe_status moe_store_put(moe_store_t store, int32_t expert, const void* w1, const void* w3,
                         const void* w2, void* stream);

/* Asynchronous load on `stream` of expert `expert`'s fp16 matrices
 * (high != 0: dst_w[3], fp16_bytes each) or low copy (dst_q[3] code_bytes,
 * dst_s[3] scale_bytes each) into device buffers.  MOE_ESTATE if the expert
 * was never put. */
moe_status moe_store_load(moe_store_t store, int32_t expert, int32_t high, void* const* dst_w,
                          void* const* dst_q, void* const* dst_s, void* stream);

/* Free the pinned storage (synchronises the device first). */
moe_status moe_store_destroy(moe_store_t store);

/* Point expert `expert` of a layer at caller-owned device copies (borrowed:
 * they must outlive their use), in stream order on `stream`: tag FP16
 * needs w[3] (fp16, layout as moe_layer_init); INT4 / INT2 need q[3], s[3]
 * with low_bits 4 / 2 (layout as moe_quantize); MISS_INT4 / MISS_INT2 need
 * all of them.  The int8-model tags (INT8, MISS_INT8_INT2) are not bindable
 * (MOE_EUNSUPPORTED).  Pointers must be 16-byte aligned.  An expert bound without
 * fp16 weights cannot take moe_set_expert_precision (MOE_ESTATE) until it
 * is bound again; moe_export_packed reports only library-built copies. */
moe_status moe_layer_bind_expert(moe_layer_t layer, int32_t expert, int32_t tag,
                                 const void* const* w, const void* const* q,
                                 const void* const* s, int32_t low_bits, void* stream);

/* ---- Stacking Computer of the Adaptive Expert Predictor ----------------
 * Section 3.3 ("Expert predictor design") and Fig. 7: gating inputs of
 * consecutive layers are similar, so the gates of the next p layers
 * applied to the current layer's gating input predict the experts those
 * layers will select.  The p gates are stacked into one [p*E, d_model]
 * matrix and evaluated as one product; per token and predicted layer j the
 * prediction is that layer's top-k (slot 0 = largest logit, exact ties to
 * the lower index) with the softmax over the K selected logits.  The walk
 * j = 1, 2, ..., p continues while every predicted expert of layer l+j is
 * in the expert cache and stops at the first layer with a missing one: its
 * missing experts are the ones to preload. */
typedef struct moe_predictor* moe_predictor_t;

/* Create a predictor for p = n_ahead layers ahead (1..8).
 *  d_model     multiple of 64, <= 16384;  n_experts 1..64;
 *  top_k       1..min(8, n_experts);  max_tokens 1..8192
 *  w_router_next  host array of n_ahead device pointers, each fp16
 *              [n_experts, d_model] (16-byte aligned): the gates of layers
 *              l+1 .. l+n_ahead.  They are copied ("stacked") into one
 *              library-owned array, so they need not outlive the call.
 * Synchronises `stream`.  *out receives the handle. */
moe_status moe_predictor_init(int32_t d_model, int32_t n_experts, int32_t top_k,
                              int32_t n_ahead, int32_t max_tokens,
                              const void* const* w_router_next, void* stream,
                              moe_predictor_t* out);

/* Predict for 1 <= n_tokens <= max_tokens tokens (one kernel launch).
 *  x           device fp16 [n_tokens, d_model]: the current gating input
 *  cached      device uint64 [n_ahead]: bit e of cached[j-1] set when
 *              expert e of layer l+j is in the expert cache
 *  pred_idx    device int32 [n_tokens, n_ahead, top_k]: predicted experts
 *  pred_w      device fp32 [n_tokens, n_ahead, top_k] or NULL: their
 *              normalised gate values
 *  first_miss  device int32 [1]: the first j in 1..n_ahead with a predicted
 *              expert not cached, 0 if every prediction is cached
 *  preload     device uint64 [1]: bitmask of the predicted experts of
 *              layer l+first_miss that are not cached (0 if none) */
moe_status moe_predict(moe_predictor_t pred, int32_t n_tokens, const void* x,
                       const uint64_t* cached, int32_t* pred_idx, float* pred_w,
                       int32_t* first_miss, uint64_t* preload, void* stream);

/* Free the predictor (synchronises the device first). */
moe_status moe_predictor_destroy(moe_predictor_t pred);

/* ---- Mixed-precision expert cache manager ---------------------------------
 * Section 3.4 ("Cache Manager design", Eq. 3) and "Cache replacement
 * policies".  Host-side bookkeeping that decides which expert copies stay
 * resident; layer_tags() turns its state into the per-expert tags of
 * moe_set_expert_precision.  No GPU work, no HIP calls.
 *
 * Experts are (layer, expert) pairs.  Two caches hold high- and
 * low-precision copies (capacities counted in experts).  Per sequence the
 * manager records for every expert t its last-use time R_t (token number),
 * use count F_t and high-precision use count H_t (low-precision uses do not
 * count in H_t); uses update the records whether they hit or miss.  A use
 * names the copy (high or low) and hits when that copy is resident; on a
 * miss the copy is inserted, and when its cache is full the resident with
 * the lowest priority (Eq. 3)
 *   p_t = w_lru R_t/T + w_lfu F_t/T + w_lhu H_t/T
 *         + w_fld (1 - ((l_t - l_i + n_layers) mod n_layers) / n_layers)
 * is evicted: T is the current token number (the three record terms are 0
 * before the first token), l_i the layer of the incoming copy; ties evict
 * the smaller key layer * n_experts + expert; residents masked by the
 * expert predictor (Section 3.3) are kept unless every resident is masked.
 * A high-precision miss adds miss_cost to the penalty, a low-precision miss
 * miss_cost * bits_lo / bits_hi.
 * One handle is not safe for concurrent use from several threads. */
typedef struct moe_cache* moe_cache_t;

typedef struct {
  int32_t n_layers, n_experts;     /* >= 1 each, product <= 2^24 */
  int32_t hi_capacity, lo_capacity;/* >= 0 (0: that cache holds nothing) */
  double w_lru, w_lfu, w_lhu, w_fld;  /* >= 0, sum 1 (within 1e-6) */
  int32_t bits_hi, bits_lo;        /* 1 <= bits_lo <= bits_hi (e.g. 16 / 4) */
  double miss_cost;                /* C: cost of one high-precision miss, >= 0 */
} moe_cache_desc;

/* Create an empty cache manager; *out receives the handle. */
moe_status moe_cache_create(const moe_cache_desc* desc, moe_cache_t* out);

/* A new sequence: T = 0 and the R, F, H records restart; contents stay. */
moe_status moe_cache_begin_sequence(moe_cache_t cache);

/* The next token: T += 1 (tokens are numbered 1, 2, ... per sequence). */
moe_status moe_cache_begin_token(moe_cache_t cache);

/* One use of expert (layer, expert) through its high (high != 0) or low
 * copy.  *hit (if non-NULL) = 1 when that copy was resident; the evicted
 * expert (or -1, -1) goes to *evicted_layer / *evicted_expert (non-NULL). */
moe_status moe_cache_access(moe_cache_t cache, int32_t layer, int32_t expert, int32_t high,
                            int32_t* hit, int32_t* evicted_layer, int32_t* evicted_expert);

/* *present = 1 when the high (high != 0) or low copy is resident. */
moe_status moe_cache_contains(moe_cache_t cache, int32_t layer, int32_t expert, int32_t high,
                              int32_t* present);

/* Mask (masked != 0) or unmask an expert against eviction (predicted
 * experts, Section 3.3); clear_masks unmasks all. */
moe_status moe_cache_set_mask(moe_cache_t cache, int32_t layer, int32_t expert, int32_t masked);
moe_status moe_cache_clear_masks(moe_cache_t cache);

/* Replay n uses (host arrays of n entries): the token number advances
 * whenever tokens[i] differs from the previous use's, and a new sequence
 * starts before use i when new_sequence (may be NULL) has new_sequence[i]
 * != 0.  hits[i] (may be NULL) = 1 for a hit; evicted[i] (may be NULL) =
 * evicted key layer * n_experts + expert or -1.  All indices are checked
 * before any use is applied. */
moe_status moe_cache_replay(moe_cache_t cache, int64_t n, const int32_t* tokens,
                            const int32_t* layers, const int32_t* experts, const int32_t* highs,
                            const uint8_t* new_sequence, int32_t* hits, int32_t* evicted);

/* Tags of the n_experts experts of one layer (host int32 array) so that the
 * Eq. 2 rule decides per token for the missing ones: bits 16/4 and 16/2
 * give FP16 when the high copy is resident, else MISS_INT4 / MISS_INT2;
 * bits 8/2 (an int8 model) give INT8, else MISS_INT8_INT2; other widths
 * MOE_EUNSUPPORTED. */
moe_status moe_cache_layer_tags(moe_cache_t cache, int32_t layer, int32_t* tags);

/* Accumulated miss penalty and counts since creation (NULL outputs skipped). */
moe_status moe_cache_stats(moe_cache_t cache, double* penalty, int64_t* hi_misses,
                           int64_t* lo_misses, int64_t* hits);

moe_status moe_cache_destroy(moe_cache_t cache);

/* Thread-local text of the last error on this thread ("" if none). */
const char* moe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
