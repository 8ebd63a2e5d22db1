/*
 * dlm.h - C ABI of the MI355X (gfx950) denoising-step library, libdlm.so.
 *
 * One call of dlm_denoise_step is one batched denoising step of a
 * masked-diffusion transformer (paper: "Background and Challenges",
 * Diffusion Language Models): the prompt plus [MASK] tokens pass through a
 * bidirectional-attention Transformer, every masked position of the active
 * block gets a prediction and a confidence (its softmax probability), the
 * positions whose confidence exceeds the request's threshold are unmasked,
 * and when none does the most confident one is unmasked alone. With
 * approximate KV caching ("Support for Approximate Caching"; "Supporting
 * Approximate KV Caching") a step is either a recompute step, which processes
 * every token and rewrites the request's cache, or a cache step, which
 * recomputes only the active block (dual cache) or the active block and the
 * positions after it (prefix cache) and reads every other key/value from the
 * cache written by the last recompute step.
 *
 * Conventions shared by every entry point:
 *  - All device memory is owned by the caller. The library never allocates or
 *    frees device memory and never synchronises a stream; work is enqueued on
 *    the stream passed in (a hipStream_t given as void*; NULL is the default
 *    stream) and results are valid once the caller has synchronised it.
 *  - dlm_model and dlm_cache are opaque host handles that borrow the caller's
 *    device pointers; those must outlive the handles. *_destroy frees host
 *    state only.
 *  - Every argument is validated on the host before anything is enqueued. On
 *    any non-OK status nothing is enqueued and no handle changes state; the
 *    reason is in dlm_last_error() (thread-local, valid until the next call on
 *    the same thread).
 *  - Handles are thread-compatible, not thread-safe: calls that share a handle
 *    must be serialised by the caller.
 *
 * Data types: DLM_BF16 models store weights, normed activations, Q/K/V and the
 * KV cache in bf16 and accumulate in fp32; the residual stream is fp32.
 * DLM_F32 models store everything in fp32. Norm gains are always fp32.
 * Matrices are row-major [out, in] (in contiguous).
 */
#ifndef DLM_H
#define DLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DLM_OK = 0,
  DLM_EINVAL = -1,        /* malformed argument (null pointer, bad shape, bad threshold) */
  DLM_ESIZE = -2,         /* a buffer is too small (workspace, cache buffer, limits)     */
  DLM_EHIP = -3,          /* a HIP runtime call failed; its message is in last_error    */
  DLM_ESTATE = -4,        /* cache step on a slot whose cache is not current             */
  DLM_EUNSUPPORTED = -5   /* configuration outside what the kernels implement           */
} dlm_status;

typedef enum { DLM_F32 = 0, DLM_BF16 = 1 } dlm_dtype;

typedef enum {
  DLM_CACHE_NONE = 0,     /* every step recomputes the whole sequence (exact)          */
  DLM_CACHE_PREFIX = 1,   /* cache steps recompute [block_start, seq_len)               */
  DLM_CACHE_DUAL = 2      /* cache steps recompute [block_start, block_start+block_len) */
} dlm_cache_mode;

enum {
  DLM_MAX_BLOCK = 64,     /* largest block length (one 64-lane wavefront per request) */
  DLM_MAX_REQ = 64,       /* largest number of requests in one step                     */
  DLM_MAX_SEQ = 8192,     /* largest sequence length                                    */
  DLM_NSTATS = 8,         /* confidence statistics per request (dlm_step_out.stats)    */
  DLM_SCRATCH_BYTES = 134217728 /* scratch of dlm_denoise_step_noalloc (128 MiB per GPU)  */
};

/* Request flag: this step is a recompute step (whole sequence, cache rewritten). */
#define DLM_REQ_REFRESH 1

/* Model shape. Supported: head_dim 64 or 128, d_model a multiple of 64, d_ffn a
 * multiple of 16,
 * n_q_heads a multiple of n_kv_heads, mask_id in [0, vocab). inv_tau scales the
 * logits before the softmax (1/temperature). */
typedef struct dlm_config {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab, mask_id;
  float rms_eps, rope_theta, inv_tau;
  int32_t dtype;          /* dlm_dtype */
} dlm_config;

/* Per-layer weights (device pointers). */
typedef struct dlm_layer_weights {
  const float* attn_norm; /* [d_model] fp32                                               */
  const void* w_qkv;      /* [(n_q_heads + 2 n_kv_heads) head_dim, d_model]: Q rows, then K, then V */
  const void* w_o;        /* [d_model, n_q_heads head_dim]                                 */
  const float* ffn_norm;  /* [d_model] fp32                                               */
  const void* w_gate_up;  /* [2 d_ffn, d_model]: gate rows, then up rows                   */
  const void* w_down;     /* [d_model, d_ffn]                                              */
} dlm_layer_weights;

typedef struct dlm_weights {
  const void* embed;      /* [vocab, d_model]                                              */
  const void* lm_head;    /* [vocab, d_model] (untied)                                     */
  const float* final_norm;/* [d_model] fp32                                               */
  const dlm_layer_weights* layers; /* host array of n_layers entries, copied by load     */
} dlm_weights;

/* One request of a batched step (host struct). Positions are 0-based within the
 * request; position j of request r lives at tokens[tok_offset + j]. The ranges
 * [tok_offset, tok_offset + seq_len) of the requests of one batch must not
 * overlap (DLM_EINVAL otherwise). */
typedef struct dlm_req {
  int32_t slot;           /* cache slot, unique within a batch                          */
  int32_t seq_len;        /* prompt + generation length                                  */
  int32_t prompt_len;     /* positions [0, prompt_len) are the prompt                    */
  int32_t block_start;    /* first position of the active block (>= prompt_len)          */
  int32_t block_len;      /* 1..DLM_MAX_BLOCK, block_start + block_len <= seq_len         */
  int32_t tok_offset;     /* offset of position 0 in the packed tokens/mask arrays       */
  int32_t flags;          /* DLM_REQ_REFRESH or 0                                        */
} dlm_req;

typedef struct dlm_batch {
  int32_t n_req;          /* 1..DLM_MAX_REQ                                              */
  const dlm_req* reqs;    /* host array [n_req]                                          */
  int32_t* tokens;        /* device, packed token ids; updated in place                  */
  uint8_t* mask;          /* device, packed, 1 = [MASK]; updated in place                */
  int32_t mode;           /* dlm_cache_mode                                              */
  float* tok_conf;        /* optional device, packed like tokens: the confidence with which
                             each position was unmasked. The step writes it for every
                             position it unmasks; positions the caller unmasks itself hold
                             what the caller wrote. Required when dlm_step_out.stats is set. */
} dlm_batch;

/* Step outputs (device). Request r's entries start at r * DLM_MAX_BLOCK. */
typedef struct dlm_step_out {
  int32_t* n_unmasked;    /* [n_req] number of positions unmasked this step              */
  int32_t* pos;           /* [n_req * DLM_MAX_BLOCK] unmasked positions, ascending        */
  int32_t* tok;           /* [n_req * DLM_MAX_BLOCK] their new tokens                     */
  float* conf;            /* [n_req * DLM_MAX_BLOCK] their confidences                    */
  float* block_conf;      /* optional [n_req * DLM_MAX_BLOCK]: confidence of every block
                             position masked at step start (index = pos - block_start),
                             -1 for positions that were already unmasked                  */
  int32_t* block_tok;     /* optional, same layout: prediction of each masked position   */
  float* stats;           /* optional [n_req * DLM_NSTATS], after this step's unmasking:
                             the Step Predictor's confidence features (paper, "Step
                             Prediction" and the appendix "Step Predictor Features") over
                             the request's output tokens, i.e. the unmasked positions of
                             [prompt_len, seq_len), each valued at batch.tok_conf:
                             [0] count n, [1] min, [2] lower quartile, [3] median, [4] mean,
                             [5] upper quartile, [6] max, [7] unmasked positions of the
                             active block. Quartiles and median interpolate linearly
                             between order statistics (p-quantile of the ascending v:
                             v[j] + (h - j)(v[j+1] - v[j]), h = (n-1)p, j = floor(h)).
                             With n = 0, [1..6] are 0. fp32; the mean is a fixed-order sum. */
} dlm_step_out;

typedef struct dlm_model dlm_model;
typedef struct dlm_cache dlm_cache;

/* Validate the configuration and record the caller's weight pointers. */
dlm_status dlm_load_weights(const dlm_config* cfg, const dlm_weights* w, dlm_model** out);
void dlm_model_destroy(dlm_model* m);

/* Workspace bytes for steps of at most max_rows recomputed rows (sum over
 * requests of the rows each step recomputes) and max_reqs requests. */
dlm_status dlm_workspace_bytes(const dlm_model* m, int32_t max_rows, int32_t max_reqs,
                               size_t* out_bytes);

/* KV cache (paper: "Support for Approximate Caching"; "Supporting Approximate
 * KV Caching", where the caches are kept in GPU memory and rebuilt by the
 * recompute steps; "Implementation"). Carve n_slots fixed KV slots of
 * max_seq_len positions out of the caller's buffer: the post-RoPE keys and
 * values of every layer, per layer a key region [slot][kv_head][pos][head_dim]
 * and a transposed value region [slot][kv_head][head_dim][pos], slots rounded
 * up to 64 positions. A request's output length is known when it arrives
 * ("Request Scheduling"), so slots are fixed-size and never paged. With
 * dev_buf == NULL only *required_bytes is written (out may then be NULL).
 * The buffer must be 256-byte aligned and hold *required_bytes (DLM_ESIZE
 * otherwise); it stays the caller's. Every slot starts invalid: its first
 * step must be a recompute step. */
dlm_status dlm_kv_cache_alloc(const dlm_model* m, int32_t n_slots, int32_t max_seq_len,
                              void* dev_buf, size_t buf_bytes, size_t* required_bytes,
                              dlm_cache** out);
void dlm_cache_destroy(dlm_cache* c);
/* Mark a slot stale (its next step must be a recompute step). */
dlm_status dlm_cache_invalidate(dlm_cache* c, int32_t slot);

/* One batched denoising step (paper: "Background and Challenges", Diffusion
 * Language Models, for the forward, the confidence and the threshold rule;
 * "SLO-aware Confidence Threshold Adjustment" for per-request thresholds; "Supporting
 * Approximate KV Caching" for recompute and cache steps). thresholds: host
 * [n_req], each in [0, 1] (DLM_EINVAL otherwise, or for a NaN).
 * Requests flagged DLM_REQ_REFRESH (all requests when mode is DLM_CACHE_NONE)
 * recompute every position and rewrite their slot; the others recompute the
 * rows their mode names and need a slot refreshed at the same block_start
 * and seq_len (else DLM_ESTATE). Masked positions of the active block get a
 * prediction, the vocabulary argmax (lowest id on ties) of the logits scaled
 * by inv_tau, and a confidence, its softmax probability; those with
 * confidence > threshold are unmasked (tokens[] and mask[] updated in place);
 * if none passes, the most confident one (lowest position on ties) is
 * unmasked. Outputs and the token/mask updates are device writes, valid once
 * the stream is synchronised. The workspace (256-byte aligned,
 * dlm_workspace_bytes for at least this step's rows and requests) is
 * scratch, overwritten by the step. */
dlm_status dlm_denoise_step(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                            const float* thresholds, const dlm_step_out* out,
                            void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the step of
 * dlm_denoise_step with no workspace argument. Its scratch is a fixed array
 * of DLM_SCRATCH_BYTES (128 MiB) built into the library, one per GPU the
 * library runs on, held until the process ends; the first call on a device
 * looks up that device's copy. A step whose workspace (dlm_workspace_bytes
 * for its rows and requests) exceeds DLM_SCRATCH_BYTES is rejected with
 * DLM_ESIZE before anything is enqueued (for example the 512-row step of a
 * 4096-wide, 32-layer bf16 model fits, a 1024-row step does not). The call
 * allocates nothing: no hipMalloc, no hipFree, no allocating library routine.
 * Every call on one GPU shares that GPU's array, which keeps the previous
 * call's contents (the step needs nothing in it to start at zero); calls that
 * overlap on one GPU (different streams, or threads without ordering between
 * them) race on it and must be serialised by the caller. Kernel timing
 * (dlm_profile_enable) does not apply to this entry point. Arguments,
 * outputs, cache rules and errors are those of dlm_denoise_step. */
dlm_status dlm_denoise_step_noalloc(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                                    const float* thresholds, const dlm_step_out* out,
                                    void* stream);

/* Recompute step without unmasking (paper: "Implementation", the caches are
 * rebuilt during recompute steps; "Request Scheduling", a request migrates or
 * resumes only at a recompute step): recompute every position of every
 * request of the batch with the batch's current tokens and mask and rewrite
 * their slots, marking each slot current for its block_start and seq_len.
 * Nothing is unmasked and no step output is written; the thresholds are not
 * needed. Used for prefill, for resuming a migrated or evicted request, or for
 * rebuilding a slot. Same validation, workspace and stream rules as
 * dlm_denoise_step. */
dlm_status dlm_cache_refresh(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                             void* workspace, size_t ws_bytes, void* stream);

/* Test hook: run the forward of a step (same rows and cache writes as
 * dlm_denoise_step, nothing unmasked) and write the scaled logits z = logits *
 * inv_tau of every active-block position: rows in request order, positions
 * ascending, logits_out [sum block_len, vocab] fp32 (device). */
dlm_status dlm_debug_logits(dlm_model* m, dlm_cache* c, const dlm_batch* b,
                            float* logits_out, void* workspace, size_t ws_bytes,
                            void* stream);

/* Test hook: the intermediate values of one layer of a step's forward (the
 * pre-norm layer of "Background and Challenges", Diffusion Language Models:
 * norm, QKV projection, rotary positions and the key/value write, full
 * bidirectional attention over the slot, output projection and residual,
 * norm, SwiGLU feed-forward and residual), copied device to device out of the
 * workspace as the step's own kernels produce them, so that every kernel can
 * be checked on the exact inputs it was given. The forward is the one of
 * dlm_denoise_step (same rows, plans and cache writes; nothing is unmasked).
 * N is the number of recomputed rows of the step, packed in request order,
 * positions ascending (a request's rows are [0, seq_len) on a recompute step,
 * [block_start, block_start + block_len) on a dual-cache step and
 * [block_start, seq_len) on a prefix-cache step). Every buffer is a device
 * pointer and optional (NULL records nothing); "model dtype" buffers hold the
 * storage type (bf16 or fp32), the others fp32:
 *   h_in   [N, d_model]       residual stream entering the layer
 *   a_attn [N, d_model]       attention-norm output (model dtype)
 *   qkv    [qkv_cap, N, (n_q_heads + 2 n_kv_heads) head_dim] fp32 output of
 *                             the QKV GEMM as K-split slices: slice s holds the
 *                             sum over the s-th of qkv_splits equal K ranges;
 *                             the consumer adds slices 0, 1, ... in order
 *   q      [N, n_q_heads head_dim]  queries after the rotary embedding (model dtype)
 *   attn_out [N, n_q_heads head_dim] attention output (model dtype)
 *   h_mid  [N, d_model]       residual stream after the output projection
 *   a_ffn  [N, d_model]       feed-forward-norm output (model dtype)
 *   act    [N, d_ffn]         silu(gate) * up (model dtype)
 *   h_out  [N, d_model]       residual stream after the down projection
 *   u      [sum block_len, d_model] final-normed rows of every active-block
 *                             position (model dtype); needs logits
 *   logits [sum block_len, vocab] scaled logits, as dlm_debug_logits
 * The keys and values of the layer are in the cache. qkv_splits (out) is the
 * number of slices the step's QKV GEMM wrote; DLM_ESIZE (nothing enqueued)
 * when qkv is given and qkv_cap is smaller. */
typedef struct dlm_trace {
  int32_t layer;          /* in [0, n_layers)                                           */
  int32_t qkv_cap;        /* slices the qkv buffer holds                                 */
  float* h_in;
  void* a_attn;
  float* qkv;
  void* q;
  void* attn_out;
  float* h_mid;
  void* a_ffn;
  void* act;
  float* h_out;
  void* u;
  float* logits;
  int32_t qkv_splits;     /* out */
} dlm_trace;
dlm_status dlm_debug_trace(dlm_model* m, dlm_cache* c, const dlm_batch* b, dlm_trace* trace,
                           void* workspace, size_t ws_bytes, void* stream);

/* The fused LM head alone: for each of m_rows final-normed hidden rows
 * (device, [m_rows, d_model] in the model dtype), conf[i] = max softmax(z_i) and
 * tok[i] = lowest argmax z_i, z_i = (u_i W_lm^T) * inv_tau. The logits are not
 * stored. Needs dlm_workspace_bytes(m, m_rows, 1) of workspace. */
dlm_status dlm_head_confidence(dlm_model* m, const void* u_rows, int32_t m_rows,
                               float* conf, int32_t* tok, void* workspace,
                               size_t ws_bytes, void* stream);

/* Test hooks for the bf16 GEMM kernel (the contraction of every projection of
 * the step: QKV, output, gate/up and down). dlm_debug_gemm_info: the output
 * tile (bm x bn) of tile configuration cfg and, in *subs, the sub-tile splits
 * it allows for a launch's last round (bit 1: halves, bit 2: quarters) and
 * bit 8 when it has no SwiGLU epilogue (its wave tiles hold an odd number of
 * column fragments); DLM_EINVAL for an unknown configuration. dlm_debug_gemm: one launch of configuration cfg,
 * a [M, K] and b [N, K] bf16, row-major and K-contiguous (device), computing
 * p[m][n] = sum_k a[m][k] b[n][k] in fp32 with the epilogue
 *   0: c [splits, M, N] fp32, slice z = the sum over k in
 *      [z K / splits, (z + 1) K / splits) (the whole p when splits is 1);
 *   1: c [M, N/2] bf16 = silu(g) * u with g = p[:, f], u = p[:, N/2 + f]
 *      (rows [0, N/2) of b are the gate weights, [N/2, N) the up weights);
 *   2: c [M, N] fp32 += p;
 * the last n_tail tiles of the launch's tile order run as `sub` (2 or 4)
 * sub-tiles (sub 0: whole tiles only); group_m > 0 selects the grouped
 * XCD-aware tile order. DLM_EINVAL (nothing enqueued) for NULL buffers,
 * non-positive sizes, K not a multiple of 64, splits below 1, above 1 with
 * epilogue 1 or 2, or not dividing the K/64 k-tiles, with epilogue 1 an N/2
 * that is not a multiple of 16 (of 32 for configurations with 32x32 MFMA
 * tiles) or a configuration without it, an unknown configuration or
 * epilogue, or a sub-tile split the configuration does not allow or with
 * n_tail beyond the tile count. */
dlm_status dlm_debug_gemm_info(int32_t cfg, int32_t* bm, int32_t* bn, int32_t* subs);
dlm_status dlm_debug_gemm(int32_t cfg, int32_t epilogue, int32_t sub, int32_t n_tail,
                          int32_t group_m, int32_t splits, const void* a, const void* b, void* c,
                          int32_t M, int32_t N, int32_t K, void* stream);

/* Kernel timing. While enabled, every kernel the library enqueues for this
 * model (or, when only_class is not NULL, every kernel of that class; see also
 * dlm_profile_sample) is timed by a pair of HIP events carried in the kernel's
 * own dispatch (start and end of the kernel; no extra commands on the
 * stream). dlm_profile_read waits for those events, adds their elapsed times
 * per kernel class into out[0 .. *n_out) (at most cap entries, in first-seen
 * order) and clears them. A class that enqueues several kernels has its first
 * one timed. The profiler state is per model and not thread-safe. */
typedef struct dlm_profile_entry {
  char name[32];          /* kernel class, e.g. "gemm_gate_up_swiglu"                  */
  int32_t calls;          /* launches timed                                             */
  double total_ms;        /* sum of their event-to-event times                          */
  int32_t launches;       /* launches of the class since the last read, timed or not    */
} dlm_profile_entry;
dlm_status dlm_profile_enable(dlm_model* m, int32_t on, const char* only_class);
dlm_status dlm_profile_read(dlm_model* m, dlm_profile_entry* out, int32_t cap, int32_t* n_out);
/* Time only the launches 0, every, 2 every, ... of each selected class (counted
 * from the last dlm_profile_enable or dlm_profile_sample call); 1 (the
 * default) times all. With every coprime to the layer count the timed
 * launches rotate through the layers at about one event pair per step.
 * DLM_EINVAL when every < 1. */
dlm_status dlm_profile_sample(dlm_model* m, int32_t every);

/* Measured ceilings (benchmark support, not part of the method). */
/* dlm_ceiling_mfma: n_blocks blocks of 4 waves, each wave running iters x 32
 * v_mfma_f32_16x16x32_bf16 over 8 independent accumulators; writes one float per wave to out
 * (device, [4 n_blocks]) and the FLOPs executed to *flop_out (host, may be
 * NULL). The caller times it on the stream. DLM_EINVAL for non-positive
 * sizes or a NULL out. */
dlm_status dlm_ceiling_mfma(int32_t n_blocks, int32_t iters, float* out, double* flop_out,
                            void* stream);
/* dlm_ceiling_copy: dst[0 .. bytes) = src[0 .. bytes) on the device with
 * 16-byte vector loads and stores (bytes moved through HBM: 2 x bytes).
 * Both pointers 16-byte aligned, bytes a multiple of 16, else DLM_EINVAL. */
dlm_status dlm_ceiling_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Message for the last non-OK status on this thread ("" if none). */
const char* dlm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DLM_H */
