/*
 * dvi.h — C ABI of the MI355X (gfx950) engine for the self-speculative decode
 * step of "Draft, Verify & Improve" (DVI, arXiv 2510.05421).
 *
 * One decoder-only transformer is split at layer k (Section 3.1): layers 1..k
 * plus a LoRA draft head propose tokens (the draft path), layers k+1..L plus
 * the frozen head verify them (the target path).  A decode step is
 *
 *     dvi_draft -> dvi_verify -> dvi_commit   [-> dvi_update_drafter]
 *
 * following Section 3.3 (rollout, verification, longest agreeing prefix,
 * replay logging) and Section 3.4 (drafter objective).
 *
 * Conventions for every entry point
 *  - Device pointers are HIP device memory (any allocator; PyTorch tensors in
 *    the Python binding).  Host pointers are ordinary host memory.  Each
 *    argument below says which.
 *  - Matrices are row-major [out_features][in_features]; bf16 arrays hold
 *    IEEE bfloat16 bit patterns, fp32 arrays IEEE float.
 *  - All work is enqueued on the stream given to dvi_create.  Calls that return
 *    host data synchronise that stream before returning.  On a stream other
 *    than the null stream, the kernels of each draft and verify call are
 *    captured once into a HIP graph per shape (batch, k_spec, variant,
 *    attention grid bucket) and replayed (see dvi_set_graphs).
 *  - Errors: a negative dvi_status; dvi_last_error() describes the last one.
 *    DVI_ERR_ARG, DVI_ERR_STATE and DVI_ERR_CAPACITY are detected on the host
 *    before anything is launched and leave the context unchanged.
 *    DVI_ERR_DEVICE (a HIP runtime failure) is sticky: destroy the context.
 *    DVI_ERR_NUMERIC means a NaN/Inf reached a vocabulary head; the step can
 *    be abandoned with dvi_abort_step.
 *  - Nothing crosses the ABI as a C++ exception.
 *
 * Memory ownership
 *  - The caller owns the weights, the LoRA tensors and one workspace of
 *    dvi_workspace_bytes() bytes; all must outlive the context.  dvi_create
 *    copies the frozen weights into the workspace in the engine's internal
 *    layout, so the caller's frozen-weight buffers may be released after
 *    dvi_create returns.  The LoRA tensors are read at every draft and updated
 *    in place by dvi_update_drafter.
 *  - The context itself (host memory) owns only bookkeeping.
 */
#ifndef DVI_H
#define DVI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dvi_ctx dvi_ctx;

typedef enum {
    DVI_OK = 0,
    DVI_ERR_ARG = -1,       /* an argument is out of range or inconsistent            */
    DVI_ERR_STATE = -2,     /* call out of order (see the state machine below)         */
    DVI_ERR_CAPACITY = -3,  /* a length, batch or k_spec exceeds the configured maximum */
    DVI_ERR_DEVICE = -4,    /* HIP runtime failure (sticky)                             */
    DVI_ERR_NUMERIC = -5    /* NaN or Inf in a head's logits                            */
} dvi_status;

typedef enum { DVI_FP32 = 0, DVI_BF16 = 1 } dvi_dtype;

/*
 * Model and capacity.  Section 3.1: layers indexed 1..L, split index k with
 * 0 < k < L (k == L is accepted only as a test relaxation).  The backbone is a
 * pre-norm decoder block: RMSNorm, rotary position embedding (rotate-half,
 * base rope_theta), grouped-query attention (n_heads divisible by n_kv_heads),
 * SwiGLU MLP, no biases.  Both heads read RMSNorm(h; final_norm).
 */
typedef struct {
    int32_t n_layers;      /* L                                                   */
    int32_t split_k;       /* k: draft = layers 1..k, verify = layers k+1..L      */
    int32_t d_model;       /* multiple of 32, at most 8192                        */
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t head_dim;      /* 64 or 128                                           */
    int32_t ffn_dim;       /* multiple of 32                                      */
    int32_t vocab;         /* multiple of 16                                      */
    float rms_eps;
    float rope_theta;
    int32_t max_batch;     /* sequences decoded together                         */
    int32_t max_seq;       /* prompt + generated + k_spec positions per sequence  */
    int32_t max_k_spec;    /* 1..16                                               */
    int32_t lora_rank;     /* r of A_s [V, r], B_s [r, d]; 1..64                  */
    float lora_gamma;      /* gamma_s                                             */
    int32_t buffer_rows;   /* replay ring capacity (rows), >= 1                   */
    dvi_dtype dtype;       /* weight / KV storage type                            */
} dvi_config;

/*
 * Frozen weights (DEVICE pointers, dtype of the config) and LoRA factors
 * (DEVICE fp32).  Per-layer arguments are HOST arrays of n_layers DEVICE
 * pointers.  W^(S) of the draft head is W^(V) (lm_head): one tensor.
 */
typedef struct {
    const void *tok_emb;                 /* [V, d]                     */
    const void *const *attn_norm;        /* n_layers x [d]             */
    const void *const *wq;               /* n_layers x [H*hd, d]       */
    const void *const *wk;               /* n_layers x [Hkv*hd, d]     */
    const void *const *wv;               /* n_layers x [Hkv*hd, d]     */
    const void *const *wo;               /* n_layers x [d, H*hd]       */
    const void *const *mlp_norm;         /* n_layers x [d]             */
    const void *const *w_gate;           /* n_layers x [F, d]          */
    const void *const *w_up;             /* n_layers x [F, d]          */
    const void *const *w_down;           /* n_layers x [d, F]          */
    const void *final_norm;              /* [d]                        */
    const void *lm_head;                 /* [V, d]   W^(V) == W^(S)    */
    float *lora_A;                       /* [V, r]   A_s, fp32         */
    float *lora_B;                       /* [r, d]   B_s, fp32         */
} dvi_weights;

/* Bytes of device workspace dvi_create needs for this configuration. */
size_t dvi_workspace_bytes(const dvi_config *cfg);

/*
 * Validate cfg, lay out the workspace (DEVICE, at least dvi_workspace_bytes,
 * 256-byte aligned) and copy the frozen weights into it.  hip_stream is a
 * hipStream_t (NULL: the default stream).  On success *out is a new context in
 * state CREATED.
 */
dvi_status dvi_create(const dvi_config *cfg, const dvi_weights *w, void *workspace, size_t ws_bytes,
                      void *hip_stream, dvi_ctx **out);

/* Release the context (host bookkeeping only; the caller frees device memory). */
void dvi_destroy(dvi_ctx *ctx);

/*
 * Prefill (Section 3.3: the shallow state is computed once from the prefix):
 * run all L layers over each sequence's prompt, fill the KV cache, and emit
 * each sequence's first token x_P = argmax p_phi(. | h_{L,P-1}).  ids: HOST
 * int32 [batch, stride], sequence b's prompt in ids[b*stride .. b*stride+lens[b]);
 * lens: HOST int32 [batch], each 1 <= lens[b] <= stride and lens[b] + 1 <= max_seq
 * (prompts may differ in length; DVI_ERR_ARG / DVI_ERR_CAPACITY otherwise);
 * first_tok: HOST int32 [batch] (out).  The first token is committed and
 * becomes each sequence's pending token, and sequence b's cache length is
 * lens[b].  Allowed in any state except DRAFTED/VERIFIED; resets all
 * sequences.  -> READY
 */
dvi_status dvi_prefill(dvi_ctx *ctx, int32_t batch, const int32_t *ids, const int32_t *lens, int32_t stride,
                       int32_t *first_tok);

/*
 * Draft (Section 3.3): k_spec serial single-token passes of layers 1..k from
 * each pending token, each followed by the LoRA draft head
 * p_theta = softmax((W^(S) + gamma A_s B_s) RMSNorm(h_k)) and its argmax
 * (ties -> lowest id), writing layer 1..k keys/values at positions
 * len..len+k_spec-1 and keeping the k_spec states h_k for the verify.
 * forced: NULL or HOST int32 [batch, k_spec] replacing the argmax (test hook).
 * drafts_out: NULL or HOST int32 [batch, k_spec].  k_spec == 1 with forced ==
 * NULL is plain autoregressive decoding: the draft head is skipped, drafts read
 * -1, every step commits the verifier's token and nothing is logged (the
 * baseline the method's speedup is measured against).  READY -> DRAFTED
 */
dvi_status dvi_draft(dvi_ctx *ctx, int32_t k_spec, const int32_t *forced, int32_t *drafts_out);

/*
 * Verify (Section 3.3): one block pass of layers k+1..L over the k_spec kept
 * states of every sequence (row i at position len+i attends to keys 0..len+i,
 * i.e. block-causal), then the frozen head and argmax y*_{t+i+1}.  The
 * verifier logits stay on the device for logging.  targets_out: NULL or HOST
 * int32 [batch, k_spec]; accept_out: NULL or HOST int32 [batch], the longest
 * agreeing prefix m.  DRAFTED -> VERIFIED
 */
dvi_status dvi_verify(dvi_ctx *ctx, int32_t *targets_out, int32_t *accept_out);

/*
 * dvi_verify for callers that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  Same semantics, arguments and results as
 * dvi_verify (bit for bit), but its device scratch (attention partials and merge counters, the
 * head's argmax partials) lives in a static array of the library, one 16 MiB copy per device that
 * the library holds until the process ends, instead of in the workspace; its kernels are launched
 * directly (no graph instantiation), and it calls no hipMalloc/hipFree.  Every context on a device
 * shares that device's array and the array keeps the last call's contents (the counters are
 * cleared by a kernel at the start of each call): calls that overlap on one device race.
 * DVI_ERR_CAPACITY, before anything is launched, when the step needs more scratch than the array
 * holds (batch*k_spec * n_heads * 64-key chunks of the longest sequence * (head_dim + 2) * 4 bytes
 * of attention partials, plus batch*k_spec * vocab/2 bytes); DVI_ERR_DEVICE if the array's address
 * could not be resolved on this device.  DRAFTED -> VERIFIED
 */
dvi_status dvi_verify_static(dvi_ctx *ctx, int32_t *targets_out, int32_t *accept_out);

/*
 * Commit (Section 3.3): per sequence m = longest agreeing prefix,
 * n = min(m+1, k_spec, max_new[b]) tokens y*_{t+1..t+n} are committed, the
 * cache length advances by n (keys/values beyond it are stale and are
 * overwritten later: that is the whole rollback), the last committed token
 * becomes pending, and replay tuples are logged for positions
 * i = 1..min(m+1, k_spec) with r = 1 for i <= m and r = 0 for i = m+1.
 * max_new: NULL (no limit) or HOST int32 [batch] tokens still wanted
 * (0 freezes a finished sequence).  forced_commit: NULL, or HOST int32
 * [batch, k_spec] replacing y* for the commit (test hook that breaks
 * losslessness on purpose, to follow another trajectory).  tokens_out: HOST
 * int32 [batch, k_spec] (entries past n are -1); n_out: HOST int32 [batch];
 * accept_out: NULL or HOST int32 [batch] receiving m.  VERIFIED -> READY
 */
dvi_status dvi_commit(dvi_ctx *ctx, const int32_t *max_new, const int32_t *forced_commit, int32_t *tokens_out,
                      int32_t *n_out, int32_t *accept_out);

/*
 * Several decode steps in one call (Section 3.3, the draft -> verify -> commit -> log loop):
 * n_steps (1..64) steps of dvi_draft + dvi_verify + dvi_commit with k_spec drafts each,
 * queued on the stream without a host synchronisation between them; each sequence's
 * remaining-token count lives on the device and the commit kernel lowers it, so a sequence
 * that reaches its max_new commits nothing further (its lanes keep computing).  Results are
 * those of n_steps separate calls, bit for bit.  max_new: NULL (no limit) or HOST int32
 * [batch].  tokens_out: HOST int32 [n_steps, batch, k_spec] (entries past n are -1); n_out:
 * HOST int32 [n_steps, batch]; accept_out: NULL or HOST int32 [n_steps, batch] receiving m.
 * No drafter update runs inside; callers that train the drafter call dvi_update_drafter
 * between calls.  The capacity check is made up front on the longest length the steps could
 * reach (each sequence grows by at most min(k_spec per step, max_new)): DVI_ERR_CAPACITY
 * if any could pass max_seq.  DVI_ERR_NUMERIC if a head produced a non-finite logit: nothing
 * is committed from that step on, the earlier steps stand, and the context is READY.
 * READY -> READY
 */
dvi_status dvi_decode_steps(dvi_ctx *ctx, int32_t k_spec, int32_t n_steps, const int32_t *max_new,
                            int32_t *tokens_out, int32_t *n_out, int32_t *accept_out);

/* Return to the last committed state from DRAFTED or VERIFIED (length reset only). */
dvi_status dvi_abort_step(dvi_ctx *ctx);

/*
 * Drafter update (Section 3.4) over all valid replay rows, with coefficients
 * already resolved by the caller's KL->RL schedule:
 *   loss = sum_i [ c_kl/n KL(p_i || q_i) - beta_i log p_i(a_i) - c_ent/n H(p_i) ]
 *   beta_i = c_ce r_i / max(n_acc,1) + c_pg (r_i - baseline) fresh_i / max(n_fresh,1)
 *   p_i = softmax(W^(S) h_i + gamma A_s B_s h_i), q_i = softmax(logits^phi_i / tau)
 * Gradients flow to A_s and B_s only; an Adam step (lr, beta1, beta2, eps,
 * step number opt_step >= 1) updates them in place unless lr == 0.  Fresh flags
 * are cleared afterwards.  grad_A_out / grad_B_out: NULL or DEVICE fp32
 * [V, r] / [r, d] receiving the gradients.  stats: NULL or HOST (out).
 * Allowed in READY.
 */
typedef struct {
    float c_kl, c_ce, c_pg, c_ent;
    float tau, baseline;
    float lr, beta1, beta2, eps;
    int32_t opt_step;
    float *grad_A_out;
    float *grad_B_out;
} dvi_update_args;

typedef struct {
    float loss, kl, ce, pg, entropy;   /* total loss and the per-term means            */
    int32_t rows, accepted, fresh;     /* valid rows, rows with r = 1, fresh rows        */
    int32_t fresh_accepted;            /* fresh rows with r = 1 (for the reward EMA)     */
} dvi_update_stats;

dvi_status dvi_update_drafter(dvi_ctx *ctx, const dvi_update_args *args, dvi_update_stats *stats);

/* Message for the last error on this context (static storage; never NULL). */
const char *dvi_last_error(const dvi_ctx *ctx);

/* ---- inspection and test hooks (synchronous; HOST outputs) -------------------------- */

/* Keys/values of one layer (0-based) and sequence at positions [pos0, pos0+npos):
 * HOST buffers [n_kv_heads, npos, head_dim] in the storage dtype. */
dvi_status dvi_read_kv(dvi_ctx *ctx, int32_t layer, int32_t seq, int32_t pos0, int32_t npos, void *k, void *v);

/* Verifier logits of the last verify: HOST fp32 [batch, k_spec, V]; right after a
 * prefill, the head logits behind each sequence's first token: [batch, 1, V]. */
dvi_status dvi_read_logits(dvi_ctx *ctx, float *out);

/* Draft-head logits of the last drafted position: HOST fp32 [batch, V]. */
dvi_status dvi_read_draft_logits(dvi_ctx *ctx, float *out);

/* Committed cache length per sequence: HOST int32 [batch]. */
dvi_status dvi_read_lengths(dvi_ctx *ctx, int32_t *len);

/* Number of valid rows in the replay ring and the ring's next write index. */
dvi_status dvi_buffer_info(dvi_ctx *ctx, int32_t *valid_rows, int32_t *next_row);

/* Replay rows [row0, row0+nrows): h HOST fp32 [nrows, d] (the stored RMSNorm(h_k)),
 * a / i / prev int32 [nrows], logits fp32 [nrows, V], r / fresh int8 [nrows].
 * Any output may be NULL. */
dvi_status dvi_read_buffer(dvi_ctx *ctx, int32_t row0, int32_t nrows, float *h, int32_t *a, float *logits,
                           int8_t *r, int8_t *fresh, int32_t *i, int32_t *prev);

/* Replace the replay ring's contents with nrows HOST rows (h fp32 [nrows, d],
 * rounded to the storage dtype; a int32; logits fp32 [nrows, V]; r, fresh int8).
 * Test hook for update parity on a synthetic buffer.  Allowed in READY. */
dvi_status dvi_write_buffer(dvi_ctx *ctx, int32_t nrows, const float *h, const int32_t *a, const float *logits,
                            const int8_t *r, const int8_t *fresh);

/*
 * Per-kernel timing probe (measurement only).  While a probe is set, every launch of
 * that kernel class is bracketed by hipEvents on the context's stream and its
 * algorithmic bytes (weights streamed once, activations in and out, keys/values read
 * and written) are added up.  which: 0 = off, then one of DVI_PROBE_*.  Setting a probe
 * clears its counters.  dvi_probe_read synchronises and returns the summed event time,
 * the launch count and the summed algorithmic bytes; at most 8192 launches are timed.
 */
enum {
    DVI_PROBE_OFF = 0, DVI_PROBE_QKV = 1, DVI_PROBE_ATTN_OUT = 2, DVI_PROBE_GATE_UP = 3,
    DVI_PROBE_DOWN = 4, DVI_PROBE_HEAD = 5, DVI_PROBE_ATTENTION = 6
};
dvi_status dvi_probe_kernel(dvi_ctx *ctx, int32_t which);
dvi_status dvi_probe_read(dvi_ctx *ctx, double *total_ms, int64_t *launches, double *bytes);

/*
 * Sampled drafting (Section 3.3 writes the draft as a sample t~ ~ p_theta; the default, tau = 0,
 * takes the argmax).  With tau > 0 every draft of dvi_draft is drawn from softmax(z / tau), z
 * the draft-head logits, by Gumbel-max: t~ = argmax_v z_v / tau - log(-log(u_v)).  u comes from
 * Philox4x64-10 (Salmon et al., SC 2011) with key (seed, 0) and counter (v / 4, b * 16 + j,
 * step, 0): word v % 4 of the block, b the sequence, j the draft index, step the decode steps
 * committed since the last dvi_prefill; u = (2 * (x >> 41) + 1) / 2^24.  Commits stay
 * exactly those of greedy decoding: only the drafts, and so the accept lengths, change.
 * dvi_read_draft_logits still returns z.  Errors: DVI_ERR_ARG for tau < 0 or not finite;
 * DVI_ERR_STATE during a step.  Drops the cached graphs.
 */
dvi_status dvi_set_sampling(dvi_ctx *ctx, float tau, uint64_t seed);

/*
 * Graph replay of the decode passes (DVI's step structure, Section 3.3: a draft of
 * k_spec shallow passes and one block verify).  enable = 1 (the default on a
 * non-null stream): dvi_draft and dvi_verify launch one captured HIP graph per
 * call, keyed by (batch, k_spec, variant, attention grid bucket); sequence lengths
 * are read on the device, so a graph stays valid as they grow, and a pass is
 * captured again only when the longest sequence enters a new 256-position bucket.
 * Results are bitwise the same as with enable = 0 (every kernel launched
 * directly).  Disabling frees the cached graphs.  Errors: DVI_ERR_ARG when
 * enabling on the null stream (which cannot be captured).  While a timing probe
 * is set, launches are direct.
 */
dvi_status dvi_set_graphs(dvi_ctx *ctx, int32_t enable);

/*
 * Streaming-read reference (measurement only): reads the caller's DEVICE buffer buf[0, bytes)
 * reps times with the same non-temporal 16-byte loads the decode GEMMs stream their weights
 * with, each pass timed by HIP events stamped at the kernel's own start and end, and returns the
 * fastest pass's rate in *gb_s (1e9 bytes per second): the practical HBM read ceiling the step's
 * kernels are compared against, beside the nominal peak.  bytes: at least 1 MiB, a multiple of
 * 16; the buffer must exceed the last-level cache for an HBM figure.  Runs on the context's
 * stream and synchronises it.  DVI_ERR_ARG on bad arguments.
 */
dvi_status dvi_measure_read_rate(dvi_ctx *ctx, const void *buf, size_t bytes, int32_t reps, double *gb_s);

/* Per-phase device time of the last call of each kind (ms, hipEvent based). */
dvi_status dvi_get_timings(dvi_ctx *ctx, double *ms_draft, double *ms_verify, double *ms_commit, double *ms_update);

#ifdef __cplusplus
}
#endif
#endif /* DVI_H */
