/*
 * wino.h - C ABI of the MI355X (gfx950) WINO decoding library.
 *
 * WINO ("Wide-In, Narrow-Out") is the revokable decoding rule for masked
 * diffusion language models of arXiv 2605.16941.  One decoding step is one
 * bidirectional transformer forward over the extended sequence
 *     [Y_left, Y_cur, Y_right, Y_shad]                      (Sec. 4.2.2)
 * followed by the draft rule (Eq. 2: unmask masked positions of Y_cur whose
 * top probability exceeds tau1) and the verify rule (Eq. 3: re-mask unmasked
 * positions whose probability, read from the shadow block at the current
 * token, is below tau2), both taken from the same forward (Eq. 4).  Blocks of
 * the response are decoded left to right (semi-autoregressive, Sec. 3).
 *
 * Conventions for every entry point
 * ---------------------------------
 * - Pointers named d_* are HIP device memory owned by the caller; h_* are host
 *   memory owned by the caller.  The library never frees caller memory.
 * - bf16 tensors are raw IEEE bfloat16 bit patterns (uint16), row-major.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Entry
 *   points that only enqueue work are asynchronous with respect to the host.
 * - No entry point aborts or prints.  Arguments are validated on the host
 *   before any GPU work is enqueued; failures return a negative wino_status
 *   and leave outputs untouched.  HIP runtime failures return WINO_ERR_HIP;
 *   the text is available from wino_last_error(ctx), and for a failed
 *   wino_create (no context) from wino_last_error(NULL) on the same thread.
 * - A context is not thread-safe; calls that overlap on one context race.
 * - Device pointers must come from the HIP runtime the library is loaded
 *   against.  A process with two copies of the runtime (the system's and one
 *   bundled with a framework) must load the framework first, so that the
 *   library's runtime dependency resolves to the framework's copy.
 *
 * Readings of points the paper leaves open (all documented with the flags):
 * greedy argmax decoding; the draft's max/argmax exclude the mask id (which
 * stays in the softmax normaliser); argmax ties go to the lowest id; strict
 * comparisons (> tau1, < tau2); forced draft of the most confident masked
 * position when none clears tau1 (Eq. 1); a per-block step cap whose last step
 * skips verification and fills every remaining mask; a block whose Y_cur
 * holds no mask is complete and receives no further steps.
 */
#ifndef WINO_H
#define WINO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WINO_OK = 0,
  WINO_ERR_INVALID_ARG = -1, /* null pointer, non-finite threshold, bad id    */
  WINO_ERR_SHAPE = -2,       /* shapes inconsistent or beyond the context     */
  WINO_ERR_HIP = -3,         /* a HIP runtime call failed                     */
  WINO_ERR_NO_MEMORY = -4,   /* workspace allocation failed                   */
  WINO_ERR_STEP_CAP = -5,    /* a block hit its step cap with cap fill off    */
  WINO_ERR_UNSUPPORTED = -6  /* shape (or fp16 weight) it has no kernels for  */
} wino_status;

typedef struct wino_ctx wino_ctx;

/* Activation types (wino_model_config.act_precision). */
#define WINO_ACT_BF16 0 /* bf16 activations, the weights as given (default)   */
#define WINO_ACT_FP16 1 /* fp16 activations and fp16 copies of the matrices   */

/* Backbone shape.  Requirements: d_model == n_heads*head_dim; head_dim is 64
 * or 128; d_model and d_ff are multiples of 64; vocab is a multiple of 256.
 * act_precision: the 16-bit type of the activations the matrix cores read
 * (normed rows, q/k/v, attention probabilities and output, the SwiGLU
 * product), accumulation being fp32 and the residual stream fp32 either way.
 * WINO_ACT_FP16 keeps three more mantissa bits, so the decision probabilities
 * move several times less from exact arithmetic (for callers whose
 * confidences sit near a threshold), at the cost of fp16 copies of every
 * weight matrix (2 bytes per parameter of the QKV, O, gate/up, down and LM
 * head matrices, allocated by wino_create beside the workspace) and of fp16
 * matrix-core throughput; weights and activations must stay within fp16's
 * range (|x| < 65504; weights of magnitude below 2^-17 move by at most
 * 2^-25 in the copy).  Zero-initialised configurations get WINO_ACT_BF16. */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ff, vocab;
  float rope_theta; /* rotate-half RoPE base                         */
  float rms_eps;    /* RMSNorm epsilon                               */
  int32_t act_precision; /* WINO_ACT_BF16 or WINO_ACT_FP16           */
} wino_model_config;

/* Weights, all bf16 device memory, row-major, one row per output feature.
 * Per-layer members are HOST arrays of n_layers device pointers; the context
 * copies the arrays, not the tensors, and the tensors must outlive it. */
typedef struct {
  const void* tok_emb;               /* [V, d]                                 */
  const void* const* attn_norm;      /* [d]      RMSNorm gain before attention */
  const void* const* w_qkv;          /* [3d, d]  rows: q (d) | k (d) | v (d)   */
  const void* const* w_o;            /* [d, d]                                  */
  const void* const* ffn_norm;       /* [d]      RMSNorm gain before the FFN   */
  const void* const* w_gate_up;      /* [2F, d]  rows: gate (F) | up (F)       */
  const void* const* w_down;         /* [d, F]                                  */
  const void* final_norm;            /* [d]                                     */
  const void* lm_head;               /* [V, d]                                  */
  const float* lm_bias;              /* fp32 [V] added to the logits, or NULL   */
} wino_weights;

/* Flags of wino_params.flags. */
#define WINO_FLAG_NO_FORCE_TOP1 0x1u /* no forced draft when nothing clears tau1 */
#define WINO_FLAG_NO_CAP_FILL 0x2u   /* the step cap ends the block unfilled     */

/* One decoding problem (Sec. 3 and Sec. 4.2): batch of independent sequences,
 * each prompt_len prompt ids followed by gen_len response ids, decoded in
 * blocks of block_len; mask_id is the [MASK] token; tau1 drafts (Eq. 2), tau2
 * verifies (Eq. 3).  tau1 >= tau2 is accepted (tau2 = 0 disables verification,
 * the paper's only-draft ablation).  max_steps caps the steps one block may
 * take (0 = block_len); on the last allowed step verification is skipped and
 * every remaining mask is drafted, unless WINO_FLAG_NO_CAP_FILL is set.
 * tokens_per_step > 0 selects the baseline decoders instead (Sec. 3): each
 * step unmasks the tokens_per_step most confident masks of Y_cur (equal
 * confidences: lower position first) - Eq. 1 greedy decoding for 1, naive
 * parallel sampling above - with no threshold, no verification and no shadow
 * block; a block then takes ceil(block_len / tokens_per_step) steps and
 * tau1, tau2, max_steps and the flags are ignored. */
typedef struct {
  int32_t batch, prompt_len, gen_len, block_len, mask_id;
  float tau1, tau2;
  int32_t max_steps;
  uint32_t flags;
  int32_t tokens_per_step;
} wino_params;

/* Per block position diagnostics of one step. */
typedef struct {
  float m_all;    /* max logit of the row the decision read                   */
  float sumexp;   /* sum over all ids of exp(z - m_all)                       */
  float z_best;   /* max logit over ids != mask_id                            */
  float z_target; /* logit of the current token (verify rows), else -inf      */
  int32_t argmax; /* lowest id reaching z_best                                */
  int32_t row_kind; /* 0 current row (draft), 1 shadow row (verify), -1 idle,
                       2 unmasked position not verified: the step ran without
                       the shadow block (tau2 <= 0, see wino_step)            */
} wino_row_stats;

/* Decision flags written per block position (uint8). */
#define WINO_KEEP 0
#define WINO_DRAFT 1
#define WINO_REMASK 2
#define WINO_FORCED 3
#define WINO_CAPFILL 4

/* Create a context for `cfg` with the given weights.  The context owns a
 * device workspace sized for up to max_batch sequences of up to max_seq =
 * prompt_len + gen_len + block_len extended rows (the current device at the
 * time of the call), and with WINO_ACT_FP16 the fp16 copies of the weight
 * matrices.  Returns WINO_ERR_NO_MEMORY if they cannot be allocated, and
 * with WINO_ACT_FP16 WINO_ERR_UNSUPPORTED if a weight matrix holds a value
 * with no finite fp16 copy (|w| > 65504, or not finite). */
wino_status wino_create(const wino_model_config* cfg, const wino_weights* w,
                        int32_t max_batch, int32_t max_seq, wino_ctx** out);
wino_status wino_destroy(wino_ctx* ctx);
/* Workspace bytes wino_create would allocate (without the fp16 weight copies
 * of WINO_ACT_FP16: 2 bytes per parameter of the weight matrices). */
size_t wino_workspace_bytes(const wino_model_config* cfg, int32_t max_batch, int32_t max_seq);

/* One WINO step (Eq. 4) for every sequence of the batch.
 *   d_tokens      int32 [batch, prompt_len+gen_len], updated in place
 *   d_block_start int32 [batch] generation-relative start of Y_cur, a multiple
 *                 of block_len; a sequence with block_start >= gen_len is done
 *   d_block_steps int32 [batch] steps already taken in the current block; in/out
 *   d_flags       uint8 [batch, block_len] decision per position, or NULL
 *   d_n_masked    int32 [batch] masks left in Y_cur after the step, or NULL
 *   d_stats       wino_row_stats [batch, block_len], or NULL
 * Sequences that are done or whose Y_cur holds no mask are left unchanged
 * (flags 0, n_masked 0).  With tau2 <= 0 no position can be re-masked (Eq. 3
 * compares a probability), so the step runs without the shadow block; the
 * decode loops below also drop it for steps in which every active sequence's
 * Y_cur is all masks (Sec. 4.2.2: the other rows never see the shadow block,
 * so the result is the same).  Asynchronous on `stream`. */
wino_status wino_step(wino_ctx* ctx, const wino_params* p, int32_t* d_tokens,
                      const int32_t* d_block_start, int32_t* d_block_steps, uint8_t* d_flags,
                      int32_t* d_n_masked, wino_row_stats* d_stats, void* stream);

/* Iterate wino_step on the current block of every sequence until none holds a
 * mask (Sec. 4.2.3); if none holds one at the start, no forward runs.
 * d_final_step int32 [batch, gen_len] (device, or NULL) is written as in
 * wino_decode.  h_steps [batch] receives the steps each sequence took.
 * Synchronises `stream` once per step. */
wino_status wino_decode_block(wino_ctx* ctx, const wino_params* p, int32_t* d_tokens,
                              const int32_t* d_block_start, int32_t* d_final_step,
                              int32_t* h_steps, void* stream);

/* Full semi-autoregressive decode (Sec. 3): every sequence advances to its
 * next block as soon as its current block holds no mask (Sec. 4.2.3); a block
 * that already holds no mask when the sequence reaches it (filled by the
 * caller, or by an earlier call) is skipped without a forward.  Returns when
 * every sequence reaches gen_len, or after max_forwards batched forwards.
 *
 * Resumable: the decode state is exactly (d_tokens, d_block_start,
 * d_block_steps).  d_block_start int32 [batch] (in/out) is each sequence's
 * current block, a multiple of block_len; gen_len means done.
 * d_block_steps int32 [batch] (device, in/out, or NULL) holds the steps
 * already taken in that block, which count toward the step cap; NULL starts
 * every block count at 0.  max_forwards > 0 stops after that many batched
 * forwards with WINO_OK, leaving a state from which a later call continues
 * exactly as the uninterrupted decode would (0 = no limit).
 *
 * d_final_step int32 [batch, gen_len] (device, or NULL) receives, for every
 * response position this call changes, the sequence's step (1-based, counted
 * from this call) at which the position last changed: from an all-mask
 * response that is the finalization step t_l of Sec. 5.1; positions never
 * changed keep the caller's values.  h_steps_per_seq [batch] (or NULL)
 * receives the steps each sequence took in this call; h_forward_passes (or
 * NULL) the number of batched forwards.  Synchronises once per step.
 * WINO_ERR_STEP_CAP: a block reached its cap with WINO_FLAG_NO_CAP_FILL set;
 * the state is left at that step. */
wino_status wino_decode(wino_ctx* ctx, const wino_params* p, int32_t* d_tokens,
                        int32_t* d_block_start, int32_t* d_block_steps, int32_t* d_final_step,
                        int32_t max_forwards, int32_t* h_steps_per_seq, int32_t* h_forward_passes,
                        void* stream);

/* Per response position quantities of a WINO+ training state (Sec. 5.2-5.3). */
typedef struct {
  float entropy;  /* H(p) = -sum_v p(v) log p(v), p = softmax of the row's logits */
  float nll;      /* -log p(target)                                             */
  float conf;     /* greedy confidence: max p over ids != mask_id               */
  int32_t argmax; /* greedy prediction: lowest id reaching conf                 */
} wino_row_loss;

/* The forward half of the WINO+ objective (Sec. 5.3, Eq. 6-7): for each
 * sequence, a plain bidirectional forward over the training state d_tokens
 * int32 [batch, prompt_len+gen_len] (no shadow block; block_len and the
 * thresholds are not used), then for every response position j the entropy
 * of its prediction, the negative log-likelihood of d_targets[b, j] (int32
 * [batch, gen_len], ids in [0, vocab)) and its greedy prediction, fused into
 * the LM head (no logits in memory).  d_out: wino_row_loss [batch, gen_len].
 * Asynchronous on `stream`. */
wino_status wino_row_losses(wino_ctx* ctx, const wino_params* p, const int32_t* d_tokens,
                            const int32_t* d_targets, wino_row_loss* d_out, void* stream);

/* Standalone decision from given bf16 logits (the fused step's epilogue on
 * materialised logits).  d_logits: bf16 [batch, 2*block_len, vocab]; rows
 * 0..block_len-1 are Y_cur, rows block_len..2*block_len-1 Y_shad.
 * d_cur_tokens int32 [batch, block_len] is updated in place by Eq. 4 (forced
 * draft per the flags; no step cap), or by the baseline rule when
 * p->tokens_per_step > 0 (shadow rows unused).  d_mask_bitmap uint8 [batch, block_len]
 * receives 1 where the token is the mask after the step.  d_flags / d_stats
 * may be NULL.  d_workspace must hold wino_epilogue_workspace_bytes(...). */
size_t wino_epilogue_workspace_bytes(int32_t batch, int32_t block_len, int32_t vocab);
wino_status wino_epilogue(const wino_params* p, int32_t vocab, const void* d_logits,
                          int32_t* d_cur_tokens, uint8_t* d_mask_bitmap, uint8_t* d_flags,
                          wino_row_stats* d_stats, void* d_workspace, size_t workspace_bytes,
                          void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * wino_epilogue without a workspace argument.  Same arguments, kernels and
 * results as wino_epilogue; its partial statistics live in a library-owned
 * device array of WINO_EPILOGUE_NOALLOC_MAX_BYTES on each GPU it runs on
 * (held until the process ends), so a call allocates and frees nothing.
 * WINO_ERR_SHAPE if wino_epilogue_workspace_bytes(batch, block_len, vocab)
 * exceeds that size (e.g. 2 MiB holds 6552 block positions at vocab
 * 126464).  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (different streams or threads) race.  Nothing in the
 * array needs to start at zero. */
#define WINO_EPILOGUE_NOALLOC_MAX_BYTES (2u << 20)
wino_status wino_epilogue_noalloc(const wino_params* p, int32_t vocab, const void* d_logits,
                                  int32_t* d_cur_tokens, uint8_t* d_mask_bitmap, uint8_t* d_flags,
                                  wino_row_stats* d_stats, void* stream);

/* Test entry points (same kernels, unfused outputs).
 * wino_debug_logits: fp32 logits [batch, 2*block_len, vocab] of the current
 *   block rows (0..Lb-1) and shadow rows (Lb..2Lb-1) for the given state.
 * wino_debug_forward: residual stream fp32 [batch, T, d] (T = prompt_len +
 *   gen_len + block_len) after the embedding and the first n_sublayers
 *   sublayers; each layer is two sublayers, attention then FFN, so
 *   n_sublayers = 2*n_layers is the full backbone before the final norm. */
wino_status wino_debug_logits(wino_ctx* ctx, const wino_params* p, const int32_t* d_tokens,
                              const int32_t* d_block_start, float* d_logits, void* stream);
wino_status wino_debug_forward(wino_ctx* ctx, const wino_params* p, const int32_t* d_tokens,
                               const int32_t* d_block_start, int32_t n_sublayers, float* d_out,
                               void* stream);

/* wino_debug_gemm: out fp32 [M, N] = A W^T for bf16 A [M, K] and W [N, K]
 *   (row-major, contiguous), the backbone GEMM kernel with a plain store.
 *   K must be a multiple of 64 and N of the tile width (128); otherwise
 *   WINO_ERR_UNSUPPORTED.  Asynchronous on `stream`. */
wino_status wino_debug_gemm(const void* d_A, const void* d_W, int32_t M, int32_t N, int32_t K,
                            float* d_out, void* stream);

/* Kernel timing with HIP events on the launch stream.  enable != 0 records a
 * pair of events around every launch of the kernel classes in `class_mask`
 * (bit i = class i, see wino_kernel_class_name).  wino_profile_read
 * synchronises, then reports per class: launches, total milliseconds and the
 * algorithmic flops and HBM bytes those launches represent; it resets the
 * counters.  Arrays have WINO_N_KERNEL_CLASSES entries. */
#define WINO_N_KERNEL_CLASSES 13
wino_status wino_profile(wino_ctx* ctx, uint32_t class_mask);
wino_status wino_profile_read(wino_ctx* ctx, int64_t* h_launches, double* h_ms,
                              double* h_flops, double* h_bytes);
const char* wino_kernel_class_name(int32_t cls);

const char* wino_status_string(wino_status s);
const char* wino_last_error(const wino_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* WINO_H */
