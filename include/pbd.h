/*
 * pbd.h -- C ABI of the PEFT-BD speculative-step library for AMD MI355X (gfx950).
 *
 * One speculative step of PEFT-BD (Sec. 3, enumerated algorithm):
 *   1-2. pbd_draft_block   -- adapter-enabled block-diffusion draft pass: the block
 *                             [anchor, mask x D] at positions t..t+D attends to the
 *                             committed prefix KV and bidirectionally inside the
 *                             block; proposes D tokens in one denoising step.
 *   3.   pbd_verify_block  -- adapter-disabled causal verify pass over
 *                             [anchor, x_1..x_D]; writes its K/V at t..t+D.
 *   4-5. pbd_accept_commit -- greedy longest-prefix acceptance (App. A.1: exact
 *                             greedy top-1 matching) and KV commit/rollback.
 * The adapter is LoRA on every linear projection of every block (App. A.2); both
 * passes have width W = D + 1 ("token width 17", Tab. profile; App. A.4).
 *
 * Conventions for every entry point:
 *  - Pointers named "device" are HIP device pointers; the library never allocates
 *    device memory.  The caller allocates the packed-weight, KV-cache and workspace
 *    buffers with the sizes the *_bytes functions return, keeps them alive while
 *    the context lives, and owns them.  The library allocates only the host-side
 *    context, freed by pbd_destroy.
 *  - Calls are asynchronous and ordered on `stream` (a hipStream_t; NULL = the
 *    legacy default stream).  Per-sequence state (seq_len, anchor) is device
 *    resident, so a step needs no host synchronisation and can be captured in a
 *    HIP graph.  A context serves one stream at a time (not thread-safe).
 *  - Return value: PBD_OK (0) or a negative PBD_ERR_*.  Errors the host can
 *    detect are reported before anything is enqueued, leaving device state
 *    untouched.  Errors only the device can detect (capacity overflow, token id
 *    out of range, forced count out of range) set bits of a sticky device status
 *    word and skip that sequence's writes; pbd_sync_status reads and clears it.
 *    pbd_last_error gives a message for the last failed call.
 *  - Token ids are int32.  Batch sequences are independent (data parallel).
 */
#ifndef PBD_H
#define PBD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pbd_ctx pbd_ctx;
typedef void* pbd_stream_t;            /* hipStream_t */

/* status codes */
#define PBD_OK               0
#define PBD_ERR_INVALID_ARG (-1)       /* null pointer, bad flag combination, bad value */
#define PBD_ERR_SHAPE       (-2)       /* shape not supported by the kernels */
#define PBD_ERR_CAPACITY    (-3)       /* batch > max_batch, buffer too small, length > max_seq */
#define PBD_ERR_STATE       (-4)       /* context not usable */
#define PBD_ERR_HIP         (-5)       /* a HIP runtime call failed */
#define PBD_ERR_UNSUPPORTED (-6)

/* data types of weights, KV cache and GEMM/attention inputs */
#define PBD_DTYPE_F32  0
#define PBD_DTYPE_BF16 1

/* pass flags: each pair may be left unset (the pass's default) but not both set */
#define PBD_PASS_DEFAULT      0u
#define PBD_PASS_ADAPTER_ON   1u       /* draft default */
#define PBD_PASS_ADAPTER_OFF  2u       /* verify default */
#define PBD_PASS_MASK_BLOCK   4u       /* draft default: bidirectional inside the block */
#define PBD_PASS_MASK_CAUSAL  8u       /* verify default */

/* precision of the activation operands fed to the bf16 matrix cores */
#define PBD_OPERANDS_BF16    0         /* rounded to bf16: refused for bf16 models (see pbd_set_operand_precision) */
#define PBD_OPERANDS_BF16X2  1         /* bf16 value plus bf16 residual: two MFMAs per weight
                                          fragment, ~16-bit operand mantissa (default for bf16) */

/* kernel classes timed by the profiling aid */
#define PBD_KCLASS_GEMM     0          /* layer projection GEMMs (q/k/v, o, gate/up, down) */
#define PBD_KCLASS_LMHEAD   1          /* tied LM head with fused argmax */
#define PBD_KCLASS_ATTN     2          /* split-KV attention */
#define PBD_KCLASS_COMBINE  3          /* split merge + O-projection operand */
#define PBD_KCLASS_NORM     4          /* unused: RMSNorm and the LoRA shrink are fused into the GEMMs */
#define PBD_KCLASS_OTHER    5          /* block assembly, final argmax */
#define PBD_KCLASS_FUSED    6          /* persistent batch-1 layer stack (all layers of a pass in one launch) */
#define PBD_KCLASS_COUNT    7

/* bits of the device status word */
#define PBD_STATUS_CAPACITY  1         /* seq_len + W > max_seq, or prompt length out of range */
#define PBD_STATUS_TOKEN     2         /* a token id outside [0, vocab) */
#define PBD_STATUS_FORCED_N  4         /* forced accepted count outside [0, D] */
#define PBD_STATUS_TIMEOUT   8         /* a bounded wait of the persistent batch-1 pass gave up:
                                          that pass's outputs are invalid */

/*
 * Model and capacity description.  The backbone is a Qwen3-style decoder
 * (RMSNorm, per-head QK RMSNorm before rotate-half RoPE, grouped-query attention,
 * SwiGLU MLP, tied embedding/LM head, no biases); the paper evaluates
 * Qwen3-0.6B (Sec. 4.1) and does not print the architecture.
 * Supported: head_dim 64 or 128; n_q_heads a multiple of n_kv_heads;
 * hidden, ffn, n_q_heads*head_dim multiples of 64; vocab a multiple of 16;
 * 0 <= block <= 32 (block = 0: width-1 passes, so that pbd_verify_block over
 * [anchor] followed by pbd_accept_commit is one plain autoregressive greedy
 * step, the baseline speculation is measured against; the unanchored verify
 * then fails with PBD_ERR_SHAPE); lora_rank in [0, 64] and a multiple of 8;
 * mask_id in [0, vocab).
 */
typedef struct pbd_config {
    int32_t n_layers;
    int32_t hidden;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn;
    int32_t vocab;
    int32_t lora_rank;      /* r */
    float   lora_alpha;     /* scale s = alpha / r (App. A.2: r = 16, alpha = 32) */
    int32_t block;          /* D, masked positions per draft (Sec. 3: D = 16); 0: autoregressive steps */
    int32_t mask_id;        /* token id of the diffusion mask */
    float   rms_eps;
    float   rope_theta;
    int32_t qk_norm;        /* 1: per-head RMSNorm of q and k before RoPE */
    int32_t dtype;          /* PBD_DTYPE_F32 or PBD_DTYPE_BF16 */
    int32_t max_batch;      /* sequences per call */
    int32_t max_seq;        /* KV capacity per sequence (positions) */
    int32_t prefill_chunk;  /* prompt rows per sequence per prefill pass: 0 (= D + 1) or
                               in [1, 1024]; max_batch * max(D + 1, prefill_chunk) <= 4096.
                               The workspace grows with it. */
} pbd_config;

/*
 * Canonical weights, all device pointers of element type `dtype`, row-major
 * [out_features][in_features] for matrices (y = W x).  LoRA (App. A.2):
 * lora_a[i] is A [r][in], lora_b[i] is B [out][r], for i in order
 * q, k, v, o, gate, up, down; y = W x + (alpha/r) B (A x) when the adapter is on.
 */
typedef struct pbd_layer_weights {
    const void *attn_norm, *q, *k, *v, *o, *q_norm, *k_norm, *mlp_norm, *gate, *up, *down;
    const void *lora_a[7];
    const void *lora_b[7];
} pbd_layer_weights;

typedef struct pbd_weights {
    const void* embed;                  /* [vocab][hidden]; also the LM head (tied) */
    const void* final_norm;             /* [hidden] */
    const pbd_layer_weights* layers;    /* HOST array of n_layers entries */
} pbd_weights;

/*
 * Buffer sizes in bytes for a configuration; 0 if the configuration is invalid.
 * All three are sized for cfg->max_batch sequences of cfg->max_seq positions:
 * the workspace serves every batch up to max_batch (a call's batch argument
 * selects how much of it a pass uses), so no per-batch size query is needed.
 * When the model qualifies for the persistent batch-1 pass (see
 * pbd_set_pass_mode), the packed weights also hold an fp16 copy of every
 * layer's projection and LoRA A fragments, which that pass streams.  A bf16
 * model whose max_batch * (block + 1) is at least 128 (draft and verify
 * passes on the large-M GEMM) also gets those copies and an fp16 copy of the
 * embedding fragments (the tied LM head), read by those passes; its
 * workspace also holds the LoRA shrink's K slices (up to eight).
 */
size_t pbd_packed_weight_bytes(const pbd_config* cfg);
size_t pbd_kv_bytes(const pbd_config* cfg);
size_t pbd_workspace_bytes(const pbd_config* cfg);

/*
 * Validate `cfg`, repack the canonical weights into `packed` (layouts chosen by
 * the library for streaming), build the RoPE table, and create a context that
 * uses `packed`, `kv` and `ws`.  The canonical weights may be freed once
 * `stream` has completed.  *out receives the context (NULL on failure).
 */
int pbd_init_weights(const pbd_config* cfg, const pbd_weights* canon,
                     void* packed, size_t packed_bytes,
                     void* kv, size_t kv_bytes,
                     void* ws, size_t ws_bytes,
                     pbd_stream_t stream, pbd_ctx** out);

/*
 * Prefill (Sec. 3: the step is stated for a given committed context x_1..x_t;
 * this call builds that context's KV cache).  Adapter-off causal pass over
 * each prompt (the committed prefix the speculative steps start from).  tokens: device int32 [batch][max_len] (row b holds
 * lengths[b] ids, the rest ignored); lengths: device int32 [batch], each in
 * [1, max_len] and with lengths[b] + D + 1 <= max_seq.  Writes the prompt K/V to
 * the cache, seq_len[b] = lengths[b] and anchor[b] = greedy next token (device
 * int32 [batch] each), which is the first generated token.
 * The prompt runs in chunks of cfg.prefill_chunk rows per sequence (D + 1 if
 * 0): per chunk, the projections run as one GEMM over batch * chunk rows, the
 * chunk's K/V are appended to the cache first, and attention reads every key
 * from the cache with a causal mask inside the chunk.
 */
int pbd_prefill(pbd_ctx* ctx, int32_t batch, const int32_t* tokens, const int32_t* lengths,
                int32_t max_len, int32_t* seq_len, int32_t* anchor, pbd_stream_t stream);

/*
 * Draft pass (Sec. 3 steps 1-2; App. A.4): block [anchor, mask x D] at positions
 * seq_len..seq_len+D; by default adapter on and bidirectional block mask.
 * seq_len, anchor: device int32 [batch] (read).  draft: device int32 [batch][D]
 * receives argmax over token ids != mask_id of block rows 1..D (ties: lowest id).
 * logits: NULL or device float [batch][D+1][vocab] receiving all rows' logits.
 * The KV cache is not written (the block K/V is scratch in the workspace).
 */
int pbd_draft_block(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                    uint32_t flags, int32_t* draft, float* logits, pbd_stream_t stream);

/*
 * Early-exit draft (the drafter whose cost the draft-cost analysis of App. A.7
 * and Tab. draft-cost-oracle varies): the same draft pass as pbd_draft_block
 * with only the first n_layers backbone layers, followed by the final RMSNorm
 * and the tied LM head.  n_layers in [1, cfg.n_layers]; n_layers = n_layers of
 * the model gives exactly pbd_draft_block.  Other arguments, outputs and
 * errors as pbd_draft_block; n_layers outside the range is PBD_ERR_INVALID_ARG.
 */
int pbd_draft_block_layers(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                           uint32_t flags, int32_t n_layers, int32_t* draft, float* logits, pbd_stream_t stream);

/*
 * Multi-step drafting for the denoising-steps ablation (Sec. 4.4, Sec. 5.3; the
 * Limitations note that the adapter was trained for one step).  The paper gives
 * no remasking rule; this one is low-confidence remasking:
 *   the block starts as D masks; pass s = 1..n_steps runs the draft pass over
 *   [anchor, y_1..y_D] (y_j = the token fixed earlier, or the mask id) and
 *   takes, for each still-masked position j, the candidate argmax of row j
 *   over v != mask id and its confidence, the log-probability of that
 *   candidate under the softmax of the whole row; it then fixes the n_s
 *   still-masked positions of highest confidence (equal confidences: lower
 *   position first), n_s = D / n_steps, plus one for s <= D % n_steps.  Fixed
 *   positions never change; after the last pass none is masked.
 * n_steps = 1 gives pbd_draft_block's tokens and logits.
 *
 * n_steps: in [1, D], else PBD_ERR_INVALID_ARG.
 * draft: device int32 [batch][D]; holds the block state between passes and the
 *   final draft at the end (its previous contents are ignored).
 * conf: NULL or device float [batch][D]: confidence at which each position was
 *   fixed.  fixed_at: NULL or device int32 [batch][D]: the pass (1-based) that
 *   fixed it.  logits: NULL or device float [batch][D+1][V], the last pass's.
 * seq_len, anchor, flags, stream, errors: as pbd_draft_block.  The KV cache is
 * not modified.  Work per call: n_steps draft passes, each followed by one
 * small remasking kernel.
 */
int pbd_draft_block_denoise(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                            uint32_t flags, int32_t n_steps, int32_t* draft, float* conf, int32_t* fixed_at,
                            float* logits, pbd_stream_t stream);

/*
 * Verify pass (Sec. 3 step 3): block [anchor, draft[b][0..D-1]] at positions
 * seq_len..seq_len+D; by default adapter off and causal mask.  Writes the block
 * K/V into the cache at positions seq_len..seq_len+D.  verify: device int32
 * [batch][D+1] receives p_0..p_D, the greedy token after each block row.
 * logits: NULL or device float [batch][D+1][vocab].  Exact greedy matching
 * (App. A.1) compares these with the drafts in pbd_accept_commit.
 * Errors and the capacity rule (seq_len + D + 1 <= max_seq, else the
 * sequence is skipped and PBD_STATUS_CAPACITY raised) as pbd_draft_block.
 */
int pbd_verify_block(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                     const int32_t* draft, uint32_t flags, int32_t* verify, float* logits,
                     pbd_stream_t stream);

/*
 * Unanchored drafting, the anchored-vs-unanchored ablation (Sec. 4.4, Sec. 5.3).
 * The paper does not define the anchor.  Reading: in the anchored step the
 * draft block is [anchor, mask x D] with the adapter on for every row; in the
 * unanchored step the block is the D masks alone at t+1..t+D, and the anchor
 * (the last committed token, position t) is context already in the cache,
 * computed as the verifier computes it.
 *
 * pbd_draft_block_unanchored runs rows [anchor, mask x D] at t..t+D in one pass:
 * the anchor row without the adapter, seeing the prefix and itself (exactly the
 * verifier's row for position t), its K/V appended to the cache at t; the mask
 * rows with the adapter (per flags), seeing the prefix, the anchor and the
 * whole block.  draft[b][j-1] = argmax of mask row j over v != mask id;
 * verify[b][0] = argmax of the anchor row over all V (the verifier's p_0).
 * verify: device int32 [batch][D+1]; only column 0 is written.  logits: NULL
 * or device float [batch][D+1][V] (row 0: the anchor row).
 *
 * pbd_verify_block_unanchored runs the D drafts alone at t+1..t+D, without the
 * adapter, causal, over the prefix including the anchor; it appends their K/V
 * at t+1..t+D and writes verify[b][j] = argmax of row j-1 over all V for
 * j = 1..D (the verifier's p_1..p_D).  logits: NULL or device float
 * [batch][D][V].  With the anchor's K/V from the draft, the pair computes the
 * same K/V and predictions p_0..p_D as pbd_verify_block over [anchor, draft];
 * pbd_accept_commit then applies unchanged.
 *
 * Flags, stream, capacity (t + D + 1 <= max_seq) and errors as
 * pbd_draft_block / pbd_verify_block.  The unanchored draft writes the cache
 * row t; call it only on a state whose anchor is not yet committed (after a
 * prefill or an accept).
 */
int pbd_draft_block_unanchored(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                               uint32_t flags, int32_t* draft, int32_t* verify, float* logits, pbd_stream_t stream);
int pbd_verify_block_unanchored(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* draft,
                                uint32_t flags, int32_t* verify, float* logits, pbd_stream_t stream);

/*
 * pbd_verify_block for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same verify pass, arguments, outputs, flags and errors, with the pass's
 * workspace regions in a static device array of PBD_NOALLOC_SCRATCH_BYTES
 * that the library holds on every device it runs on until the process ends,
 * instead of in the workspace given to pbd_init_weights (the device status
 * word stays there).  It runs one kernel per operator whatever
 * pbd_set_pass_mode chose, and allocates nothing.  The context's device must
 * be current (else PBD_ERR_STATE).  A context whose pass needs more scratch
 * than the array holds (about 12 MiB per sequence of max_batch at the
 * Qwen3-0.6B shape) gets PBD_ERR_CAPACITY.  All calls on one device share
 * the array: calls that overlap on a device (other streams, other threads,
 * other contexts) race and must be serialised by the caller.
 */
#define PBD_NOALLOC_SCRATCH_BYTES (32u << 20)
int pbd_verify_block_noalloc(pbd_ctx* ctx, int32_t batch, const int32_t* seq_len, const int32_t* anchor,
                             const int32_t* draft, uint32_t flags, int32_t* verify, float* logits,
                             pbd_stream_t stream);

/*
 * Acceptance and commit (Sec. 3 steps 4-5; App. A.1).  For each sequence:
 * n = largest k <= D with draft[i-1] == verify[i-1] for all i <= k (or
 * forced_n[b] if forced_n != NULL, device int32 [batch], each in [0, D]);
 * out_tokens[b][0..n] = draft[0..n-1], verify[n] (device int32 [batch][D+1];
 * entries past n are set to -1); n_accepted[b] = n (device int32 [batch]);
 * seq_len[b] += n + 1 and anchor[b] = verify[b][n] (in/out, device).  Cache rows
 * seq_len..seq_len+n written by the verify are kept; later rows are rolled back
 * (they lie past the new seq_len and are overwritten by the next verify).
 */
int pbd_accept_commit(pbd_ctx* ctx, int32_t batch, const int32_t* draft, const int32_t* verify,
                      const int32_t* forced_n, int32_t* seq_len, int32_t* anchor,
                      int32_t* n_accepted, int32_t* out_tokens, pbd_stream_t stream);

/*
 * Wait for `stream`, read and clear the device status word.  *status receives
 * the PBD_STATUS_* bits raised since the last call (0 = none); the return
 * value is the call's own PBD_OK / PBD_ERR_* code (a HIP failure while
 * reading is reported there, not mixed into the status bits).
 */
int pbd_sync_status(pbd_ctx* ctx, pbd_stream_t stream, int32_t* status);

/* ------------------------------------------------------------------------
 * Implementation controls.  The calls below are not part of the step's
 * interface (they change no result beyond fp32 rounding, or they only
 * measure): kernel tuning, operand precision and the profiling aid.
 * ------------------------------------------------------------------------ */

/*
 * Attention split tuning: prefix keys per split-KV work item of the step
 * passes (a positive multiple of 16), or 0 (default) for automatic: 256,
 * doubled while batch * n_kv_heads * ceil(max_seq / keys) exceeds 1280 work
 * items or ceil(max_seq / keys) exceeds 16 splits.  Prefill chunks use at
 * least 1024.  Other values: PBD_ERR_INVALID_ARG.
 */
int pbd_set_attn_keys_per_split(pbd_ctx* ctx, int32_t keys);

/*
 * Attention layout tuning.  mode 1: each split-KV work item runs as one
 * work-group per 16 query rows (shorter per-wave instruction chains, more
 * work-groups, K/V read once per group); 0: one work-group takes all G*W query
 * rows of a KV head; -1 (default): 1 when G*W needs at most three 16-row
 * tiles or batch * n_kv_heads * (splits at max_seq) < 256, else 0.  Results
 * are identical up to fp32 rounding.
 * Other modes: PBD_ERR_INVALID_ARG.
 */
int pbd_set_attn_query_split(pbd_ctx* ctx, int32_t mode);

/*
 * Precision of the GEMM activation operands.  bf16 models run with
 * PBD_OPERANDS_BF16X2 (value + residual, the default); PBD_OPERANDS_BF16
 * returns PBD_ERR_UNSUPPORTED for them, because single bf16 activation
 * operands put the Qwen3-0.6B-shape logits outside the 2e-2 bound.  fp32
 * models accept either value and ignore it.  Other values:
 * PBD_ERR_INVALID_ARG.  Independently of this setting, draft and verify
 * passes of 128 or more rows (batches of 8+) and the persistent batch-1
 * pass take single fp16 operands (11 significant bits) against fp16 weight
 * copies, within the same parity bound; prefill chunks keep the pair.
 */
int pbd_set_operand_precision(pbd_ctx* ctx, int32_t mode);

/*
 * Pass execution mode.  0 (default): batch-1 draft and verify passes of the
 * Qwen3-0.6B layer shape (bf16, hidden 1024, 16 query / 8 KV heads of 128,
 * FFN 3072, LoRA rank <= 16, D + 1 <= 32 rows, max_seq <= 4960, on a
 * 256-CU device) run their layer stack as one persistent kernel; other
 * passes use one kernel per operator.  1: one kernel per operator always.
 * The persistent kernel feeds its matrix cores fp16 activations (11
 * significant bits) and an fp16 copy of the packed weights (exact for bf16
 * weights of magnitude >= 2^-14), the per-operator kernels a bf16 value plus
 * bf16 residual per activation; both stay within the step's parity bound of
 * the float64 reference.  Other values: PBD_ERR_INVALID_ARG.
 */
int pbd_set_pass_mode(pbd_ctx* ctx, int32_t mode);

/*
 * Bound of each wait inside the persistent pass, in polls (0: the default,
 * about a quarter of a second).  A wait that runs out sets
 * PBD_STATUS_TIMEOUT, releases every other wait and lets the kernel finish;
 * the pass's outputs are then invalid.  polls = 1 also makes every
 * work-group of the persistent pass first wait on a word that nothing ever
 * sets, so that the bounded-wait path is always taken (for tests of it).
 * Negative: PBD_ERR_INVALID_ARG.
 */
int pbd_set_wait_limit(pbd_ctx* ctx, int32_t polls);

/*
 * Profiling aid: while enabled, every kernel of a pass is launched with a pair
 * of HIP events attached to its dispatch (hipExtLaunchKernel), which record the
 * kernel's own start and end on the call's stream.  Use it with direct calls,
 * not under stream capture.  pbd_profile_enable(ctx, on) also discards earlier
 * records.  pbd_profile_read waits for the last recorded event and returns the
 * summed kernel time and the launch count of kernel class `kclass`
 * (PBD_KCLASS_*) since the last enable.
 */
int pbd_profile_enable(pbd_ctx* ctx, int32_t on);
int pbd_profile_read(pbd_ctx* ctx, int32_t kclass, double* total_ms, int64_t* launches);

/*
 * Profiling aid of the persistent batch-1 pass: copies the stage timestamps
 * of the last such pass on ctx to the host (synchronises the device).  out:
 * host uint64 array of max_entries; entry (((g * 32 + r) * 64 + l) * 8 + s)
 * * 4 + k is, for rank r of XCD group g in layer l < 64 and stage s (R, Q,
 * A, M, O, R2, GU, D), the device clock (100 MHz) when the stage's wait
 * began (k = 0), when its inputs were ready (k = 1), when its compute waves
 * finished (k = 2; Q, O, GU), when its weight fragments were in LDS (k = 2;
 * D) and when its flag was published (k = 3; R, Q, A, M, R2, GU).
 * l = n_layers holds the final norm's start and end (stage 0, k = 0 and 1).
 * Entries not recorded hold stale values.  *n_written
 * receives min(max_entries, 524288).
 */
int pbd_profile_stage_times(pbd_ctx* ctx, uint64_t* out, int32_t max_entries, int32_t* n_written);

/* Message of the last failed call on ctx (or of the last failed init if ctx is NULL). */
const char* pbd_last_error(const pbd_ctx* ctx);

/* Free the host context.  Device buffers stay the caller's. */
void pbd_destroy(pbd_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* PBD_H */
