/*
 * nld.h -- block-decode step of linear self-speculation on AMD MI355X (gfx950).
 *
 * Method: arXiv 2607.05722, Sec. 3.3 ("Mode 3: Self-Speculation Decoding",
 * linear self-speculation).  A block of k tokens per sequence runs one
 * forward pass of a decoder-only transformer against the sequence's prefix
 * KV cache.  In the diffusion *draft* pass the block attends bidirectionally
 * within itself (block-wise diffusion, Sec. 2.1); in the AR *verify* pass it
 * is causal (Sec. 2.2, Sec. 3.1).  The longest draft prefix that matches the
 * AR predictions is accepted and the AR prediction at the first rejected
 * position is committed as one extra token (Sec. 3.3; the first-mismatch
 * index j* of the same section).
 *
 * Block layout.  Row 0 of a block is the *anchor*: the last committed token,
 * whose K/V is not cached yet.  Rows 1..k-1 hold mask tokens (draft) or the
 * draft tokens d_1..d_{k-1} (verify), so the speculative width is k-1 (the
 * paper's Tab. 10 pairs draft length 31 with blocks of 32).  Block row j sits
 * at absolute position P_b + j, where P_b is the sequence's committed length.
 * Draft token d_j is the argmax of draft row j; verify row j predicts the
 * token at position P_b + j + 1.  A step commits L+1 tokens, 0 <= L <= k-1.
 *
 * Conventions for every call:
 *  - All array arguments are DEVICE pointers unless marked "host".  The
 *    caller allocates and owns every buffer (weights, cache, workspace,
 *    outputs); the library never allocates or frees device memory and keeps
 *    no pointer after a call returns, except the weight pointers a model
 *    handle borrows (they must outlive the handle).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Calls only enqueue work; they never synchronize except
 *    nld_read_device_status.
 *  - bf16 means IEEE bfloat16 bit patterns (uint16).  Matrices are row-major.
 *  - Argument checks run on the host before anything is enqueued; a failing
 *    call enqueues nothing and returns a negative nld_status, with a message
 *    available from nld_last_error() (thread-local).
 *  - Conditions only the device can see (a token id outside [0, vocab), a
 *    block that would run past the cache capacity, max_len < P_b + k) set bits
 *    of a sticky status word in the workspace; the offending write is
 *    skipped, never performed out of bounds.  Read it with
 *    nld_read_device_status.
 *  - Concurrent calls on one workspace race; give each stream its own.
 */
#ifndef NLD_H
#define NLD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NLD_OK = 0,
    NLD_ERR_INVALID_ARG = -1,   /* null pointer, non-positive size, value out of range */
    NLD_ERR_SHAPE = -2,         /* a size the kernels do not support (see each call) */
    NLD_ERR_CAPACITY = -3,      /* workspace too small */
    NLD_ERR_HIP = -4,           /* a HIP runtime call failed; message has the HIP error */
    NLD_ERR_UNSUPPORTED = -5,   /* no gfx950 device, or an unsupported mode */
    NLD_ERR_DEVICE = -6         /* nld_read_device_status found a device-side error bit */
} nld_status;

/* Device status bits (sticky, OR-ed together). */
#define NLD_DEV_BAD_TOKEN 0x1u     /* a token id outside [0, vocab) was replaced by 0 */
#define NLD_DEV_CAPACITY 0x2u      /* P_b + k > max_len: the block's K/V rows at or past max_len were not
                                      written, and a commit that would pass max_len stops the length there */
#define NLD_DEV_BAD_LENGTH 0x4u    /* a negative committed length was read */
#define NLD_DEV_MASK_LEFT 0x8u     /* nld_refresh_block found a mask token in block rows 1..k-1 */

typedef enum {
    NLD_MODE_VERIFY = 0,   /* AR verify: causal within the block */
    NLD_MODE_DRAFT = 1     /* diffusion draft: block rows >= bidir_from see the whole block */
} nld_mode;

/* Architecture of the decoder.  Pre-norm RMSNorm, rotate-half RoPE (pairs
 * (i, i + head_dim/2), angle pos * rope_base^(-2i/head_dim)), GQA attention
 * with scale 1/sqrt(head_dim) where query head h reads KV head
 * h / (n_q_heads / n_kv_heads), SwiGLU FFN silu(x Wg) * (x Wu) then Wd,
 * residual connections, final RMSNorm, untied LM head; no biases. */
typedef struct {
    int32_t n_layers;
    int32_t hidden;        /* multiple of 32 */
    int32_t n_q_heads;
    int32_t n_kv_heads;    /* divides n_q_heads */
    int32_t head_dim;      /* 64 or 128 */
    int32_t ffn;           /* multiple of 8 */
    int32_t vocab;
    float rope_base;
    float rms_eps;
    int32_t mask_token_id; /* token placed in draft rows 1..k-1 */
    /* LoRA-enhanced drafter (Sec. 3.3): an adapter on the O projection used only by
     * draft-mode passes (the draft pass, denoising steps, nld_block_forward with
     * NLD_MODE_DRAFT); verify passes never read it.  A draft pass adds
     * lora_scale * B (A o) to the O projection's output, A = lora_a [lora_rank][n_q_heads*head_dim],
     * B = lora_b [hidden][lora_rank] (standard LoRA, lora_scale = alpha / rank; the paper
     * uses rank 128, alpha 512).  lora_rank 0 (no adapter) or a multiple of 32 up to 512. */
    int32_t lora_rank;
    float lora_scale;
} nld_config;

/* Per-layer weights.  Norm gains are plain bf16 vectors; matrices must be in
 * the packed layouts produced by the nld_pack_* calls below. */
typedef struct {
    const void* attn_norm;   /* bf16 [hidden] */
    const void* w_qkv;       /* nld_pack_qkv(Wq, Wk, Wv) */
    const void* w_o;         /* nld_pack_linear(Wo [hidden][n_q_heads*head_dim]) */
    const void* ffn_norm;    /* bf16 [hidden] */
    const void* w_gate_up;   /* nld_pack_gate_up(Wg, Wu) */
    const void* w_down;      /* nld_pack_linear(Wd [hidden][ffn]) */
    const void* lora_a;      /* nld_pack_linear(A [lora_rank][n_q_heads*head_dim]); NULL when lora_rank = 0 */
    const void* lora_b;      /* nld_pack_linear(B [hidden][lora_rank]); NULL when lora_rank = 0 */
} nld_layer_weights;

typedef struct {
    const void* embed;                 /* bf16 [vocab][hidden], row-major (not packed) */
    const void* final_norm;            /* bf16 [hidden] */
    const void* lm_head;               /* nld_pack_linear(W_lm [vocab][hidden]) */
    const nld_layer_weights* layers;   /* host array [n_layers]; copied by nld_model_create */
} nld_weights;

/* KV cache.  K and V of every layer, sequence and KV head, bf16:
 *   k: [n_layers][batch][n_kv_heads][max_len][head_dim]
 *   v: [n_layers][batch][n_kv_heads][max_len/64][head_dim][64]
 *      (64-position tiles, each stored transposed: head_dim rows of 64 positions)
 * lengths[b] = P_b, the committed length of sequence b.  Rows at positions
 * >= P_b are scratch: a verify pass writes its block's K/V rows to positions
 * [P_b, P_b + k) (a draft pass writes no cache row), and only
 * nld_verify_accept (by L+1: the anchor row and the accepted draft rows) and
 * nld_refresh_block (by k-1) advance lengths, which commits those rows; the
 * rest are overwritten by later passes.  A length never advances past max_len:
 * a commit that would (its rows at or past max_len were not written) stops at
 * max_len and sets NLD_DEV_CAPACITY, so every row below lengths[b] is valid.
 * Within a pass the block attends to its own keys and values from a
 * higher-precision copy in the workspace (bf16 value plus bf16 remainder),
 * so the cache rows are only what a commit keeps. */
typedef struct {
    void* k;
    void* v;
    int32_t* lengths;   /* device int32 [batch] */
    int32_t batch;
    int32_t max_len;    /* multiple of 64 */
} nld_kv_cache;

typedef struct nld_model nld_model;   /* opaque handle; borrows the weight pointers */

/* Message for the last non-OK status returned on this thread. */
const char* nld_last_error(void);
const char* nld_status_string(int32_t status);

/* Validate `cfg` and the weight pointers (host-side only) and build a handle.
 * Errors: INVALID_ARG (null pointer, non-positive size, a negative or
 * non-finite LoRA setting, missing adapter weights when lora_rank > 0), SHAPE
 * (hidden not a multiple of 32, head_dim not 64/128, n_q_heads not a multiple
 * of n_kv_heads, ffn not a multiple of 8, lora_rank not a multiple of 32).
 * No device call is made. */
nld_status nld_model_create(const nld_config* cfg, const nld_weights* w, nld_model** out);
void nld_model_destroy(nld_model* m);

/* ---- weight packing (one-time, on the device) ------------------------------
 * Packed layout: the output features are cut into tiles of 16, the input
 * features into steps of 32 (zero-padded); tile t, step s is one contiguous
 * 1 KiB block whose 16-byte lane l holds W[16t + l%16][32s + 8(l/16) .. +8]
 * -- one MFMA B-operand per wavefront load.  Sizes come from
 * nld_packed_bytes.  Source matrices are bf16 row-major [out][in]; source and
 * destination must not overlap. */
#define NLD_PACK_LINEAR 0
#define NLD_PACK_QKV 1       /* rows of each 16-column tile pair RoPE partners (i, i + head_dim/2) */
#define NLD_PACK_GATE_UP 2   /* each 16-column tile holds 8 gate rows then the same 8 up rows */
size_t nld_packed_bytes(int32_t kind, const nld_config* cfg, int32_t out_dim, int32_t in_dim);
/* out_dim x in_dim matrix w.  Errors: INVALID_ARG, SHAPE (in_dim % 8 != 0). */
nld_status nld_pack_linear(const void* w, int32_t out_dim, int32_t in_dim, void* packed, void* stream);
/* wq [n_q_heads*head_dim][hidden], wk/wv [n_kv_heads*head_dim][hidden]. */
nld_status nld_pack_qkv(const nld_config* cfg, const void* wq, const void* wk, const void* wv, void* packed,
                        void* stream);
/* wg, wu [ffn][hidden]. */
nld_status nld_pack_gate_up(const nld_config* cfg, const void* wg, const void* wu, void* packed, void* stream);

/* ---- workspace -------------------------------------------------------------
 * Bytes of scratch one call with this batch, block size and cache capacity
 * needs (activations, attention partials, argmax partials, counters, status
 * word).  nld_workspace_init must run once on a new workspace before its
 * first use (it clears the counters and the status word). */
size_t nld_workspace_bytes(const nld_model* m, int32_t batch, int32_t k, int32_t max_len);
nld_status nld_workspace_init(void* workspace, size_t ws_bytes, void* stream);

/* ---- the block-decode step ---------------------------------------------------
 * One forward pass over tokens[batch][k] (block row j at position P_b + j):
 * embedding -> n_layers x (RMSNorm, QKV, RoPE, K/V write (verify: cache rows
 * [P_b, P_b+k)), block-masked GQA attention over the P_b + k keys, O +
 * residual, RMSNorm, SwiGLU, down + residual) -> final RMSNorm -> LM head ->
 * per-row argmax (lowest index among equal maxima).
 * mode: NLD_MODE_VERIFY (block causal) or NLD_MODE_DRAFT (rows j >= bidir_from
 * see every block column, rows below it are causal); bidir_from in [0, k].
 * logits (optional) f32 [batch][k][vocab]; argmax (optional) int32 [batch][k].
 * lengths are not changed.
 * Errors: INVALID_ARG (null model/cache/tokens/workspace, batch < 1,
 * k < 1 or k > 64, bad mode/bidir_from, kv->batch != batch), SHAPE
 * (n_q_heads/n_kv_heads * k > 256), CAPACITY (ws_bytes too small). */
nld_status nld_block_forward(const nld_model* m, const nld_kv_cache* kv, const int32_t* tokens, int32_t batch,
                             int32_t k, int32_t mode, int32_t bidir_from, float* logits, int32_t* argmax,
                             void* workspace, size_t ws_bytes, void* stream);

/* Diffusion draft (Sec. 3.3): runs the draft pass over [anchor[b], mask x (k-1)]
 * and writes draft[b][j-1] = argmax of draft row j, j = 1..k-1 (k >= 2).
 * logits optional as above.  The cache is not written; lengths unchanged.
 * Errors as nld_block_forward. */
nld_status nld_draft(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor, int32_t batch, int32_t k,
                     int32_t bidir_from, int32_t* draft, float* logits, void* workspace, size_t ws_bytes,
                     void* stream);

/* AR verify + acceptance (Sec. 3.3): runs the causal pass over
 * [anchor[b], draft[b][0..k-2]], takes a_j = argmax of verify row j, accepts
 * L_b = the number of leading j in 1..k-1 with draft[b][j-1] == a_{j-1}, and
 * writes accept_len[b] = L_b, committed[b][0..k) = d_1..d_{L_b}, a_{L_b},
 * then -1 padding, next_anchor[b] = a_{L_b}, and lengths[b] += L_b + 1 (the
 * anchor row and the accepted draft rows become committed cache rows).
 * next_anchor may be the same buffer as anchor (it is written last), which
 * keeps a decode loop on the device.
 * With k = 1 this is one step of AR decoding (Sec. 3.1); draft may then be NULL.
 * logits optional.  Errors as nld_block_forward. */
nld_status nld_verify_accept(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor,
                             const int32_t* draft, int32_t batch, int32_t k, int32_t* accept_len,
                             int32_t* committed, int32_t* next_anchor, float* logits, void* workspace,
                             size_t ws_bytes, void* stream);

/* Argmax + acceptance alone, from given logits f32 [batch][k][vocab] and
 * draft int32 [batch][k-1] (NULL when k = 1): writes argmax [batch][k] and the
 * same accept_len / committed / next_anchor as nld_verify_accept.  Does not
 * touch any cache.  workspace must be initialized and hold at least
 * nld_accept_workspace_bytes(batch, k).  Errors: INVALID_ARG, CAPACITY. */
size_t nld_accept_workspace_bytes(int32_t batch, int32_t k);
nld_status nld_accept_from_logits(const float* logits, const int32_t* draft, int32_t batch, int32_t k,
                                  int32_t vocab, int32_t* argmax, int32_t* accept_len, int32_t* committed,
                                  int32_t* next_anchor, void* workspace, size_t ws_bytes, void* stream);

/* ---- a decoding loop on the device ---------------------------------------------
 * n_steps decoding steps enqueued back to back with no host synchronisation (the
 * sequence can be captured into a graph and replayed): with k >= 2 each step is
 * linear self-speculation, nld_draft then nld_verify_accept (Sec. 3.3); with
 * k = 1 each step is one AR decoding step (Sec. 3.1).  anchor [batch] is
 * read by each step and overwritten with its next anchor; step s writes
 * accept_len[s][batch] and committed[s][batch][k] as nld_verify_accept does, and
 * every step advances lengths.  The drafts live in the workspace.  The cache
 * needs room for n_steps * k more rows per sequence (else NLD_DEV_CAPACITY).
 * Errors as nld_block_forward, plus INVALID_ARG for n_steps < 1 or a NULL
 * anchor/accept_len/committed. */
nld_status nld_decode_steps(const nld_model* m, const nld_kv_cache* kv, int32_t* anchor, int32_t batch, int32_t k,
                            int32_t n_steps, int32_t bidir_from, int32_t* accept_len, int32_t* committed,
                            void* workspace, size_t ws_bytes, void* stream);

/* Host-only choice between AR decoding and self-speculation for the next steps
 * (AR is the mode for high concurrency, Sec. 3.1, where a self-speculation step
 * stops paying for its second pass): returns k_ss when expected_committed
 * tokens per self-speculation step of ss_step_ms beat one token per AR step of
 * ar_step_ms, else 1.  The caller measures both step times at its batch size
 * and tracks expected_committed (the mean of L+1 over recent steps).  Returns 1
 * for non-positive times or k_ss < 2. */
int32_t nld_choose_block(float ar_step_ms, float ss_step_ms, float expected_committed, int32_t k_ss);

/* ---- quadratic self-speculation (Sec. 3.4, Appendix C) -------------------------
 * One forward pass that both verifies the previous step's speculative tokens and
 * drafts the next ones for every possible acceptance length.  The block of each
 * sequence is the chain [anchor, s_1 .. s_{k-1}] (Mode 3's verify block: chain
 * element c at position P_b + c) followed by one group of k mask tokens per chain
 * element (mask r = 1..k of group c at position P_b + c + r): k(k+1) rows.  Every
 * row sees the cached prefix; chain row c sees chain elements 0..c; a mask of
 * group c sees chain elements 0..c and its own group's masks.  Chain rows predict
 * the next position (AR); masks predict their own position (diffusion).
 * Verifier token v_i of position P_b + i (i = 1..k): argmax of
 * lambda * softmax(chain row i-1) + (1 - lambda) * softmax(mask 1 of group i-1),
 * lowest index on ties (lambda = 1: AR verification; 0: diffusion).  Then
 * Mode 3's acceptance: L = longest prefix with s_i = v_i, committed[b] =
 * s_1..s_L, v_{L+1}, -1 padded to k; lengths[b] += L+1 (the chain rows' K/V,
 * written to cache rows [P_b, P_b + k), become committed); next_anchor[b] =
 * v_{L+1}; next_spec[b][r-2] = argmax of mask r of group L, r = 2..k (the tokens
 * at positions P_b + L + 2 .. P_b + L + k, right after the next anchor).
 * spec / next_spec int32 [batch][k-1] (next_spec may alias spec, next_anchor may
 * alias anchor); accept_len [batch]; committed [batch][k]; logits (optional) f32
 * [batch][k(k+1)][vocab] in block-row order.  The first step's speculative
 * tokens come from nld_draft.  The LoRA adapter is not used by this pass.
 * The workspace must hold nld_quad_workspace_bytes(m, batch, k, max_len)
 * (initialized with nld_workspace_init).
 * Errors: INVALID_ARG (k outside [2, NLD_QUAD_MAX_K], lambda outside [0, 1] or
 * NaN, a NULL pointer, and the checks of nld_block_forward for k(k+1) rows),
 * SHAPE ((n_q_heads/n_kv_heads) * k(k+1) > 256), CAPACITY (workspace). */
#define NLD_QUAD_MAX_K 7   /* k(k+1) block rows must fit one 64-key stage of the block attention */
size_t nld_quad_workspace_bytes(const nld_model* m, int32_t batch, int32_t k, int32_t max_len);
nld_status nld_quad_step(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor, const int32_t* spec,
                         int32_t batch, int32_t k, float lambda, int32_t* accept_len, int32_t* committed,
                         int32_t* next_anchor, int32_t* next_spec, float* logits, void* workspace, size_t ws_bytes,
                         void* stream);

/* ---- Mode 2: block-wise diffusion denoising (Sec. 3.2) -----------------------
 * Confidence-based decoding of one block per sequence: the block starts as
 * [anchor, mask x (k-1)] and each denoising step, one diffusion (draft) pass
 * over the current block, fills in some of its masked rows; when no mask is
 * left, a refresh recomputes the block's K/V with the causal mask (the clean
 * stream is strictly causal, Sec. 2.2) and commits it, and the next block
 * starts from the last decoded token as its anchor.
 * A masked row is denoised to the argmax of its logits over every token except
 * mask_token_id (a mask is never a decoded value), with confidence = that
 * token's softmax probability over the same tokens. */

/* One denoising step.  block: int32 [batch][k], in/out; row 0 is the anchor,
 * rows 1..k-1 hold mask_token_id (still masked) or an earlier step's token.
 * Runs the draft pass (rows >= bidir_from see every block column) and commits,
 * per sequence, every masked row whose confidence exceeds `threshold`
 * (strictly); when none does, the most confident masked row (the lowest row
 * among equal confidences), so a step with a mask left commits at least one.
 * Writes n_committed[b] (rows filled by this step) and n_masked[b] (masks
 * left); confidence (optional) f32 [batch][k] gets every row's confidence and
 * logits (optional) the pass's raw logits.  The cache and lengths are not
 * touched.  A block with no mask left is returned unchanged (n_committed 0).
 * Errors as nld_block_forward, plus INVALID_ARG for k < 2, a NULL
 * block/n_committed/n_masked or a NaN threshold. */
nld_status nld_denoise_step(const nld_model* m, const nld_kv_cache* kv, int32_t* block, int32_t batch, int32_t k,
                            int32_t bidir_from, float threshold, int32_t* n_committed, int32_t* n_masked,
                            float* confidence, float* logits, void* workspace, size_t ws_bytes, void* stream);

/* K/V refresh of completed blocks: a causal pass over block [batch][k] that
 * writes every layer's K/V rows [P_b, P_b + k) and then commits k-1 of them
 * (lengths[b] += k-1: the anchor and rows 1..k-2), with next_anchor[b] =
 * block[b][k-1].  Only the K/V projections run in the last layer and the LM
 * head does not run (nothing after the last K/V write is needed).  A mask
 * token left in rows 1..k-1 sets NLD_DEV_MASK_LEFT (the rows are still
 * committed).  Errors as nld_block_forward, plus INVALID_ARG for k < 2. */
nld_status nld_refresh_block(const nld_model* m, const nld_kv_cache* kv, const int32_t* block, int32_t batch,
                             int32_t k, int32_t* next_anchor, void* workspace, size_t ws_bytes, void* stream);

/* The denoising step's decision alone, from given logits f32 [batch][k][vocab]:
 * argmax (optional) int32 [batch][k] and confidence (optional) f32 [batch][k]
 * over the tokens other than mask_token_id, and the same in-place commit into
 * block [batch][k] with n_committed / n_masked as nld_denoise_step.  Needs no
 * workspace.  Errors: INVALID_ARG (NULL pointer, batch < 1, k outside [2, 64],
 * vocab < 2, mask_token_id outside [0, vocab), NaN threshold). */
nld_status nld_commit_from_logits(const float* logits, int32_t* block, int32_t batch, int32_t k, int32_t vocab,
                                  int32_t mask_token_id, float threshold, int32_t* argmax, int32_t* n_committed,
                                  int32_t* n_masked, float* confidence, void* stream);

/* ---- tracing aid -------------------------------------------------------------
 * While enabled, every kernel launch made by the block-decode calls records a
 * pair of HIP events on its own dispatch (hipExtLaunchKernel), so the times are
 * those of the kernels themselves, without launch gaps (do not enable it while
 * a stream is being captured into a graph).  nld_trace_read synchronizes on
 * those events and returns, per kernel class, the summed milliseconds and the
 * number of class instances since the last read (host arrays of length n >=
 * NLD_TRACE_CLASSES), then clears the record.  An instance is one step of the
 * pass: the attention class holds the attention and merge kernels, the O
 * projection class also the LoRA down-projection when an adapter runs. */
#define NLD_TRACE_EMBED 0
#define NLD_TRACE_QKV 1
#define NLD_TRACE_ATTENTION 2
#define NLD_TRACE_O_PROJ 3
#define NLD_TRACE_GATE_UP 4
#define NLD_TRACE_DOWN 5
#define NLD_TRACE_LM_HEAD 6
#define NLD_TRACE_ARGMAX 7
#define NLD_TRACE_CLASSES 8
nld_status nld_trace_enable(int32_t on);
nld_status nld_trace_read(float* ms, int32_t* counts, int32_t n);

/* Synchronizes `stream`, copies the sticky device status word to *host_bits
 * (host pointer) and clears it.  Returns NLD_ERR_DEVICE if any bit was set. */
nld_status nld_read_device_status(void* workspace, uint32_t* host_bits, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the verify
 * + acceptance step of nld_verify_accept with no workspace argument.  Its
 * scratch is a static device array of NLD_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends; the call
 * itself allocates and frees nothing.  Arguments and results are those of
 * nld_verify_accept (same kernels, same launch plan).  device_status
 * (optional device uint32) receives this call's device status bits
 * (NLD_DEV_*); the scratch's own status word is cleared at the start of every
 * call.  All calls on one GPU share that GPU's scratch array, which keeps the
 * last call's contents: calls that overlap on one GPU (several streams or
 * threads) race and must be serialized by the caller.
 * Errors as nld_verify_accept; NLD_ERR_CAPACITY when the scratch this batch,
 * k and max_len need (nld_workspace_bytes) exceeds NLD_NOALLOC_SCRATCH_BYTES
 * (it holds batch 1 at k <= 16 for the 8B and 14B shapes). */
#define NLD_NOALLOC_SCRATCH_BYTES (64u << 20)
nld_status nld_verify_accept_noalloc(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor,
                                     const int32_t* draft, int32_t batch, int32_t k, int32_t* accept_len,
                                     int32_t* committed, int32_t* next_anchor, float* logits,
                                     uint32_t* device_status, void* stream);

/* HBM streaming-read probe, a measurement aid (not a step of the method): reads
 * `bytes` (a multiple of 1024) from device buffer `buf` with `grid` workgroups of
 * `waves` (1..16) wavefronts, each wavefront load one contiguous 1 KiB block (the
 * weight streams' pattern) and each lane keeping `depth` (4, 8, 16 or 32) loads
 * in flight; workgroup b writes a checksum to device word sink[b] (grid words).
 * Bytes over the time of the launch (events on `stream`) is the read rate this
 * pattern reaches.  Errors: INVALID_ARG, HIP. */
nld_status nld_hbm_read_probe(const void* buf, size_t bytes, int32_t grid, int32_t waves, int32_t depth,
                              uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* NLD_H */
