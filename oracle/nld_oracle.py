"""CPU oracle for one block-decode step of linear self-speculation.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the package smoke check and the
CPU-baseline leg of the benchmark use it.  It shares no code with the GPU
path; the two meet only in the seeded input generator (``synth``).

What it computes (arXiv 2607.05722):

* Linear self-speculation, Sec. 3.3 ("Mode 3: Self-Speculation Decoding"):
  a diffusion *draft* pass over a block that holds mask tokens after the
  verified prefix, then an AR *verify* pass over the draft tokens with causal
  attention that reuses the prefix KV cache, then acceptance of the longest
  draft prefix that matches the AR predictions plus one token from the AR
  prediction at the first rejected position.
* The attention pattern follows Sec. 2.1 (block-wise diffusion objective:
  bidirectional within a block, causal across blocks) and Sec. 2.2 (the clean
  stream is strictly causal).
* Mode 1 (Sec. 3.1), AR decoding, is the verify pass with a one-token block.
* The first-mismatch index j* of the LoRA paragraph in Sec. 3.3 restates the
  acceptance rule and is the form used here.
* The LoRA-enhanced drafter of Sec. 3.3: an adapter on the attention's O
  projection that only the diffusion (draft-mode) passes use, the AR pathway
  left unchanged.  Standard LoRA form: the O projection's output gains
  (alpha / r) * B A o for rank r, A [r][q_dim], B [hidden][r].
* Mode 2 (Sec. 3.2), block-wise diffusion denoising with confidence-based
  sampling: repeated draft passes over a block that commit masked positions by
  a confidence threshold, then a causal K/V refresh of the completed block
  (its readings are listed with those functions at the end of this module).

Readings where the paper is silent or its indices do not close (listed with
reasons in the design notes of the repository):

* Block layout: a block of ``k`` rows is ``[anchor, r_1 .. r_{k-1}]``.  The
  anchor is the last committed token, whose K/V is not cached yet; the
  ``r_j`` are mask tokens (draft) or draft tokens (verify).  The speculative
  width is k-1 (Tab. 10 uses draft length 31 with blocks of 32) and one step
  commits between 1 and k tokens.  With k = 1 the verify pass is AR decoding.
* Draft token d_j is the argmax of draft row j (a mask at a position predicts
  the token at that same position, as in the diffusion objective of Sec. 2.1);
  verify row j predicts the token at the next position (AR shift).
* Draft mask: block rows j >= bidir_from see every block column (default 0:
  the whole block is bidirectional); other rows are causal.
* Decoder architecture (not specified by the paper; taken from the workload
  statement): pre-norm RMSNorm (eps 1e-6) -> QKV -> rotate-half RoPE (base
  1e4, angles in float64, absolute 0-based positions) -> GQA softmax attention
  with scale 1/sqrt(head_dim) (query head h uses KV head h // (Hq/Hkv)) ->
  O projection + residual -> RMSNorm -> SwiGLU FFN silu(h Wg) * (h Wu) ->
  down projection + residual; final RMSNorm -> untied LM head.  No biases.
* Argmax takes the first index of the maximum (ties to the lowest index).

Arithmetic runs in float32 by default (the precision the reference oracle is
specified in); ``dtype=np.float64`` gives a second instantiation used to
bound this oracle's own rounding error.  Weights and cached K/V arrive as
bfloat16 bit patterns and are widened exactly.
"""
from __future__ import annotations

import numpy as np

DRAFT = "draft"
VERIFY = "verify"


# ----------------------------------------------------------------------------- elementary pieces
def bf16_bits_to_float(bits: np.ndarray, dtype=np.float32) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32/float64."""
    f = (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    return f.astype(dtype, copy=False)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding.

    x: [..., rows, heads, D]; positions: integer array broadcastable to the
    rows axis.  Pair (i, i + D/2) is rotated by angle pos * base^(-2i/D).
    """
    d = x.shape[-1]
    half = d // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / d)
    ang = np.asarray(positions, dtype=np.float64)[..., None] * inv_freq      # [..., rows, half]
    cos = np.cos(ang).astype(x.dtype)[..., None, :]                           # [..., rows, 1, half]
    sin = np.sin(ang).astype(x.dtype)[..., None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax_attention(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, visible: np.ndarray) -> np.ndarray:
    """softmax(q K^T / sqrt(D) restricted to visible columns) V.

    q: [rows, D]; keys/vals: [n, D]; visible: bool [rows, n] (every row has at
    least one visible column).
    """
    d = q.shape[-1]
    s = (q @ keys.T) / np.sqrt(np.asarray(d, dtype=q.dtype))
    s = np.where(visible, s, -np.inf)
    s = s - np.max(s, axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / np.sum(p, axis=-1, keepdims=True)
    return p @ vals


def block_visibility(prefix_len: int, k: int, mode: str, bidir_from: int = 0) -> np.ndarray:
    """Which of the prefix_len + k key positions each block row may attend to.

    Every block row sees the whole cached prefix (causal across blocks).  Within
    the block, verify rows are causal (column c visible iff c <= row); draft
    rows at or after ``bidir_from`` see every block column (bidirectional), the
    rows before it stay causal.
    """
    vis = np.zeros((k, prefix_len + k), dtype=bool)
    vis[:, :prefix_len] = True
    for j in range(k):
        for c in range(k):
            if c <= j or (mode == DRAFT and j >= bidir_from):
                vis[j, prefix_len + c] = True
    return vis


def lora_scale(shape) -> float:
    """LoRA output scale alpha / r (Sec. 3.3 uses r = 128, alpha = 512)."""
    return float(shape.lora_alpha) / float(shape.lora_rank)


def argmax_first(logits: np.ndarray) -> np.ndarray:
    """Index of the first maximum along the last axis."""
    return np.argmax(logits, axis=-1).astype(np.int32)


# ----------------------------------------------------------------------------- model + cache
class OracleWeights:
    """Float views of a synthetic model, widened from bf16 one layer at a time."""

    def __init__(self, shape, source, dtype=np.float32):
        self.shape, self.src, self.dtype = shape, source, dtype

    def layer(self, l: int) -> dict:
        w = self.src.layer(l)
        return {name: bf16_bits_to_float(v, self.dtype) for name, v in w.items()}

    def embed_rows(self, token_ids: np.ndarray) -> np.ndarray:
        return bf16_bits_to_float(self.src.embed[np.asarray(token_ids)], self.dtype)

    def final_norm(self) -> np.ndarray:
        return bf16_bits_to_float(self.src.final_norm, self.dtype)

    def lm_head(self) -> np.ndarray:
        return bf16_bits_to_float(self.src.lm_head, self.dtype)


class OracleKV:
    """Per-layer K/V of every sequence plus its committed length P_b.

    k[l], v[l]: [batch, n_kv_heads, capacity, head_dim] in the oracle's dtype.
    Rows at or beyond lengths[b] are not part of the committed state.
    """

    def __init__(self, shape, batch: int, capacity: int, dtype=np.float32):
        self.shape, self.batch, self.capacity, self.dtype = shape, batch, capacity, dtype
        kvshape = (batch, shape.n_kv_heads, capacity, shape.head_dim)
        self.k = [np.zeros(kvshape, dtype=dtype) for _ in range(shape.n_layers)]
        self.v = [np.zeros(kvshape, dtype=dtype) for _ in range(shape.n_layers)]
        self.lengths = np.zeros(batch, dtype=np.int64)

    def set_prefix_bf16(self, layer: int, k_bits: np.ndarray, v_bits: np.ndarray, lengths) -> None:
        """Load given cached K/V ([batch, kv_heads, P, D] bf16 bits) as the prefix."""
        n = k_bits.shape[2]
        self.k[layer][:, :, :n] = bf16_bits_to_float(k_bits, self.dtype)
        self.v[layer][:, :, :n] = bf16_bits_to_float(v_bits, self.dtype)
        self.lengths[:] = np.asarray(lengths)

    def copy(self) -> "OracleKV":
        c = OracleKV.__new__(OracleKV)
        c.shape, c.batch, c.capacity, c.dtype = self.shape, self.batch, self.capacity, self.dtype
        c.k = [a.copy() for a in self.k]
        c.v = [a.copy() for a in self.v]
        c.lengths = self.lengths.copy()
        return c


# ----------------------------------------------------------------------------- one block forward
def block_forward(weights: OracleWeights, kv: OracleKV, tokens: np.ndarray, mode: str,
                  bidir_from: int = 0, positions: np.ndarray | None = None,
                  rows_for_logits=None, block_vis: np.ndarray | None = None):
    """One forward pass of a k-token block per sequence against the cached prefix.

    tokens: int [batch, k].  Returns (logits [batch, k, vocab], new_k, new_v)
    where new_k/new_v[l] are the block's rotated keys and values,
    [batch, n_kv_heads, k, head_dim].  The cache itself is not modified (what
    to commit is decided by acceptance).  ``positions`` overrides the default
    block positions P_b + j.  ``rows_for_logits`` (optional list of row
    indices) restricts the LM head to those rows; other rows get NaN.
    ``block_vis`` (bool [k, k]) overrides which block columns each block row
    sees (every row still sees the whole prefix); the LoRA adapter then takes
    no part (it belongs to the draft pass).
    """
    s = weights.shape
    dt = weights.dtype
    tokens = np.asarray(tokens)
    B, k = tokens.shape
    G = s.n_q_heads // s.n_kv_heads
    if positions is None:
        positions = kv.lengths[:, None] + np.arange(k)[None, :]
    positions = np.asarray(positions)

    x = weights.embed_rows(tokens)                                   # [B, k, H]
    new_k, new_v = [], []
    for l in range(s.n_layers):
        w = weights.layer(l)
        h = rms_norm(x, w["attn_norm"], s.rms_eps)
        q = (h @ w["wq"].T).reshape(B, k, s.n_q_heads, s.head_dim)
        kb = (h @ w["wk"].T).reshape(B, k, s.n_kv_heads, s.head_dim)
        vb = (h @ w["wv"].T).reshape(B, k, s.n_kv_heads, s.head_dim)
        q = rope(q, positions, s.rope_base)
        kb = rope(kb, positions, s.rope_base)
        new_k.append(np.ascontiguousarray(kb.transpose(0, 2, 1, 3)))
        new_v.append(np.ascontiguousarray(vb.transpose(0, 2, 1, 3)))

        o = np.zeros((B, k, s.n_q_heads, s.head_dim), dtype=dt)
        for b in range(B):
            p_b = int(kv.lengths[b])
            if block_vis is None:
                vis = block_visibility(p_b, k, mode, bidir_from)
            else:
                vis = np.concatenate([np.ones((k, p_b), dtype=bool), np.asarray(block_vis, dtype=bool)], axis=1)
            for g in range(s.n_kv_heads):
                keys = np.concatenate([kv.k[l][b, g, :p_b], kb[b, :, g]], axis=0)
                vals = np.concatenate([kv.v[l][b, g, :p_b], vb[b, :, g]], axis=0)
                for hq in range(g * G, (g + 1) * G):
                    o[b, :, hq] = softmax_attention(q[b, :, hq], keys, vals, vis)
        o2 = o.reshape(B, k, s.q_dim)
        x = x + o2 @ w["wo"].T
        if mode == DRAFT and block_vis is None and "lora_a" in w:
            x = x + lora_scale(s) * ((o2 @ w["lora_a"].T) @ w["lora_b"].T)

        h = rms_norm(x, w["ffn_norm"], s.rms_eps)
        act = silu(h @ w["w_gate"].T) * (h @ w["w_up"].T)
        x = x + act @ w["w_down"].T

    hf = rms_norm(x, weights.final_norm(), s.rms_eps)
    lm = weights.lm_head()
    if rows_for_logits is None:
        logits = hf @ lm.T
    else:
        logits = np.full((B, k, s.vocab), np.nan, dtype=dt)
        for r in rows_for_logits:
            logits[:, r] = hf[:, r] @ lm.T
    return logits, new_k, new_v


def full_forward(weights: OracleWeights, seq_tokens: np.ndarray, visible: np.ndarray,
                 positions: np.ndarray | None = None, lora_rows: np.ndarray | None = None) -> np.ndarray:
    """Recompute every position from tokens with an explicit attention mask (no cache).

    seq_tokens: int [batch, T]; visible: bool [T, T] (row attends to column);
    lora_rows: optional bool [T], the rows that take the draft-pathway LoRA
    (the block rows of a draft pass).  Returns logits [batch, T, vocab].  This
    is the plain definition the cached block pass must reproduce.
    """
    s = weights.shape
    B, T = seq_tokens.shape
    G = s.n_q_heads // s.n_kv_heads
    if positions is None:
        positions = np.broadcast_to(np.arange(T), (B, T))
    x = weights.embed_rows(seq_tokens)
    for l in range(s.n_layers):
        w = weights.layer(l)
        h = rms_norm(x, w["attn_norm"], s.rms_eps)
        q = rope((h @ w["wq"].T).reshape(B, T, s.n_q_heads, s.head_dim), positions, s.rope_base)
        kk = rope((h @ w["wk"].T).reshape(B, T, s.n_kv_heads, s.head_dim), positions, s.rope_base)
        vv = (h @ w["wv"].T).reshape(B, T, s.n_kv_heads, s.head_dim)
        o = np.zeros((B, T, s.n_q_heads, s.head_dim), dtype=weights.dtype)
        for b in range(B):
            for hq in range(s.n_q_heads):
                g = hq // G
                o[b, :, hq] = softmax_attention(q[b, :, hq], kk[b, :, g], vv[b, :, g], visible)
        o2 = o.reshape(B, T, s.q_dim)
        x = x + o2 @ w["wo"].T
        if lora_rows is not None and "lora_a" in w:
            x = x + np.asarray(lora_rows)[None, :, None] * (lora_scale(s) * ((o2 @ w["lora_a"].T) @ w["lora_b"].T))
        h = rms_norm(x, w["ffn_norm"], s.rms_eps)
        x = x + (silu(h @ w["w_gate"].T) * (h @ w["w_up"].T)) @ w["w_down"].T
    return rms_norm(x, weights.final_norm(), s.rms_eps) @ weights.lm_head().T


def sequence_visibility(prefix_len: int, k: int, mode: str, bidir_from: int = 0) -> np.ndarray:
    """[T, T] mask for full_forward over prefix + block: causal prefix, block rows per mode."""
    T = prefix_len + k
    vis = np.tril(np.ones((T, T), dtype=bool))
    vis[prefix_len:] = block_visibility(prefix_len, k, mode, bidir_from)
    return vis


# ----------------------------------------------------------------------------- decoding steps
def accept(draft: np.ndarray, ar_pred: np.ndarray):
    """Longest-prefix acceptance with one bonus token, for one sequence.

    draft[j-1] = d_j (j = 1..k-1) are the draft tokens at positions P+1..P+k-1;
    ar_pred[j] = a_j is the AR prediction of verify row j, i.e. for position
    P+j+1.  With j* the first j where d_j != a_{j-1}, the accepted length is
    L = j* - 1, or k - 1 when no mismatch exists.  The committed tokens are
    d_1..d_L followed by the bonus a_L (the AR token at the first rejected
    position, or after the last draft).  Returns (L, committed list, bonus).
    """
    k = len(ar_pred)
    j_star = None
    for j in range(1, k):
        if draft[j - 1] != ar_pred[j - 1]:
            j_star = j
            break
    L = (k - 1) if j_star is None else j_star - 1
    bonus = int(ar_pred[L])
    committed = [int(t) for t in draft[:L]] + [bonus]
    return L, committed, bonus


def commit(kv: OracleKV, new_k, new_v, n_rows) -> None:
    """Append the first n_rows[b] block rows of every layer to the cache."""
    for b in range(kv.batch):
        p, n = int(kv.lengths[b]), int(n_rows[b])
        if p + n > kv.capacity:
            raise ValueError("cache capacity exceeded")
        for l in range(len(new_k)):
            kv.k[l][b, :, p:p + n] = new_k[l][b, :, :n]
            kv.v[l][b, :, p:p + n] = new_v[l][b, :, :n]
        kv.lengths[b] = p + n


def draft_block(anchor: np.ndarray, k: int, mask_id: int) -> np.ndarray:
    """[anchor, mask x (k-1)] per sequence."""
    blk = np.full((len(anchor), k), mask_id, dtype=np.int32)
    blk[:, 0] = anchor
    return blk


def verify_block(anchor: np.ndarray, drafts: np.ndarray) -> np.ndarray:
    """[anchor, d_1 .. d_{k-1}] per sequence."""
    return np.concatenate([np.asarray(anchor, dtype=np.int32)[:, None],
                           np.asarray(drafts, dtype=np.int32)], axis=1)


def draft_pass(weights, kv, anchor, k, bidir_from=0):
    """Diffusion draft: d_j = argmax of draft row j for j = 1..k-1.  Returns (drafts, logits)."""
    logits, _, _ = block_forward(weights, kv, draft_block(anchor, k, weights.shape.mask_token_id),
                                 DRAFT, bidir_from)
    return argmax_first(logits)[:, 1:], logits


def verify_pass(weights, kv, anchor, drafts):
    """AR verify over [anchor, drafts] with the causal mask.  Returns (a, logits, new_k, new_v)."""
    logits, nk, nv = block_forward(weights, kv, verify_block(anchor, drafts), VERIFY)
    return argmax_first(logits), logits, nk, nv


def self_spec_step(weights, kv, anchor, k, bidir_from=0):
    """One linear self-speculation step; commits accepted rows into ``kv``.

    Returns dict with drafts, verify argmax, accept lengths L, committed tokens
    (per sequence lists) and the next anchors.
    """
    drafts, dlogits = draft_pass(weights, kv, anchor, k, bidir_from)
    a, vlogits, nk, nv = verify_pass(weights, kv, anchor, drafts)
    Ls, committed, nxt = [], [], []
    for b in range(len(anchor)):
        L, c, bonus = accept(drafts[b], a[b])
        Ls.append(L)
        committed.append(c)
        nxt.append(bonus)
    commit(kv, nk, nv, np.asarray(Ls) + 1)
    return {"drafts": drafts, "ar": a, "L": np.asarray(Ls, dtype=np.int32), "committed": committed,
            "next_anchor": np.asarray(nxt, dtype=np.int32), "draft_logits": dlogits, "verify_logits": vlogits}


def ar_step(weights, kv, token):
    """Mode 1: one AR decoding step (a one-token verify pass) that commits its row."""
    logits, nk, nv = block_forward(weights, kv, np.asarray(token, dtype=np.int32)[:, None], VERIFY)
    commit(kv, nk, nv, np.ones(kv.batch, dtype=np.int64))
    return argmax_first(logits)[:, 0], logits


def prefill(weights, kv, prefix_tokens, chunk: int = 0):
    """Causal prefill of a token prefix into an empty cache (verify passes, all rows committed)."""
    prefix_tokens = np.asarray(prefix_tokens, dtype=np.int32)
    T = prefix_tokens.shape[1]
    chunk = chunk or T
    for c0 in range(0, T, chunk):
        blk = prefix_tokens[:, c0:c0 + chunk]
        _, nk, nv = block_forward(weights, kv, blk, VERIFY)
        commit(kv, nk, nv, np.full(kv.batch, blk.shape[1]))


# ----------------------------------------------------------------------------- Mode 2: diffusion denoising
# Block-wise diffusion decoding with confidence-based sampling (Sec. 3.2): a block
# starts as masks after the verified prefix, each denoising step is one draft pass
# over the block that commits some masked positions, and once no mask is left the
# block's K/V is refreshed and decoding moves to the next block.
#
# Readings (the paper names the procedure and cites its source for the details):
#
# * Block layout as in Mode 3: ``[anchor, r_1 .. r_{k-1}]`` with the anchor at
#   position P (its K/V not yet cached); r_j is a mask or a token committed by an
#   earlier step, and a step over the block denoises the masked r_j in place.
# * A masked position is denoised to the most probable token other than the mask
#   token itself (a mask is never a decoded value); its confidence is that token's
#   softmax probability over the same vocabulary (all tokens except the mask).
# * Commit rule: every masked position whose confidence exceeds the threshold
#   (strictly); when none does, the single most confident one (the lowest row
#   among equal confidences), so each step commits at least one position -- the
#   fallback the SOL construction of Sec. 4.1 also states for greedy acceptance.
# * Refresh: the clean stream is strictly causal (Sec. 2.2), so a completed block's
#   K/V is recomputed by a causal (verify-mode) pass over it.  Rows 0..k-2 (the
#   anchor and the first k-2 decoded tokens) are committed; the last decoded token
#   becomes the next block's anchor, as after a full acceptance in Mode 3.
def denoising_logits(logits: np.ndarray, mask_id: int) -> np.ndarray:
    """The logits over which a masked position is denoised: the mask token's own logit removed (-inf)."""
    z = np.array(logits, dtype=np.float64, copy=True)
    z[..., mask_id] = -np.inf
    return z


def top1_confidence(logits: np.ndarray) -> np.ndarray:
    """Softmax probability of the most probable token, float64: 1 / sum_v exp(z_v - max_v z_v).

    Entries at -inf take no part (probability 0)."""
    z = np.asarray(logits, dtype=np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return 1.0 / np.sum(np.exp(z - m), axis=-1)


def threshold_commit(block: np.ndarray, pred: np.ndarray, conf: np.ndarray, threshold: float, mask_id: int):
    """One denoising step's commit for one sequence.

    block: int [k] (row 0 the anchor, rows >= 1 a committed token or ``mask_id``);
    pred/conf: per-row denoised token and its confidence.  Returns (new block,
    sorted list of the rows committed by this step).
    """
    block = np.asarray(block)
    masked = [j for j in range(1, len(block)) if block[j] == mask_id]
    chosen = [j for j in masked if conf[j] > threshold]
    if masked and not chosen:
        best = masked[0]
        for j in masked[1:]:
            if conf[j] > conf[best]:
                best = j
        chosen = [best]
    out = block.copy()
    for j in chosen:
        out[j] = pred[j]
    return out, chosen


def denoise_step(weights, kv, block: np.ndarray, threshold: float, bidir_from: int = 0):
    """One denoising step for every sequence: a draft (bidirectional) pass over the current block, then
    the commit rule.  The cache is not modified.  Returns dict with the new block, committed rows per
    sequence, per-row prediction and confidence, and the pass's raw logits."""
    mask_id = weights.shape.mask_token_id
    block = np.asarray(block, dtype=np.int32)
    logits, _, _ = block_forward(weights, kv, block, DRAFT, bidir_from)
    z = denoising_logits(logits, mask_id)
    pred = argmax_first(z)
    conf = top1_confidence(z)
    new_block = block.copy()
    committed = []
    for b in range(block.shape[0]):
        new_block[b], rows = threshold_commit(block[b], pred[b], conf[b], threshold, mask_id)
        committed.append(rows)
    return {"block": new_block, "committed": committed, "pred": pred, "conf": conf, "logits": logits}


def refresh(weights, kv, block: np.ndarray) -> np.ndarray:
    """K/V refresh of completed blocks: a causal pass over ``block`` whose rows 0..k-2 are committed to
    ``kv``.  Returns the next anchors (the blocks' last tokens)."""
    block = np.asarray(block, dtype=np.int32)
    B, k = block.shape
    if np.any(block[:, 1:] == weights.shape.mask_token_id):
        raise ValueError("refresh of a block that still holds a mask")
    _, nk, nv = block_forward(weights, kv, block, VERIFY)
    commit(kv, nk, nv, np.full(B, k - 1))
    return block[:, k - 1].copy()


def diffusion_block(weights, kv, anchor, k: int, threshold: float, bidir_from: int = 0):
    """Mode 2 over one block per sequence: denoising steps until no mask is left, then the refresh.

    Returns (decoded block [batch, k], number of denoising steps, next anchors)."""
    block = draft_block(np.asarray(anchor), k, weights.shape.mask_token_id)
    steps = 0
    while np.any(block[:, 1:] == weights.shape.mask_token_id):
        block = denoise_step(weights, kv, block, threshold, bidir_from)["block"]
        steps += 1
    return block, steps, refresh(weights, kv, block)


# ----------------------------------------------------------------------------- quadratic self-speculation
# Quadratic self-speculation (Sec. 3.4, Appendix C): one forward pass verifies the
# previous step's speculative tokens causally, as Mode 3's verify pass does, and in
# the same pass drafts the next ones for every possible acceptance length (a group of
# mask tokens after each element of the verified chain, bidirectional within the
# group), with an optional AR-diffusion ensemble verifier.
#
# Readings (the appendix's indices do not close; these keep Mode 3's conventions):
#
# * The chain is Mode 3's verify block [anchor, s_1 .. s_{k-1}] (the anchor at
#   position P).  After chain element c (position P + c) come k mask tokens at
#   positions P + c + 1 .. P + c + k -- one group per chain element, so that fresh
#   drafts exist for every acceptance length 0 .. k-1.  Block rows: the chain first,
#   then mask r (1..k) of group c at row k + c*k + r - 1; k(k+1) rows in all.
# * Attention: every row sees the cached prefix; chain row c sees chain elements
#   0..c (causal); a mask of group c sees chain elements 0..c and every mask of its
#   own group (bidirectional within the group), nothing else.
# * Predictions: chain row c is AR (it predicts position P + c + 1); mask r of group
#   c predicts the token at its own position P + c + r, as Mode 3's draft rows do.
# * The verifier of the token at position P + i (i = 1..k) mixes the AR distribution
#   of chain row i - 1 with the diffusion distribution of mask 1 of group i - 1 (the
#   mask at that same position): lambda * p_AR + (1 - lambda) * p_diff; v_i is its
#   argmax (lowest index on ties).  lambda = 1 is plain AR verification.
# * Acceptance as in Mode 3: L = longest prefix of s_1..s_{k-1} with s_i = v_i.  The
#   chain rows 0..L (anchor and accepted tokens) are committed, the next anchor is
#   v_{L+1}, and the next speculative tokens are the argmax of masks 2..k of group L
#   (positions P + L + 2 .. P + L + k, right after the next anchor).
# * The LoRA adapter (a draft-pass feature) is not used by this pass.
# * The first step's speculative tokens come from a Mode 3 draft pass.
def quad_rows(k: int) -> int:
    """Block rows of a quadratic pass with chain length k: k chain rows + k groups of k masks."""
    return k * (k + 1)


def quad_layout(k: int):
    """Per block row: (position offset from P, group, is_chain).  Group of a chain row c is c."""
    off, grp, chain = [], [], []
    for c in range(k):
        off.append(c)
        grp.append(c)
        chain.append(True)
    for c in range(k):
        for r in range(1, k + 1):
            off.append(c + r)
            grp.append(c)
            chain.append(False)
    return np.asarray(off), np.asarray(grp), np.asarray(chain)


def quad_block_visibility(k: int) -> np.ndarray:
    """bool [R, R]: which block columns each block row of the quadratic layout sees."""
    off, grp, chain = quad_layout(k)
    R = quad_rows(k)
    vis = np.zeros((R, R), dtype=bool)
    for i in range(R):
        for j in range(R):
            if chain[j]:
                vis[i, j] = j <= grp[i]                        # chain columns 0..c (chain row c: causal)
            else:
                vis[i, j] = (not chain[i]) and grp[j] == grp[i]   # the own group's masks
    return vis


def quad_tokens(anchor: np.ndarray, spec: np.ndarray, k: int, mask_id: int) -> np.ndarray:
    """[anchor, s_1 .. s_{k-1}, mask x k^2] per sequence."""
    B = len(anchor)
    if np.shape(spec) != (B, k - 1):
        raise ValueError("spec must hold k-1 tokens per sequence")
    t = np.full((B, quad_rows(k)), mask_id, dtype=np.int32)
    t[:, :k] = verify_block(anchor, spec)
    return t


def quad_forward(weights, kv, anchor, spec, k):
    """The quadratic pass.  Returns (logits [B, R, V], new_k, new_v) with the block's rows in layout order."""
    off, _, _ = quad_layout(k)
    positions = kv.lengths[:, None] + off[None, :]
    return block_forward(weights, kv, quad_tokens(anchor, spec, k, weights.shape.mask_token_id), VERIFY,
                         positions=positions, block_vis=quad_block_visibility(k))


def softmax64(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - np.max(z, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def ensemble_argmax(ar_logits: np.ndarray, diff_logits: np.ndarray, lam: float) -> np.ndarray:
    """argmax of lambda * softmax(AR) + (1 - lambda) * softmax(diffusion) over the last axis (float64,
    first index of the maximum)."""
    p = lam * softmax64(ar_logits) + (1.0 - lam) * softmax64(diff_logits)
    return np.argmax(p, axis=-1).astype(np.int32)


def quad_verifier(logits: np.ndarray, k: int, lam: float) -> np.ndarray:
    """v [B, k]: v[:, i-1] is the verifier's token for position P + i, i = 1..k."""
    ar = logits[:, 0:k]                                 # chain rows 0..k-1
    diff = logits[:, [k + c * k for c in range(k)]]     # mask 1 of groups 0..k-1
    return ensemble_argmax(ar, diff, lam)


def quad_step(weights, kv, anchor, spec, k: int, lam: float = 1.0):
    """One quadratic self-speculation step; commits the accepted chain rows into ``kv``.

    spec: int [B, k-1], the previous step's speculative tokens.  Returns dict with the logits,
    verifier tokens v, accept lengths L, committed tokens, next anchors and next speculative tokens."""
    anchor = np.asarray(anchor, dtype=np.int32)
    spec = np.asarray(spec, dtype=np.int32)
    logits, nk, nv = quad_forward(weights, kv, anchor, spec, k)
    v = quad_verifier(logits, k, lam)
    am = argmax_first(logits)
    Ls, committed, nxt, nspec = [], [], [], []
    for b in range(len(anchor)):
        L, c, bonus = accept(spec[b], v[b])
        Ls.append(L)
        committed.append(c)
        nxt.append(bonus)
        nspec.append(am[b, [k + L * k + r - 1 for r in range(2, k + 1)]])
    commit(kv, nk, nv, np.asarray(Ls) + 1)
    return {"logits": logits, "v": v, "L": np.asarray(Ls, dtype=np.int32), "committed": committed,
            "next_anchor": np.asarray(nxt, dtype=np.int32), "next_spec": np.asarray(nspec, dtype=np.int32).reshape(len(anchor), k - 1)}
