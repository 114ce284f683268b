"""Pins of the CPU oracle against what the paper and mathematics fix (no GPU).

Each test names the invariant it pins.  A plausible mistake in the oracle
(wrong mask, wrong RoPE pairing or position, transposed weight, wrong GQA
grouping, off-by-one in acceptance) fails at least one of them.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import nld_oracle as O
from synth.workloads import LazyWeights, ModelShape, SHAPE_TINY, tokens as synth_tokens

# a small decoder for fast pins: 2 layers, GQA group 2, odd vocab
MINI = ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96, vocab=97)


def mini_weights(dtype=np.float64, seed=11, shape=MINI):
    return O.OracleWeights(shape, LazyWeights(shape, seed), dtype)


def prefilled(w, prefix_tokens, capacity=None):
    kv = O.OracleKV(w.shape, prefix_tokens.shape[0], capacity or prefix_tokens.shape[1] + 40, w.dtype)
    O.prefill(w, kv, prefix_tokens)
    return kv


def rel(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


# ----------------------------------------------------------------------------- elementary closed forms
def test_rope_hand_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "rope_d4_pos1.json")))
    x = np.array(g["x"], dtype=np.float64).reshape(1, 1, 4)
    out = O.rope(x, np.array([g["position"]]), g["base"]).reshape(-1)
    np.testing.assert_allclose(out, g["expected"], rtol=0, atol=1e-15)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 2, 16))
    np.testing.assert_array_equal(O.rope(x, np.zeros(3, dtype=int), 1e4), x)        # position 0 = identity
    r = O.rope(x, np.array([5, 900, 70000]), 1e4)
    np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # <rope(q, m), rope(k, n)> depends only on m - n
    q, k = rng.standard_normal((1, 1, 16)), rng.standard_normal((1, 1, 16))
    d1 = np.sum(O.rope(q, np.array([17]), 1e4) * O.rope(k, np.array([5]), 1e4))
    d2 = np.sum(O.rope(q, np.array([1012]), 1e4) * O.rope(k, np.array([1000]), 1e4))
    assert abs(d1 - d2) < 1e-11


def test_rmsnorm_and_swiglu_closed_forms():
    c = np.full((1, 8), 3.0)
    np.testing.assert_allclose(O.rms_norm(c, np.full(8, 2.0), 1e-6), 2 * 3 / np.sqrt(9 + 1e-6), rtol=1e-15)
    np.testing.assert_allclose(O.rms_norm(np.array([[3.0, 4.0]]), np.ones(2), 0.0),
                               [[3 / np.sqrt(12.5), 4 / np.sqrt(12.5)]], rtol=1e-15)
    assert O.silu(np.array(0.0)) == 0.0
    np.testing.assert_allclose(O.silu(np.array([40.0, -40.0, 1.0])), [40.0, 0.0, 1 / (1 + np.exp(-1))], atol=1e-15)


def test_attention_closed_forms():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((6, 4))
    keys = np.tile(rng.standard_normal((1, 4)), (6, 1))            # all keys equal -> uniform weights
    q = rng.standard_normal((3, 4))
    vis = O.block_visibility(3, 3, O.VERIFY)                         # rows see 4, 5, 6 keys
    out = O.softmax_attention(q, keys, v, vis)
    for j in range(3):
        np.testing.assert_allclose(out[j], v[:4 + j].mean(axis=0), rtol=1e-13)
    vis1 = np.zeros((3, 6), dtype=bool)
    vis1[:, 2] = True                                                # one visible key -> its value
    np.testing.assert_allclose(O.softmax_attention(q, rng.standard_normal((6, 4)), v, vis1), np.tile(v[2], (3, 1)))


def test_block_visibility_patterns():
    v = O.block_visibility(2, 3, O.VERIFY)
    assert v.tolist() == [[1, 1, 1, 0, 0], [1, 1, 1, 1, 0], [1, 1, 1, 1, 1]]
    assert O.block_visibility(2, 3, O.DRAFT).all()
    d1 = O.block_visibility(2, 3, O.DRAFT, bidir_from=1)
    assert d1.tolist() == [[1, 1, 1, 0, 0], [1, 1, 1, 1, 1], [1, 1, 1, 1, 1]]


def test_argmax_ties_and_signed_zero():
    assert O.argmax_first(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert O.argmax_first(np.array([-0.0, 0.0])) == 0
    assert O.argmax_first(np.array([0.0, -0.0])) == 0
    assert O.argmax_first(np.array([-1.0, -0.0, 0.0, -2.0])) == 1
    assert O.argmax_first(np.full(7, 0.25)) == 0


# ----------------------------------------------------------------------------- acceptance rule
def test_accept_hand_examples(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "accept_examples.json")))
    for c in g["cases"]:
        L, committed, bonus = O.accept(np.array(c["draft"], dtype=int), np.array(c["ar"], dtype=int))
        assert L == c["L"] and committed == c["committed"] and bonus == c["committed"][-1], c


@pytest.mark.parametrize("V,k", [(2, 1), (2, 2), (2, 4), (3, 3), (3, 4), (4, 3)])
def test_accept_exhaustive_brute_force(V, k):
    """Every (draft, AR) pair over a tiny vocabulary: L is the longest matching prefix."""
    for draft in itertools.product(range(V), repeat=k - 1):
        for ar in itertools.product(range(V), repeat=k):
            L, committed, bonus = O.accept(np.array(draft, dtype=int), np.array(ar, dtype=int))
            longest = max(l for l in range(k) if list(draft[:l]) == list(ar[:l]))
            assert L == longest
            assert committed == list(draft[:L]) + [ar[L]] and bonus == ar[L]
            assert 1 <= len(committed) <= k


# ----------------------------------------------------------------------------- the block pass
@pytest.fixture(scope="module")
def mini():
    w = mini_weights()
    prefix = synth_tokens(MINI, 5, "pin.prefix", (2, 13))
    block = synth_tokens(MINI, 5, "pin.block", (2, 6))
    return w, prefix, block


def test_verify_k1_equals_ar_full_recompute(mini):
    """P1: a one-token verify pass over the cache equals plain causal decoding recomputed from tokens."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    logits, _, _ = O.block_forward(w, kv, block[:, :1], O.VERIFY)
    seq = np.concatenate([prefix, block[:, :1]], axis=1)
    full = O.full_forward(w, seq, np.tril(np.ones((14, 14), dtype=bool)))
    np.testing.assert_allclose(logits[:, 0], full[:, -1], rtol=1e-10, atol=1e-12)


def test_verify_equals_sequential_ar_steps(mini):
    """P2: one causal verify pass over k tokens equals k teacher-forced one-token steps (logits and K/V)."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    logits, nk, nv = O.block_forward(w, kv, block, O.VERIFY)
    kv2 = kv.copy()
    for j in range(block.shape[1]):
        _, lj = O.ar_step(w, kv2, block[:, j])
        np.testing.assert_allclose(logits[:, j], lj[:, 0], rtol=1e-10, atol=1e-12)
    P = prefix.shape[1]
    for l in range(MINI.n_layers):
        np.testing.assert_allclose(kv2.k[l][:, :, P:P + 6], nk[l], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(kv2.v[l][:, :, P:P + 6], nv[l], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("bidir_from", [0, 1, 3])
def test_draft_equals_full_attention(mini, bidir_from):
    """P3: the draft pass equals full recompute over [prefix ; block] with the block rows bidirectional."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    logits, _, _ = O.block_forward(w, kv, block, O.DRAFT, bidir_from)
    seq = np.concatenate([prefix, block], axis=1)
    full = O.full_forward(w, seq, O.sequence_visibility(13, 6, O.DRAFT, bidir_from))
    np.testing.assert_allclose(logits, full[:, 13:], rtol=1e-10, atol=1e-12)
    causal = O.full_forward(w, seq, O.sequence_visibility(13, 6, O.VERIFY))
    assert rel(full[:, 13:], causal[:, 13:]) > 1e-3          # the masks really differ


def test_draft_mask_degenerate_cases(mini):
    """P4: draft with k=1, or with bidir_from=k, is exactly the verify pass."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    a = O.block_forward(w, kv, block[:, :1], O.DRAFT)[0]
    b = O.block_forward(w, kv, block[:, :1], O.VERIFY)[0]
    np.testing.assert_array_equal(a, b)
    a = O.block_forward(w, kv, block, O.DRAFT, bidir_from=6)[0]
    b = O.block_forward(w, kv, block, O.VERIFY)[0]
    np.testing.assert_array_equal(a, b)


def test_verify_rows_ignore_later_rows(mini):
    """P5: verify row i does not depend on block tokens at rows > i (causality)."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    base = O.block_forward(w, kv, block, O.VERIFY)[0]
    changed = block.copy()
    changed[:, 4:] = (changed[:, 4:] + 7) % (MINI.vocab - 1)
    alt = O.block_forward(w, kv, changed, O.VERIFY)[0]
    np.testing.assert_allclose(alt[:, :4], base[:, :4], rtol=1e-12, atol=1e-13)
    assert rel(alt[:, 4:], base[:, 4:]) > 1e-3
    alt_d = O.block_forward(w, kv, changed, O.DRAFT)[0]
    base_d = O.block_forward(w, kv, block, O.DRAFT)[0]
    assert rel(alt_d[:, :4], base_d[:, :4]) > 1e-4            # the draft rows do see later rows


def test_draft_permutation_equivariance(mini):
    """P6: permuting block tokens together with their positions permutes the draft rows."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    P = prefix.shape[1]
    pos = P + np.arange(6)[None, :].repeat(2, axis=0)
    perm = np.array([3, 0, 5, 1, 4, 2])
    base = O.block_forward(w, kv, block, O.DRAFT, positions=pos)[0]
    alt = O.block_forward(w, kv, block[:, perm], O.DRAFT, positions=pos[:, perm])[0]
    np.testing.assert_allclose(alt, base[:, perm], rtol=1e-10, atol=1e-12)


def test_position_shift_invariance():
    """P7: shifting every position of prefix and block by a constant leaves the logits unchanged."""
    w = mini_weights()
    seq = synth_tokens(MINI, 6, "pin.shift", (1, 10))
    vis = O.sequence_visibility(7, 3, O.DRAFT)
    a = O.full_forward(w, seq, vis, positions=np.arange(10)[None])
    b = O.full_forward(w, seq, vis, positions=1000 + np.arange(10)[None])
    np.testing.assert_allclose(a, b, rtol=1e-8, atol=1e-10)


def test_gqa_equals_mha_with_replicated_kv_heads(mini):
    """GQA grouping: query head h reads KV head h // (Hq/Hkv); equal to MHA with replicated K/V projections."""
    w, prefix, block = mini
    mha_shape = ModelShape(**{**MINI.__dict__, "n_kv_heads": MINI.n_q_heads})

    class Replicated:
        def __init__(self, src):
            self.src = src
            self.embed, self.lm_head, self.final_norm = src.embed, src.lm_head, src.final_norm

        def layer(self, l):
            d = dict(self.src.layer(l))
            G, D = MINI.n_q_heads // MINI.n_kv_heads, MINI.head_dim
            for name in ("wk", "wv"):
                heads = d[name].reshape(MINI.n_kv_heads, D, MINI.hidden)
                d[name] = np.repeat(heads, G, axis=0).reshape(-1, MINI.hidden)
            return d

    wm = O.OracleWeights(mha_shape, Replicated(LazyWeights(MINI, 11)), np.float64)
    seq = np.concatenate([prefix, block], axis=1)
    vis = O.sequence_visibility(13, 6, O.VERIFY)
    np.testing.assert_allclose(O.full_forward(w, seq, vis), O.full_forward(wm, seq, vis), rtol=1e-10, atol=1e-12)


def _torch_reference_logits(shape, src, seq, visible):
    """The same decoder written with PyTorch library routines (F.linear's [out][in] weights, F.rms_norm,
    scaled_dot_product_attention with an explicit mask, F.silu) and RoPE as a complex rotation."""
    def t(bits):
        return torch.from_numpy(O.bf16_bits_to_float(bits, np.float64))

    T = seq.shape[1]
    D, half = shape.head_dim, shape.head_dim // 2
    inv = torch.tensor([shape.rope_base ** (-2.0 * i / D) for i in range(half)], dtype=torch.float64)
    rot = torch.polar(torch.ones(T, half, dtype=torch.float64), torch.arange(T, dtype=torch.float64)[:, None] * inv)

    def rope_c(x):                                   # x [B, T, H, D]; pair (i, i+D/2) as one complex number
        z = torch.complex(x[..., :half], x[..., half:]) * rot[None, :, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    x = t(src.embed)[torch.from_numpy(seq.astype(np.int64))]
    mask = torch.from_numpy(visible)
    G = shape.n_q_heads // shape.n_kv_heads
    for l in range(shape.n_layers):
        w = {k: t(v) for k, v in src.layer(l).items()}
        h = F.rms_norm(x, (shape.hidden,), w["attn_norm"], eps=shape.rms_eps)
        B = x.shape[0]
        q = rope_c(F.linear(h, w["wq"]).view(B, T, shape.n_q_heads, D)).transpose(1, 2)
        k = rope_c(F.linear(h, w["wk"]).view(B, T, shape.n_kv_heads, D)).transpose(1, 2)
        v = F.linear(h, w["wv"]).view(B, T, shape.n_kv_heads, D).transpose(1, 2)
        k = k.repeat_interleave(G, dim=1)
        v = v.repeat_interleave(G, dim=1)
        o = F.scaled_dot_product_attention(q, k, v, attn_mask=mask).transpose(1, 2).reshape(B, T, -1)
        x = x + F.linear(o, w["wo"])
        h = F.rms_norm(x, (shape.hidden,), w["ffn_norm"], eps=shape.rms_eps)
        x = x + F.linear(F.silu(F.linear(h, w["w_gate"])) * F.linear(h, w["w_up"]), w["w_down"])
    x = F.rms_norm(x, (shape.hidden,), t(src.final_norm), eps=shape.rms_eps)
    return F.linear(x, t(src.lm_head)).numpy()


@pytest.mark.parametrize("mode", [O.VERIFY, O.DRAFT])
def test_block_pass_matches_torch_library_decoder(mini, mode):
    """The cached block pass equals the decoder built from PyTorch library layers (weight layout,
    norm placement, SwiGLU, GQA and attention masking)."""
    w, prefix, block = mini
    kv = prefilled(w, prefix)
    logits = O.block_forward(w, kv, block, mode)[0]
    seq = np.concatenate([prefix, block], axis=1)
    ref = _torch_reference_logits(MINI, LazyWeights(MINI, 11), seq, O.sequence_visibility(13, 6, mode))
    np.testing.assert_allclose(logits, ref[:, 13:], rtol=1e-9, atol=1e-11)


class _GainSwap:
    """Weights of `src` with RMSNorm gain vectors moved: 'swap<l>' exchanges layer l's attention and FFN
    gains, 'final<-attn1' puts layer 1's attention gain at the final norm, 'attn1<-attn0' repeats layer
    0's attention gain in layer 1."""

    def __init__(self, src, kind):
        self.src, self.kind = src, kind
        self.embed, self.lm_head = src.embed, src.lm_head
        self.final_norm = src.layer(1)["attn_norm"] if kind == "final<-attn1" else src.final_norm

    def layer(self, l):
        d = dict(self.src.layer(l))
        if self.kind == "swap%d" % l:
            d["attn_norm"], d["ffn_norm"] = d["ffn_norm"], d["attn_norm"]
        if self.kind == "attn1<-attn0" and l == 1:
            d["attn_norm"] = self.src.layer(0)["attn_norm"]
        return d


@pytest.mark.parametrize("kind", ["swap0", "swap1", "final<-attn1", "attn1<-attn0"])
def test_misplaced_gain_moves_logits_beyond_the_tolerance(kind):
    """The workloads draw every RMSNorm gain vector separately (bf16(1 + 0.1 z)), so a gain used at the
    wrong place changes the tiny workload's logits by more than five times the 2e-2 parity tolerance:
    a GPU path with such a mistake cannot pass the parity tests."""
    src = LazyWeights(SHAPE_TINY, 0)
    prefix = synth_tokens(SHAPE_TINY, 0, "tiny.prefix", (1, 128))
    block = synth_tokens(SHAPE_TINY, 0, "tiny.block", (1, 8))
    outs = []
    for s in (src, _GainSwap(src, kind)):
        w = O.OracleWeights(SHAPE_TINY, s, np.float64)
        kv = O.OracleKV(SHAPE_TINY, 1, 256, np.float64)
        O.prefill(w, kv, prefix)
        outs.append(O.block_forward(w, kv, block, O.VERIFY)[0])
    assert rel(outs[1], outs[0]) > 5 * 2e-2


def test_fp32_oracle_close_to_fp64():
    """P13: on the tiny workload the float32 oracle is within 1e-4 (normwise) of the float64 one."""
    src = LazyWeights(SHAPE_TINY, 0)
    prefix = synth_tokens(SHAPE_TINY, 0, "pin.p13.prefix", (1, 32))
    block = synth_tokens(SHAPE_TINY, 0, "pin.p13.block", (1, 8))
    outs = []
    for dt in (np.float32, np.float64):
        w = O.OracleWeights(SHAPE_TINY, src, dt)
        kv = prefilled(w, prefix)
        outs.append(O.block_forward(w, kv, block, O.DRAFT)[0])
    assert rel(outs[0].astype(np.float64), outs[1]) < 1e-4


# ----------------------------------------------------------------------------- decoding loop
def test_self_speculation_reproduces_greedy_ar():
    """Greedy verification makes self-speculation commit exactly the greedy AR continuation, and the
    cache it builds equals the one AR decoding builds (only accepted rows are committed)."""
    w = mini_weights()
    prefix = synth_tokens(MINI, 9, "pin.ss.prefix", (2, 9))
    k, steps = 5, 4
    kv_ss = prefilled(w, prefix[:, :-1], capacity=64)
    kv_ar = kv_ss.copy()
    anchor = prefix[:, -1].copy()
    out_ss = [[] for _ in range(2)]
    for _ in range(steps):
        r = O.self_spec_step(w, kv_ss, anchor, k)
        for b in range(2):
            assert 0 <= r["L"][b] <= k - 1
            out_ss[b] += r["committed"][b]
        anchor = r["next_anchor"]
    n = min(len(o) for o in out_ss)
    tok = prefix[:, -1].copy()
    out_ar = [[] for _ in range(2)]
    for _ in range(n):
        tok, _ = O.ar_step(w, kv_ar, tok)
        for b in range(2):
            out_ar[b].append(int(tok[b]))
    for b in range(2):
        assert out_ss[b][:n] == out_ar[b]


def test_planted_drafts_are_fully_accepted():
    """Drafts equal to the greedy AR continuation are accepted in full (L = k-1), the bonus is the next
    AR token, and the committed cache rows equal those of AR decoding."""
    w = mini_weights()
    prefix = synth_tokens(MINI, 10, "pin.plant.prefix", (1, 9))
    k = 6
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    kv_ar = kv.copy()
    tok, greedy = prefix[:, -1].copy(), []
    for _ in range(k):
        tok, _ = O.ar_step(w, kv_ar, tok)
        greedy.append(int(tok[0]))
    a, _, nk, nv = O.verify_pass(w, kv, prefix[:, -1], np.array([greedy[:k - 1]]))
    L, committed, bonus = O.accept(np.array(greedy[:k - 1]), a[0])
    assert L == k - 1 and committed == greedy and bonus == greedy[-1]
    O.commit(kv, nk, nv, [L + 1])
    for l in range(MINI.n_layers):
        np.testing.assert_allclose(kv.k[l][:, :, :int(kv.lengths[0])], kv_ar.k[l][:, :, :int(kv.lengths[0])],
                                   rtol=1e-10, atol=1e-12)


def test_chunked_prefill_equals_single_pass():
    w = mini_weights()
    prefix = synth_tokens(MINI, 12, "pin.chunk", (1, 20))
    a = prefilled(w, prefix)
    b = O.OracleKV(MINI, 1, 60, np.float64)
    O.prefill(w, b, prefix, chunk=7)
    for l in range(MINI.n_layers):
        np.testing.assert_allclose(a.k[l], b.k[l], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(a.v[l], b.v[l], rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------------- Mode 2: diffusion denoising
def test_top1_confidence_closed_forms():
    """Confidence is the softmax probability of the top token: 1/V for equal logits, 3/4 for logits
    (log 3, 0), 1/2 for two equal maxima with the rest excluded, invariant to a shift, and equal to the
    maximum of torch's softmax on random rows."""
    V = 97
    np.testing.assert_allclose(O.top1_confidence(np.zeros((2, V))), 1.0 / V, rtol=1e-15)
    np.testing.assert_allclose(O.top1_confidence(np.array([np.log(3.0), 0.0])), 0.75, rtol=1e-15)
    z = np.full(V, -np.inf)
    z[[4, 60]] = 1.5
    np.testing.assert_allclose(O.top1_confidence(z), 0.5, rtol=1e-15)
    rng = np.random.default_rng(3)
    r = rng.standard_normal((5, V)) * 4
    np.testing.assert_allclose(O.top1_confidence(r + 123.25), O.top1_confidence(r), rtol=1e-13)
    lib = torch.softmax(torch.from_numpy(r), dim=-1).max(dim=-1).values.numpy()
    np.testing.assert_allclose(O.top1_confidence(r), lib, rtol=1e-13)


def test_denoising_never_decodes_the_mask_token():
    """With the mask token's logit the largest of its row, the denoised token is the best other token and
    its confidence is the softmax over the vocabulary without the mask token (torch on the reduced row)."""
    V, mask_id = 50, 49
    rng = np.random.default_rng(4)
    r = rng.standard_normal((3, V))
    r[:, mask_id] = 10.0
    z = O.denoising_logits(r, mask_id)
    assert np.all(O.argmax_first(z) == np.argmax(r[:, :mask_id], axis=-1))
    lib = torch.softmax(torch.from_numpy(r[:, :mask_id]), dim=-1).max(dim=-1).values.numpy()
    np.testing.assert_allclose(O.top1_confidence(z), lib, rtol=1e-13)


@pytest.mark.parametrize("threshold", [-1.0, 0.0, 0.3, 0.5, 0.7, 0.95, 1.0])
def test_threshold_commit_exhaustive(threshold):
    """Every mask pattern of a k=5 block and every assignment of confidences from a small set (ties
    included): the committed rows are exactly the masked rows above the threshold, or else the first of
    the most confident masked rows; other rows and the anchor keep their tokens."""
    M = 99
    levels = [0.1, 0.5, 0.9]
    for pattern in itertools.product([False, True], repeat=4):
        block = np.array([7] + [M if m else 20 + j for j, m in enumerate(pattern)])
        pred = np.array([0, 31, 32, 33, 34])
        for cs in itertools.product(levels, repeat=4):
            conf = np.array([0.0] + list(cs))
            out, rows = O.threshold_commit(block, pred, conf, threshold, M)
            masked = [j for j in range(1, 5) if pattern[j - 1]]
            above = [j for j in masked if conf[j] > threshold]
            if above:
                assert rows == above
            elif masked:
                top = max(conf[j] for j in masked)
                assert rows == [min(j for j in masked if conf[j] == top)]
            else:
                assert rows == []
            for j in range(5):
                assert out[j] == (pred[j] if j in rows else block[j])


def test_threshold_commit_monotone_in_threshold():
    """A lower threshold commits a superset of the rows a higher one commits (when both commit by
    threshold), and a threshold of 1 or more commits exactly one row per step."""
    rng = np.random.default_rng(5)
    M = 1000
    for _ in range(200):
        k = int(rng.integers(2, 12))
        block = np.where(rng.random(k) < 0.7, M, 5)
        block[0] = 3
        conf = rng.random(k)
        pred = rng.integers(0, M, k)
        hi_rows = O.threshold_commit(block, pred, conf, 0.8, M)[1]
        lo_rows = O.threshold_commit(block, pred, conf, 0.4, M)[1]
        if any(conf[j] > 0.8 for j in hi_rows):
            assert set(hi_rows) <= set(lo_rows)
        n_masked = int(np.sum(block[1:] == M))
        assert len(O.threshold_commit(block, pred, conf, 1.0, M)[1]) == min(1, n_masked)


@pytest.fixture(scope="module")
def mode2():
    w = mini_weights()
    prefix = synth_tokens(MINI, 14, "pin.m2.prefix", (2, 11))
    return w, prefix


def test_diffusion_threshold_below_zero_is_one_draft_pass(mode2):
    """With every confidence above the threshold the block is decoded in one step, to the argmax (mask
    token excluded) of one draft pass over [anchor, masks] -- the Mode 3 draft pass."""
    w, prefix = mode2
    k = 6
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    logits, _, _ = O.block_forward(w, kv, O.draft_block(prefix[:, -1], k, MINI.mask_token_id), O.DRAFT)
    expect = np.argmax(np.where(np.arange(MINI.vocab) == MINI.mask_token_id, -np.inf, logits), axis=-1)[:, 1:]
    block, steps, nxt = O.diffusion_block(w, kv, prefix[:, -1], k, threshold=-1.0)
    assert steps == 1
    np.testing.assert_array_equal(block[:, 1:], expect)
    np.testing.assert_array_equal(block[:, 0], prefix[:, -1])
    np.testing.assert_array_equal(nxt, block[:, -1])


def test_diffusion_threshold_one_decodes_one_token_per_step(mode2):
    """A threshold no probability exceeds gives one commit per step (k-1 steps), each the most confident
    remaining mask -- decoding one token at a time in confidence order."""
    w, prefix = mode2
    k = 5
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    block = O.draft_block(prefix[:, -1], k, MINI.mask_token_id)
    for step in range(k - 1):
        r = O.denoise_step(w, kv, block, threshold=1.0)
        for b in range(2):
            assert len(r["committed"][b]) == 1
            j = r["committed"][b][0]
            masked = [i for i in range(1, k) if block[b, i] == MINI.mask_token_id]
            assert j in masked and r["conf"][b, j] == max(r["conf"][b, i] for i in masked)
        block = r["block"]
    assert not np.any(block == MINI.mask_token_id)
    assert np.all(kv.lengths == prefix.shape[1] - 1)            # denoising never writes the cache


@pytest.mark.parametrize("threshold", [0.02, 0.05, 0.2])
def test_diffusion_refresh_equals_causal_recompute(mode2, threshold):
    """After a block is decoded and refreshed the cache holds P + k - 1 rows, the next anchor is the
    block's last token, and an AR step from it equals plain causal decoding recomputed from all tokens
    (no cache).  Any threshold finishes the block in at most k - 1 steps."""
    w, prefix = mode2
    k = 6
    P = prefix.shape[1] - 1
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    block, steps, nxt = O.diffusion_block(w, kv, prefix[:, -1], k, threshold)
    assert 1 <= steps <= k - 1
    assert np.all(kv.lengths == P + k - 1)
    np.testing.assert_array_equal(nxt, block[:, -1])
    tok_ar, logits_ar = O.ar_step(w, kv, nxt)
    seq = np.concatenate([prefix[:, :-1], block], axis=1)
    T = seq.shape[1]
    full = O.full_forward(w, seq, np.tril(np.ones((T, T), dtype=bool)))
    np.testing.assert_allclose(logits_ar[:, 0], full[:, -1], rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(tok_ar, O.argmax_first(full[:, -1]))


def test_refresh_rejects_an_incomplete_block(mode2):
    w, prefix = mode2
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    with pytest.raises(ValueError):
        O.refresh(w, kv, O.draft_block(prefix[:, -1], 4, MINI.mask_token_id))


# ----------------------------------------------------------------------------- LoRA-enhanced drafter
MINI_LORA = ModelShape(**{**MINI.__dict__, "lora_rank": 8, "lora_alpha": 32.0})


class _MergedLoRA(O.OracleWeights):
    """The same model with each adapter merged into the O projection, W_o + (alpha/r) B A (float64)."""

    def layer(self, l):
        w = super().layer(l)
        w["wo"] = w["wo"] + (self.shape.lora_alpha / self.shape.lora_rank) * (w.pop("lora_b") @ w.pop("lora_a"))
        return w


@pytest.fixture(scope="module")
def lora_mini():
    w = O.OracleWeights(MINI_LORA, LazyWeights(MINI_LORA, 11), np.float64)
    base = mini_weights()            # same seed and names: the same base weights without the adapter
    prefix = synth_tokens(MINI, 15, "pin.lora.prefix", (2, 12))
    block = synth_tokens(MINI, 15, "pin.lora.block", (2, 6))
    return w, base, prefix, block


def test_lora_leaves_the_verify_pass_unchanged(lora_mini):
    """The adapter belongs to the diffusion pathway only: verify logits and K/V equal the base model's."""
    w, base, prefix, block = lora_mini
    a = O.block_forward(w, prefilled(w, prefix), block, O.VERIFY)
    b = O.block_forward(base, prefilled(base, prefix), block, O.VERIFY)
    np.testing.assert_array_equal(a[0], b[0])
    for l in range(MINI.n_layers):
        np.testing.assert_array_equal(a[1][l], b[1][l])


def test_lora_draft_equals_merged_weights(lora_mini):
    """A draft pass with the adapter equals a draft pass whose O projection is W_o + (alpha/r) B A (the
    adapter merged into the weight), and differs from the base model's draft."""
    w, base, prefix, block = lora_mini
    merged = _MergedLoRA(MINI_LORA, LazyWeights(MINI_LORA, 11), np.float64)
    kv = prefilled(base, prefix)               # the prefix cache is AR-pathway: the same for all three
    got = O.block_forward(w, kv, block, O.DRAFT)[0]
    ref = O.block_forward(merged, kv, block, O.DRAFT)[0]
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)
    assert rel(O.block_forward(base, kv, block, O.DRAFT)[0], ref) > 1e-3


def test_lora_draft_equals_full_recompute(lora_mini):
    """The cached draft pass with the adapter equals full recompute over [prefix; block] where only the
    block rows take the adapter and the block is bidirectional."""
    w, base, prefix, block = lora_mini
    kv = prefilled(base, prefix)
    got = O.block_forward(w, kv, block, O.DRAFT)[0]
    P, k = prefix.shape[1], block.shape[1]
    seq = np.concatenate([prefix, block], axis=1)
    full = O.full_forward(w, seq, O.sequence_visibility(P, k, O.DRAFT), lora_rows=np.arange(P + k) >= P)
    np.testing.assert_allclose(got, full[:, P:], rtol=1e-10, atol=1e-12)


class _LowRankO(O.OracleWeights):
    """MINI_LORA with a rank-r output projection W_o = B0 A0 in every layer and, with `cancel`, the adapter
    A = A0, B = -(r / alpha) B0; without it, no adapter and W_o = 0 (float64)."""

    def __init__(self, cancel):
        super().__init__(MINI_LORA, LazyWeights(MINI_LORA, 11), np.float64)
        self.cancel = cancel

    def layer(self, l):
        w = super().layer(l)
        s, r = self.shape, self.shape.lora_rank
        a0 = 0.02 * synth.normal_f64(11, "pin.lowrank.a%d" % l, (r, s.q_dim))
        b0 = 0.35 * synth.normal_f64(11, "pin.lowrank.b%d" % l, (s.hidden, r))
        del w["lora_a"], w["lora_b"]
        if self.cancel:
            w["wo"] = b0 @ a0
            w["lora_a"], w["lora_b"] = a0, -(r / s.lora_alpha) * b0
        else:
            w["wo"] = np.zeros_like(w["wo"])
        return w


def test_lora_scale_cancels_a_low_rank_output_projection(lora_mini):
    """Pins the adapter's output scale alpha/r (Sec. 3.3: rank 128 with alpha 512) by a closed form rather
    than by restating it: with a rank-r O projection W_o = B0 A0 and the adapter A = A0, B = -(r/alpha) B0,
    the draft pathway's projection W_o + scale * B A vanishes exactly when scale = alpha/r, so the draft
    pass equals that of the model with W_o = 0; the verify pass keeps W_o and differs from it."""
    _, base, prefix, block = lora_mini
    kv = prefilled(base, prefix)
    cancel, zero = _LowRankO(True), _LowRankO(False)
    d_cancel = O.block_forward(cancel, kv, block, O.DRAFT)[0]
    d_zero = O.block_forward(zero, kv, block, O.DRAFT)[0]
    np.testing.assert_allclose(d_cancel, d_zero, rtol=1e-9, atol=1e-11)
    assert rel(O.block_forward(cancel, kv, block, O.VERIFY)[0], O.block_forward(zero, kv, block, O.VERIFY)[0]) > 1e-3


# ----------------------------------------------------------------------------- quadratic self-speculation
def test_quad_layout_hand_example():
    """The quadratic layout for chain length k = 2 (Sec. 3.4, Appendix C, in this build's reading):
    rows [anchor, s_1, g0.m1, g0.m2, g1.m1, g1.m2] at offsets [0, 1, 1, 2, 2, 3] from P; chain rows are
    causal, a mask sees the chain up to its group's element and its own group."""
    off, grp, chain = O.quad_layout(2)
    assert O.quad_rows(2) == 6
    assert off.tolist() == [0, 1, 1, 2, 2, 3]
    assert grp.tolist() == [0, 1, 0, 0, 1, 1]
    assert chain.tolist() == [True, True, False, False, False, False]
    expected = np.array([[1, 0, 0, 0, 0, 0],
                         [1, 1, 0, 0, 0, 0],
                         [1, 0, 1, 1, 0, 0],
                         [1, 0, 1, 1, 0, 0],
                         [1, 1, 0, 0, 1, 1],
                         [1, 1, 0, 0, 1, 1]], dtype=bool)
    np.testing.assert_array_equal(O.quad_block_visibility(2), expected)


@pytest.fixture(scope="module")
def quad_mini():
    w = mini_weights(seed=13)
    prefix = synth_tokens(MINI, 13, "pin.quad.prefix", (2, 11))
    spec = synth_tokens(MINI, 13, "pin.quad.spec", (2, 3))
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    return w, kv, prefix[:, -1].copy(), spec, prefix[:, :-1]


def test_quad_chain_rows_equal_the_verify_pass(quad_mini):
    """The chain rows of a quadratic pass are Mode 3's verify pass over [anchor, s_1 .. s_{k-1}]: same
    logits and same K/V rows (the masks after them are invisible to them)."""
    w, kv, anchor, spec, _ = quad_mini
    k = 4
    logits, nk, nv = O.quad_forward(w, kv, anchor, spec, k)
    _, vlogits, vk, vv = O.verify_pass(w, kv, anchor, spec)
    np.testing.assert_allclose(logits[:, :k], vlogits, rtol=1e-10, atol=1e-12)
    for l in range(MINI.n_layers):
        np.testing.assert_allclose(nk[l][:, :, :k], vk[l], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(nv[l][:, :, :k], vv[l], rtol=1e-10, atol=1e-12)


def test_quad_groups_equal_draft_passes(quad_mini):
    """Group c of a quadratic pass is Mode 3's draft pass over [chain_0 .. chain_c, mask x k] with the chain
    rows causal (bidir_from = c + 1): the same positions, keys and mask, so the same logits."""
    w, kv, anchor, spec, _ = quad_mini
    k = 4
    logits, _, _ = O.quad_forward(w, kv, anchor, spec, k)
    chain = O.verify_block(anchor, spec)
    for c in range(k):
        blk = np.concatenate([chain[:, :c + 1], np.full((2, k), MINI.mask_token_id, dtype=np.int32)], axis=1)
        dl, _, _ = O.block_forward(w, kv, blk, O.DRAFT, bidir_from=c + 1)
        rows = [k + c * k + r for r in range(k)]
        np.testing.assert_allclose(logits[:, rows], dl[:, c + 1:], rtol=1e-10, atol=1e-12)


def test_quad_equals_full_recompute(quad_mini):
    """The cached quadratic pass equals recomputing [prefix ; quadratic block] from tokens with the explicit
    mask (prefix causal, block rows as the layout says) and the layout's positions."""
    w, kv, anchor, spec, prefix = quad_mini
    k = 3
    spec = spec[:, :k - 1]
    logits, _, _ = O.quad_forward(w, kv, anchor, spec, k)
    P = int(kv.lengths[0])
    R = O.quad_rows(k)
    toks = np.concatenate([prefix, O.quad_tokens(anchor, spec, k, MINI.mask_token_id)], axis=1)
    vis = np.tril(np.ones((P + R, P + R), dtype=bool))
    vis[P:, P:] = O.quad_block_visibility(k)
    off, _, _ = O.quad_layout(k)
    pos = np.broadcast_to(np.concatenate([np.arange(P), P + off]), (2, P + R))
    full = O.full_forward(w, toks, vis, positions=pos)
    np.testing.assert_allclose(logits, full[:, P:], rtol=1e-10, atol=1e-12)


def test_ensemble_argmax_closed_forms():
    """lambda = 1 is the AR argmax, lambda = 0 the diffusion argmax; a two-token example by hand:
    p_AR = (0.7, 0.3), p_diff = (0.2, 0.8) mix to (0.45, 0.55) at lambda = 0.5 and (0.55, 0.45) at 0.7;
    equal mixtures tie to the lower index."""
    rng = np.random.default_rng(3)
    a, d = rng.standard_normal((5, 40)), rng.standard_normal((5, 40))
    np.testing.assert_array_equal(O.ensemble_argmax(a, d, 1.0), O.argmax_first(a))
    np.testing.assert_array_equal(O.ensemble_argmax(a, d, 0.0), O.argmax_first(d))
    la, ld = np.log([[0.7, 0.3]]), np.log([[0.2, 0.8]])
    assert O.ensemble_argmax(la, ld, 0.5)[0] == 1
    assert O.ensemble_argmax(la, ld, 0.7)[0] == 0
    assert O.ensemble_argmax(np.log([[0.5, 0.5]]), np.log([[0.5, 0.5]]), 0.3)[0] == 0


def test_quad_self_speculation_reproduces_greedy_ar():
    """With the AR verifier (lambda = 1), quadratic self-speculation commits exactly the greedy AR
    continuation and builds the same cache, whatever its speculative tokens were."""
    w = mini_weights(seed=14)
    prefix = synth_tokens(MINI, 14, "pin.qss.prefix", (2, 9))
    k, steps = 4, 5
    kv_q = prefilled(w, prefix[:, :-1], capacity=64)
    kv_ar = kv_q.copy()
    anchor = prefix[:, -1].copy()
    spec, _ = O.draft_pass(w, kv_q, anchor, k)            # the first speculative tokens: a Mode 3 draft
    out = [[] for _ in range(2)]
    for _ in range(steps):
        r = O.quad_step(w, kv_q, anchor, spec, k, lam=1.0)
        for b in range(2):
            assert 0 <= r["L"][b] <= k - 1
            out[b] += r["committed"][b][:-1]               # anchor's successors up to the bonus
            out[b].append(r["committed"][b][-1])
        anchor, spec = r["next_anchor"], r["next_spec"]
    n = min(len(o) for o in out)
    tok = prefix[:, -1].copy()
    ar = [[] for _ in range(2)]
    for _ in range(n):
        tok, _ = O.ar_step(w, kv_ar, tok)
        for b in range(2):
            ar[b].append(int(tok[b]))
    for b in range(2):
        assert out[b][:n] == ar[b]
    m = int(min(kv_q.lengths))
    for l in range(MINI.n_layers):
        np.testing.assert_allclose(kv_q.k[l][:, :, :m], kv_ar.k[l][:, :, :m], rtol=1e-9, atol=1e-11)


def test_quad_planted_spec_fully_accepted():
    """Speculative tokens equal to the greedy AR continuation are accepted in full (L = k - 1); the next
    anchor is the next greedy token and the next speculative tokens come from the last group's masks."""
    w = mini_weights(seed=15)
    prefix = synth_tokens(MINI, 15, "pin.qplant.prefix", (1, 9))
    k = 4
    kv = prefilled(w, prefix[:, :-1], capacity=64)
    kv_ar = kv.copy()
    tok, greedy = prefix[:, -1].copy(), []
    for _ in range(k):
        tok, _ = O.ar_step(w, kv_ar, tok)
        greedy.append(int(tok[0]))
    r = O.quad_step(w, kv, prefix[:, -1], np.array([greedy[:k - 1]]), k, lam=1.0)
    assert r["L"][0] == k - 1 and r["committed"][0] == greedy and r["next_anchor"][0] == greedy[-1]
    am = O.argmax_first(r["logits"])
    assert r["next_spec"][0].tolist() == [int(am[0, k + (k - 1) * k + i]) for i in range(1, k)]
