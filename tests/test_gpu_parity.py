"""GPU parity of the block-decode step against the CPU oracle, through the C ABI.

Bar: logits within 2e-2 normwise relative error of the fp32 oracle; argmax and
acceptance bit-exact on identical logits; integer-exact where every value is an
exactly representable small integer.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import nld_oracle as O
from synth.workloads import LazyWeights, ModelShape, SHAPE_TINY, WORKLOADS, tokens as synth_tokens, prefix_kv

from gpu_common import (ArraySource, BF16_ONE, check_argmax, int_to_bf16_bits, log, rel_err)

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def R():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime
    return runtime


# ----------------------------------------------------------------------------- integer-exact pins
def _int_model(shape: ModelShape, seed: int, wv_int=False, lm_range=8):
    """Zero layer weights (so the residual stream is the embedding), embeddings of +-1, gains 1,
    small-integer LM head (and optionally small-integer Wv)."""
    h = shape.hidden
    zero = lambda o, i: np.zeros((o, i), dtype=np.uint16)
    sign = synth.uniform_int(seed, "int.embed", (shape.vocab, h), 0, 1)
    embed = np.where(sign == 1, BF16_ONE, np.uint16(0xBF80)).astype(np.uint16)
    lm = int_to_bf16_bits(synth.uniform_int(seed, "int.lm", (shape.vocab, h), -lm_range, lm_range))
    layers = []
    for l in range(shape.n_layers):
        wv = int_to_bf16_bits(synth.uniform_int(seed, "int.wv%d" % l, (shape.kv_dim, h), -1, 1)) if wv_int \
            else zero(shape.kv_dim, h)
        layers.append({"attn_norm": synth.bf16_ones(h), "wq": zero(shape.q_dim, h), "wk": zero(shape.kv_dim, h),
                       "wv": wv, "wo": zero(h, shape.q_dim), "ffn_norm": synth.bf16_ones(h),
                       "w_gate": zero(shape.ffn, h), "w_up": zero(shape.ffn, h), "w_down": zero(h, shape.ffn)})
    return ArraySource(layers, embed, lm, synth.bf16_ones(h))


INT_SHAPE = ModelShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=96, vocab=1000,
                       rms_eps=0.0)


@pytest.mark.parametrize("k", [1, 8, 12, 28, 40, 64])
def test_lm_head_integer_exact(R, k):
    """Embedding gather, LM-head packing/tiling (ragged vocab 1000) and the fused argmax: the logits are
    exact integers on both sides, so they must agree bit for bit, ties included (lowest index wins)."""
    shape, seed = INT_SHAPE, 21
    src = _int_model(shape, seed)
    tok = synth_tokens(shape, seed, "int.tokens", (2, k))
    w = O.OracleWeights(shape, src, np.float64)
    kv = O.OracleKV(shape, 2, 64, np.float64)
    ref, _, _ = O.block_forward(w, kv, tok, O.VERIFY)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 2, 64)
    ws = R.Workspace(model, 2, k, 64)
    logits, am = R.block_forward(model, cache, ws, torch.from_numpy(tok).cuda(), R.VERIFY)
    g = logits.cpu().numpy()
    assert np.array_equal(g, ref.astype(np.float32)), "max diff %g" % np.max(np.abs(g - ref))
    assert np.array_equal(am.cpu().numpy(), O.argmax_first(ref))
    assert R.read_device_status(ws) == 0


@pytest.mark.parametrize("prefix,k", [(0, 8), (5, 8), (61, 8), (5, 24), (61, 56)])
def test_qkv_value_rows_integer_exact(R, prefix, k):
    """QKV packing, the V cache's transposed 64-position tiles and the cache row addressing: with +-1
    activations and {-1,0,1} Wv the block's V rows are exact integers; K rows are zero.  24 and 56
    rows run the QKV projection on the 17..64-row kernel (K slices met through the workspace)."""
    shape, seed = INT_SHAPE, 22
    src = _int_model(shape, seed, wv_int=True)
    tok = synth_tokens(shape, seed, "int.tokens", (1, k))
    w = O.OracleWeights(shape, src, np.float64)
    kv = O.OracleKV(shape, 1, 128, np.float64)
    kv.lengths[:] = prefix
    _, nk, nv = O.block_forward(w, kv, tok, O.VERIFY)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 1, 128)
    cache.set_lengths([prefix])
    ws = R.Workspace(model, 1, k, 128)
    R.block_forward(model, cache, ws, torch.from_numpy(tok).cuda(), R.VERIFY, want_logits=False)
    kg, vg = cache.read_kv(0, prefix, prefix + k)
    f = lambda bits: O.bf16_bits_to_float(bits, np.float64)
    assert np.array_equal(f(vg), nv[0]), "V rows differ"
    assert np.array_equal(f(kg), nk[0])
    assert int(cache.lengths.cpu()[0]) == prefix        # a block pass never commits


# ----------------------------------------------------------------------------- argmax + acceptance
def test_accept_from_logits_bit_exact(R):
    """Argmax and longest-prefix acceptance on identical (oracle-side) logits, with planted exact ties,
    signed zeros and drafts planted to give every acceptance length 0..k-1."""
    B, k, V = 9, 8, 5003
    z = synth.normal_f64(5, "acc.logits", (B, k, V)).astype(np.float32)
    z[0, 2, [5, 900, 4000]] = 7.5                     # exact three-way tie -> lowest index
    z[1, 0, :] = -1.0
    z[1, 0, 3], z[1, 0, 1] = 0.0, -0.0                # -0.0 == +0.0: first index wins
    a = O.argmax_first(z)
    drafts = synth.uniform_int(5, "acc.drafts", (B, k - 1), 0, V - 1)
    for b in range(B):                                 # sequence b accepts exactly min(b, k-1) drafts
        L = min(b, k - 1)
        drafts[b, :L] = a[b, :L]
        if L < k - 1:
            drafts[b, L] = (a[b, L] + 1) % V
    out = R.accept_from_logits(torch.from_numpy(z).cuda(), torch.from_numpy(drafts).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(out["argmax"].cpu().numpy(), a)
    assert a[0, 2] == 5 and a[1, 0] == 1
    for b in range(B):
        L, committed, bonus = O.accept(drafts[b], a[b])
        assert int(out["accept_len"][b]) == L == min(b, k - 1)
        assert out["committed"][b].cpu().tolist() == committed + [-1] * (k - len(committed))
        assert int(out["next_anchor"][b]) == bonus


# ----------------------------------------------------------------------------- tiny workload (real prefix)
@pytest.fixture(scope="module")
def tiny(R):
    wl = WORKLOADS["tiny"]
    shape, seed = wl.shape, wl.seed
    src = LazyWeights(shape, seed)
    prefix = synth_tokens(shape, seed, "tiny.prefix", (1, wl.prefix_len))
    block = synth_tokens(shape, seed, "tiny.block", (1, 8))
    w = O.OracleWeights(shape, src, np.float32)
    okv = O.OracleKV(shape, 1, 256, np.float32)
    O.prefill(w, okv, prefix)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 1, 256)
    ws16 = R.Workspace(model, 1, 16, 256)
    pt = torch.from_numpy(prefix).cuda()
    for c0 in range(0, wl.prefix_len, 16):               # causal prefill = verify passes, every row committed
        R.block_forward(model, cache, ws16, pt[:, c0:c0 + 16].contiguous(), R.VERIFY, want_logits=False)
        cache.lengths += 16
    torch.cuda.synchronize()
    return dict(shape=shape, src=src, w=w, okv=okv, model=model, cache=cache, prefix=prefix, block=block)


def test_tiny_prefill_cache(R, tiny):
    """The GPU's own prefill writes K/V rows within tolerance of the oracle's cache."""
    t = tiny
    for l in range(t["shape"].n_layers):
        kg, vg = t["cache"].read_kv(l, 0, 128)
        assert rel_err(O.bf16_bits_to_float(kg), t["okv"].k[l][:, :, :128]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), t["okv"].v[l][:, :, :128]) < TOL


@pytest.mark.parametrize("mode,bidir_from", [(O.VERIFY, 0), (O.DRAFT, 0), (O.DRAFT, 1), (O.DRAFT, 5)])
def test_tiny_block_pass(R, tiny, mode, bidir_from):
    t = tiny
    ref, _, _ = O.block_forward(t["w"], t["okv"], t["block"], mode, bidir_from)
    ws = R.Workspace(t["model"], 1, 8, 256)
    logits, am = R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(t["block"]).cuda(),
                                 R.VERIFY if mode == O.VERIFY else R.DRAFT, bidir_from)
    g = logits.cpu().numpy()
    e = rel_err(g, ref)
    log("tiny %s bidir_from=%d: rel err %.3e" % (mode, bidir_from, e))
    assert e <= TOL
    near = check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    log("  near-tie argmax rows differing: %s" % near)
    assert int(t["cache"].lengths.cpu()[0]) == 128


@pytest.mark.parametrize("kind", ["swap0", "final<-attn1"])
def test_tiny_misplaced_gain_fails_parity(R, tiny, kind):
    """Negative control of the gain path: the device pass of a model whose RMSNorm gains were moved
    (layer 0's attention and FFN gains swapped; layer 1's attention gain at the final norm) is far
    outside the tolerance against the oracle of the true model, while the true model passes."""
    from test_oracle_pins import _GainSwap
    t = tiny
    bad = R.DeviceModel(t["shape"], _GainSwap(t["src"], kind))
    ref, _, _ = O.block_forward(t["w"], t["okv"], t["block"], O.VERIFY)
    ws = R.Workspace(bad, 1, 8, 256)
    logits, _ = R.block_forward(bad, t["cache"], ws, torch.from_numpy(t["block"]).cuda(), R.VERIFY)
    e = rel_err(logits.cpu().numpy(), ref)
    log("tiny with gains moved (%s) against the true oracle: rel err %.3e" % (kind, e))
    assert e > 5 * TOL
    bad.close()


def test_tiny_self_speculation_loop(R, tiny):
    """Three paper-loop steps (draft -> verify -> accept -> commit) on both sides from the same prefix."""
    t = tiny
    shape = t["shape"]
    okv = t["okv"].copy()
    k = 8
    anchor = synth_tokens(shape, 0, "tiny.anchor", (1,))
    model = t["model"]
    cache = R.DeviceCache(shape, 1, 256)
    cache.k.copy_(t["cache"].k)
    cache.v.copy_(t["cache"].v)
    cache.lengths.copy_(t["cache"].lengths)
    ws = R.Workspace(model, 1, k, 256)
    a_o, a_g = anchor.copy(), torch.from_numpy(anchor).cuda()
    for step in range(3):
        ref = O.self_spec_step(t["w"], okv, a_o, k)
        d, dl = R.draft(model, cache, ws, a_g, k, want_logits=True)
        e_d = rel_err(dl.cpu().numpy(), ref["draft_logits"])
        assert e_d <= TOL
        assert np.array_equal(d.cpu().numpy(), ref["drafts"]), "drafts differ (step %d)" % step
        out = R.verify_accept(model, cache, ws, a_g, d, k, want_logits=True)
        e_v = rel_err(out["logits"].cpu().numpy(), ref["verify_logits"])
        assert e_v <= TOL
        L = int(out["accept_len"].cpu()[0])
        assert L == int(ref["L"][0])
        assert out["committed"][0].cpu().tolist()[:L + 1] == ref["committed"][0]
        assert int(cache.lengths.cpu()[0]) == int(okv.lengths[0])
        a_o, a_g = ref["next_anchor"], out["next_anchor"]
        assert int(a_g.cpu()[0]) == int(a_o[0])
        log("tiny step %d: L=%d draft err %.2e verify err %.2e" % (step, L, e_d, e_v))
    assert R.read_device_status(ws) == 0


def test_tiny_planted_drafts_full_accept(R, tiny):
    """Drafts equal to the oracle's greedy AR continuation are accepted in full (L = k-1) and the
    committed rows advance the cache by k."""
    t = tiny
    k = 8
    okv = t["okv"].copy()
    anchor = synth_tokens(t["shape"], 0, "tiny.anchor", (1,))
    tok, greedy = anchor.copy(), []
    for _ in range(k):
        tok, _ = O.ar_step(t["w"], okv, tok)
        greedy.append(int(tok[0]))
    drafts = np.array([greedy[:k - 1]], dtype=np.int32)
    cache = R.DeviceCache(t["shape"], 1, 256)
    cache.k.copy_(t["cache"].k)
    cache.v.copy_(t["cache"].v)
    cache.lengths.copy_(t["cache"].lengths)
    ws = R.Workspace(t["model"], 1, k, 256)
    out = R.verify_accept(t["model"], cache, ws, torch.from_numpy(anchor).cuda(), torch.from_numpy(drafts).cuda(),
                          k)
    assert int(out["accept_len"].cpu()[0]) == k - 1
    assert out["committed"][0].cpu().tolist() == greedy
    assert int(cache.lengths.cpu()[0]) == 128 + k
    kg, _ = cache.read_kv(0, 0, 128 + k)
    assert rel_err(O.bf16_bits_to_float(kg), okv.k[0][:, :, :128 + k]) < TOL


def _tiny_cache_copy(R, t):
    cache = R.DeviceCache(t["shape"], 1, 256)
    cache.k.copy_(t["cache"].k)
    cache.v.copy_(t["cache"].v)
    cache.lengths.copy_(t["cache"].lengths)
    return cache


def test_tiny_decode_steps_equal_single_calls(R, tiny):
    """nld_decode_steps (n steps enqueued at once, anchor updated in place) equals n draft + verify_accept
    call pairs bit for bit: accept lengths, committed tokens, anchors, lengths and cache rows."""
    t = tiny
    k, n = 8, 3
    anchor = synth_tokens(t["shape"], 0, "tiny.anchor", (1,))
    ca, cb = _tiny_cache_copy(R, t), _tiny_cache_copy(R, t)
    wa, wb = R.Workspace(t["model"], 1, k, 256), R.Workspace(t["model"], 1, k, 256)
    a_a, a_b = torch.from_numpy(anchor.copy()).cuda(), torch.from_numpy(anchor.copy()).cuda()
    outs = R.decode_steps(t["model"], ca, wa, a_a, k, n)
    acc, com = [], []
    for _ in range(n):
        d, _ = R.draft(t["model"], cb, wb, a_b, k)
        o = R.verify_accept(t["model"], cb, wb, a_b, d, k, outs={
            "accept_len": torch.empty(1, dtype=torch.int32, device="cuda"),
            "committed": torch.empty((1, k), dtype=torch.int32, device="cuda"), "next_anchor": a_b})
        acc.append(o["accept_len"].clone())
        com.append(o["committed"].clone())
    assert torch.equal(outs["accept_len"], torch.stack(acc))
    assert torch.equal(outs["committed"], torch.stack(com))
    assert torch.equal(a_a, a_b) and torch.equal(ca.lengths, cb.lengths)
    end = int(ca.lengths.cpu()[0])
    assert end >= 128 + n
    for l in range(t["shape"].n_layers):
        assert all(np.array_equal(x, y) for x, y in zip(ca.read_kv(l, 0, end), cb.read_kv(l, 0, end)))
    assert R.read_device_status(wa) == 0


def test_tiny_decode_steps_against_the_oracle(R, tiny):
    """nld_decode_steps at k = 8 for 3 steps (drafts kept on the device) against three oracle
    self-speculation steps: accept lengths, committed tokens, the anchor left in place, the lengths and
    every layer's committed K/V rows."""
    t = tiny
    k, n = 8, 3
    okv = t["okv"].copy()
    anchor = synth_tokens(t["shape"], 0, "tiny.anchor", (1,))
    a_o, refs = anchor.copy(), []
    for _ in range(n):
        ref = O.self_spec_step(t["w"], okv, a_o, k)
        refs.append(ref)
        a_o = ref["next_anchor"]
    cache = _tiny_cache_copy(R, t)
    ws = R.Workspace(t["model"], 1, k, 256)
    a_g = torch.from_numpy(anchor.copy()).cuda()
    outs = R.decode_steps(t["model"], cache, ws, a_g, k, n)
    acc, com = outs["accept_len"].cpu().numpy(), outs["committed"].cpu().numpy()
    for s, ref in enumerate(refs):
        L = int(ref["L"][0])
        assert acc[s, 0] == L, "step %d" % s
        assert com[s, 0].tolist() == ref["committed"][0] + [-1] * (k - L - 1), "step %d" % s
    assert int(a_g.cpu()[0]) == int(a_o[0])
    end = int(okv.lengths[0])
    assert int(cache.lengths.cpu()[0]) == end
    for l in range(t["shape"].n_layers):
        kg, vg = cache.read_kv(l, 0, end)
        assert rel_err(O.bf16_bits_to_float(kg), okv.k[l][:, :, :end]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), okv.v[l][:, :, :end]) < TOL
    assert R.read_device_status(ws) == 0
    log("tiny decode loop: accept lengths %s" % acc[:, 0].tolist())


def test_tiny_decode_steps_ar_mode(R, tiny):
    """With k = 1 the loop is AR decoding: the committed tokens are the oracle's greedy continuation."""
    t = tiny
    n = 5
    okv = t["okv"].copy()
    tok = synth_tokens(t["shape"], 0, "tiny.anchor", (1,))
    greedy = []
    for _ in range(n):
        tok, _ = O.ar_step(t["w"], okv, tok)
        greedy.append(int(tok[0]))
    cache = _tiny_cache_copy(R, t)
    ws = R.Workspace(t["model"], 1, 1, 256)
    a = torch.from_numpy(synth_tokens(t["shape"], 0, "tiny.anchor", (1,))).cuda()
    outs = R.decode_steps(t["model"], cache, ws, a, 1, n)
    assert outs["committed"][:, 0, 0].cpu().tolist() == greedy
    assert np.all(outs["accept_len"].cpu().numpy() == 0)
    assert int(a.cpu()[0]) == greedy[-1] and int(cache.lengths.cpu()[0]) == 128 + n
    assert R.read_device_status(ws) == 0


def test_draft_with_bidir_from_k_is_the_verify_pass(R, tiny):
    """A draft pass whose bidirectional rows start at k has the causal mask: its logits equal the verify
    pass's bit for bit (the draft still writes no cache row)."""
    t = tiny
    bt = torch.from_numpy(t["block"]).cuda()
    ws = R.Workspace(t["model"], 1, 8, 256)
    cache = _tiny_cache_copy(R, t)
    before = cache.read_kv(0, 128, 136)
    d = R.block_forward(t["model"], cache, ws, bt, R.DRAFT, 8)[0]
    assert all(np.array_equal(x, y) for x, y in zip(before, cache.read_kv(0, 128, 136)))
    v = R.block_forward(t["model"], cache, ws, bt, R.VERIFY)[0]
    assert torch.equal(d, v)


def test_capacity_error_is_reported_not_written(R, tiny):
    """A block that would run past max_len sets the capacity bit; no row beyond the cache is written.
    A commit that would pass max_len stops the length at max_len: with drafts planted to be accepted in
    full (L = 7 from length 124 in a cache of 128 rows) the length ends at 128, the capacity bit is set,
    and cache rows 124..127 hold the verify pass's K/V, which equal the oracle's."""
    t = tiny
    k = 8
    cache = R.DeviceCache(t["shape"], 1, 128)
    cache.set_lengths([124])
    ws = R.Workspace(t["model"], 1, k, 128)
    R.block_forward(t["model"], cache, ws, torch.from_numpy(t["block"]).cuda(), R.VERIFY, want_logits=False)
    assert R.read_device_status(ws) & 0x2
    assert R.read_device_status(ws) == 0        # reading clears the sticky bits

    okv = t["okv"].copy()
    okv.lengths[:] = 124
    anchor = synth_tokens(t["shape"], 0, "tiny.cap.anchor", (1,))
    tok, greedy = anchor.copy(), []
    for _ in range(k):
        tok, _ = O.ar_step(t["w"], okv, tok)
        greedy.append(int(tok[0]))
    cache.k[:, :, :, :128].copy_(t["cache"].k[:, :, :, :128])
    cache.v.copy_(t["cache"].v[:, :, :, :2])
    cache.set_lengths([124])
    drafts = np.array([greedy[:k - 1]], dtype=np.int32)
    out = R.verify_accept(t["model"], cache, ws, torch.from_numpy(anchor).cuda(), torch.from_numpy(drafts).cuda(), k)
    assert int(out["accept_len"].cpu()[0]) == k - 1
    assert out["committed"][0].cpu().tolist() == greedy
    assert int(cache.lengths.cpu()[0]) == 128
    assert R.read_device_status(ws) & 0x2
    for l in range(t["shape"].n_layers):
        kg, vg = cache.read_kv(l, 0, 128)
        assert rel_err(O.bf16_bits_to_float(kg), okv.k[l][:, :, :128]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), okv.v[l][:, :, :128]) < TOL


def test_bad_token_is_reported(R, tiny):
    t = tiny
    bad = t["block"].copy()
    bad[0, 3] = 5000
    ws = R.Workspace(t["model"], 1, 8, 256)
    R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(bad).cuda(), R.VERIFY, want_logits=False)
    assert R.read_device_status(ws) & 0x1


# ----------------------------------------------------------------------------- one 8B-shaped layer + LM head
@pytest.mark.parametrize("mode", [O.VERIFY, O.DRAFT])
def test_tiny_ragged_batch_attention_items(R, monkeypatch, mode):
    """A ragged batch (committed lengths 0, 70, 128, 1 and 248: an empty prefix, one key, split boundaries
    and a block that ends at max_len) with the attention's length-aware work items (the default for
    batches: only splits holding committed keys get a workgroup, the merge reads only those) and with
    the plain grid over max_len: both within tolerance of the oracle and equal up to the fp32
    rounding of the merge."""
    wl = WORKLOADS["tiny"]
    shape, seed = wl.shape, wl.seed
    lengths = np.array([0, 70, 128, 1, 256 - 8])
    B, k, max_len = len(lengths), 8, 256
    src = LazyWeights(shape, seed)
    w = O.OracleWeights(shape, src, np.float32)
    okv = O.OracleKV(shape, B, max_len, np.float32)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, B, max_len)
    for l in range(shape.n_layers):
        kb, vb = prefix_kv(shape, seed, l, B, int(lengths.max()))
        okv.set_prefix_bf16(l, kb, vb, lengths)
        cache.load_prefix(l, kb, vb)
    cache.set_lengths(lengths)
    tok = synth_tokens(shape, seed, "tiny.ragged", (B, k))
    ref, _, _ = O.block_forward(w, okv, tok, mode)
    out = {}
    for items in ("1", "0"):
        monkeypatch.setenv("NLD_ATTN_NO_ITEMS", "0" if items == "1" else "1")
        ws = R.Workspace(model, B, k, max_len)
        logits, am = R.block_forward(model, cache, ws, torch.from_numpy(tok).cuda(),
                                     R.VERIFY if mode == O.VERIFY else R.DRAFT)
        g = logits.cpu().numpy()
        e = rel_err(g, ref)
        log("tiny ragged batch %s, %s: rel err %.3e" % (mode, "items" if items == "1" else "grid", e))
        assert e <= TOL
        check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
        assert R.read_device_status(ws) == 0
        out[items] = g
    assert rel_err(out["1"], out["0"]) < 1e-5
    assert cache.lengths.cpu().numpy().tolist() == lengths.tolist()


@pytest.fixture(scope="module")
def layer8b(R):
    wl = WORKLOADS["8b_layer"]
    shape, seed, P = wl.shape, wl.seed, wl.prefix_len
    src = LazyWeights(shape, seed)
    kb, vb = prefix_kv(shape, seed, 0, 1, P)
    w = O.OracleWeights(shape, src, np.float32)
    okv = O.OracleKV(shape, 1, P + 64, np.float32)
    okv.set_prefix_bf16(0, kb, vb, [P])
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 1, P + 64)
    cache.load_prefix(0, kb, vb)
    cache.set_lengths([P])
    return dict(shape=shape, w=w, okv=okv, model=model, cache=cache, seed=seed)


@pytest.mark.parametrize("k", [8, 16, 32, 64])
@pytest.mark.parametrize("mode", [O.VERIFY, O.DRAFT])
def test_8b_layer_block_pass(R, layer8b, k, mode):
    t = layer8b
    shape = t["shape"]
    tok = synth_tokens(shape, t["seed"], "8b_layer.block%d" % k, (1, k))
    ref, nk, nv = O.block_forward(t["w"], t["okv"], tok, mode)
    ws = R.Workspace(t["model"], 1, k, t["cache"].max_len)
    before = t["cache"].read_kv(0, 2048, 2048 + k)
    logits, am = R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(tok).cuda(),
                                 R.VERIFY if mode == O.VERIFY else R.DRAFT)
    g = logits.cpu().numpy()
    e = rel_err(g, ref)
    log("8b_layer k=%d %s: rel err %.3e" % (k, mode, e))
    assert e <= TOL
    check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    kg, vg = t["cache"].read_kv(0, 2048, 2048 + k)
    if mode == O.VERIFY:     # the verify pass leaves its K/V rows in the uncommitted cache rows
        assert rel_err(O.bf16_bits_to_float(kg), nk[0]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), nv[0]) < TOL
    else:                    # a draft pass writes no cache row
        assert np.array_equal(kg, before[0]) and np.array_equal(vg, before[1])
    assert R.read_device_status(ws) == 0


@pytest.mark.parametrize("env", ["NLD_ATTN_LATE=0", "NLD_ATTN_LATE=1", "NLD_STREAM_NW_RESID=8"])
def test_8b_layer_alternative_launch_paths(R, layer8b, monkeypatch, env):
    """The launch paths kept selectable beside the defaults: a prefix split's stages 1 and 2 requested
    together with stage 0 or stage 2 alone deferred, and the 16-row O projection on 8 wavefronts.
    Each gives the same pass as the default within the fp32 rounding of its reductions, and is within
    tolerance of the oracle, in both masks."""
    t = layer8b
    shape, k = t["shape"], 16
    name, value = env.split("=")
    tok = torch.from_numpy(synth_tokens(shape, t["seed"], "8b_layer.alt.block", (1, k))).cuda()
    for mode in (O.VERIFY, O.DRAFT):
        ref = O.block_forward(t["w"], t["okv"], tok.cpu().numpy(), mode)[0]
        gm = R.VERIFY if mode == O.VERIFY else R.DRAFT
        ws = R.Workspace(t["model"], 1, k, t["cache"].max_len)
        monkeypatch.delenv(name, raising=False)
        base = R.block_forward(t["model"], t["cache"], ws, tok, gm)[0].cpu().numpy()
        monkeypatch.setenv(name, value)
        alt = R.block_forward(t["model"], t["cache"], ws, tok, gm)[0].cpu().numpy()
        monkeypatch.delenv(name, raising=False)
        e = rel_err(alt, ref)
        log("8b_layer k=16 %s %s: rel err %.3e, against the default path %.3e" % (mode, env, e, rel_err(alt, base)))
        assert e <= TOL
        if name == "NLD_ATTN_LATE":   # the same arithmetic in the same order: only when loads are issued
            assert np.array_equal(alt, base)
        else:
            assert rel_err(alt, base) < 1e-4
        assert R.read_device_status(ws) == 0


@pytest.mark.parametrize("mode", [O.VERIFY, O.DRAFT])
def test_8b_layer_long_cache_block_pass(R, layer8b, mode):
    """A cache whose capacity (16384) is eight times its committed prefix (2048): one sequence's prefix
    splits are cut from the committed length on the device, not from the capacity.  Within tolerance of
    the oracle, and equal to the same pass over a cache of capacity 2112 up to the fp32 rounding of the
    merge (the split boundaries differ)."""
    t = layer8b
    shape, k = t["shape"], 16
    P = 2048
    cache = R.DeviceCache(shape, 1, 16384)
    kb, vb = prefix_kv(shape, t["seed"], 0, 1, P)
    cache.load_prefix(0, kb, vb)
    cache.set_lengths([P])
    tok = synth_tokens(shape, t["seed"], "8b_layer.long%d" % k, (1, k))
    ref, nk, nv = O.block_forward(t["w"], t["okv"], tok, mode)
    out = {}
    for name, c in (("long", cache), ("short", t["cache"])):
        ws = R.Workspace(t["model"], 1, k, c.max_len)
        logits, am = R.block_forward(t["model"], c, ws, torch.from_numpy(tok).cuda(),
                                     R.VERIFY if mode == O.VERIFY else R.DRAFT)
        g = logits.cpu().numpy()
        e = rel_err(g, ref)
        log("8b_layer %s cache (capacity %d) k=%d %s: rel err %.3e" % (name, c.max_len, k, mode, e))
        assert e <= TOL
        check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
        assert R.read_device_status(ws) == 0
        out[name] = g
    assert rel_err(out["long"], out["short"]) < 1e-5
    if mode == O.VERIFY:
        kg, vg = cache.read_kv(0, P, P + k)
        assert rel_err(O.bf16_bits_to_float(kg), nk[0]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), nv[0]) < TOL


@pytest.fixture(scope="module")
def layer8b_b4(R):
    """One 8B-shaped layer, batch 4 with ragged prefixes: 128 block rows at k=32 (the tiled GEMM path)."""
    wl = WORKLOADS["8b_layer"]
    shape, seed = wl.shape, wl.seed
    lengths = np.array([2048, 1000, 64, 1537])
    src = LazyWeights(shape, seed)
    kb, vb = prefix_kv(shape, seed, 0, 4, int(lengths.max()))
    w = O.OracleWeights(shape, src, np.float32)
    okv = O.OracleKV(shape, 4, 2048 + 64, np.float32)
    okv.set_prefix_bf16(0, kb, vb, lengths)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 4, 2048 + 64)
    cache.load_prefix(0, kb, vb)
    cache.set_lengths(lengths)
    return dict(shape=shape, w=w, okv=okv, model=model, cache=cache, seed=seed, lengths=lengths)


@pytest.mark.parametrize("mode", [O.VERIFY, O.DRAFT])
def test_8b_layer_batched_block_pass(R, layer8b_b4, mode):
    """128 rows (batch 4, k=32, ragged prefixes 64..2048): every projection runs on the tiled MFMA GEMM;
    logits, argmax and the verify pass's K/V rows against the oracle."""
    t = layer8b_b4
    shape, k = t["shape"], 32
    tok = synth_tokens(shape, t["seed"], "8b_layer.b4.block", (4, k))
    ref, nk, nv = O.block_forward(t["w"], t["okv"], tok, mode)
    ws = R.Workspace(t["model"], 4, k, t["cache"].max_len)
    logits, am = R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(tok).cuda(),
                                 R.VERIFY if mode == O.VERIFY else R.DRAFT)
    g = logits.cpu().numpy()
    e = rel_err(g, ref)
    log("8b_layer batch 4 k=32 %s: rel err %.3e" % (mode, e))
    assert e <= TOL
    check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    if mode == O.VERIFY:
        for b, P in enumerate(t["lengths"]):
            kg, vg = t["cache"].read_kv(0, int(P), int(P) + k)
            assert rel_err(O.bf16_bits_to_float(kg[b:b + 1]), nk[0][b:b + 1]) < TOL
            assert rel_err(O.bf16_bits_to_float(vg[b:b + 1]), nv[0][b:b + 1]) < TOL
    assert R.read_device_status(ws) == 0


def test_8b_layer_tile_gemm_k_slices(R, layer8b_b4, monkeypatch):
    """The tiled GEMM with K slices (by default at 128 rows: O and down 8 slices, QKV 5, met through the
    workspace by the last-arriving workgroup) against the same GEMM unsliced: both within tolerance of
    the oracle, equal up to the fp32 rounding of the slice sums, and the sliced result bit-identical over
    repeated passes whatever order the slices finish in."""
    t = layer8b_b4
    shape, k = t["shape"], 32
    tok = torch.from_numpy(synth_tokens(shape, t["seed"], "8b_layer.b4.kslices", (4, k))).cuda()
    ref, _, _ = O.block_forward(t["w"], t["okv"], tok.cpu().numpy(), O.DRAFT)
    out = {}
    for ks in ("1", None):
        for kind in ("O", "DOWN", "QKV"):
            if ks is None:
                monkeypatch.delenv("NLD_TILE_KSPLIT_" + kind, raising=False)
            else:
                monkeypatch.setenv("NLD_TILE_KSPLIT_" + kind, ks)
        ws = R.Workspace(t["model"], 4, k, t["cache"].max_len)
        runs = [R.block_forward(t["model"], t["cache"], ws, tok, R.DRAFT)[0].cpu().numpy() for _ in range(3)]
        assert R.read_device_status(ws) == 0
        e = rel_err(runs[0], ref)
        log("8b_layer batch 4 k=32 tile GEMM %s: rel err %.3e" % ("unsliced" if ks else "K slices", e))
        assert e <= TOL
        for r in runs[1:]:
            assert np.array_equal(r, runs[0])
        out[ks] = runs[0]
    d = rel_err(out[None], out["1"])
    log("  sliced vs unsliced: %.3e" % d)
    assert d < 1e-4


# ----------------------------------------------------------------------------- split-K residual GEMM
@pytest.mark.parametrize("ksplit,ct", [(1, 4), (2, 2), (3, 4), (8, 4), (8, 2)])
def test_tiny_split_k_residual_gemm(R, tiny, monkeypatch, ksplit, ct):
    """QKV, O and down projections cut into ksplit K slices (ragged: the tiny down projection has 22
    k-steps, so 8 slices of 3 leave the last one a single step and some wavefronts none) of ct column
    tiles, the slices meeting through the last-arriving workgroup; verify and draft passes against the
    oracle."""
    t = tiny
    monkeypatch.setenv("NLD_SPLITK", str(ksplit))
    monkeypatch.setenv("NLD_SPLITK_CT", str(ct))
    ws = R.Workspace(t["model"], 1, 8, 256)
    for mode in (O.VERIFY, O.DRAFT):
        ref, _, _ = O.block_forward(t["w"], t["okv"], t["block"], mode)
        logits, am = R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(t["block"]).cuda(),
                                     R.VERIFY if mode == O.VERIFY else R.DRAFT)
        g = logits.cpu().numpy()
        e = rel_err(g, ref)
        log("tiny split-K ksplit=%d ct=%d %s: rel err %.3e" % (ksplit, ct, mode, e))
        assert e <= TOL
        check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    assert R.read_device_status(ws) == 0


@pytest.mark.parametrize("k,qkv", [(16, ""), (32, ""), (16, "4,2"), (32, "3,3")])
def test_8b_layer_split_k_repeatable(R, layer8b, monkeypatch, k, qkv):
    """The split-K projections' result does not depend on which workgroup arrives last: ten verify
    passes over the same block give bit-identical logits (a partial read before it was visible
    would change them), within tolerance of the oracle.  `qkv` also puts the QKV projection on
    the split-K kernel (ct tiles, ksplit slices)."""
    if qkv:
        monkeypatch.setenv("NLD_SPLITK_QKV", qkv)
    t = layer8b
    shape = t["shape"]
    tok = synth_tokens(shape, t["seed"], "8b_layer.block%d" % k, (1, k))
    ref, _, _ = O.block_forward(t["w"], t["okv"], tok, O.VERIFY)
    ws = R.Workspace(t["model"], 1, k, t["cache"].max_len)
    tt = torch.from_numpy(tok).cuda()
    first, _ = R.block_forward(t["model"], t["cache"], ws, tt, R.VERIFY)
    first = first.cpu().numpy()
    assert rel_err(first, ref) <= TOL
    for i in range(9):
        again, _ = R.block_forward(t["model"], t["cache"], ws, tt, R.VERIFY)
        assert np.array_equal(again.cpu().numpy(), first), "pass %d differs" % (i + 1)
    assert R.read_device_status(ws) == 0


@pytest.mark.parametrize("k,ksplit", [(24, 3), (40, 3), (64, 8), (24, 0), (56, 0)])
def test_tiny_split_k_many_rows(R, tiny, monkeypatch, k, ksplit):
    """17..64 rows.  ksplit > 0: every projection (QKV, O, gate/up, down) on the split-K kernel with two
    or four row tiles (four: one accumulator per tile for both operand halves), ksplit ragged K slices.
    ksplit = 0: the default plan, the multi-tile kernel that holds the operand's K slice in registers
    (the LM head too).  Verify and draft passes against the oracle."""
    t = tiny
    if ksplit:
        monkeypatch.setenv("NLD_NO_NORMK", "1")
        monkeypatch.setenv("NLD_SPLITK", str(ksplit))
    block = synth_tokens(t["shape"], 0, "tiny.block%d" % k, (1, k))
    ws = R.Workspace(t["model"], 1, k, 256)
    for mode in (O.VERIFY, O.DRAFT):
        ref, _, _ = O.block_forward(t["w"], t["okv"], block, mode)
        logits, am = R.block_forward(t["model"], t["cache"], ws, torch.from_numpy(block).cuda(),
                                     R.VERIFY if mode == O.VERIFY else R.DRAFT)
        g = logits.cpu().numpy()
        e = rel_err(g, ref)
        log("tiny split-K k=%d ksplit=%d %s: rel err %.3e" % (k, ksplit, mode, e))
        assert e <= TOL
        check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    assert R.read_device_status(ws) == 0
