"""GPU parity of quadratic self-speculation (Sec. 3.4, Appendix C) against the CPU oracle, through the C ABI.

Bar: logits within 2e-2 normwise relative error of the fp32 oracle; the verifier, acceptance, commit and
next speculative tokens bit-exact against the rule applied to the GPU's own logits (the ensemble verifier
up to rows whose two best mixed probabilities lie within the fp32 rounding of the mixture); against the
oracle's own decisions wherever no near tie makes them ambiguous.
"""
import numpy as np
import pytest
import torch

from oracle import nld_oracle as O
from synth.workloads import LazyWeights, WORKLOADS, tokens as synth_tokens, prefix_kv

from gpu_common import log, rel_err

pytestmark = pytest.mark.gpu

TOL = 2e-2
MIX_REL = 1e-5   # fp32 mixture of two softmax values: relative rounding well below this


@pytest.fixture(scope="module")
def R():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime
    return runtime


def mixed_probs(ar: np.ndarray, diff: np.ndarray, lam: float) -> np.ndarray:
    return lam * O.softmax64(ar) + (1.0 - lam) * O.softmax64(diff)


def rule_on_logits(logits: np.ndarray, spec: np.ndarray, k: int, lam: float):
    """Verifier tokens, acceptance and next speculative tokens from given logits [B][k(k+1)][V], plus the
    positions whose ensemble decision is a near tie (two best mixed probabilities within MIX_REL)."""
    B = logits.shape[0]
    v = O.quad_verifier(logits, k, lam)
    near = np.zeros((B, k), dtype=bool)
    if 0.0 < lam < 1.0:
        p = mixed_probs(logits[:, :k], logits[:, [k + c * k for c in range(k)]], lam)
        top2 = np.sort(p, axis=-1)[..., -2:]
        near = (top2[..., 1] - top2[..., 0]) <= MIX_REL * top2[..., 1]
    am = O.argmax_first(logits)
    out = []
    for b in range(B):
        L, committed, bonus = O.accept(spec[b], v[b])
        nspec = [int(am[b, k + L * k + r - 1]) for r in range(2, k + 1)]
        out.append((L, committed, bonus, nspec))
    return out, near


def check_step(res, logits_g, spec, k, lam, P, cache):
    """The GPU's decisions equal the rule applied to its own logits (near ensemble ties excepted) and the
    chain rows it committed advanced the lengths."""
    rule, near = rule_on_logits(logits_g, spec, k, lam)
    L_g = res["accept_len"].cpu().numpy()
    com = res["committed"].cpu().numpy()
    na = res["next_anchor"].cpu().numpy()
    ns = res["next_spec"].cpu().numpy()
    lens = cache.lengths.cpu().numpy()
    for b, (L, committed, bonus, nspec) in enumerate(rule):
        if near[b, :L + 1].any():
            log("  sequence %d: ensemble near tie among positions 1..%d, decision not compared" % (b, L + 1))
            continue
        assert int(L_g[b]) == L, (b, int(L_g[b]), L)
        assert com[b].tolist() == committed + [-1] * (k - len(committed))
        assert int(na[b]) == bonus
        assert ns[b].tolist() == nspec
        assert int(lens[b]) == int(P[b]) + L + 1


@pytest.fixture(scope="module")
def tiny(R):
    wl = WORKLOADS["tiny"]
    shape, seed = wl.shape, wl.seed
    src = LazyWeights(shape, seed)
    prefix = synth_tokens(shape, seed, "tiny.prefix", (1, wl.prefix_len))
    w = O.OracleWeights(shape, src, np.float32)
    okv = O.OracleKV(shape, 1, 256, np.float32)
    O.prefill(w, okv, prefix)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, 1, 256)
    ws16 = R.Workspace(model, 1, 16, 256)
    pt = torch.from_numpy(prefix).cuda()
    for c0 in range(0, wl.prefix_len, 16):
        R.block_forward(model, cache, ws16, pt[:, c0:c0 + 16].contiguous(), R.VERIFY, want_logits=False)
        cache.lengths += 16
    torch.cuda.synchronize()
    return dict(shape=shape, w=w, okv=okv, model=model, cache=cache)


def _cache_copy(R, t, max_len=256):
    cache = R.DeviceCache(t["shape"], 1, max_len)
    cache.k.copy_(t["cache"].k)
    cache.v.copy_(t["cache"].v)
    cache.lengths.copy_(t["cache"].lengths)
    return cache


@pytest.mark.parametrize("k,lam", [(3, 1.0), (7, 1.0), (7, 0.0), (7, 0.5), (2, 0.3)])
def test_tiny_quad_step(R, tiny, k, lam):
    """One quadratic pass on the tiny model: logits of all k(k+1) rows, the chain rows' cache writes, the
    verifier, acceptance, commit and next speculative tokens."""
    t = tiny
    shape = t["shape"]
    anchor = synth_tokens(shape, 0, "quad.anchor", (1,))
    spec = synth_tokens(shape, 0, "quad.spec%d" % k, (1, k - 1))
    okv = t["okv"].copy()
    ref_logits, nk, nv = O.quad_forward(t["w"], okv, anchor, spec, k)
    cache = _cache_copy(R, t)
    ws = R.QuadWorkspace(t["model"], 1, k, 256)
    res = R.quad_step(t["model"], cache, ws, torch.from_numpy(anchor).cuda(), torch.from_numpy(spec).cuda(), k, lam,
                      want_logits=True)
    g = res["logits"].cpu().numpy()
    e = rel_err(g, ref_logits)
    log("tiny quad k=%d lambda=%.1f: rel err %.3e, L=%d" % (k, lam, e, int(res["accept_len"].cpu()[0])))
    assert e <= TOL
    check_step(res, g, spec, k, lam, [128], cache)
    kg, vg = cache.read_kv(0, 128, 128 + k)
    assert rel_err(O.bf16_bits_to_float(kg), nk[0][:, :, :k]) < TOL
    assert rel_err(O.bf16_bits_to_float(vg), nv[0][:, :, :k]) < TOL
    # the oracle's own decision agrees (its verifier tokens are not near ties at this error level)
    ref = O.quad_step(t["w"], okv, anchor, spec, k, lam)
    assert int(res["accept_len"].cpu()[0]) == int(ref["L"][0])
    assert int(res["next_anchor"].cpu()[0]) == int(ref["next_anchor"][0])
    assert res["next_spec"].cpu().numpy().tolist() == ref["next_spec"].tolist()
    assert R.read_device_status(ws) == 0


def test_tiny_quad_planted_and_loop(R, tiny):
    """Speculative tokens equal to the greedy AR continuation are accepted in full; then four steps of the
    decoding loop run with the outputs aliased to the inputs (anchor and speculative tokens updated in
    place), committing exactly what the oracle's loop commits."""
    t = tiny
    shape, k = t["shape"], 5
    okv = t["okv"].copy()
    anchor = synth_tokens(shape, 0, "quad.loop.anchor", (1,))
    okv_ar = okv.copy()
    tok, greedy = anchor.copy(), []
    for _ in range(k):
        tok, _ = O.ar_step(t["w"], okv_ar, tok)
        greedy.append(int(tok[0]))
    cache = _cache_copy(R, t)
    ws = R.QuadWorkspace(t["model"], 1, k, 256)
    a_g = torch.from_numpy(anchor).cuda()
    s_g = torch.tensor([greedy[:k - 1]], dtype=torch.int32, device="cuda")
    res = R.quad_step(t["model"], cache, ws, a_g, s_g, k, 1.0, outs={"next_anchor": a_g, "next_spec": s_g})
    assert int(res["accept_len"].cpu()[0]) == k - 1
    assert res["committed"][0].cpu().tolist() == greedy
    assert int(a_g.cpu()[0]) == greedy[-1]
    r0 = O.quad_step(t["w"], okv, anchor, np.array([greedy[:k - 1]], dtype=np.int32), k, 1.0)
    a_o, s_o = r0["next_anchor"], r0["next_spec"]
    assert s_g.cpu().numpy().tolist() == s_o.tolist()
    for step in range(4):
        ref = O.quad_step(t["w"], okv, a_o, s_o, k, 1.0)
        res = R.quad_step(t["model"], cache, ws, a_g, s_g, k, 1.0, outs={"next_anchor": a_g, "next_spec": s_g})
        L = int(res["accept_len"].cpu()[0])
        assert L == int(ref["L"][0])
        assert res["committed"][0].cpu().tolist()[:L + 1] == ref["committed"][0]
        assert int(a_g.cpu()[0]) == int(ref["next_anchor"][0])
        assert s_g.cpu().numpy().tolist() == ref["next_spec"].tolist()
        assert int(cache.lengths.cpu()[0]) == int(okv.lengths[0])
        a_o, s_o = ref["next_anchor"], ref["next_spec"]
        log("tiny quad loop step %d: L=%d" % (step, L))
    assert R.read_device_status(ws) == 0


@pytest.fixture(scope="module")
def layer8b(R):
    wl = WORKLOADS["8b_layer"]
    shape, seed = wl.shape, wl.seed
    src = LazyWeights(shape, seed)
    return dict(shape=shape, src=src, w=O.OracleWeights(shape, src, np.float32), model=R.DeviceModel(shape, src),
                seed=seed, P=wl.prefix_len)


@pytest.mark.parametrize("batch,lam", [(1, 1.0), (1, 0.5), (2, 0.5)])
def test_8b_layer_quad_step(R, layer8b, batch, lam):
    """One 8B-shaped layer + LM head, k = 7 (56 block rows per sequence: the streamed GEMMs at batch 1,
    the tiled GEMMs at batch 2 with ragged prefixes): logits, chain K/V rows and decisions."""
    t = layer8b
    shape, k, P = t["shape"], 7, t["P"]
    lengths = np.array([P, 1111][:batch])
    kb, vb = prefix_kv(shape, t["seed"], 0, batch, P)
    okv = O.OracleKV(shape, batch, P + 64, np.float32)
    okv.set_prefix_bf16(0, kb, vb, lengths)
    cache = R.DeviceCache(shape, batch, P + 64)
    cache.load_prefix(0, kb, vb)
    cache.set_lengths(lengths)
    anchor = synth_tokens(shape, t["seed"], "quad.anchor", (batch,))
    spec = synth_tokens(shape, t["seed"], "quad.spec", (batch, k - 1))
    ref_logits, nk, nv = O.quad_forward(t["w"], okv, anchor, spec, k)
    ws = R.QuadWorkspace(t["model"], batch, k, cache.max_len)
    res = R.quad_step(t["model"], cache, ws, torch.from_numpy(anchor).cuda(), torch.from_numpy(spec).cuda(), k, lam,
                      want_logits=True)
    g = res["logits"].cpu().numpy()
    e = rel_err(g, ref_logits)
    log("8b_layer quad batch=%d k=%d lambda=%.1f: rel err %.3e" % (batch, k, lam, e))
    assert e <= TOL
    check_step(res, g, spec, k, lam, lengths, cache)
    for b in range(batch):
        Pb = int(lengths[b])
        kg, vg = cache.read_kv(0, Pb, Pb + k)
        assert rel_err(O.bf16_bits_to_float(kg[b:b + 1]), nk[0][b:b + 1, :, :k]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg[b:b + 1]), nv[0][b:b + 1, :, :k]) < TOL
    assert R.read_device_status(ws) == 0
