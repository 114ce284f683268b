"""GPU parity of Mode 2, block-wise diffusion denoising with confidence-based sampling (Sec. 3.2),
against the CPU oracle, through the C ABI.

Every denoising step runs on both sides from the same block (the oracle's, uploaded), so the two
trajectories cannot drift apart.  Bar:
* logits within 2e-2 normwise relative error of the fp32 oracle;
* the device's confidences within 1e-5 of those recomputed from its own logits, and within the bound
  a logit error e implies (|d ln c| <= 2e) of the oracle's;
* the commit bit-exact given the device's own argmax and confidences (the decision taken in the
  same precision on both sides), and equal to the oracle's commit on every sequence where no
  confidence lies within that bound of the threshold (or, for the fallback, of another masked row's);
* the refresh's K/V rows within 2e-2 of the oracle's, lengths and next anchors exact.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import nld_oracle as O
from synth.workloads import LazyWeights, WORKLOADS, prefix_kv, tokens as synth_tokens

from gpu_common import decision_near_tie, log, log_conf_bound, own_commit, rel_err

pytestmark = pytest.mark.gpu

TOL = 2e-2
CONF_SELF_RTOL = 1e-5


@pytest.fixture(scope="module")
def R():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime
    return runtime


def pick_threshold(conf: np.ndarray, rows_mask: np.ndarray) -> float:
    """A threshold that splits the given confidences near their median, placed in the widest relative gap
    among the middle half so that no confidence sits close to it."""
    c = np.sort(np.log(conf[rows_mask]))
    lo, hi = len(c) // 4, max(len(c) // 4 + 1, (3 * len(c)) // 4)
    gaps = c[lo + 1:hi + 1] - c[lo:hi]
    i = lo + int(np.argmax(gaps))
    return float(np.exp(0.5 * (c[i] + c[i + 1])))


def compare_step(block_in, gpu, ref, threshold, mask_id, what):
    """Check one denoising step (see the module docstring).  Returns the near-tie sequences."""
    g_logits = gpu["logits"].cpu().numpy()
    g_conf = gpu["confidence"].cpu().numpy()
    g_block = gpu["block"].cpu().numpy()
    e = rel_err(g_logits, ref["logits"])
    err_abs = e * float(np.max(np.abs(ref["logits"])))
    assert e <= TOL, "%s: logits rel err %.3e" % (what, e)
    own_conf = O.top1_confidence(O.denoising_logits(g_logits, mask_id))
    np.testing.assert_allclose(g_conf, own_conf, rtol=CONF_SELF_RTOL, err_msg=what + ": confidence vs own logits")
    d = log_conf_bound(err_abs)
    assert np.all(np.abs(np.log(g_conf.astype(np.float64)) - np.log(ref["conf"])) <= d + 1e-6), \
        what + ": confidence vs oracle beyond the logit-error bound"
    expect_own, _ = own_commit(block_in, g_logits, g_conf, threshold, mask_id)
    assert np.array_equal(g_block, expect_own), what + ": commit differs from the rule on the device's own values"
    near = decision_near_tie(block_in, ref["logits"], ref["conf"], threshold, mask_id, err_abs)
    for b in range(block_in.shape[0]):
        if b not in near:
            assert np.array_equal(g_block[b], ref["block"][b]), "%s: sequence %d commit differs" % (what, b)
    n_after = np.sum(g_block[:, 1:] == mask_id, axis=1)
    n_before = np.sum(block_in[:, 1:] == mask_id, axis=1)
    assert np.array_equal(gpu["n_masked"].cpu().numpy(), n_after)
    assert np.array_equal(gpu["n_committed"].cpu().numpy(), n_before - n_after)
    log("%s: rel err %.2e, committed %s, near-tie sequences %s" % (what, e, (n_before - n_after).tolist(), near))
    return near


def gpu_step(R, model, cache, ws, block_np, threshold):
    blk = torch.from_numpy(np.ascontiguousarray(block_np, dtype=np.int32)).cuda()
    out = R.denoise_step(model, cache, ws, blk, threshold, want_logits=True)
    out["block"] = blk
    return out


# ----------------------------------------------------------------------------- the decision alone
def test_commit_from_logits(R):
    """Confidence, argmax without the mask token and the threshold commit on identical logits, with
    planted cases: the mask token's logit the largest of its row, equal confidences everywhere (the
    fallback takes the first masked row), a block with no mask left, partly committed blocks and an
    exact top-2 tie."""
    B, k, V = 6, 16, 5003
    mask = V - 1
    z = (3.0 * synth.normal_f64(7, "m2.logits", (B, k, V))).astype(np.float32)
    z[0, 3, mask] = 50.0
    z[1, :, :] = z[1, 0, :]
    z[5, 6, [100, 2000]] = 40.0
    block = synth.uniform_int(7, "m2.block", (B, k), 0, V - 2).astype(np.int32)
    block[:, 1:] = mask
    block[2, 1:] = synth.uniform_int(7, "m2.done", (k - 1,), 0, V - 2)
    block[4, 1:8] = synth.uniform_int(7, "m2.part", (7,), 0, V - 2)
    ref_z = O.denoising_logits(z, mask)
    ref_pred, ref_conf = O.argmax_first(ref_z), O.top1_confidence(ref_z)
    assert ref_pred[0, 3] != mask and ref_pred[5, 6] == 100
    for tau in [pick_threshold(ref_conf, np.broadcast_to(block == mask, ref_conf.shape)), -1.0, 2.0]:
        blk = torch.from_numpy(block.copy()).cuda()
        out = R.commit_from_logits(torch.from_numpy(z).cuda(), blk, mask, tau)
        g_block, g_conf = blk.cpu().numpy(), out["confidence"].cpu().numpy()
        assert np.array_equal(out["argmax"].cpu().numpy(), ref_pred)
        np.testing.assert_allclose(g_conf, ref_conf, rtol=CONF_SELF_RTOL)
        expect = block.copy()
        for b in range(B):
            expect[b], rows = O.threshold_commit(block[b], ref_pred[b], ref_conf[b], tau, mask)
            assert int(out["n_committed"][b]) == len(rows)
        assert np.array_equal(g_block, expect), "tau %g" % tau
        assert np.array_equal(out["n_masked"].cpu().numpy(), np.sum(expect[:, 1:] == mask, axis=1))
        assert int(out["n_committed"][2]) == 0
        if tau == 2.0:
            assert np.array_equal(out["n_committed"].cpu().numpy(), [1, 1, 0, 1, 1, 1])
            assert g_block[1, 1] == ref_pred[1, 1] and np.all(g_block[1, 2:] == mask)   # equal confidences
        if tau == -1.0:
            assert not np.any(g_block[:, 1:] == mask)


# ----------------------------------------------------------------------------- tiny workload (real prefix)
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
    for c0 in range(0, wl.prefix_len, 16):               # causal prefill = verify passes, every row committed
        R.block_forward(model, cache, ws16, pt[:, c0:c0 + 16].contiguous(), R.VERIFY, want_logits=False)
        cache.lengths += 16
    torch.cuda.synchronize()
    return dict(shape=shape, w=w, okv=okv, model=model, cache=cache)


def test_tiny_diffusion_block_and_refresh(R, tiny):
    """A whole Mode 2 block (k=8) on the tiny model: every denoising step from the oracle's block, the
    refresh of the finished block (K/V rows of both layers, lengths, next anchor), then one AR step on
    the refreshed cache."""
    t = tiny
    shape, k = t["shape"], 8
    mask = shape.mask_token_id
    okv = t["okv"].copy()
    cache = R.DeviceCache(shape, 1, 256)
    cache.k.copy_(t["cache"].k)
    cache.v.copy_(t["cache"].v)
    cache.lengths.copy_(t["cache"].lengths)
    ws = R.Workspace(t["model"], 1, k, 256)
    anchor = synth_tokens(shape, 0, "tiny.m2.anchor", (1,))
    block = O.draft_block(anchor, k, mask)
    first = O.denoise_step(t["w"], okv, block, 1.0)
    tau = pick_threshold(first["conf"], block == mask)
    steps = 0
    while np.any(block[:, 1:] == mask):
        ref = O.denoise_step(t["w"], okv, block, tau)
        gpu = gpu_step(R, t["model"], cache, ws, block, tau)
        compare_step(block, gpu, ref, tau, mask, "tiny step %d" % steps)
        block = ref["block"]
        steps += 1
        assert steps <= k - 1
    P = int(okv.lengths[0])
    nxt_o = O.refresh(t["w"], okv, block)
    nxt_g = R.refresh_block(t["model"], cache, ws, torch.from_numpy(block).cuda())
    assert int(nxt_g.cpu()[0]) == int(nxt_o[0]) == int(block[0, -1])
    assert int(cache.lengths.cpu()[0]) == int(okv.lengths[0]) == P + k - 1
    for l in range(shape.n_layers):
        kg, vg = cache.read_kv(l, P, P + k - 1)
        assert rel_err(O.bf16_bits_to_float(kg), okv.k[l][:, :, P:P + k - 1]) < TOL
        assert rel_err(O.bf16_bits_to_float(vg), okv.v[l][:, :, P:P + k - 1]) < TOL
    tok_o, logit_o = O.ar_step(t["w"], okv, nxt_o)
    out = R.verify_accept(t["model"], cache, ws, nxt_g, None, 1, want_logits=True)
    e = rel_err(out["logits"].cpu().numpy()[:, 0], logit_o[:, 0])
    log("tiny: %d denoising steps at threshold %.3g; AR step after refresh rel err %.2e" % (steps, tau, e))
    assert e <= TOL
    assert R.read_device_status(ws) == 0


def test_refresh_reports_a_mask_left(R, tiny):
    t = tiny
    k = 8
    cache = R.DeviceCache(t["shape"], 1, 256)
    cache.set_lengths([128])
    ws = R.Workspace(t["model"], 1, k, 256)
    blk = O.draft_block(synth_tokens(t["shape"], 0, "tiny.m2.anchor", (1,)), k, t["shape"].mask_token_id)
    R.refresh_block(t["model"], cache, ws, torch.from_numpy(blk).cuda())
    assert R.read_device_status(ws) & 0x8


# ----------------------------------------------------------------------------- 8B-shaped layer, batch 1 and 2
@pytest.fixture(scope="module")
def layer8b2(R):
    wl = WORKLOADS["8b_layer"]
    shape, seed, P = wl.shape, wl.seed, wl.prefix_len
    src = LazyWeights(shape, seed)
    kb, vb = prefix_kv(shape, seed, 0, 2, P)
    w = O.OracleWeights(shape, src, np.float32)
    model = R.DeviceModel(shape, src)
    return dict(shape=shape, w=w, kb=kb, vb=vb, P=P, model=model, seed=seed)


@pytest.mark.parametrize("batch", [1, 2])
def test_8b_layer_denoising_and_refresh(R, layer8b2, batch):
    """One 8B-shaped layer + the 151936-token LM head, k=16: two denoising steps and the refresh.  Batch 1
    runs the LM head on the normed multi-tile kernel, batch 2 (32 rows) on the streamed kernel."""
    t = layer8b2
    shape, k, P = t["shape"], 16, t["P"]
    mask = shape.mask_token_id
    okv = O.OracleKV(shape, batch, P + 64, np.float32)
    okv.set_prefix_bf16(0, t["kb"][:batch], t["vb"][:batch], [P] * batch)
    cache = R.DeviceCache(shape, batch, P + 64)
    cache.load_prefix(0, t["kb"][:batch], t["vb"][:batch])
    cache.set_lengths([P] * batch)
    ws = R.Workspace(t["model"], batch, k, P + 64)
    anchor = synth_tokens(shape, t["seed"], "8b_layer.m2.anchor", (batch,))
    block = O.draft_block(anchor, k, mask)
    first = O.denoise_step(t["w"], okv, block, 1.0)
    tau = pick_threshold(first["conf"], block == mask)
    for step in range(2):
        ref = O.denoise_step(t["w"], okv, block, tau)
        gpu = gpu_step(R, t["model"], cache, ws, block, tau)
        compare_step(block, gpu, ref, tau, mask, "8b_layer batch %d step %d" % (batch, step))
        block = ref["block"]
    block[:, 1:] = np.where(block[:, 1:] == mask, synth_tokens(shape, t["seed"], "8b_layer.m2.fill", (batch, k - 1)),
                            block[:, 1:])
    O.refresh(t["w"], okv, block)
    nxt = R.refresh_block(t["model"], cache, ws, torch.from_numpy(block).cuda())
    assert np.array_equal(nxt.cpu().numpy(), block[:, -1])
    assert np.all(cache.lengths.cpu().numpy() == P + k - 1)
    kg, vg = cache.read_kv(0, P, P + k - 1)
    assert rel_err(O.bf16_bits_to_float(kg), okv.k[0][:, :, P:P + k - 1]) < TOL
    assert rel_err(O.bf16_bits_to_float(vg), okv.v[0][:, :, P:P + k - 1]) < TOL
    assert R.read_device_status(ws) == 0
