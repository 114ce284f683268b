"""GPU parity at the full workload sizes, on the launch configuration the benchmark times.

The oracle cannot afford every sequence of the large batches, so it recomputes a
sample of sequences (every sequence's block is independent of the others) and the
comparison covers those sequences' logits, argmax and acceptance.  All inputs come
from the seeded generator; the oracle never sees a GPU result.
"""
import numpy as np
import pytest
import torch

from oracle import nld_oracle as O
from synth.workloads import LazyWeights, ModelShape, WORKLOADS, prefix_kv, tokens as synth_tokens

from gpu_common import check_argmax, log, rel_err

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def R():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime
    return runtime


class SubBatch:
    """Prefix K/V of a subset of a batch's sequences, drawn from the full-batch generator."""

    def __init__(self, wl, seqs):
        self.wl, self.seqs = wl, list(seqs)
        self.lengths = wl.prefix_lengths()

    def fill(self, okv, cache_gpu, max_prefix):
        shape = self.wl.shape
        for l in range(shape.n_layers):
            kb, vb = prefix_kv(shape, self.wl.seed, l, self.wl.batch, max_prefix)
            cache_gpu.load_prefix(l, kb, vb)
            okv.set_prefix_bf16(l, kb[self.seqs], vb[self.seqs], self.lengths[self.seqs])
            del kb, vb


def _setup(R, name, seqs):
    wl = WORKLOADS[name]
    shape, k, B = wl.shape, wl.k_values[0], wl.batch
    plens = wl.prefix_lengths()
    maxp = int(plens.max())
    max_len = (maxp + 2 * k + 63) // 64 * 64
    src = LazyWeights(shape, wl.seed, keep=True)
    log("%s: building model" % name)
    model = R.DeviceModel(shape, src)
    cache = R.DeviceCache(shape, B, max_len)
    okv = O.OracleKV(shape, len(seqs), max_len, np.float32)
    SubBatch(wl, seqs).fill(okv, cache, maxp)
    cache.set_lengths(plens)
    w = O.OracleWeights(shape, src, np.float32)
    return wl, shape, k, B, plens, max_len, model, cache, okv, w


def test_8b_full_self_speculation_step(R):
    """36-layer 8B stack, batch 1, prefix 4096, k=16: draft pass, verify pass, acceptance and commit."""
    wl, shape, k, B, plens, max_len, model, cache, okv, w = _setup(R, "8b", [0])
    anchor = synth_tokens(shape, wl.seed, "test.8b.anchor", (1,))
    ws = R.Workspace(model, B, k, max_len)
    a_g = torch.from_numpy(anchor).cuda()
    d_g, dl = R.draft(model, cache, ws, a_g, k, want_logits=True)
    gd = d_g.cpu().numpy()
    log("8b: oracle draft pass")
    od, ref_d = O.draft_pass(w, okv, anchor, k)
    e_d = rel_err(dl.cpu().numpy(), ref_d)
    log("8b: draft rel err %.3e" % e_d)
    assert e_d <= TOL
    # draft tokens: argmax of GPU draft logits; equal to the oracle's except on near-ties
    near = check_argmax(gd, dl.cpu().numpy()[:, 1:], ref_d[:, 1:], e_d * np.max(np.abs(ref_d)))
    log("8b: near-tie draft rows differing: %s" % near)
    # verify on the oracle's drafts (GPU and oracle consume the same drafts)
    drafts = od.astype(np.int32)
    out = R.verify_accept(model, cache, ws, a_g, torch.from_numpy(drafts).cuda(), k, want_logits=True)
    log("8b: oracle verify pass")
    a, ref_v, nk, nv = O.verify_pass(w, okv, anchor, drafts)
    g_v = out["logits"].cpu().numpy()
    e_v = rel_err(g_v, ref_v)
    log("8b: verify rel err %.3e" % e_v)
    assert e_v <= TOL
    # acceptance is bit-exact given the GPU's own argmax; equal to the oracle's away from near-ties
    g_a = np.argmax(g_v, axis=-1).astype(np.int32)
    L, committed, bonus = O.accept(drafts[0], g_a[0])
    assert int(out["accept_len"].cpu()[0]) == L
    assert out["committed"][0].cpu().tolist()[:L + 1] == committed
    assert int(out["next_anchor"].cpu()[0]) == bonus
    assert int(cache.lengths.cpu()[0]) == int(plens[0]) + L + 1
    check_argmax(g_a, g_v, ref_v, e_v * np.max(np.abs(ref_v)))
    kg, vg = cache.read_kv(shape.n_layers - 1, int(plens[0]), int(plens[0]) + k)
    assert rel_err(O.bf16_bits_to_float(kg), nk[-1]) < TOL
    assert rel_err(O.bf16_bits_to_float(vg), nv[-1]) < TOL
    assert R.read_device_status(ws) == 0


def test_8b_batch32_ragged_verify(R):
    """36-layer 8B, batch 32 with ragged prefixes in [512, 8192], k=16, verify mask: sequences with the
    shortest, the longest and a middle prefix are recomputed by the oracle."""
    wl = WORKLOADS["8b_batch32"]
    plens = wl.prefix_lengths()
    order = np.argsort(plens, kind="stable")
    seqs = [int(order[0]), int(order[-1]), int(order[len(order) // 2])]
    wl, shape, k, B, plens, max_len, model, cache, okv, w = _setup(R, "8b_batch32", seqs)
    blk = synth_tokens(shape, wl.seed, "test.8b_batch32.block", (B, k))
    ws = R.Workspace(model, B, k, max_len)
    logits, am = R.block_forward(model, cache, ws, torch.from_numpy(blk).cuda(), R.VERIFY)
    g = logits.cpu().numpy()[seqs]
    log("8b_batch32: oracle verify pass over sequences %s (prefixes %s)" % (seqs, plens[seqs].tolist()))
    ref, _, _ = O.block_forward(w, okv, blk[seqs], O.VERIFY)
    e = rel_err(g, ref)
    log("8b_batch32: rel err %.3e" % e)
    assert e <= TOL
    check_argmax(am.cpu().numpy()[seqs], g, ref, e * np.max(np.abs(ref)))
    # every sequence's argmax is the first maximum of its own logits
    assert np.array_equal(am.cpu().numpy(), np.argmax(logits.cpu().numpy(), axis=-1))
    assert R.read_device_status(ws) == 0


def test_14b_self_speculation_step(R):
    """40-layer 14B shape, batch 8, prefix 16384, k=32: draft + verify + acceptance; sequences 0 and 5
    are recomputed by the oracle."""
    seqs = [0, 5]
    wl, shape, k, B, plens, max_len, model, cache, okv, w = _setup(R, "14b", seqs)
    anchor = synth_tokens(shape, wl.seed, "test.14b.anchor", (B,))
    ws = R.Workspace(model, B, k, max_len)
    a_g = torch.from_numpy(anchor).cuda()
    d_g, dl = R.draft(model, cache, ws, a_g, k, want_logits=True)
    log("14b: oracle draft pass")
    od, ref_d = O.draft_pass(w, okv, anchor[seqs], k)
    e_d = rel_err(dl.cpu().numpy()[seqs], ref_d)
    log("14b: draft rel err %.3e" % e_d)
    assert e_d <= TOL
    drafts = synth_tokens(shape, wl.seed, "test.14b.drafts", (B, k - 1))
    drafts[seqs] = od
    out = R.verify_accept(model, cache, ws, a_g, torch.from_numpy(drafts).cuda(), k, want_logits=True)
    log("14b: oracle verify pass")
    a, ref_v, _, _ = O.verify_pass(w, okv, anchor[seqs], drafts[seqs])
    g_v = out["logits"].cpu().numpy()
    e_v = rel_err(g_v[seqs], ref_v)
    log("14b: verify rel err %.3e" % e_v)
    assert e_v <= TOL
    g_a = np.argmax(g_v, axis=-1).astype(np.int32)
    for b in range(B):
        L, committed, bonus = O.accept(drafts[b], g_a[b])
        assert int(out["accept_len"].cpu()[b]) == L
        assert out["committed"][b].cpu().tolist()[:L + 1] == committed
        assert int(cache.lengths.cpu()[b]) == int(plens[b]) + L + 1
    check_argmax(g_a[seqs], g_v[seqs], ref_v, e_v * np.max(np.abs(ref_v)))
    assert R.read_device_status(ws) == 0


def test_8b_full_denoising_step_and_refresh(R):
    """Mode 2 at the full 8B size (36 layers, prefix 4096, k=16): one denoising step from [anchor, masks]
    at a threshold every confidence exceeds (the whole block is decoded at once), then the refresh of the
    oracle's decoded block, compared on the K/V rows of every layer, the lengths and the next anchor."""
    wl, shape, k, B, plens, max_len, model, cache, okv, w = _setup(R, "8b", [0])
    mask = shape.mask_token_id
    anchor = synth_tokens(shape, wl.seed, "test.8b.m2.anchor", (1,))
    block = O.draft_block(anchor, k, mask)
    ws = R.Workspace(model, B, k, max_len)
    blk = torch.from_numpy(block.copy()).cuda()
    out = R.denoise_step(model, cache, ws, blk, -1.0, want_logits=True)
    log("8b: oracle denoising step")
    ref = O.denoise_step(w, okv, block, -1.0)
    g = out["logits"].cpu().numpy()
    e = rel_err(g, ref["logits"])
    log("8b: denoising rel err %.3e" % e)
    assert e <= TOL
    err_abs = e * float(np.max(np.abs(ref["logits"])))
    g_conf = out["confidence"].cpu().numpy()
    np.testing.assert_allclose(g_conf, O.top1_confidence(O.denoising_logits(g, mask)), rtol=1e-5)
    assert np.all(np.abs(np.log(g_conf.astype(np.float64)) - np.log(ref["conf"])) <= 2 * err_abs + 1e-6)
    g_block = blk.cpu().numpy()
    own = O.argmax_first(O.denoising_logits(g, mask))
    assert np.array_equal(g_block[:, 1:], own[:, 1:]) and g_block[0, 0] == anchor[0]
    assert int(out["n_committed"].cpu()[0]) == k - 1 and int(out["n_masked"].cpu()[0]) == 0
    near = check_argmax(own[:, 1:], np.where(np.arange(shape.vocab) == mask, -np.inf, g)[:, 1:],
                        O.denoising_logits(ref["logits"], mask)[:, 1:], err_abs)
    log("8b: near-tie denoised rows differing: %s" % near)
    assert int(cache.lengths.cpu()[0]) == int(plens[0])          # denoising never commits
    P = int(plens[0])
    dec = ref["block"]
    nxt = R.refresh_block(model, cache, ws, torch.from_numpy(dec).cuda())
    log("8b: oracle refresh")
    nxt_o = O.refresh(w, okv, dec)
    assert int(nxt.cpu()[0]) == int(nxt_o[0])
    assert int(cache.lengths.cpu()[0]) == P + k - 1 == int(okv.lengths[0])
    for l in range(shape.n_layers):
        kg, vg = cache.read_kv(l, P, P + k - 1)
        assert rel_err(O.bf16_bits_to_float(kg), okv.k[l][:, :, P:P + k - 1]) < TOL, "layer %d K" % l
        assert rel_err(O.bf16_bits_to_float(vg), okv.v[l][:, :, P:P + k - 1]) < TOL, "layer %d V" % l
    assert R.read_device_status(ws) == 0


def test_8b_full_lora_draft(R):
    """The 36-layer 8B draft pass with the paper's adapter (rank 128, alpha 512) attached to the benchmark's
    weights, against the oracle with the same adapter."""
    from synth.workloads import lora_weights
    wl, shape, k, B, plens, max_len, model, cache, okv, _ = _setup(R, "8b", [0])
    lshape = ModelShape(**{**shape.__dict__, "lora_rank": 128, "lora_alpha": 512.0})
    src = LazyWeights(shape, wl.seed, keep=False)

    class Src:
        embed, lm_head, final_norm = src.embed, src.lm_head, src.final_norm

        @staticmethod
        def layer(l):
            return {**src.layer(l), **lora_weights(lshape, wl.seed, l)}

    lmodel = model.with_lora(lshape, lambda l: lora_weights(lshape, wl.seed, l))
    anchor = synth_tokens(shape, wl.seed, "test.8b.lora.anchor", (1,))
    ws = R.Workspace(lmodel, B, k, max_len)
    d, dl = R.draft(lmodel, cache, ws, torch.from_numpy(anchor).cuda(), k, want_logits=True)
    log("8b: oracle draft pass with the adapter")
    od, ref = O.draft_pass(O.OracleWeights(lshape, Src, np.float32), okv, anchor, k)
    g = dl.cpu().numpy()
    e = rel_err(g, ref)
    log("8b lora: draft rel err %.3e" % e)
    assert e <= TOL
    near = check_argmax(d.cpu().numpy(), g[:, 1:], ref[:, 1:], e * np.max(np.abs(ref)))
    log("8b lora: near-tie draft rows differing: %s" % near)
    assert R.read_device_status(ws) == 0


def test_8b_full_quad_step(R):
    """36-layer 8B stack, batch 1, prefix 4096: one quadratic self-speculation step with chain length 7
    (56 block rows, the benchmark's quadratic configuration) and the lambda = 0.5 ensemble verifier, its
    speculative tokens from the oracle's own draft pass: logits of all rows and the decisions against the
    rule on the GPU's own logits."""
    from test_gpu_quad import check_step
    wl, shape, _, B, plens, max_len, model, cache, okv, w = _setup(R, "8b", [0])
    k, lam = 7, 0.5
    anchor = synth_tokens(shape, wl.seed, "test.8b.quad.anchor", (1,))
    log("8b quad: oracle draft pass for the speculative tokens")
    spec, _ = O.draft_pass(w, okv, anchor, k)
    spec = spec.astype(np.int32)
    ws = R.QuadWorkspace(model, B, k, max_len)
    res = R.quad_step(model, cache, ws, torch.from_numpy(anchor).cuda(), torch.from_numpy(spec).cuda(), k, lam,
                      want_logits=True)
    g = res["logits"].cpu().numpy()
    log("8b quad: oracle quadratic pass")
    ref, _, _ = O.quad_forward(w, okv, anchor, spec, k)
    e = rel_err(g, ref)
    log("8b quad k=%d lambda=%.1f: rel err %.3e, L=%d" % (k, lam, e, int(res["accept_len"].cpu()[0])))
    assert e <= TOL
    check_step(res, g, spec, k, lam, plens, cache)
    assert R.read_device_status(ws) == 0
