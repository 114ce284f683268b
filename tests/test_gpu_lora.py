"""GPU parity of the LoRA-enhanced drafter (Sec. 3.3): an adapter on the O projection that only
draft-mode passes use.  Bar: draft logits within 2e-2 normwise of the fp32 oracle with the adapter;
verify passes bit-identical to the same weights without it (the AR pathway is unchanged)."""
import numpy as np
import pytest
import torch

from oracle import nld_oracle as O
from synth.workloads import LazyWeights, ModelShape, SHAPE_TINY, WORKLOADS, lora_weights, prefix_kv, \
    tokens as synth_tokens

from gpu_common import check_argmax, log, rel_err

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def R():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime
    return runtime


class WithLoRA:
    """A weight source: the base model's tensors plus each layer's adapter (generated alone)."""

    def __init__(self, base, lora_shape, seed):
        self.base, self.lora_shape, self.seed = base, lora_shape, seed

    def layer(self, l):
        return {**self.base.layer(l), **lora_weights(self.lora_shape, self.seed, l)}

    def __getattr__(self, name):          # embed, lm_head, final_norm
        return getattr(self.base, name)


def _lora(shape, rank, alpha):
    return ModelShape(**{**shape.__dict__, "lora_rank": rank, "lora_alpha": alpha})


def test_tiny_lora_draft_verify_and_denoise(R):
    """Tiny model with a rank-32 adapter (scale 4): draft pass (bidir_from 0 and 1) and a denoising step
    against the oracle; verify logits identical to the base model's; the draft differs from the base's."""
    wl = WORKLOADS["tiny"]
    shape, seed = wl.shape, wl.seed
    lshape = _lora(shape, 32, 128.0)
    src = LazyWeights(shape, seed)
    lsrc = WithLoRA(src, lshape, seed)
    prefix = synth_tokens(shape, seed, "tiny.prefix", (1, wl.prefix_len))
    block = synth_tokens(shape, seed, "tiny.lora.block", (1, 8))
    w = O.OracleWeights(lshape, lsrc, np.float32)
    okv = O.OracleKV(lshape, 1, 256, np.float32)
    O.prefill(w, okv, prefix)
    base = R.DeviceModel(shape, src)
    model = base.with_lora(lshape, lambda l: lora_weights(lshape, seed, l))
    cache = R.DeviceCache(shape, 1, 256)
    ws = R.Workspace(model, 1, 16, 256)
    pt = torch.from_numpy(prefix).cuda()
    for c0 in range(0, wl.prefix_len, 16):
        R.block_forward(model, cache, ws, pt[:, c0:c0 + 16].contiguous(), R.VERIFY, want_logits=False)
        cache.lengths += 16
    bt = torch.from_numpy(block).cuda()
    for bidir_from in (0, 1):
        ref, _, _ = O.block_forward(w, okv, block, O.DRAFT, bidir_from)
        logits, am = R.block_forward(model, cache, ws, bt, R.DRAFT, bidir_from)
        g = logits.cpu().numpy()
        e = rel_err(g, ref)
        log("tiny lora draft bidir_from=%d: rel err %.3e" % (bidir_from, e))
        assert e <= TOL
        check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
        g_base = R.block_forward(base, cache, ws, bt, R.DRAFT, bidir_from)[0].cpu().numpy()
        assert rel_err(g_base, ref) > 10 * e               # the adapter is in effect
    v_lora = R.block_forward(model, cache, ws, bt, R.VERIFY)[0].cpu().numpy()
    v_base = R.block_forward(base, cache, ws, bt, R.VERIFY)[0].cpu().numpy()
    assert np.array_equal(v_lora, v_base)
    ref_v, _, _ = O.block_forward(w, okv, block, O.VERIFY)
    assert rel_err(v_lora, ref_v) <= TOL
    # a denoising step runs the draft pathway too
    blk = O.draft_block(block[:, 0], 8, shape.mask_token_id)
    ref = O.denoise_step(w, okv, blk, -1.0)
    out = R.denoise_step(model, cache, ws, torch.from_numpy(blk).cuda(), -1.0, want_logits=True)
    assert rel_err(out["logits"].cpu().numpy(), ref["logits"]) <= TOL
    assert R.read_device_status(ws) == 0


@pytest.fixture(scope="module")
def layer8b_lora(R):
    wl = WORKLOADS["8b_layer"]
    shape, seed, P = wl.shape, wl.seed, wl.prefix_len
    lshape = _lora(shape, 128, 512.0)
    src = LazyWeights(shape, seed)
    lsrc = WithLoRA(src, lshape, seed)
    kb, vb = prefix_kv(shape, seed, 0, 2, P)
    w = O.OracleWeights(lshape, lsrc, np.float32)
    base = R.DeviceModel(shape, src)
    model = base.with_lora(lshape, lambda l: lora_weights(lshape, seed, l))
    return dict(shape=shape, w=w, kb=kb, vb=vb, P=P, base=base, model=model, seed=seed)


@pytest.mark.parametrize("batch", [1, 2])
def test_8b_layer_lora_draft(R, layer8b_lora, batch):
    """One 8B-shaped layer with the paper's adapter size (rank 128, alpha 512), k=16: draft parity at batch
    1 (16 rows) and 2 (32 rows, two row tiles in the adapter and O projection), verify unchanged."""
    t = layer8b_lora
    shape, k, P = t["shape"], 16, t["P"]
    okv = O.OracleKV(shape, batch, P + 64, np.float32)
    okv.set_prefix_bf16(0, t["kb"][:batch], t["vb"][:batch], [P] * batch)
    cache = R.DeviceCache(shape, batch, P + 64)
    cache.load_prefix(0, t["kb"][:batch], t["vb"][:batch])
    cache.set_lengths([P] * batch)
    ws = R.Workspace(t["model"], batch, k, P + 64)
    tok = synth_tokens(shape, t["seed"], "8b_layer.lora.block", (batch, k))
    ref, _, _ = O.block_forward(t["w"], okv, tok, O.DRAFT)
    logits, am = R.block_forward(t["model"], cache, ws, torch.from_numpy(tok).cuda(), R.DRAFT)
    g = logits.cpu().numpy()
    e = rel_err(g, ref)
    log("8b_layer lora batch %d: draft rel err %.3e" % (batch, e))
    assert e <= TOL
    check_argmax(am.cpu().numpy(), g, ref, e * np.max(np.abs(ref)))
    tt = torch.from_numpy(tok).cuda()
    v_lora = R.block_forward(t["model"], cache, ws, tt, R.VERIFY)[0].cpu().numpy()
    v_base = R.block_forward(t["base"], cache, ws, tt, R.VERIFY)[0].cpu().numpy()
    assert np.array_equal(v_lora, v_base)
    assert R.read_device_status(ws) == 0
