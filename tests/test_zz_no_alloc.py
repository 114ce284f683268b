"""The allocation-free verify entry point (nld_verify_accept_noalloc) against nld_verify_accept.

Both run the same kernels with the same launch plan, the first on the library's static per-device
scratch array and the second on a caller-owned workspace, so every output must agree bit for bit:
logits, argmax-derived acceptance, committed tokens, next anchors, lengths, every cache row and the
device status bits.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_05722_amd import _lib as C
from synth.workloads import LazyWeights, WORKLOADS, prefix_kv, tokens as synth_tokens


def _fake_model(hidden, n_layers, q, kv, ffn, vocab):
    cfg = C.Config(n_layers, hidden, q, kv, 128, ffn, vocab, 1e4, 1e-6, vocab - 1, 0, 0.0)
    fake = 0x1000
    layers = (C.LayerWeights * n_layers)(*[C.LayerWeights(fake, fake, fake, fake, fake, fake) for _ in range(n_layers)])
    w = C.Weights(fake, fake, fake, layers)
    h = ctypes.c_void_p()
    C.check(C.load().nld_model_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(h)))
    return h


def test_noalloc_rejects_calls_beyond_its_scratch():
    """Host-side checks (no GPU needed): a call whose scratch exceeds the static array is refused with
    NLD_ERR_CAPACITY and a message naming the limit; a call that fits but has a NULL output is refused
    before anything touches the device."""
    lib = C.load()
    h = _fake_model(4096, 36, 32, 8, 12288, 151936)
    fake = 0x2000
    big = C.KVCache(fake, fake, fake, 4, 8192)
    st = lib.nld_verify_accept_noalloc(h, ctypes.byref(big), fake, fake, 4, 16, fake, fake, fake, None, None, None)
    assert st == C.NLD_ERR_CAPACITY
    assert b"allocation-free" in lib.nld_last_error() and str(C.NLD_NOALLOC_SCRATCH_BYTES).encode() in lib.nld_last_error()
    assert lib.nld_workspace_bytes(h, 4, 16, 8192) > C.NLD_NOALLOC_SCRATCH_BYTES
    one = C.KVCache(fake, fake, fake, 1, 4608)
    assert lib.nld_workspace_bytes(h, 1, 16, 4608) <= C.NLD_NOALLOC_SCRATCH_BYTES
    st = lib.nld_verify_accept_noalloc(h, ctypes.byref(one), None, fake, 1, 16, fake, fake, fake, None, None, None)
    assert st == C.NLD_ERR_INVALID_ARG
    lib.nld_model_destroy(h)


@pytest.mark.gpu
def test_noalloc_verify_equals_workspace_verify():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_05722_amd import runtime as R
    wl = WORKLOADS["tiny"]
    shape, seed, max_len = wl.shape, wl.seed, 256
    model = R.DeviceModel(shape, LazyWeights(shape, seed))

    def cache_with(lengths):
        c = R.DeviceCache(shape, len(lengths), max_len)
        for l in range(shape.n_layers):
            kb, vb = prefix_kv(shape, seed, l, len(lengths), int(max(lengths)))
            c.load_prefix(l, kb, vb)
        c.set_lengths(lengths)
        return c

    # two calls in a row, the second smaller; the first has a sequence whose block runs past max_len
    # (capacity bit set, length stopped at max_len), the second must see its own, clear status
    for call, (lengths, k, want_status) in enumerate([([100, 37, 250], 8, C.NLD_DEV_CAPACITY), ([60, 3], 4, 0)]):
        B = len(lengths)
        print("no-alloc call %d: batch %d, k %d, lengths %s" % (call, B, k, lengths), flush=True)
        ca, cb = cache_with(lengths), cache_with(lengths)
        anchor = torch.from_numpy(synth_tokens(shape, seed, "noalloc.anchor%d" % call, (B,))).cuda()
        drafts = torch.from_numpy(synth_tokens(shape, seed, "noalloc.drafts%d" % call, (B, k - 1))).cuda()
        ws = R.Workspace(model, B, k, max_len)
        ref = R.verify_accept(model, ca, ws, anchor.clone(), drafts, k, want_logits=True)
        status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        got = R.verify_accept_noalloc(model, cb, anchor.clone(), drafts, k, want_logits=True, device_status=status)
        torch.cuda.synchronize()
        assert torch.equal(got["logits"], ref["logits"])
        for name in ("accept_len", "committed", "next_anchor"):
            assert torch.equal(got[name], ref[name]), name
        assert torch.equal(cb.lengths, ca.lengths)
        assert torch.equal(cb.k, ca.k) and torch.equal(cb.v, ca.v)
        ws_bits = ctypes.c_uint32(0)
        C.load().nld_read_device_status(ctypes.c_void_p(ws.ptr), ctypes.byref(ws_bits), ctypes.c_void_p(R.stream_handle()))
        assert int(status.cpu()[0]) == ws_bits.value == want_status
        if want_status:
            assert int(cb.lengths.cpu().max()) <= max_len
    model.close()
