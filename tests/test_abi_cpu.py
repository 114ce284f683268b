"""The C-ABI library loads, exports every function include/nld.h declares, and validates
arguments on the host (no GPU needed: every call here fails before anything is enqueued)."""
import ctypes
import os
import re

import pytest

from paper_2607_05722_amd import _lib as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "nld.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nld_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = C.load()
    names = declared_functions()
    assert len(names) >= 16
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(C.EXPORTED)


def test_status_strings():
    lib = C.load()
    assert lib.nld_status_string(0) == b"ok"
    assert lib.nld_status_string(-3) == b"workspace too small"


def fake_model(**over):
    cfg = dict(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=688, vocab=1024,
               rope_base=1e4, rms_eps=1e-6, mask_token_id=1023)
    cfg.update(over)
    c = C.Config(**cfg)
    fake = 0x1000
    layers = (C.LayerWeights * cfg["n_layers"])(*[C.LayerWeights(fake, fake, fake, fake, fake, fake)
                                                  for _ in range(cfg["n_layers"])])
    w = C.Weights(fake, fake, fake, layers)
    h = ctypes.c_void_p()
    st = C.load().nld_model_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(h))
    return st, h, c


def test_model_create_validates_config():
    lib = C.load()
    st, h, _ = fake_model()
    assert st == C.NLD_OK and h.value
    lib.nld_model_destroy(h)
    assert fake_model(hidden=100)[0] == C.NLD_ERR_SHAPE
    assert fake_model(head_dim=96)[0] == C.NLD_ERR_SHAPE
    assert fake_model(n_q_heads=5)[0] == C.NLD_ERR_SHAPE
    assert fake_model(ffn=690)[0] == C.NLD_ERR_SHAPE
    assert fake_model(vocab=0)[0] == C.NLD_ERR_INVALID_ARG
    assert fake_model(mask_token_id=1024)[0] == C.NLD_ERR_INVALID_ARG
    assert b"mask_token_id" in lib.nld_last_error()


def test_model_create_rejects_null_weights():
    lib = C.load()
    c = C.Config(1, 256, 4, 2, 64, 688, 1024, 1e4, 1e-6, 1023)
    layers = (C.LayerWeights * 1)(C.LayerWeights(1, 1, 0, 1, 1, 1))
    w = C.Weights(1, 1, 1, layers)
    h = ctypes.c_void_p()
    assert lib.nld_model_create(ctypes.byref(c), ctypes.byref(w), ctypes.byref(h)) == C.NLD_ERR_INVALID_ARG
    assert b"layer 0" in lib.nld_last_error()


def test_sizes():
    lib = C.load()
    st, h, c = fake_model()
    # packed: 16-column tiles x 32-deep steps x 1 KiB
    assert lib.nld_packed_bytes(C.NLD_PACK_LINEAR, ctypes.byref(c), 1000, 256) == 63 * 8 * 1024
    assert lib.nld_packed_bytes(C.NLD_PACK_LINEAR, ctypes.byref(c), 256, 688) == 16 * 22 * 1024
    assert lib.nld_packed_bytes(C.NLD_PACK_QKV, ctypes.byref(c), 512, 256) == 32 * 8 * 1024
    assert lib.nld_packed_bytes(C.NLD_PACK_GATE_UP, ctypes.byref(c), 688, 256) == 86 * 8 * 1024
    ws = lib.nld_workspace_bytes(h, 1, 8, 256)
    assert ws > 0 and ws % 256 == 0
    assert lib.nld_workspace_bytes(h, 2, 8, 256) > ws
    assert lib.nld_workspace_bytes(h, 0, 8, 256) == 0
    lib.nld_model_destroy(h)


@pytest.mark.parametrize("case,expect", [
    ("batch0", C.NLD_ERR_INVALID_ARG), ("k0", C.NLD_ERR_INVALID_ARG), ("k65", C.NLD_ERR_INVALID_ARG),
    ("mode", C.NLD_ERR_INVALID_ARG), ("bidir", C.NLD_ERR_INVALID_ARG), ("maxlen", C.NLD_ERR_INVALID_ARG),
    ("kvbatch", C.NLD_ERR_INVALID_ARG), ("ws", C.NLD_ERR_CAPACITY), ("rows", C.NLD_ERR_SHAPE),
    ("tokens", C.NLD_ERR_INVALID_ARG),
])
def test_block_forward_validation(case, expect):
    lib = C.load()
    st, h, c = fake_model(n_q_heads=16, n_kv_heads=2) if case == "rows" else fake_model()
    assert st == C.NLD_OK
    batch, k, mode, bidir, max_len = 1, 8, C.NLD_MODE_VERIFY, 0, 256
    kvb = 1
    if case == "batch0":
        batch = 0
    if case == "k0":
        k = 0
    if case == "k65":
        k = 65
    if case == "mode":
        mode = 7
    if case == "bidir":
        bidir = 9
    if case == "maxlen":
        max_len = 100
    if case == "kvbatch":
        kvb = 2
    if case == "rows":
        k = 64          # 8 query heads per KV head x 64 rows > 256
    kv = C.KVCache(0x1000, 0x1000, 0x1000, kvb, max_len)
    need = lib.nld_workspace_bytes(h, max(batch, 1), max(1, min(k, 64)), 256)
    ws_bytes = 1024 if case == "ws" else need
    tokens = 0 if case == "tokens" else 0x1000
    r = lib.nld_block_forward(h, ctypes.byref(kv), tokens, batch, k, mode, bidir, None, None, 0x1000, ws_bytes, None)
    assert r == expect, lib.nld_last_error()
    lib.nld_model_destroy(h)


def test_draft_and_verify_validation():
    lib = C.load()
    st, h, c = fake_model()
    kv = C.KVCache(0x1000, 0x1000, 0x1000, 1, 256)
    need = lib.nld_workspace_bytes(h, 1, 8, 256)
    p = 0x1000
    assert lib.nld_draft(h, ctypes.byref(kv), p, 1, 1, 0, p, None, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_draft(h, ctypes.byref(kv), 0, 1, 8, 0, p, None, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_verify_accept(h, ctypes.byref(kv), p, None, 1, 8, p, p, p, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert b"draft" in lib.nld_last_error()
    assert lib.nld_verify_accept(h, ctypes.byref(kv), p, p, 1, 8, None, p, p, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert lib.nld_accept_from_logits(p, p, 1, 8, 100, p, p, p, p, p, 4, None) == C.NLD_ERR_CAPACITY
    assert lib.nld_accept_from_logits(p, None, 1, 8, 100, p, p, p, p, p, 4096, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_pack_linear(p, 16, 20, p, None) == C.NLD_ERR_SHAPE
    lib.nld_model_destroy(h)


def test_lora_config_validation():
    lib = C.load()
    assert fake_model(lora_rank=48, lora_scale=4.0)[0] == C.NLD_ERR_SHAPE
    assert fake_model(lora_rank=544, lora_scale=4.0)[0] == C.NLD_ERR_SHAPE
    assert fake_model(lora_rank=-32, lora_scale=4.0)[0] == C.NLD_ERR_INVALID_ARG
    assert fake_model(lora_rank=32, lora_scale=float("inf"))[0] == C.NLD_ERR_INVALID_ARG
    # a rank without adapter weights (fake_model leaves lora_a / lora_b NULL)
    assert fake_model(lora_rank=32, lora_scale=4.0)[0] == C.NLD_ERR_INVALID_ARG
    assert b"lora" in lib.nld_last_error()


def test_mode2_and_decode_loop_validation():
    lib = C.load()
    st, h, c = fake_model()
    kv = C.KVCache(0x1000, 0x1000, 0x1000, 1, 256)
    need = lib.nld_workspace_bytes(h, 1, 8, 256)
    p = 0x1000
    nan = float("nan")
    # denoising step: k >= 2, non-NULL block/outputs, threshold not NaN, bidir_from range, workspace size
    assert lib.nld_denoise_step(h, ctypes.byref(kv), p, 1, 1, 0, 0.9, p, p, None, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert lib.nld_denoise_step(h, ctypes.byref(kv), None, 1, 8, 0, 0.9, p, p, None, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert lib.nld_denoise_step(h, ctypes.byref(kv), p, 1, 8, 0, nan, p, p, None, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert lib.nld_denoise_step(h, ctypes.byref(kv), p, 1, 8, 9, 0.9, p, p, None, None, p, need, None) == \
        C.NLD_ERR_INVALID_ARG
    assert lib.nld_denoise_step(h, ctypes.byref(kv), p, 1, 8, 0, 0.9, p, p, None, None, p, 64, None) == \
        C.NLD_ERR_CAPACITY
    assert lib.nld_refresh_block(h, ctypes.byref(kv), p, 1, 1, p, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_refresh_block(h, ctypes.byref(kv), p, 1, 8, None, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_commit_from_logits(p, p, 1, 8, 1, 0, 0.9, None, p, p, None, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_commit_from_logits(p, p, 1, 8, 100, 100, 0.9, None, p, p, None, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_commit_from_logits(p, p, 1, 8, 100, 99, nan, None, p, p, None, None) == C.NLD_ERR_INVALID_ARG
    # decode loop
    assert lib.nld_decode_steps(h, ctypes.byref(kv), p, 1, 8, 0, 0, p, p, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_decode_steps(h, ctypes.byref(kv), None, 1, 8, 2, 0, p, p, p, need, None) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_decode_steps(h, ctypes.byref(kv), p, 1, 8, 2, 0, p, p, p, 64, None) == C.NLD_ERR_CAPACITY
    lib.nld_model_destroy(h)


def test_choose_block_rule():
    """Self-speculation wins when its expected committed tokens per ms beat one token per AR step."""
    lib = C.load()
    assert lib.nld_choose_block(1.0, 2.0, 3.0, 16) == 16        # 1.5 tokens/ms > 1 token/ms
    assert lib.nld_choose_block(1.0, 2.0, 1.5, 16) == 1         # 0.75 < 1
    assert lib.nld_choose_block(1.0, 2.0, 2.0, 16) == 1         # a tie keeps AR
    assert lib.nld_choose_block(0.0, 2.0, 9.0, 16) == 1
    assert lib.nld_choose_block(1.0, 2.0, 9.0, 1) == 1


def test_quad_step_validation():
    """Quadratic self-speculation: k in [2, 7], lambda in [0, 1] (not NaN), non-NULL arguments, the
    quadratic workspace size, and the GQA row limit on k(k+1) block rows."""
    lib = C.load()
    st, h, c = fake_model()
    kv = C.KVCache(0x1000, 0x1000, 0x1000, 1, 256)
    p = 0x1000
    need = lib.nld_quad_workspace_bytes(h, 1, 4, 256)
    assert need > lib.nld_workspace_bytes(h, 1, 20, 256)         # plus the ensemble verifier's buffers
    assert lib.nld_quad_workspace_bytes(h, 1, 1, 256) == 0
    assert lib.nld_quad_workspace_bytes(h, 1, 8, 256) == 0
    args = lambda k=4, lam=0.5, anchor=p, spec=p, ws=need: (h, ctypes.byref(kv), anchor, spec, 1, k, lam, p, p, p, p,
                                                            None, p, ws, None)
    assert lib.nld_quad_step(*args(k=1)) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_quad_step(*args(k=8)) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_quad_step(*args(lam=1.5)) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_quad_step(*args(lam=float("nan"))) == C.NLD_ERR_INVALID_ARG
    assert b"lambda" in lib.nld_last_error()
    assert lib.nld_quad_step(*args(spec=None)) == C.NLD_ERR_INVALID_ARG
    assert lib.nld_quad_step(*args(ws=lib.nld_workspace_bytes(h, 1, 20, 256))) == C.NLD_ERR_CAPACITY
    lib.nld_model_destroy(h)
    st, h, c = fake_model(n_q_heads=16, n_kv_heads=2)             # 8 x 7 x 8 rows per KV head > 256
    kv = C.KVCache(0x1000, 0x1000, 0x1000, 1, 256)
    big = lib.nld_quad_workspace_bytes(h, 1, 7, 256)
    assert lib.nld_quad_step(h, ctypes.byref(kv), p, p, 1, 7, 1.0, p, p, p, p, None, p, big, None) == C.NLD_ERR_SHAPE
    lib.nld_model_destroy(h)
