"""Python binding of libnld: device buffers (PyTorch-ROCm) + C-ABI calls.

PyTorch only provides device memory and the stream; every step of the
block-decode path runs in libnld's HIP kernels.  Functions here marshal
arguments: they allocate outputs, pass raw pointers and check statuses.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib as C

__all__ = ["DeviceModel", "DeviceCache", "Workspace", "block_forward", "draft", "verify_accept",
           "accept_from_logits", "verify_accept_noalloc", "denoise_step", "refresh_block", "commit_from_logits", "read_device_status",
           "stream_handle", "VERIFY", "DRAFT"]

VERIFY = C.NLD_MODE_VERIFY
DRAFT = C.NLD_MODE_DRAFT


def stream_handle(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _bits_to_device(bits: np.ndarray, device) -> torch.Tensor:
    """bf16 bit patterns (uint16, host) -> int16 tensor on the device (bitwise copy)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device)


def _ptr(t) -> int:
    return 0 if t is None else t.data_ptr()


def make_config(shape) -> C.Config:
    rank = int(getattr(shape, "lora_rank", 0))
    scale = float(shape.lora_alpha) / rank if rank else 0.0
    return C.Config(shape.n_layers, shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                    shape.vocab, float(shape.rope_base), float(shape.rms_eps), int(shape.mask_token_id), rank, scale)


def _pack_lora(lib, shape, rank, device, w, packed, s):
    """Pack one layer's adapter: lora_a [rank][q_dim] and lora_b [hidden][rank] (row-major bits)."""
    qd, h = shape.q_dim, shape.hidden
    a, b = _bits_to_device(w["lora_a"], device), _bits_to_device(w["lora_b"], device)
    la, lb = packed(C.NLD_PACK_LINEAR, rank, qd), packed(C.NLD_PACK_LINEAR, h, rank)
    C.check(lib.nld_pack_linear(_ptr(a), rank, qd, _ptr(la), s))
    C.check(lib.nld_pack_linear(_ptr(b), h, rank, _ptr(lb), s))
    torch.cuda.current_stream().synchronize()
    return la, lb


class DeviceModel:
    """Uploads a model's row-major bf16 weights and packs them with the library's pack kernels.

    ``source`` provides ``layer(l)`` (dict of row-major [out][in] uint16 arrays
    named attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down),
    ``embed``, ``lm_head`` and ``final_norm``.
    """

    def __init__(self, shape, source, device="cuda"):
        self.lib = C.load()
        self.shape, self.device = shape, torch.device(device)
        self.cfg = make_config(shape)
        s = stream_handle()
        keep = []

        def packed(kind, out_dim, in_dim):
            n = self.lib.nld_packed_bytes(kind, ctypes.byref(self.cfg), out_dim, in_dim)
            assert n > 0
            t = torch.empty(n, dtype=torch.uint8, device=self.device)
            keep.append(t)
            return t

        h, qd, kvd, f = shape.hidden, shape.q_dim, shape.kv_dim, shape.ffn
        layers = (C.LayerWeights * shape.n_layers)()
        for l in range(shape.n_layers):
            w = source.layer(l)
            an, fn = _bits_to_device(w["attn_norm"], self.device), _bits_to_device(w["ffn_norm"], self.device)
            keep += [an, fn]
            wq, wk, wv = (_bits_to_device(w[n], self.device) for n in ("wq", "wk", "wv"))
            qkv = packed(C.NLD_PACK_QKV, qd + 2 * kvd, h)
            C.check(self.lib.nld_pack_qkv(ctypes.byref(self.cfg), _ptr(wq), _ptr(wk), _ptr(wv), _ptr(qkv), s))
            wo = _bits_to_device(w["wo"], self.device)
            o = packed(C.NLD_PACK_LINEAR, h, qd)
            C.check(self.lib.nld_pack_linear(_ptr(wo), h, qd, _ptr(o), s))
            wg, wu = _bits_to_device(w["w_gate"], self.device), _bits_to_device(w["w_up"], self.device)
            gu = packed(C.NLD_PACK_GATE_UP, f, h)
            C.check(self.lib.nld_pack_gate_up(ctypes.byref(self.cfg), _ptr(wg), _ptr(wu), _ptr(gu), s))
            wd = _bits_to_device(w["w_down"], self.device)
            dn = packed(C.NLD_PACK_LINEAR, h, f)
            C.check(self.lib.nld_pack_linear(_ptr(wd), h, f, _ptr(dn), s))
            la = lb = None
            if self.cfg.lora_rank:
                la, lb = self._pack_lora(w, packed, s)
            torch.cuda.current_stream().synchronize()     # row-major sources are freed below
            del wq, wk, wv, wo, wg, wu, wd
            layers[l] = C.LayerWeights(_ptr(an), _ptr(qkv), _ptr(o), _ptr(fn), _ptr(gu), _ptr(dn), _ptr(la), _ptr(lb))
        self.embed = _bits_to_device(source.embed, self.device)
        self.final_norm = _bits_to_device(source.final_norm, self.device)
        lm = _bits_to_device(source.lm_head, self.device)
        self.lm_head = packed(C.NLD_PACK_LINEAR, shape.vocab, h)
        C.check(self.lib.nld_pack_linear(_ptr(lm), shape.vocab, h, _ptr(self.lm_head), s))
        torch.cuda.current_stream().synchronize()
        del lm
        self._keep, self._layers = keep, layers
        self.weights = C.Weights(_ptr(self.embed), _ptr(self.final_norm), _ptr(self.lm_head), layers)
        handle = ctypes.c_void_p()
        C.check(self.lib.nld_model_create(ctypes.byref(self.cfg), ctypes.byref(self.weights), ctypes.byref(handle)))
        self.handle = handle

    def _pack_lora(self, w, packed, s):
        return _pack_lora(self.lib, self.shape, self.cfg.lora_rank, self.device, w, packed, s)

    def with_lora(self, lora_shape, lora_layer):
        """A second handle over these weights with a draft-pathway adapter attached.  lora_shape: this
        model's shape with lora_rank / lora_alpha set; lora_layer(l) -> dict with lora_a, lora_b bits."""
        view = ModelView(self, lora_shape)
        keep = []

        def packed(kind, out_dim, in_dim):
            n = self.lib.nld_packed_bytes(kind, ctypes.byref(view.cfg), out_dim, in_dim)
            t = torch.empty(n, dtype=torch.uint8, device=self.device)
            keep.append(t)
            return t

        s = stream_handle()
        layers = (C.LayerWeights * self.shape.n_layers)()
        for l in range(self.shape.n_layers):
            base = self._layers[l]
            la, lb = _pack_lora(self.lib, lora_shape, view.cfg.lora_rank, self.device, lora_layer(l), packed, s)
            layers[l] = C.LayerWeights(base.attn_norm, base.w_qkv, base.w_o, base.ffn_norm, base.w_gate_up,
                                       base.w_down, _ptr(la), _ptr(lb))
        view.finish(layers, keep)
        return view

    def close(self):
        if getattr(self, "handle", None):
            self.lib.nld_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class ModelView:
    """A model handle that borrows a DeviceModel's weights (see DeviceModel.with_lora)."""

    def __init__(self, base: DeviceModel, shape):
        self.base, self.shape, self.device, self.lib = base, shape, base.device, base.lib
        self.cfg = make_config(shape)
        self.handle = None

    def finish(self, layers, keep):
        self._layers, self._keep = layers, keep
        b = self.base
        self.weights = C.Weights(_ptr(b.embed), _ptr(b.final_norm), _ptr(b.lm_head), layers)
        handle = ctypes.c_void_p()
        C.check(self.lib.nld_model_create(ctypes.byref(self.cfg), ctypes.byref(self.weights), ctypes.byref(handle)))
        self.handle = handle

    def close(self):
        if getattr(self, "handle", None):
            self.lib.nld_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DeviceCache:
    """KV cache in the library's layout (see nld_kv_cache in include/nld.h)."""

    def __init__(self, shape, batch: int, max_len: int, device="cuda"):
        assert max_len % 64 == 0
        self.shape, self.batch, self.max_len = shape, batch, max_len
        L, H, D = shape.n_layers, shape.n_kv_heads, shape.head_dim
        dev = torch.device(device)
        self.k = torch.zeros((L, batch, H, max_len, D), dtype=torch.int16, device=dev)
        self.v = torch.zeros((L, batch, H, max_len // 64, D, 64), dtype=torch.int16, device=dev)
        self.lengths = torch.zeros(batch, dtype=torch.int32, device=dev)
        self.struct = C.KVCache(_ptr(self.k), _ptr(self.v), _ptr(self.lengths), batch, max_len)

    def load_prefix(self, layer: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        """Write cached K/V given as [batch][kv_heads][P][head_dim] bf16 bits into positions [0, P)."""
        P = k_bits.shape[2]
        assert P <= self.max_len
        kd = _bits_to_device(k_bits, self.k.device)
        self.k[layer, :, :, :P] = kd
        vd = _bits_to_device(v_bits, self.v.device)
        P64 = (P + 63) // 64 * 64
        vpad = torch.zeros((self.batch, self.shape.n_kv_heads, P64, self.shape.head_dim), dtype=torch.int16,
                           device=self.v.device)
        vpad[:, :, :P] = vd
        tiles = vpad.view(self.batch, self.shape.n_kv_heads, P64 // 64, 64, self.shape.head_dim).transpose(-1, -2)
        self.v[layer, :, :, :P64 // 64] = tiles

    def set_lengths(self, lengths) -> None:
        self.lengths.copy_(torch.as_tensor(np.asarray(lengths, dtype=np.int32)))

    def read_kv(self, layer: int, start: int, stop: int):
        """Host copies of K/V rows [start, stop) as [batch][kv_heads][n][head_dim] bf16 bits (uint16)."""
        k = self.k[layer, :, :, start:stop].cpu().numpy().view(np.uint16)
        vt = self.v[layer].transpose(-1, -2).reshape(self.batch, self.shape.n_kv_heads, self.max_len,
                                                     self.shape.head_dim)
        v = vt[:, :, start:stop].contiguous().cpu().numpy().view(np.uint16)
        return k, v


class Workspace:
    def __init__(self, model: DeviceModel, batch: int, k: int, max_len: int):
        lib = C.load()
        self.nbytes = lib.nld_workspace_bytes(model.handle, batch, k, max_len)
        assert self.nbytes > 0
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=model.device)
        C.check(lib.nld_workspace_init(_ptr(self.buf), self.nbytes, stream_handle()))

    @property
    def ptr(self) -> int:
        return _ptr(self.buf)


class QuadWorkspace(Workspace):
    """Workspace of quadratic self-speculation steps with chain length k (k(k+1) block rows)."""

    def __init__(self, model: DeviceModel, batch: int, k: int, max_len: int):
        lib = C.load()
        self.nbytes = lib.nld_quad_workspace_bytes(model.handle, batch, k, max_len)
        assert self.nbytes > 0
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=model.device)
        C.check(lib.nld_workspace_init(_ptr(self.buf), self.nbytes, stream_handle()))


def block_forward(model, cache, ws, tokens: torch.Tensor, mode: int, bidir_from: int = 0, want_logits=True):
    """One block pass.  tokens: int32 [batch][k] on the device.  Returns (logits or None, argmax)."""
    batch, k = tokens.shape
    dev = model.device
    logits = torch.empty((batch, k, model.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
    argmax = torch.empty((batch, k), dtype=torch.int32, device=dev)
    C.check(C.load().nld_block_forward(model.handle, ctypes.byref(cache.struct), _ptr(tokens), batch, k, mode,
                                       bidir_from, _ptr(logits), _ptr(argmax), ws.ptr, ws.nbytes, stream_handle()))
    return logits, argmax


def draft(model, cache, ws, anchor: torch.Tensor, k: int, bidir_from: int = 0, want_logits=False, out=None):
    """Diffusion draft over [anchor, mask x (k-1)].  Returns (drafts int32 [batch][k-1], logits or None)."""
    batch = anchor.shape[0]
    dev = model.device
    d = out if out is not None else torch.empty((batch, k - 1), dtype=torch.int32, device=dev)
    logits = torch.empty((batch, k, model.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
    C.check(C.load().nld_draft(model.handle, ctypes.byref(cache.struct), _ptr(anchor), batch, k, bidir_from, _ptr(d),
                               _ptr(logits), ws.ptr, ws.nbytes, stream_handle()))
    return d, logits


def verify_accept(model, cache, ws, anchor: torch.Tensor, drafts, k: int, want_logits=False, outs=None):
    """AR verify + acceptance.  Returns dict of device tensors (accept_len, committed, next_anchor, logits)."""
    batch = anchor.shape[0]
    dev = model.device
    if outs is None:
        outs = {"accept_len": torch.empty(batch, dtype=torch.int32, device=dev),
                "committed": torch.empty((batch, k), dtype=torch.int32, device=dev),
                "next_anchor": torch.empty(batch, dtype=torch.int32, device=dev)}
    logits = torch.empty((batch, k, model.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
    C.check(C.load().nld_verify_accept(model.handle, ctypes.byref(cache.struct), _ptr(anchor), _ptr(drafts), batch, k,
                                       _ptr(outs["accept_len"]), _ptr(outs["committed"]), _ptr(outs["next_anchor"]),
                                       _ptr(logits), ws.ptr, ws.nbytes, stream_handle()))
    outs = dict(outs)
    outs["logits"] = logits
    return outs


def verify_accept_noalloc(model, cache, anchor: torch.Tensor, drafts, k: int, want_logits=False, outs=None,
                          device_status=None):
    """verify_accept without a workspace: the library's static per-device scratch array stands in for it.
    ``device_status`` (optional int32 device tensor of one element) receives the call's status bits."""
    batch = anchor.shape[0]
    dev = model.device
    if outs is None:
        outs = {"accept_len": torch.empty(batch, dtype=torch.int32, device=dev),
                "committed": torch.empty((batch, k), dtype=torch.int32, device=dev),
                "next_anchor": torch.empty(batch, dtype=torch.int32, device=dev)}
    logits = torch.empty((batch, k, model.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
    C.check(C.load().nld_verify_accept_noalloc(model.handle, ctypes.byref(cache.struct), _ptr(anchor), _ptr(drafts),
                                               batch, k, _ptr(outs["accept_len"]), _ptr(outs["committed"]),
                                               _ptr(outs["next_anchor"]), _ptr(logits), _ptr(device_status),
                                               stream_handle()))
    outs = dict(outs)
    outs["logits"] = logits
    return outs


def accept_from_logits(logits: torch.Tensor, drafts, device="cuda"):
    """Argmax + acceptance from given f32 logits [batch][k][vocab] and int32 drafts [batch][k-1]."""
    lib = C.load()
    batch, k, vocab = logits.shape
    n = lib.nld_accept_workspace_bytes(batch, k)
    ws = torch.zeros(n, dtype=torch.uint8, device=device)
    out = {"argmax": torch.empty((batch, k), dtype=torch.int32, device=device),
           "accept_len": torch.empty(batch, dtype=torch.int32, device=device),
           "committed": torch.empty((batch, k), dtype=torch.int32, device=device),
           "next_anchor": torch.empty(batch, dtype=torch.int32, device=device)}
    C.check(lib.nld_accept_from_logits(_ptr(logits), _ptr(drafts), batch, k, vocab, _ptr(out["argmax"]),
                                       _ptr(out["accept_len"]), _ptr(out["committed"]), _ptr(out["next_anchor"]),
                                       _ptr(ws), n, stream_handle()))
    return out


def denoise_step(model, cache, ws, block: torch.Tensor, threshold: float, bidir_from: int = 0, want_logits=False,
                 outs=None):
    """One Mode 2 denoising step; ``block`` (int32 [batch][k], device) is updated in place.
    Returns dict of device tensors: n_committed, n_masked, confidence [batch][k], logits (or None)."""
    batch, k = block.shape
    dev = model.device
    if outs is None:
        outs = {"n_committed": torch.empty(batch, dtype=torch.int32, device=dev),
                "n_masked": torch.empty(batch, dtype=torch.int32, device=dev),
                "confidence": torch.empty((batch, k), dtype=torch.float32, device=dev)}
    logits = torch.empty((batch, k, model.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
    C.check(C.load().nld_denoise_step(model.handle, ctypes.byref(cache.struct), _ptr(block), batch, k, bidir_from,
                                      float(threshold), _ptr(outs["n_committed"]), _ptr(outs["n_masked"]),
                                      _ptr(outs.get("confidence")), _ptr(logits), ws.ptr, ws.nbytes, stream_handle()))
    outs = dict(outs)
    outs["logits"] = logits
    return outs


def refresh_block(model, cache, ws, block: torch.Tensor, next_anchor=None):
    """Causal K/V refresh of completed blocks (commits k-1 rows).  Returns next_anchor (int32 [batch])."""
    batch, k = block.shape
    nxt = next_anchor if next_anchor is not None else torch.empty(batch, dtype=torch.int32, device=model.device)
    C.check(C.load().nld_refresh_block(model.handle, ctypes.byref(cache.struct), _ptr(block), batch, k, _ptr(nxt),
                                       ws.ptr, ws.nbytes, stream_handle()))
    return nxt


def commit_from_logits(logits: torch.Tensor, block: torch.Tensor, mask_token_id: int, threshold: float):
    """The denoising commit from given f32 logits [batch][k][vocab]; ``block`` is updated in place."""
    batch, k, vocab = logits.shape
    dev = logits.device
    out = {"argmax": torch.empty((batch, k), dtype=torch.int32, device=dev),
           "n_committed": torch.empty(batch, dtype=torch.int32, device=dev),
           "n_masked": torch.empty(batch, dtype=torch.int32, device=dev),
           "confidence": torch.empty((batch, k), dtype=torch.float32, device=dev)}
    C.check(C.load().nld_commit_from_logits(_ptr(logits), _ptr(block), batch, k, vocab, mask_token_id,
                                            float(threshold), _ptr(out["argmax"]), _ptr(out["n_committed"]),
                                            _ptr(out["n_masked"]), _ptr(out["confidence"]), stream_handle()))
    return out


def decode_steps(model, cache, ws, anchor: torch.Tensor, k: int, n_steps: int, bidir_from: int = 0, outs=None):
    """n_steps decoding steps on the device (self-speculation for k >= 2, AR for k = 1); ``anchor`` is
    updated in place.  Returns dict: accept_len [n_steps][batch], committed [n_steps][batch][k]."""
    batch = anchor.shape[0]
    dev = model.device
    if outs is None:
        outs = {"accept_len": torch.empty((n_steps, batch), dtype=torch.int32, device=dev),
                "committed": torch.empty((n_steps, batch, k), dtype=torch.int32, device=dev)}
    C.check(C.load().nld_decode_steps(model.handle, ctypes.byref(cache.struct), _ptr(anchor), batch, k, n_steps,
                                      bidir_from, _ptr(outs["accept_len"]), _ptr(outs["committed"]), ws.ptr,
                                      ws.nbytes, stream_handle()))
    return outs


def quad_step(model, cache, ws, anchor: torch.Tensor, spec: torch.Tensor, k: int, lam: float = 1.0,
              want_logits=False, outs=None):
    """One quadratic self-speculation step over [anchor, spec] and k groups of k masks.  Returns dict of
    device tensors: accept_len, committed [batch][k], next_anchor, next_spec [batch][k-1], logits or None
    ([batch][k(k+1)][vocab]).  ``outs`` may pass next_anchor=anchor and next_spec=spec to update in place."""
    batch = anchor.shape[0]
    dev = model.device
    o = dict(outs or {})
    o.setdefault("accept_len", torch.empty(batch, dtype=torch.int32, device=dev))
    o.setdefault("committed", torch.empty((batch, k), dtype=torch.int32, device=dev))
    o.setdefault("next_anchor", torch.empty(batch, dtype=torch.int32, device=dev))
    o.setdefault("next_spec", torch.empty((batch, k - 1), dtype=torch.int32, device=dev))
    logits = torch.empty((batch, k * (k + 1), model.shape.vocab), dtype=torch.float32, device=dev) \
        if want_logits else None
    C.check(C.load().nld_quad_step(model.handle, ctypes.byref(cache.struct), _ptr(anchor), _ptr(spec), batch, k,
                                   float(lam), _ptr(o["accept_len"]), _ptr(o["committed"]), _ptr(o["next_anchor"]),
                                   _ptr(o["next_spec"]), _ptr(logits), ws.ptr, ws.nbytes, stream_handle()))
    o["logits"] = logits
    return o


def choose_block(ar_step_ms: float, ss_step_ms: float, expected_committed: float, k_ss: int) -> int:
    return int(C.load().nld_choose_block(ar_step_ms, ss_step_ms, expected_committed, k_ss))


def read_device_status(ws) -> int:
    bits = ctypes.c_uint32(0)
    st = C.load().nld_read_device_status(ws.ptr, ctypes.byref(bits), stream_handle())
    if st not in (C.NLD_OK, C.NLD_ERR_DEVICE):
        C.check(st)
    return int(bits.value)
