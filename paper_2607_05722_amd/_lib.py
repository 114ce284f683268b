"""ctypes declarations of libnld's C ABI (include/nld.h).  Marshalling only."""
from __future__ import annotations

import ctypes
import os

from . import buildlib as _build

c_i32, c_u32, c_f32, c_sz, c_vp = ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p

NLD_OK = 0
NLD_ERR_INVALID_ARG = -1
NLD_ERR_SHAPE = -2
NLD_ERR_CAPACITY = -3
NLD_ERR_HIP = -4
NLD_ERR_UNSUPPORTED = -5
NLD_ERR_DEVICE = -6

NLD_MODE_VERIFY = 0
NLD_MODE_DRAFT = 1

NLD_DEV_BAD_TOKEN = 0x1
NLD_DEV_CAPACITY = 0x2
NLD_DEV_BAD_LENGTH = 0x4
NLD_DEV_MASK_LEFT = 0x8

NLD_PACK_LINEAR = 0
NLD_PACK_QKV = 1
NLD_PACK_GATE_UP = 2

EXPORTED = [
    "nld_last_error", "nld_status_string", "nld_model_create", "nld_model_destroy", "nld_packed_bytes",
    "nld_pack_linear", "nld_pack_qkv", "nld_pack_gate_up", "nld_workspace_bytes", "nld_workspace_init",
    "nld_block_forward", "nld_draft", "nld_verify_accept", "nld_accept_workspace_bytes",
    "nld_accept_from_logits", "nld_denoise_step", "nld_refresh_block", "nld_commit_from_logits",
    "nld_decode_steps", "nld_choose_block", "nld_quad_workspace_bytes", "nld_quad_step",
    "nld_read_device_status", "nld_trace_enable", "nld_trace_read", "nld_verify_accept_noalloc",
    "nld_hbm_read_probe",
]

NLD_NOALLOC_SCRATCH_BYTES = 64 << 20

TRACE_CLASSES = ["embed", "qkv", "attention", "o_proj", "gate_up", "down", "lm_head", "argmax"]


class Config(ctypes.Structure):
    _fields_ = [("n_layers", c_i32), ("hidden", c_i32), ("n_q_heads", c_i32), ("n_kv_heads", c_i32),
                ("head_dim", c_i32), ("ffn", c_i32), ("vocab", c_i32), ("rope_base", c_f32),
                ("rms_eps", c_f32), ("mask_token_id", c_i32), ("lora_rank", c_i32), ("lora_scale", c_f32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", c_vp), ("w_qkv", c_vp), ("w_o", c_vp), ("ffn_norm", c_vp),
                ("w_gate_up", c_vp), ("w_down", c_vp), ("lora_a", c_vp), ("lora_b", c_vp)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", c_vp), ("final_norm", c_vp), ("lm_head", c_vp), ("layers", ctypes.POINTER(LayerWeights))]


class KVCache(ctypes.Structure):
    _fields_ = [("k", c_vp), ("v", c_vp), ("lengths", c_vp), ("batch", c_i32), ("max_len", c_i32)]


class NLDError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s (%d): %s" % (_status_name(status), status, message))
        self.status = status


_lib = None


def _status_name(st):
    return {0: "NLD_OK", -1: "NLD_ERR_INVALID_ARG", -2: "NLD_ERR_SHAPE", -3: "NLD_ERR_CAPACITY",
            -4: "NLD_ERR_HIP", -5: "NLD_ERR_UNSUPPORTED", -6: "NLD_ERR_DEVICE"}.get(st, "?")


def lib_path() -> str:
    return _build.LIB


def load(path: str = None):
    """Load libnld.so (building it first only when it does not exist).  `path` (first call only) loads
    another build of the same ABI instead, such as the timeline build of timeline.py."""
    global _lib
    if _lib is not None:
        return _lib
    if path is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
    L = ctypes.CDLL(path)
    P = ctypes.POINTER
    L.nld_last_error.restype = ctypes.c_char_p
    L.nld_last_error.argtypes = []
    L.nld_status_string.restype = ctypes.c_char_p
    L.nld_status_string.argtypes = [c_i32]
    L.nld_model_create.restype = c_i32
    L.nld_model_create.argtypes = [P(Config), P(Weights), P(c_vp)]
    L.nld_model_destroy.restype = None
    L.nld_model_destroy.argtypes = [c_vp]
    L.nld_packed_bytes.restype = c_sz
    L.nld_packed_bytes.argtypes = [c_i32, P(Config), c_i32, c_i32]
    L.nld_pack_linear.restype = c_i32
    L.nld_pack_linear.argtypes = [c_vp, c_i32, c_i32, c_vp, c_vp]
    L.nld_pack_qkv.restype = c_i32
    L.nld_pack_qkv.argtypes = [P(Config), c_vp, c_vp, c_vp, c_vp, c_vp]
    L.nld_pack_gate_up.restype = c_i32
    L.nld_pack_gate_up.argtypes = [P(Config), c_vp, c_vp, c_vp, c_vp]
    L.nld_workspace_bytes.restype = c_sz
    L.nld_workspace_bytes.argtypes = [c_vp, c_i32, c_i32, c_i32]
    L.nld_workspace_init.restype = c_i32
    L.nld_workspace_init.argtypes = [c_vp, c_sz, c_vp]
    L.nld_block_forward.restype = c_i32
    L.nld_block_forward.argtypes = [c_vp, P(KVCache), c_vp, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.nld_draft.restype = c_i32
    L.nld_draft.argtypes = [c_vp, P(KVCache), c_vp, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.nld_verify_accept.restype = c_i32
    L.nld_verify_accept.argtypes = [c_vp, P(KVCache), c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz,
                                    c_vp]
    L.nld_accept_workspace_bytes.restype = c_sz
    L.nld_accept_workspace_bytes.argtypes = [c_i32, c_i32]
    L.nld_accept_from_logits.restype = c_i32
    L.nld_accept_from_logits.argtypes = [c_vp, c_vp, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.nld_quad_workspace_bytes.restype = c_sz
    L.nld_quad_workspace_bytes.argtypes = [c_vp, c_i32, c_i32, c_i32]
    L.nld_quad_step.restype = c_i32
    L.nld_quad_step.argtypes = [c_vp, P(KVCache), c_vp, c_vp, c_i32, c_i32, c_f32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                c_sz, c_vp]
    L.nld_denoise_step.restype = c_i32
    L.nld_denoise_step.argtypes = [c_vp, P(KVCache), c_vp, c_i32, c_i32, c_i32, c_f32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                   c_sz, c_vp]
    L.nld_refresh_block.restype = c_i32
    L.nld_refresh_block.argtypes = [c_vp, P(KVCache), c_vp, c_i32, c_i32, c_vp, c_vp, c_sz, c_vp]
    L.nld_commit_from_logits.restype = c_i32
    L.nld_commit_from_logits.argtypes = [c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_f32, c_vp, c_vp, c_vp, c_vp, c_vp]
    L.nld_decode_steps.restype = c_i32
    L.nld_decode_steps.argtypes = [c_vp, P(KVCache), c_vp, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.nld_choose_block.restype = c_i32
    L.nld_choose_block.argtypes = [c_f32, c_f32, c_f32, c_i32]
    L.nld_read_device_status.restype = c_i32
    L.nld_read_device_status.argtypes = [c_vp, P(c_u32), c_vp]
    L.nld_trace_enable.restype = c_i32
    L.nld_trace_enable.argtypes = [c_i32]
    L.nld_trace_read.restype = c_i32
    L.nld_trace_read.argtypes = [P(c_f32), P(c_i32), c_i32]
    L.nld_hbm_read_probe.restype = c_i32
    L.nld_hbm_read_probe.argtypes = [c_vp, c_sz, c_i32, c_i32, c_i32, c_vp, c_vp]
    L.nld_verify_accept_noalloc.restype = c_i32
    L.nld_verify_accept_noalloc.argtypes = [c_vp, P(KVCache), c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                            c_vp]
    _lib = L
    return L


def check(status: int) -> None:
    if status != NLD_OK:
        raise NLDError(status, load().nld_last_error().decode())
