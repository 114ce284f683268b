"""Synthetic workloads for the block-decode step.

Five workloads, shapes as stated for the method's 8B- and 14B-class
decoder-only models (no trained weights exist here, so every tensor is a
seeded draw):

* ``tiny``      -- 2 layers, hidden 256, 4/2 heads, head_dim 64, FFN 688,
                   vocab 1024; batch 1; a real 128-token prefix (prefilled by
                   each side); block k=8 whose tokens are uniform ids.
* ``8b_layer``  -- one 8B-shaped layer + LM head; batch 1; prefix K/V
                   N(0,1) of length 2048; k in {8, 16, 32}.
* ``8b``        -- 36 layers, 8B shapes; batch 1; prefix 4096; k=16.
* ``8b_batch32``-- 36 layers; batch 32, ragged prefixes uniform in
                   [512, 8192]; k=16; verify mask.
* ``14b``       -- 40 layers, hidden 5120, 40/8 heads, FFN 17408; batch 8,
                   prefix 16384; k=32.

Weights are N(0, 0.02) bfloat16, stored [out_features][in_features]; every
RMSNorm gain vector (each layer's attention and FFN norms, the final norm) is its
own seeded draw bf16(1 + 0.1 z), so that a gain applied at the wrong place shows
in the output; the LM head is a separate matrix from the embedding.  The
mask token is id vocab-1; block and prefix tokens are uniform over
[0, vocab-2] so they never collide with it.  Nothing here computes any part
of the forward pass.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import gain_bf16, normal_bf16, uniform_int


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    init_std: float = 0.02
    lora_rank: int = 0          # draft-pathway LoRA on the O projection (0: none)
    lora_alpha: float = 0.0
    norm_gain_std: float = 0.1  # RMSNorm gains are bf16(1 + norm_gain_std * z), one draw per vector

    @property
    def mask_token_id(self) -> int:
        return self.vocab - 1

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_weight_bytes(self) -> int:
        h, f = self.hidden, self.ffn
        return 2 * (h * (self.q_dim + 2 * self.kv_dim) + self.q_dim * h + 2 * f * h + f * h)

    def weight_bytes(self) -> int:
        """bf16 bytes of every weight streamed once by one pass (layers + LM head)."""
        return self.n_layers * self.layer_weight_bytes() + 2 * self.vocab * self.hidden


SHAPE_TINY = ModelShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=688, vocab=1024)
SHAPE_8B = ModelShape(n_layers=36, hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128, ffn=12288, vocab=151936)
SHAPE_14B = ModelShape(n_layers=40, hidden=5120, n_q_heads=40, n_kv_heads=8, head_dim=128, ffn=17408, vocab=151936)


@dataclass
class Workload:
    name: str
    shape: ModelShape
    seed: int
    batch: int
    k_values: List[int]
    prefix_kind: str                  # "prefill" (real token prefix) or "random_kv" (N(0,1) K/V)
    prefix_len: int = 0               # uniform prefix length (ignored when ragged)
    ragged: Optional[tuple] = None    # (lo, hi) for per-sequence prefix lengths
    modes: tuple = ("draft", "verify")
    paper_loop: bool = True           # run draft -> verify -> accept
    note: str = ""

    def prefix_lengths(self) -> np.ndarray:
        if self.ragged is not None:
            return uniform_int(self.seed, "prefix_lengths", (self.batch,), self.ragged[0], self.ragged[1])
        return np.full(self.batch, self.prefix_len, dtype=np.int32)


WORKLOADS = {
    "tiny": Workload("tiny", SHAPE_TINY, seed=0, batch=1, k_values=[8], prefix_kind="prefill", prefix_len=128),
    "8b_layer": Workload("8b_layer", ModelShape(**{**SHAPE_8B.__dict__, "n_layers": 1}), seed=1, batch=1,
                         k_values=[8, 16, 32], prefix_kind="random_kv", prefix_len=2048, paper_loop=False),
    "8b": Workload("8b", SHAPE_8B, seed=2, batch=1, k_values=[16], prefix_kind="random_kv", prefix_len=4096),
    "8b_batch32": Workload("8b_batch32", SHAPE_8B, seed=3, batch=32, k_values=[16], prefix_kind="random_kv",
                           ragged=(512, 8192), modes=("verify",), paper_loop=False),
    "14b": Workload("14b", SHAPE_14B, seed=4, batch=8, k_values=[32], prefix_kind="random_kv", prefix_len=16384),
}


# ----------------------------------------------------------------------------- weights
def layer_weights(shape: ModelShape, seed: int, layer: int) -> dict:
    """Row-major [out][in] bf16 bit patterns of one decoder layer (plus lora_a [rank][q_dim] and
    lora_b [hidden][rank] when the shape has a LoRA rank; both N(0, init_std) so that the adapter is
    not the identity a fresh LoRA would be)."""
    h, s, p = shape.hidden, shape.init_std, "layer%d." % layer
    w = {
        "attn_norm": gain_bf16(seed, p + "attn_norm", h, shape.norm_gain_std),
        "wq": normal_bf16(seed, p + "wq", (shape.q_dim, h), s),
        "wk": normal_bf16(seed, p + "wk", (shape.kv_dim, h), s),
        "wv": normal_bf16(seed, p + "wv", (shape.kv_dim, h), s),
        "wo": normal_bf16(seed, p + "wo", (h, shape.q_dim), s),
        "ffn_norm": gain_bf16(seed, p + "ffn_norm", h, shape.norm_gain_std),
        "w_gate": normal_bf16(seed, p + "w_gate", (shape.ffn, h), s),
        "w_up": normal_bf16(seed, p + "w_up", (shape.ffn, h), s),
        "w_down": normal_bf16(seed, p + "w_down", (h, shape.ffn), s),
    }
    if shape.lora_rank:
        w.update(lora_weights(shape, seed, layer))
    return w


def lora_weights(shape: ModelShape, seed: int, layer: int) -> dict:
    """The draft-pathway adapter of one layer alone: lora_a [rank][q_dim], lora_b [hidden][rank]."""
    p, s = "layer%d." % layer, shape.init_std
    return {"lora_a": normal_bf16(seed, p + "lora_a", (shape.lora_rank, shape.q_dim), s),
            "lora_b": normal_bf16(seed, p + "lora_b", (shape.hidden, shape.lora_rank), s)}


def embed_weights(shape: ModelShape, seed: int) -> np.ndarray:
    return normal_bf16(seed, "embed", (shape.vocab, shape.hidden), shape.init_std)


def lm_head_weights(shape: ModelShape, seed: int) -> np.ndarray:
    return normal_bf16(seed, "lm_head", (shape.vocab, shape.hidden), shape.init_std)


def final_norm_weights(shape: ModelShape, seed: int) -> np.ndarray:
    return gain_bf16(seed, "final_norm", shape.hidden, shape.norm_gain_std)


class LazyWeights:
    """Dict-like access to a model's weights, generated on first use per layer.

    ``keep=False`` regenerates on every access so that large models can be
    streamed layer by layer without holding every layer in host memory.
    """

    def __init__(self, shape: ModelShape, seed: int, keep: bool = True):
        self.shape, self.seed, self.keep = shape, seed, keep
        self._layers = {}
        self._embed = self._lm = None

    def layer(self, l: int) -> dict:
        if l in self._layers:
            return self._layers[l]
        w = layer_weights(self.shape, self.seed, l)
        if self.keep:
            self._layers[l] = w
        return w

    @property
    def embed(self) -> np.ndarray:
        if self._embed is None:
            self._embed = embed_weights(self.shape, self.seed)
        return self._embed

    @property
    def lm_head(self) -> np.ndarray:
        if self._lm is None:
            self._lm = lm_head_weights(self.shape, self.seed)
        return self._lm

    @property
    def final_norm(self) -> np.ndarray:
        return final_norm_weights(self.shape, self.seed)


# ----------------------------------------------------------------------------- K/V and tokens
def prefix_kv(shape: ModelShape, seed: int, layer: int, batch: int, length: int):
    """N(0,1) bf16 K and V for one layer, logical layout [batch][kv_head][length][head_dim].

    These stand for keys that are already position-rotated, as a cache holds them.
    Sequence b uses the first P_b rows when lengths are ragged.
    """
    shp = (batch, shape.n_kv_heads, length, shape.head_dim)
    k = normal_bf16(seed, "layer%d.prefix_k" % layer, shp, 1.0)
    v = normal_bf16(seed, "layer%d.prefix_v" % layer, shp, 1.0)
    return k, v


def tokens(shape: ModelShape, seed: int, name: str, count_shape) -> np.ndarray:
    """Token ids uniform over [0, vocab-2] (never the mask id)."""
    return uniform_int(seed, name, count_shape, 0, shape.vocab - 2)
