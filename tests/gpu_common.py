"""Shared helpers of the GPU parity tests: build both sides from the same seeded inputs.

Nothing computed on the GPU is ever fed to the oracle: the oracle sees only the
generator's outputs (and its own results); the GPU sees the same generator
outputs, or oracle results uploaded as inputs.
"""
from __future__ import annotations

import sys

import numpy as np

from oracle import nld_oracle as O


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    """Normwise error ||g - o||_inf / ||o||_inf."""
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(np.asarray(gpu, dtype=np.float64) - ref)) / np.max(np.abs(ref)))


def top2_margin(logits: np.ndarray) -> np.ndarray:
    """Gap between the largest and second-largest logit of every row (last axis)."""
    part = np.partition(logits, -2, axis=-1)
    return part[..., -1] - part[..., -2]


def check_argmax(gpu_argmax: np.ndarray, gpu_logits: np.ndarray, ref_logits: np.ndarray, tol_abs: float):
    """GPU argmax must be the first maximum of the GPU's own logits (exact), and equal the oracle's
    argmax on every row whose oracle top-2 margin exceeds twice the measured logit error.
    Returns the list of near-tie rows where the two argmaxes differ."""
    own = np.argmax(gpu_logits, axis=-1)
    assert np.array_equal(gpu_argmax, own), "argmax kernel disagrees with the GPU's own logits"
    ref_am = O.argmax_first(ref_logits)
    margin = top2_margin(ref_logits.astype(np.float64))
    differ = gpu_argmax != ref_am
    near = margin <= 2.0 * tol_abs
    bad = differ & ~near
    assert not bad.any(), "argmax differs on rows with margin > 2*err: %s" % (np.argwhere(bad).tolist(),)
    return np.argwhere(differ).tolist()


class ArraySource:
    """Weights given as explicit arrays (same protocol as synth.workloads.LazyWeights)."""

    def __init__(self, layers, embed, lm_head, final_norm):
        self._layers, self.embed, self.lm_head, self.final_norm = layers, embed, lm_head, final_norm

    def layer(self, l):
        return self._layers[l]


BF16_ONE = np.uint16(0x3F80)
BF16_MINUS_ONE = np.uint16(0xBF80)


def int_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Exact bf16 bits of small integers (|v| <= 256)."""
    v = np.asarray(v, dtype=np.float32)
    assert np.all(np.abs(v) <= 256)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


# ----------------------------------------------------------------------------- Mode 2 decisions
def log_conf_bound(err_abs: float) -> float:
    """Largest change of ln(confidence) that a logit error of at most err_abs can cause: the top logit and
    the log-sum-exp each move by at most err_abs."""
    return 2.0 * err_abs


def own_commit(block_in: np.ndarray, gpu_logits: np.ndarray, gpu_conf: np.ndarray, threshold: float, mask_id: int):
    """The commit rule applied to the GPU's own logits (argmax without the mask token) and its own
    confidences -- what the device must have decided, bit for bit."""
    pred = O.argmax_first(O.denoising_logits(gpu_logits, mask_id))
    out = block_in.copy()
    for b in range(block_in.shape[0]):
        out[b], _ = O.threshold_commit(block_in[b], pred[b], np.asarray(gpu_conf[b], dtype=np.float64), threshold,
                                       mask_id)
    return out, pred


def decision_near_tie(block_in: np.ndarray, ref_logits: np.ndarray, ref_conf: np.ndarray, threshold: float,
                      mask_id: int, err_abs: float) -> list:
    """Sequences whose commit a logit error of err_abs could change: a masked row's confidence within the
    implied bound of the threshold, two masked rows' confidences that close when the fallback decides, or
    a masked row whose top-2 logit gap (mask token excluded) is within 2 err_abs."""
    d = log_conf_bound(err_abs)
    z = O.denoising_logits(ref_logits, mask_id)
    part = np.partition(z, -2, axis=-1)
    gap = part[..., -1] - part[..., -2]
    near = []
    for b in range(block_in.shape[0]):
        masked = [j for j in range(1, block_in.shape[1]) if block_in[b, j] == mask_id]
        lc = np.log(np.asarray([ref_conf[b, j] for j in masked]))
        lt = np.log(threshold) if threshold > 0 else -np.inf
        hit = any(abs(c - lt) <= d for c in lc)
        if masked and not np.any(lc > lt + d) and len(lc) > 1:
            top = np.sort(lc)[::-1]
            hit = hit or (top[0] - top[1] <= 2 * d)
        hit = hit or any(gap[b, j] <= 2 * err_abs for j in masked)
        if hit:
            near.append(b)
    return near
