"""Per-workgroup phase timeline of one block pass (a diagnostic, not part of the product path).

    python -m paper_2607_05722_amd.timeline [--workload 8b] [--k 16] [--mode verify|draft] [--env K=V ...]

Builds the timeline variant of the library (libnld_timeline.so: the same sources compiled with
-DNLD_TIMELINE, so that thread 0 of every workgroup records the 100 MHz real-time counter at the
phase boundaries of each kernel), runs five passes of the workload's block to warm up and one
recorded pass, and prints, for the last layer's kernels, when their workgroups started and ended and
the median / p90 / max of each phase, in microseconds from the first workgroup start of that layer's
QKV GEMM.  The passes are eager launches (no graph), so the gaps between kernels include the launch
overhead of the host.  Phases:

    qkv, gate_up   0-1 operand, first weight tile and row statistics in; 1-2 tiles and epilogues
                   (17..64 rows: 0-1 main loop; 1-2 completed tiles reduced and finished)
    attention      0-1 committed length known; 1-2 first key stage in LDS; 2-3 stages; 3-4 partials out
    combine        0-1 the whole merge
    o_proj         0-1 main loop; 1-2 reduction and residual epilogue
    down           0-1 main loop; 1-2 partial stored and counted in (the last arriver then finishes)
"""
from __future__ import annotations

import argparse
import ctypes
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

CLASSES = [(0, "qkv", 3), (1, "attention", 5), (2, "combine", 2), (4, "o_proj", 3), (3, "gate_up", 3), (5, "down", 3)]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="8b")
    ap.add_argument("--k", type=int, default=0)
    ap.add_argument("--mode", default="verify", choices=("verify", "draft"))
    ap.add_argument("--env", nargs="*", default=[], help="library environment settings, NAME=VALUE")
    args = ap.parse_args()
    for kv in args.env:
        name, value = kv.split("=", 1)
        os.environ[name] = value

    import torch   # first: the library then binds to the HIP runtime torch has loaded
    from paper_2607_05722_amd import buildlib
    path = buildlib.TIMELINE_LIB if os.path.exists(buildlib.TIMELINE_LIB) else buildlib.build(timeline=True)
    from paper_2607_05722_amd import _lib as C
    lib = C.load(path)
    lib.nld_timeline_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t]
    lib.nld_timeline_read.restype = ctypes.c_int
    from paper_2607_05722_amd import runtime as R
    from synth.workloads import LazyWeights, WORKLOADS, prefix_kv, tokens

    wl = WORKLOADS[args.workload]
    shape, k = wl.shape, args.k or wl.k_values[0]
    P = int(wl.prefix_lengths()[0])
    max_len = (P + k + 63) // 64 * 64 + 512
    model = R.DeviceModel(shape, LazyWeights(shape, wl.seed, keep=False))
    cache = R.DeviceCache(shape, 1, max_len)
    for l in range(shape.n_layers):
        kb, vb = prefix_kv(shape, wl.seed, l, 1, P)
        cache.load_prefix(l, kb, vb)
    cache.set_lengths([P])
    ws = R.Workspace(model, 1, k, max_len)
    tok = torch.from_numpy(tokens(shape, wl.seed, "timeline.block", (1, k))).cuda()
    mode = R.VERIFY if args.mode == "verify" else R.DRAFT
    for _ in range(5):
        R.block_forward(model, cache, ws, tok, mode, want_logits=False)
    torch.cuda.synchronize()
    assert lib.nld_timeline_read(None, 0) == 0
    torch.cuda.synchronize()
    R.block_forward(model, cache, ws, tok, mode, want_logits=False)
    torch.cuda.synchronize()
    ts = np.zeros((8, 8192, 8), dtype=np.uint64)
    assert lib.nld_timeline_read(ts.ctypes.data, ts.nbytes) == 0
    assert R.read_device_status(ws) == 0

    used = {c: ts[c][:, 0] > 0 for c, _, _ in CLASSES}
    t0 = int(ts[0][used[0]][:, 0].min())
    print("%s, batch 1, prefix %d, k=%d, %s pass: last layer, us from its QKV's first workgroup start "
          "(s_memrealtime, 10 ns ticks; eager launches)" % (wl.name, P, k, args.mode))
    for c, name, nph in CLASSES:
        a = ts[c][used[c]].astype(np.int64)
        if a.shape[0] == 0:
            continue
        rel = (a[:, :nph] - t0) / 100.0
        end = rel[:, nph - 1]
        end = end[a[:, nph - 1] > 0]
        print("%-9s workgroups %4d  start min %7.2f med %7.2f max %7.2f | end min %7.2f med %7.2f max %7.2f" % (
            name, a.shape[0], rel[:, 0].min(), np.median(rel[:, 0]), rel[:, 0].max(), end.min(), np.median(end),
            end.max()))
        for p in range(1, nph):
            ok = (a[:, p] > 0) & (a[:, p - 1] > 0)
            if ok.any():
                d = (a[ok, p] - a[ok, p - 1]) / 100.0
                print("    phase %d-%d: %4d workgroups  med %6.2f  p90 %6.2f  max %6.2f us" % (
                    p - 1, p, ok.sum(), np.median(d), np.percentile(d, 90), d.max()))


if __name__ == "__main__":
    main()
