"""Benchmark of the block-decode step (draft pass + verify pass + acceptance) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 8b] [--k 16] [--max-len L] [--no-cpu-baseline]
                    [--no-extras] [--no-large] [--no-graph] [--copy-calibration-mib N]

A step is one linear self-speculation step over the synthetic workload: the
diffusion draft pass over [anchor, mask x (k-1)], the causal verify pass over
[anchor, drafts], the argmax, the longest-prefix acceptance and the commit of
the accepted rows, all on the device (the next step's anchor stays on the
device).  The timed steps replay one captured HIP graph.

value = block tokens pushed through block-decode passes per second
      = 2 passes x batch x k per step / step time.
Also timed (not part of value), each replayed from its own captured graph:
"mode2" -- one Mode 2 denoising step over [anchor, mask x (k-1)] at threshold
0.9 and one K/V refresh of a completed block; "lora_draft" -- a draft pass with
and without the LoRA-enhanced drafter's adapter (rank 128) on the O projection;
"quad_ss" -- one quadratic self-speculation step (chain length 7, 56 block rows)
with the AR verifier and with the lambda = 0.5 ensemble, beside one linear step
(draft + verify) of the same speculative width; "block_k32" -- one linear step
at block size 32 (the paper's main block length) over the same prefix;
"verify_pass_ms" -- the verify pass alone; "layer_microbench" -- one 8B-shaped
layer + LM head at k = 8, 16, 32; "large_configs" -- the 8b_batch32 and 14b
steps with random weights drawn on the GPU (--no-large skips them).
"hbm_stream_ceiling" is what the library's hand-written read stream reaches on
the same box (the practical HBM ceiling the step is compared with).
"roofline" is the dominant kernel's: algorithmic bytes per launch over its
average launch time from HIP events recorded on every dispatch of three eager
steps, and its HBM traffic from the committed counter summary while the kernel
sources match it.  "cpu_baseline" times the CPU oracle on a bounded sample.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "block-decode tokens/sec at 1 MI355X; % of HBM roofline (8B-shape, k=16, bs=1)"
HBM_PEAK_GBS = 8000.0


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def kernel_bytes(shape, batch, k, prefix_lens):
    """Algorithmic HBM bytes per launch of each kernel class: bf16 weights once, K/V read once,
    activations read and written once."""
    M, H, F, V = batch * k, shape.hidden, shape.ffn, shape.vocab
    QD, KVD = shape.q_dim, shape.kv_dim
    kv_keys = int(np.sum(np.asarray(prefix_lens) + k))
    return {
        "embed": M * H * (2 + 4 + 2),
        "qkv": 2 * H * (QD + 2 * KVD) + 2 * M * H + 2 * M * QD + 2 * 2 * M * KVD,
        "attention": 2 * 2 * kv_keys * KVD + 2 * M * QD * 2,
        "o_proj": 2 * QD * H + 2 * M * QD + 4 * M * H * 2 + 2 * M * H,
        "gate_up": 2 * H * 2 * F + 2 * M * H + 2 * M * F,
        "down": 2 * F * H + 2 * M * F + 4 * M * H * 2 + 2 * M * H,
        "lm_head": 2 * V * H + 2 * M * H,
        "argmax": 0,
    }


def pass_bytes(shape, batch, k, prefix_lens):
    kb = kernel_bytes(shape, batch, k, prefix_lens)
    return kb["embed"] + shape.n_layers * (kb["qkv"] + kb["attention"] + kb["o_proj"] + kb["gate_up"] + kb["down"]) \
        + kb["lm_head"]


MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16


def pass_flops(shape, batch, k, prefix_lens):
    """Algorithmic flops of one pass: 2 per weight element and block row, plus 4 * head_dim per query head,
    block row and visible key (every block row counted against the whole prefix + block)."""
    M, H, F, V = batch * k, shape.hidden, shape.ffn, shape.vocab
    QD, KVD, L = shape.q_dim, shape.kv_dim, shape.n_layers
    w_elems = L * (H * (QD + 2 * KVD) + QD * H + 2 * H * F + F * H) + V * H
    keys = int(np.sum(np.asarray(prefix_lens) + k)) * k
    return 2 * M * w_elems + 4 * shape.n_q_heads * shape.head_dim * L * keys


def refresh_bytes(shape, batch, k, prefix_lens):
    """A refresh runs every layer's QKV but stops after the last one: no attention, FFN or LM head after it."""
    kb = kernel_bytes(shape, batch, k, prefix_lens)
    return kb["embed"] + shape.n_layers * kb["qkv"] \
        + (shape.n_layers - 1) * (kb["attention"] + kb["o_proj"] + kb["gate_up"] + kb["down"])


def graph_ms(fn, reps):
    """Mean ms of fn() replayed `reps` times from a captured graph (one eager call and one replay first)."""
    import torch
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.current_stream()):
        fn()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def mode2_timing(R, model, cache, ws, anchor, block_full, k, reps, threshold=0.9):
    """Mean ms of one denoising step (block reset to [anchor, masks] first) and of one refresh (lengths reset
    first, so every replay refreshes the same rows), each from a captured graph replayed `reps` times."""
    import torch
    B = anchor.shape[0]
    dev = anchor.device
    blk0 = torch.full((B, k), model.shape.mask_token_id, dtype=torch.int32, device=dev)
    blk0[:, 0] = anchor
    blk = blk0.clone()
    outs = {"n_committed": torch.empty(B, dtype=torch.int32, device=dev),
            "n_masked": torch.empty(B, dtype=torch.int32, device=dev),
            "confidence": torch.empty((B, k), dtype=torch.float32, device=dev)}
    nxt = torch.empty(B, dtype=torch.int32, device=dev)
    len0 = cache.lengths.clone()

    def denoise():
        blk.copy_(blk0)
        R.denoise_step(model, cache, ws, blk, threshold, outs=outs)

    def refresh():
        cache.lengths.copy_(len0)
        R.refresh_block(model, cache, ws, block_full, next_anchor=nxt)

    res = {name: graph_ms(fn, reps) for name, fn in (("denoise_step", denoise), ("refresh", refresh))}
    committed = int(outs["n_committed"].sum().item())
    cache.lengths.copy_(len0)
    torch.cuda.synchronize()
    return res, committed


LORA_RANK, LORA_ALPHA = 128, 512.0     # the adapter size of the LoRA-enhanced drafter (Sec. 3.3)


def lora_timing(R, model, cache, ws, anchor, k, reps, wl):
    """Mean ms of a plain draft pass and of a draft pass with a rank-128 adapter on the O projection
    attached to the same weights (seeded adapter weights), each replayed from a captured graph."""
    import torch
    from synth.workloads import ModelShape, lora_weights
    lshape = ModelShape(**{**model.shape.__dict__, "lora_rank": LORA_RANK, "lora_alpha": LORA_ALPHA})
    lmodel = model.with_lora(lshape, lambda l: lora_weights(lshape, wl.seed, l))
    lws = R.Workspace(lmodel, anchor.shape[0], k, cache.max_len)      # holds the adapter's intermediate too
    B = anchor.shape[0]
    d = torch.empty((B, k - 1), dtype=torch.int32, device=anchor.device)
    res = {"draft": graph_ms(lambda: R.draft(model, cache, ws, anchor, k, out=d), reps),
           "lora_draft": graph_ms(lambda: R.draft(lmodel, cache, lws, anchor, k, out=d), reps)}
    res["status"] = R.read_device_status(lws)
    lmodel.close()
    return res


def traced_kernels(fn, n):
    """Per kernel class: mean duration (us) of each launch and launches per call, over n eager calls of fn
    with launch tracing on (HIP events recorded on each kernel's own dispatch)."""
    import ctypes
    import torch
    from paper_2607_05722_amd import _lib as C
    lib = C.load()
    lib.nld_trace_enable(1)
    for _ in range(n):
        fn()
    torch.cuda.synchronize()
    ms = (ctypes.c_float * 8)()
    cnt = (ctypes.c_int32 * 8)()
    C.check(lib.nld_trace_read(ms, cnt, 8))
    lib.nld_trace_enable(0)
    return {name: {"avg_us": round(ms[i] / cnt[i] * 1e3, 2), "launches_per_call": cnt[i] // n}
            for i, name in enumerate(C.TRACE_CLASSES) if cnt[i]}


QUAD_K = 7   # chain length of the quadratic layout: k(k+1) = 56 block rows per sequence


def quad_timing(R, model, cache, anchor, reps):
    """Mean ms of one quadratic self-speculation step (chain length QUAD_K; AR verifier and the lambda = 0.5
    ensemble) and of one linear step (draft + verify) at the same speculative width, each replayed from a
    captured graph with the lengths reset first, so that every replay runs over the same prefix."""
    import torch
    k, B, dev = QUAD_K, anchor.shape[0], anchor.device
    qws = R.QuadWorkspace(model, B, k, cache.max_len)
    lws = R.Workspace(model, B, k, cache.max_len)
    a0 = anchor.clone()
    spec0 = torch.empty((B, k - 1), dtype=torch.int32, device=dev)
    R.draft(model, cache, lws, a0, k, out=spec0)        # the first speculative tokens: a linear draft
    len0 = cache.lengths.clone()
    i32 = lambda *shp: torch.empty(shp, dtype=torch.int32, device=dev)
    oq = {"accept_len": i32(B), "committed": i32(B, k), "next_anchor": i32(B), "next_spec": i32(B, k - 1)}
    ol = {"accept_len": i32(B), "committed": i32(B, k), "next_anchor": i32(B)}
    d = i32(B, k - 1)

    def quad(lam):
        cache.lengths.copy_(len0)
        R.quad_step(model, cache, qws, a0, spec0, k, lam, outs=oq)

    def linear():
        cache.lengths.copy_(len0)
        R.draft(model, cache, lws, a0, k, out=d)
        R.verify_accept(model, cache, lws, a0, d, k, outs=ol)

    res = {"quad_ar": graph_ms(lambda: quad(1.0), reps), "quad_ensemble": graph_ms(lambda: quad(0.5), reps),
           "linear": graph_ms(linear, reps)}
    res["kernels_us"] = traced_kernels(lambda: quad(0.5), 3)
    res["status"] = R.read_device_status(qws) | R.read_device_status(lws)
    cache.lengths.copy_(len0)
    torch.cuda.synchronize()
    return res


def block_size_timing(R, model, cache, anchor, reps, k):
    """Mean ms of one linear self-speculation step (draft + verify + accept) at block size k, replayed from a
    captured graph with the lengths reset first, so that every replay runs over the same prefix."""
    import torch
    B, dev = anchor.shape[0], anchor.device
    ws = R.Workspace(model, B, k, cache.max_len)
    a0 = anchor.clone()
    len0 = cache.lengths.clone()
    i32 = lambda *shp: torch.empty(shp, dtype=torch.int32, device=dev)
    outs = {"accept_len": i32(B), "committed": i32(B, k), "next_anchor": i32(B)}
    d = i32(B, k - 1)

    def linear():
        cache.lengths.copy_(len0)
        R.draft(model, cache, ws, a0, k, out=d)
        R.verify_accept(model, cache, ws, a0, d, k, outs=outs)

    ms = graph_ms(linear, reps)
    kernels = traced_kernels(linear, 3)
    status = R.read_device_status(ws)
    cache.lengths.copy_(len0)
    torch.cuda.synchronize()
    return ms, kernels, status


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [d.get("num_threads", 0) for d in threadpool_info() if d.get("user_api") == "blas"]
        return max(n) if n else os.cpu_count()
    except Exception:
        return os.cpu_count()


def cpu_baseline(wl, k, min_seconds=10.0, max_passes=8):
    """Time the CPU oracle's verify pass over the full model (batch 1 of the workload, every layer + LM head).

    Passes repeat until at least `min_seconds` of CPU work have been timed (two passes at least)."""
    from oracle import nld_oracle as O
    from synth.workloads import LazyWeights, prefix_kv, tokens

    shape = wl.shape
    P = int(wl.prefix_lengths()[0])
    src = LazyWeights(shape, wl.seed, keep=True)
    for l in range(shape.n_layers):
        src.layer(l)
    _ = src.embed, src.lm_head
    w = O.OracleWeights(shape, src, np.float32)
    kv = O.OracleKV(shape, 1, P + k, np.float32)
    for l in range(shape.n_layers):
        kb, vb = prefix_kv(shape, wl.seed, l, 1, P)
        kv.set_prefix_bf16(l, kb[:1], vb[:1], [P])
    blk = tokens(shape, wl.seed, "bench.cpu.block", (1, k))
    times = []
    while len(times) < max_passes and (len(times) < 2 or sum(times) < min_seconds):
        t0 = time.perf_counter()
        O.block_forward(w, kv, blk, O.VERIFY)
        times.append(time.perf_counter() - t0)
        log("oracle verify pass %d: %.2f s" % (len(times), times[-1]))
    total = sum(times)
    return {
        "value": round(k * len(times) / total, 4), "unit": "block tokens/s", "cores": int(blas_threads()),
        "kind": "oracle", "cpu_model": cpu_model_name(), "host_cpus": os.cpu_count(),
        "sample": "fp32 numpy oracle, %d full verify passes (batch 1 of the workload, k=%d, prefix %d, all %d layers "
                  "+ LM head), %.1f s in total" % (len(times), k, P, shape.n_layers, total),
    }


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    for name in ("kernels.hip", "nld_internal.h"):
        with open(os.path.join(ROOT, "paper_2607_05722_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None when that summary is
    missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", "%s_8b_hbm_traffic.md" % kernel)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                key, val = line[2:].split(": ", 1)
                vals[key.strip()] = val.strip().strip("`")
    if vals.get("kernel sources sha256[:16]") != kernel_source_digest():
        return None
    try:
        return int(vals["HBM bytes per launch (read + write)"])
    except (KeyError, ValueError):
        return None


def hbm_ceiling():
    """What a plain read stream reaches on this part: the library's streaming probe (one contiguous 1 KiB
    block per wavefront load, 16 loads in flight per lane) over 2 GiB at several grid shapes, each launch
    reading a different region of an 8 GiB pool so that none finds its data in the memory-side cache.
    Also the time of 16, 50 and 200 MiB reads, whose intercept is the fixed cost of one launch."""
    import torch
    from paper_2607_05722_amd import _lib as C
    lib = C.load()
    pool_bytes = 8 << 30
    pool = torch.ones(pool_bytes // 4, dtype=torch.float32, device="cuda")
    sink = torch.zeros(65536, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream

    def run(nbytes, grid, waves, depth, reps):
        offs = [((i * nbytes) % (pool_bytes - nbytes)) // 1024 * 1024 for i in range(reps + 1)]
        C.check(lib.nld_hbm_read_probe(pool.data_ptr() + offs[0], nbytes, grid, waves, depth, sink.data_ptr(), s))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            C.check(lib.nld_hbm_read_probe(pool.data_ptr() + offs[i + 1], nbytes, grid, waves, depth, sink.data_ptr(),
                                           s))
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3   # us per launch

    shapes = {}
    for grid, waves, depth in ((256, 16, 16), (512, 16, 16), (1024, 16, 16), (2048, 16, 16)):
        us = run(2 << 30, grid, waves, depth, 4)
        shapes["%dx%dx%d" % (grid, waves, depth)] = round((2 << 30) / (us * 1e-6) / 1e9, 1)
    sizes = {mib: run(mib << 20, 256, 16, 16, 10) for mib in (16, 50, 200)}
    slope = (sizes[200] - sizes[50]) / (150 << 20)              # us per byte
    del pool
    torch.cuda.empty_cache()
    best = max(shapes, key=shapes.get)
    return {"read_GBps": shapes[best], "frac": round(shapes[best] / HBM_PEAK_GBS, 4),
            "grid_x_waves_x_depth": best, "by_shape_GBps": shapes,
            "us_per_launch": {"%d MiB" % m: round(v, 2) for m, v in sizes.items()},
            "fixed_us_per_launch": round(sizes[50] - slope * (50 << 20), 2),
            "marginal_GBps": round(1e-3 / slope, 1),
            "note": "nld_hbm_read_probe, launches timed back to back with events (launch gaps included)"}


def verify_pass_timing(R, model, cache, ws, anchor, k, reps):
    """Mean ms of one verify pass (verify + argmax + acceptance + commit) replayed from a captured graph with
    the lengths reset first, on drafts from one draft pass."""
    import torch
    B, dev = anchor.shape[0], anchor.device
    a0 = anchor.clone()
    d = torch.empty((B, k - 1), dtype=torch.int32, device=dev)
    R.draft(model, cache, ws, a0, k, out=d)
    len0 = cache.lengths.clone()
    outs = {"accept_len": torch.empty(B, dtype=torch.int32, device=dev),
            "committed": torch.empty((B, k), dtype=torch.int32, device=dev),
            "next_anchor": torch.empty(B, dtype=torch.int32, device=dev)}

    def verify():
        cache.lengths.copy_(len0)
        R.verify_accept(model, cache, ws, a0, d, k, outs=outs)

    ms = graph_ms(verify, reps)
    cache.lengths.copy_(len0)
    torch.cuda.synchronize()
    return ms


def large_config(R, name, reps=8):
    """One draft + verify + accept step of a many-row configuration (8b_batch32: 32 ragged sequences of the
    8B stack, 512 block rows; 14b: 8 sequences of the 14B stack at k = 32, 256 rows), replayed from a captured
    graph with the lengths reset first: step and verify-pass times, their fractions of the HBM roofline on
    the pass bytes, the algorithmic MFMA rate, and the per-kernel times of three traced steps.  Weights come
    from the seeded generator; the K/V caches are filled on the device with seeded N(0, 1) bf16 values
    (torch's generator: only the timing is measured here; the parity tests use the oracle's inputs)."""
    import torch
    from synth.workloads import LazyWeights, WORKLOADS, tokens
    wl = WORKLOADS[name]
    shape, k, B = wl.shape, wl.k_values[0], wl.batch
    plens = wl.prefix_lengths()
    max_len = int(-(-(int(plens.max()) + 2 * k) // 64) * 64)
    t0 = time.perf_counter()
    model = R.DeviceModel(shape, LazyWeights(shape, wl.seed, keep=False))
    cache = R.DeviceCache(shape, B, max_len)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1000 + wl.seed)
    for l in range(shape.n_layers):
        for t in (cache.k[l], cache.v[l]):
            t.view(torch.bfloat16).copy_(torch.randn(t.shape, generator=gen, device="cuda", dtype=torch.float32))
    cache.set_lengths(plens)
    ws = R.Workspace(model, B, k, max_len)
    torch.cuda.synchronize()
    log("%s: model and cache ready in %.1f s" % (name, time.perf_counter() - t0))
    dev = torch.device("cuda")
    a0 = torch.from_numpy(tokens(shape, wl.seed, "bench.%s.anchor" % name, (B,))).to(dev)
    len0 = cache.lengths.clone()
    i32 = lambda *shp: torch.empty(shp, dtype=torch.int32, device=dev)
    d, outs = i32(B, k - 1), {"accept_len": i32(B), "committed": i32(B, k), "next_anchor": i32(B)}

    def step():
        cache.lengths.copy_(len0)
        R.draft(model, cache, ws, a0, k, out=d)
        R.verify_accept(model, cache, ws, a0, d, k, outs=outs)

    step_ms = graph_ms(step, reps)
    verify_ms = verify_pass_timing(R, model, cache, ws, a0, k, reps)
    kernels = traced_kernels(step, 3)
    status = R.read_device_status(ws)
    pb, pf = pass_bytes(shape, B, k, plens), pass_flops(shape, B, k, plens)
    res = {
        "workload": "%s: %d layers, hidden %d, %d/%d heads, ffn %d; batch %d, prefix %s, k=%d" % (
            name, shape.n_layers, shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.ffn, B,
            "ragged %d..%d" % wl.ragged if wl.ragged else int(plens[0]), k),
        "rows_per_pass": B * k,
        "step_ms": round(step_ms, 3), "verify_pass_ms": round(verify_ms, 3),
        "block_tokens_per_s": round(2.0 * B * k / (step_ms * 1e-3), 1),
        "step_hbm_frac": round(2 * pb / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "algorithmic_TFLOPs": round(2 * pf / (step_ms * 1e-3) / 1e12, 1),
        "mfma_frac_of_bf16_peak": round(2 * pf / (step_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "note": "split activation operands: the issued MFMA work is about twice the algorithmic",
        "kernels_us": kernels, "device_status": status,
    }
    model.close()
    del model, cache, ws
    torch.cuda.empty_cache()
    return res


def cpu_model_name():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def layer_microbench(R, reps=20):
    """One 8B-shaped layer + LM head (batch 1, prefix 2048, seeded weights and K/V): mean ms of a verify
    pass and of a draft pass at k = 8, 16 and 32, each replayed from a captured graph."""
    import torch
    from synth.workloads import LazyWeights, WORKLOADS, prefix_kv, tokens
    wl = WORKLOADS["8b_layer"]
    shape, P = wl.shape, wl.prefix_len
    model = R.DeviceModel(shape, LazyWeights(shape, wl.seed, keep=False))
    cache = R.DeviceCache(shape, 1, P + 64)
    kb, vb = prefix_kv(shape, wl.seed, 0, 1, P)
    cache.load_prefix(0, kb, vb)
    cache.set_lengths([P])
    out = {}
    for k in wl.k_values:
        ws = R.Workspace(model, 1, k, P + 64)
        tok = torch.from_numpy(tokens(shape, wl.seed, "bench.layer.block%d" % k, (1, k))).cuda()
        res = {}
        for name, mode in (("verify", R.VERIFY), ("draft", R.DRAFT)):
            ms = graph_ms(lambda: R.block_forward(model, cache, ws, tok, mode, want_logits=False), reps)
            res[name + "_pass_ms"] = round(ms, 4)
            res[name + "_hbm_frac"] = round(pass_bytes(shape, 1, k, [P]) / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        out["k=%d" % k] = res
    model.close()
    return out


def copy_calibration(mib, reps=3):
    """Plain device-to-device copies of a known size, for scaling the counters of a --pmc run."""
    import torch
    n = mib * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("copy calibration: %d x copy of %d MiB (read %d KiB, write %d KiB per dispatch)" % (reps, mib, mib * 1024,
                                                                                             mib * 1024))
    del src, dst


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="8b")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--k", type=int, default=0, help="block size (default: the workload's first)")
    ap.add_argument("--max-len", type=int, default=0,
                    help="KV cache capacity in positions (default: the prefix plus the steps' growth)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the Mode 2 and LoRA timings (counter runs use this: eager launches only)")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the 8b_batch32 and 14b step timings of the extras")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run plain copies of this many MiB (reference dispatches for counter runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_05722_amd import _lib as C
    from paper_2607_05722_amd import runtime as R
    from synth.workloads import LazyWeights, WORKLOADS, prefix_kv, tokens

    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib)
    wl = WORKLOADS[args.workload]
    shape, k, B = wl.shape, (args.k or wl.k_values[0]), wl.batch
    if not 1 <= k <= 64:
        sys.exit("--k must be in [1, 64]")
    plens = wl.prefix_lengths()
    steps, warmup = args.steps, args.warmup
    max_len = int(-(-(int(plens.max()) + (steps + warmup + 6) * k) // 64) * 64)
    if args.max_len:
        if args.max_len < max_len or args.max_len % 64:
            sys.exit("--max-len must be a multiple of 64 and at least %d" % max_len)
        max_len = args.max_len
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.perf_counter()
    model = R.DeviceModel(shape, LazyWeights(shape, wl.seed, keep=False))
    log("weights generated, uploaded and packed in %.1f s" % (time.perf_counter() - t0))
    cache = R.DeviceCache(shape, B, max_len)
    for l in range(shape.n_layers):
        kb, vb = prefix_kv(shape, wl.seed, l, B, int(plens.max()))
        cache.load_prefix(l, kb, vb)
    cache.set_lengths(plens)
    ws = R.Workspace(model, B, k, max_len)
    anchor = torch.from_numpy(tokens(shape, wl.seed, "bench.anchor", (B,))).to(dev)
    drafts = torch.empty((B, k - 1), dtype=torch.int32, device=dev)
    outs = {"accept_len": torch.empty(B, dtype=torch.int32, device=dev),
            "committed": torch.empty((B, k), dtype=torch.int32, device=dev),
            "next_anchor": anchor}                        # in place: the loop never leaves the device
    torch.cuda.synchronize()
    log("cache filled (prefix %s), max_len %d, workspace %.1f MB" % (
        plens.tolist() if B <= 4 else "%d..%d" % (plens.min(), plens.max()), max_len, ws.nbytes / 1e6))

    committed_total = torch.zeros(1, dtype=torch.int64, device=dev)

    def step():
        R.draft(model, cache, ws, anchor, k, out=drafts)
        R.verify_accept(model, cache, ws, anchor, drafts, k, outs=outs)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        graph = None
        if not args.no_graph:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                step()
            graph.replay()
        torch.cuda.synchronize()
        len0 = cache.lengths.clone()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        # one event between consecutive steps: the whole region gives the mean, the pairs the percentiles
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps - 1)]
        e0.record()
        for i in range(steps):
            if graph is not None:
                graph.replay()
            else:
                step()
            if i < steps - 1:
                marks[i].record()
        e1.record()
        torch.cuda.synchronize()
        elapsed_ms = e0.elapsed_time(e1)
        bounds = [e0] + marks + [e1]
        per_step = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(steps)])
        committed = int((cache.lengths - len0).sum().item())
        status = R.read_device_status(ws)

        # per-kernel durations: every launch of a few eager steps records HIP events on its own dispatch
        lib = C.load()
        lib.nld_trace_enable(1)
        trace_steps = 3
        for _ in range(trace_steps):
            step()
        torch.cuda.synchronize()
        import ctypes
        ms = (ctypes.c_float * 8)()
        cnt = (ctypes.c_int32 * 8)()
        C.check(lib.nld_trace_read(ms, cnt, 8))
        lib.nld_trace_enable(0)

        verify_ms = verify_pass_timing(R, model, cache, ws, anchor, k, max(5, steps // 2)) if graph is not None \
            else None
        m2_ms = lora_ms = quad_ms = layer_ms = k32_ms = None
        if not args.no_extras:
            block_full = torch.from_numpy(tokens(shape, wl.seed, "bench.m2.block", (B, k))).to(dev)
            m2_ms, m2_committed = mode2_timing(R, model, cache, ws, anchor, block_full, k, max(5, steps // 2))
            lora_ms = lora_timing(R, model, cache, ws, anchor, k, max(5, steps // 2), wl)
            quad_ms = quad_timing(R, model, cache, anchor, max(5, steps // 2))
            k32_ms, k32_kernels, k32_status = block_size_timing(R, model, cache, anchor, max(5, steps // 2), 32)
            status |= k32_status
            layer_ms = layer_microbench(R)
            status |= R.read_device_status(ws) | lora_ms["status"] | quad_ms["status"]

    ms_per_step = elapsed_ms / steps
    value = 2.0 * B * k / (ms_per_step * 1e-3)
    bytes_step = 2 * pass_bytes(shape, B, k, plens)
    kb = kernel_bytes(shape, B, k, plens)
    kernels = {}
    for i, name in enumerate(C.TRACE_CLASSES):
        if cnt[i]:
            avg_ms = ms[i] / cnt[i]
            kernels[name] = {"avg_us": round(avg_ms * 1e3, 2), "launches_per_step": cnt[i] // trace_steps,
                             "GBps": round(kb[name] / (avg_ms * 1e-3) / 1e9, 1) if kb[name] else None}
    dom = max((n for n in kernels), key=lambda n: kernels[n]["avg_us"] * kernels[n]["launches_per_step"])
    dom_avg_s = kernels[dom]["avg_us"] * 1e-6
    achieved = kb[dom] / dom_avg_s / 1e9
    traffic = measured_traffic(dom) if args.workload == "8b" and k == wl.k_values[0] else None
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "block tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "step_ms_percentiles": {"p10": round(float(np.percentile(per_step, 10)), 4),
                                "p50": round(float(np.percentile(per_step, 50)), 4),
                                "p90": round(float(np.percentile(per_step, 90)), 4)},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "%s: %d layers, hidden %d, %d/%d heads, head_dim %d, ffn %d, vocab %d; batch %d, "
                               "prefix %s, block k=%d; step = draft pass + verify pass + accept"
                               % (wl.name, shape.n_layers, shape.hidden, shape.n_q_heads, shape.n_kv_heads,
                                  shape.head_dim, shape.ffn, shape.vocab, B,
                                  int(plens[0]) if wl.ragged is None else "ragged %d..%d" % wl.ragged, k),
                   "graph": graph is not None, "kv_capacity": max_len},
        "verify_pass_ms": round(verify_ms, 4) if verify_ms is not None else None,
        "verify_pass_block_tokens_per_s": round(B * k / (verify_ms * 1e-3), 1) if verify_ms is not None else None,
        "verify_pass_hbm_frac": round(pass_bytes(shape, B, k, plens) / (verify_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        if verify_ms is not None else None,
        "step_hbm_GBps": round(bytes_step / (ms_per_step * 1e-3) / 1e9, 1),
        "step_hbm_frac": round(bytes_step / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "algorithmic_bytes_per_step": int(bytes_step),
        "mfma": {"algorithmic_TFLOPs": round(2 * pass_flops(shape, B, k, plens) / (ms_per_step * 1e-3) / 1e12, 2),
                 "frac_of_bf16_peak": round(2 * pass_flops(shape, B, k, plens) / (ms_per_step * 1e-3) / 1e12
                                            / MFMA_BF16_PEAK_TFLOPS, 4),
                 "note": "split activation operands run two MFMAs per product: the issued MFMA work is about twice this"},
        "committed_tokens_per_s": round(committed / (elapsed_ms * 1e-3), 1),
        "device_status": status,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "bytes_per_launch": int(kb[dom]), "avg_launch_us": kernels[dom]["avg_us"]},
        "kernels": kernels,
    }
    if m2_ms is not None:
        res["mode2"] = {
            "denoise_step_ms": round(m2_ms["denoise_step"], 4),
            "denoise_hbm_frac": round(pass_bytes(shape, B, k, plens) / (m2_ms["denoise_step"] * 1e-3) / 1e9
                                      / HBM_PEAK_GBS, 4),
            "refresh_ms": round(m2_ms["refresh"], 4),
            "refresh_hbm_frac": round(refresh_bytes(shape, B, k, plens) / (m2_ms["refresh"] * 1e-3) / 1e9
                                      / HBM_PEAK_GBS, 4),
            "threshold": 0.9,
            "first_step_commits": m2_committed,
        }
        res["lora_draft"] = {
            "rank": LORA_RANK, "alpha": LORA_ALPHA,
            "draft_pass_ms": round(lora_ms["draft"], 4),
            "lora_draft_pass_ms": round(lora_ms["lora_draft"], 4),
            "lora_draft_hbm_frac": round((pass_bytes(shape, B, k, plens) + shape.n_layers * 2 * LORA_RANK
                                          * (shape.q_dim + shape.hidden)) / (lora_ms["lora_draft"] * 1e-3) / 1e9
                                         / HBM_PEAK_GBS, 4),
        }
    if not args.no_extras:
        res["hbm_stream_ceiling"] = hbm_ceiling()   # what a plain read stream reaches on this part
        res["step_frac_of_stream_ceiling"] = round(res["step_hbm_GBps"] / res["hbm_stream_ceiling"]["read_GBps"], 4)
        res["layer_microbench"] = layer_ms
    if k32_ms is not None:
        res["block_k32"] = {
            "step_ms": round(k32_ms, 4),
            "block_tokens_per_s": round(2.0 * B * 32 / (k32_ms * 1e-3), 1),
            "hbm_frac": round(2 * pass_bytes(shape, B, 32, plens) / (k32_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "kernels": k32_kernels,
        }
    if quad_ms is not None:
        R_q = QUAD_K * (QUAD_K + 1)
        res["quad_ss"] = {
            "k": QUAD_K, "block_rows": R_q,
            "step_ms_ar_verifier": round(quad_ms["quad_ar"], 4),
            "step_ms_ensemble_lambda_0.5": round(quad_ms["quad_ensemble"], 4),
            "linear_step_ms_same_width": round(quad_ms["linear"], 4),
            "quad_hbm_frac": round(pass_bytes(shape, B, R_q, plens) / (quad_ms["quad_ar"] * 1e-3) / 1e9
                                   / HBM_PEAK_GBS, 4),
            "kernels": quad_ms["kernels_us"],
        }
    if not args.no_extras or not args.no_cpu_baseline:
        model.close()
        del model, cache, ws
        torch.cuda.empty_cache()
    if not args.no_extras and not args.no_large:
        with torch.cuda.stream(torch.cuda.Stream()):     # graphs are captured on a non-default stream
            res["large_configs"] = {name: large_config(R, name) for name in ("8b_batch32", "14b")}
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, k)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
