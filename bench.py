#!/usr/bin/env python3
"""Benchmark of the three-stage W4A16 decoder layer on one MI355X.

One step = the whole hot path once on the Llama-3-8B-shaped layer (hidden 4096,
32/8 heads, head_dim 128, FFN 14336, W4A16 group 128, RoPE base 5e5):
    prefill     T = 512 tokens
    prefill_kv  T = 128 new tokens over a 1024-token history
    decode      B = 1 at context 2048
The steps rotate over several device copies of the layer (each with its own
KV cache) so that the working set exceeds the 256 MB Infinity Cache and the
weights stream from HBM, as they do across the layers of a real model.

Printed: one JSON line.  ``value`` is decode layer-steps/s (the stage the
paper measures); prefill and prefill_kv TFLOP/s are under ``stages``.  The
roofline object covers the kernel that takes the largest share of a step (the
prefill gate/up GEMM); the whole persistent decode launch is reported beside it.
Those two kernels are timed with the library's HIP-event pairs on the odd
timed steps; the stage times (and ``value``) come from the even steps, whose
stages carry no inner event pairs.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
PEAK_MFMA_TFLOPS = 2500.0        # dense bf16 / fp16 MFMA

# HBM traffic per launch of the rooflined kernels: FETCH_SIZE and WRITE_SIZE
# (rocprofv3 --pmc, one pass each, over "bench.py --steps 2 --warmup 1
# --no-cpu-baseline"), each divided by what the same counter reads per byte
# for a plain device copy of known size ("bench.py --copy-calibration").
# Keyed by the SHA-256 of the kernel's source files: once one of them changes
# the figure no longer describes the kernel and is reported as null.
TRAFFIC = {
    "prefill_gate_up": {"bytes": 133422111,
                       "sha256": "3fa3926b717144d4ea4b0b0ca528a12e6caf890a2d6ec484b0423c5891d5d57b"},
    "decode_fused": {"bytes": 129701867,
                    "sha256": "985571db4c7d43acd42e4ae51d0160981fb071c7f8b918ce78cb4e09154ec129"},
}
CSRC = os.path.join(ROOT, "paper_2607_15865_amd", "csrc")


TRAFFIC_SOURCES = {
    "prefill_gate_up": ("gemm_w4.hip", "common.h", "launch.h"),
    "decode_fused": ("decode_fused.hip", "decode_fused.h", "gemv_core.h", "common.h", "launch.h"),
}


def source_hash(key):
    import hashlib
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES[key]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic(key):
    """Measured HBM bytes per launch of a kernel, or None if one of its
    sources has changed since the counters were taken."""
    t = TRAFFIC.get(key)
    if not t or source_hash(key) != t["sha256"]:
        return None
    return t["bytes"]


def copy_calibration():
    """A plain device-to-device copy of 512 MiB, four times: the reference
    reading for FETCH_SIZE and WRITE_SIZE (each copy reads and writes
    exactly 512 MiB)."""
    import torch
    n = 512 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "copies": 4}), flush=True)
    return 0

WORKLOAD = dict(name="llama8b", prefill_T=512, pkv_T=128, pkv_L=1024, decode_B=1, decode_ctx=2048)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- algorithmic work

def linear_shapes(cfg):
    from paper_2607_15865_amd import synth
    return [cfg.linear_shape(n) for n in synth.LINEARS]


def weight_bytes(cfg, names=None, fmt="int4"):
    """Bytes of the linears' weights in a storage format: int4 codes + fp16
    group scales; int8 codes + one fp16 scale (and, "int8a", one zero point)
    per column; bf16 values."""
    from paper_2607_15865_amd import synth
    tot = 0
    for n in (names or synth.LINEARS):
        K, N = cfg.linear_shape(n)
        if fmt == "int4":
            tot += N * K // 2 + 2 * N * math.ceil(K / cfg.group_size)
        elif fmt in ("int8", "int8a"):
            tot += N * K + 2 * N + (N if fmt == "int8a" else 0)
        else:
            tot += 2 * N * K
    return tot


def stage_flops(cfg, M, T, L, B):
    """2 * rows * weights of the seven linears + attention on causal pairs."""
    params = sum(K * N for K, N in linear_shapes(cfg))
    attn = 4 * cfg.head_dim * cfg.n_heads * B * (T * L + T * (T + 1) / 2)
    return 2 * M * params + attn


def stage_bytes(cfg, M, T, L, B, fmt="int4"):
    """Weights (int4 + fp16 scales, or the other formats') + norm weights + KV
    read of the history and the new entries + KV write + fp32 hidden states
    in and out."""
    kv_row = 2 * 2 * cfg.n_kv_heads * cfg.head_dim          # K and V, bf16
    return (weight_bytes(cfg, fmt=fmt) + 4 * cfg.hidden + kv_row * B * (L + T) + kv_row * B * T
            + 8 * M * cfg.hidden)


# ---------------------------------------------------------------- extras

def extras(cfg, layers, caches, binding, synth, stream, reps=30):
    """Timed after the bench steps, outside them: speculative-decode
    verification (prefill_kv of T = 2, 4, 8 draft tokens over a 2048-token
    history) and a 4096-token prompt as one prefill against 4 segments of 1024
    (one prefill, three prefill_kv).  Median of `reps` calls rotating over the
    device copies, HIP events on the library's stream."""
    import numpy as np
    import torch
    h0 = layers[0].handle
    sp = stream.cuda_stream
    L, Tp, chunk = 2048, cfg.max_seq, 1024
    ws_bytes = max([binding.layer_workspace_size(h0, 1, 1, T, L) for T in (2, 4, 8)]
                   + [binding.layer_workspace_size(h0, 0, 1, Tp, 0),
                      binding.layer_prefill_chunked_workspace_size(h0, Tp, chunk)])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

    def f32(bits):
        u = bits.astype(np.uint32) << 16
        return torch.from_numpy(u.view(np.float32).copy()).cuda()

    def median_us(call):
        ts = []
        for i in range(reps + 2):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call(i)
            e1.record(stream)
            e1.synchronize()
            if i >= 2:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts))

    res = {"verify": {}}
    for T in (2, 4, 8):
        x = f32(synth.activations(cfg, synth.TID_X_PREFILL_KV, T))
        y = torch.empty_like(x)
        pos = torch.arange(L, L + T, dtype=torch.int32, device="cuda")

        def call(i, x=x, y=y, pos=pos, T=T):
            k, v = caches[i % len(layers)]
            binding.check(binding.layer_prefill_kv(layers[i % len(layers)].handle, x, pos, T, L, k, v, y, ws,
                                                   ws_bytes, sp))
        us = median_us(call)
        by = stage_bytes(cfg, T, T, L, 1)
        res["verify"][f"T{T}"] = {"hist": L, "us": round(us, 2), "mbytes": round(by / 1e6, 2),
                                  "gbps": round(by / (us * 1e-6) / 1e9, 1),
                                  "frac_hbm": round(by / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    x = f32(synth.activations(cfg, synth.TID_X_PREFILL, Tp))
    y = torch.empty_like(x)
    pos = torch.arange(Tp, dtype=torch.int32, device="cuda")
    fl = stage_flops(cfg, Tp, Tp, 0, 1)

    def one(i):
        k, v = caches[i % len(layers)]
        binding.check(binding.layer_prefill(layers[i % len(layers)].handle, x, pos, Tp, k, v, y, ws, ws_bytes, sp))

    def seg(i):
        k, v = caches[i % len(layers)]
        binding.check(binding.layer_prefill_chunked(layers[i % len(layers)].handle, x, pos, Tp, chunk, k, v, y, ws,
                                                    ws_bytes, sp))
    for name, call in (("prefill_4096", one), ("prefill_4096_in_4x1024", seg)):
        us = median_us(call)
        res[name] = {"ms": round(us / 1e3, 4), "gflop": round(fl / 1e9, 1),
                     "tflops": round(fl / (us * 1e-6) / 1e12, 1),
                     "frac_mfma": round(fl / (us * 1e-6) / 1e12 / PEAK_MFMA_TFLOPS, 4)}
    return res


# ---------------------------------------------------------------- other workloads

def reports(binding, synth, stream, reps=20):
    """The other workloads' stages, timed after the bench steps (outside
    them): the Qwen-7B-shaped layer's prefill of 2048 tokens and its decode at
    context 8192 with 1 and 8 rows (3 rotating copies of weights and 8-row
    caches, 258 MB each), and the Qwen-0.5B-shaped layer's prefill of 256,
    prefill_kv of 64 over 256 and decode at context 512 (68 copies of 7.7 MB,
    so the rotation exceeds the 256 MB last-level cache; these calls are
    launch-bound).  Median of `reps` calls, HIP events on the library's
    stream; synthetic seeded weights, N(0,1) caches."""
    import numpy as np
    import torch
    sp = stream.cuda_stream

    def f32(bits):
        u = bits.astype(np.uint32) << 16
        return torch.from_numpy(u.view(np.float32).copy()).cuda()

    def median_us(call):
        ts = []
        for i in range(reps + 2):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call(i)
            e1.record(stream)
            e1.synchronize()
            if i >= 2:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts))

    def flops_entry(cfg, us, M, T, L):
        fl = stage_flops(cfg, M, T, L, 1)
        return {"us": round(us, 2), "gflop": round(fl / 1e9, 2), "tflops": round(fl / (us * 1e-6) / 1e12, 1),
                "frac_mfma": round(fl / (us * 1e-6) / 1e12 / PEAK_MFMA_TFLOPS, 4)}

    def bytes_entry(cfg, us, B, ctx, M=None, T=1):
        by = stage_bytes(cfg, M or B, T, ctx, B)
        return {"us": round(us, 2), "mbytes": round(by / 1e6, 2), "gbps": round(by / (us * 1e-6) / 1e9, 1),
                "frac_hbm": round(by / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}

    out = {}
    for name, ncp, Bmax in (("qwen7b", 3, 8), ("qwen05b", 68, 1)):
        cfg = synth.CONFIGS[name]
        run = synth.RUNS[name]
        log(f"bench: {name} report ({ncp} copies)")
        w = synth.make_layer(cfg)
        layers = [binding.Layer(cfg, w) for _ in range(ncp)]
        kb, vb = synth.kv_fill(cfg, Bmax)
        caches = [(torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
                  for _ in range(ncp)]
        h0 = layers[0].handle
        Tp, ctx = run["prefill_T"], run["decode_ctx"]
        need = [binding.layer_workspace_size(h0, 0, 1, Tp, 0)]
        need += [binding.layer_workspace_size(h0, 2, B, 1, ctx) for B in run["decode_B"]]
        if run["pkv_T"]:
            need.append(binding.layer_workspace_size(h0, 1, 1, run["pkv_T"], run["pkv_hist"]))
        ws_bytes = max(need)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        res = {}
        xp = f32(synth.activations(cfg, synth.TID_X_PREFILL, Tp))
        yp = torch.empty_like(xp)
        pp = torch.arange(Tp, dtype=torch.int32, device="cuda")

        def pre(i):
            k, v = caches[i % ncp]
            binding.check(binding.layer_prefill(layers[i % ncp].handle, xp, pp, Tp, k, v, yp, ws, ws_bytes, sp))
        res[f"prefill_T{Tp}"] = flops_entry(cfg, median_us(pre), Tp, Tp, 0)
        if run["pkv_T"]:
            Tk, Lk = run["pkv_T"], run["pkv_hist"]
            xk = f32(synth.activations(cfg, synth.TID_X_PREFILL_KV, Tk))
            yk = torch.empty_like(xk)
            pk = torch.arange(Lk, Lk + Tk, dtype=torch.int32, device="cuda")

            def pkv(i):
                k, v = caches[i % ncp]
                binding.check(binding.layer_prefill_kv(layers[i % ncp].handle, xk, pk, Tk, Lk, k, v, yk, ws, ws_bytes,
                                                       sp))
            us = median_us(pkv)
            res[f"prefill_kv_T{Tk}_over_{Lk}"] = dict(flops_entry(cfg, us, Tk, Tk, Lk),
                                                     **{k2: v2 for k2, v2 in bytes_entry(cfg, us, 1, Lk, Tk, Tk).items()
                                                        if k2 != "us"})
        for B in run["decode_B"]:
            xd = f32(synth.activations(cfg, synth.TID_X_DECODE, B))
            yd = torch.empty_like(xd)
            cd = torch.full((B,), ctx, dtype=torch.int32, device="cuda")

            def dec(i, xd=xd, yd=yd, cd=cd, B=B):
                k, v = caches[i % ncp]
                binding.check(binding.layer_decode(layers[i % ncp].handle, xd, cd, cd, ctx, None, B, k, v, yd, ws,
                                                   ws_bytes, sp))
            res[f"decode_B{B}_ctx{ctx}"] = bytes_entry(cfg, median_us(dec), B, ctx)
        out[name] = res
        torch.cuda.synchronize()
        for lay in layers:
            if lay.error():
                raise RuntimeError(f"{name}: a device error flag was raised")
            lay.close()
        del caches, ws
    return out


# ---------------------------------------------------------------- weight formats

def formats(binding, synth, stream, reps=20):
    """The paper's other direct-through weight modes on the Llama-3-8B-shaped
    layer, timed after the bench steps (outside them): INT8 symmetric, INT8
    asymmetric (per-column scales) and BF16 weights, each through prefill
    T = 512, prefill_kv T = 128 over 1024 and decode B = 1 at context 2048
    (the decode kernel sequence: the persistent launch takes INT4 only).
    Rotation over 2 device copies (440 MB or 872 MB, beyond the 256 MB
    last-level cache).  Median of `reps` calls, HIP events on the library's
    stream; synthetic seeded weights, N(0,1) cache."""
    import numpy as np
    import torch
    sp = stream.cuda_stream
    cfg = synth.CONFIGS[WORKLOAD["name"]]
    Tp, Tk, Lk, ctx = WORKLOAD["prefill_T"], WORKLOAD["pkv_T"], WORKLOAD["pkv_L"], WORKLOAD["decode_ctx"]

    def f32(bits):
        u = bits.astype(np.uint32) << 16
        return torch.from_numpy(u.view(np.float32).copy()).cuda()

    def median_us(call):
        ts = []
        for i in range(reps + 2):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call(i)
            e1.record(stream)
            e1.synchronize()
            if i >= 2:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts))

    kb, vb = synth.kv_fill(cfg, 1)
    xp = f32(synth.activations(cfg, synth.TID_X_PREFILL, Tp))
    xk = f32(synth.activations(cfg, synth.TID_X_PREFILL_KV, Tk))
    xd = f32(synth.activations(cfg, synth.TID_X_DECODE, 1))
    yp, yk, yd = torch.empty_like(xp), torch.empty_like(xk), torch.empty_like(xd)
    pp = torch.arange(Tp, dtype=torch.int32, device="cuda")
    pk = torch.arange(Lk, Lk + Tk, dtype=torch.int32, device="cuda")
    cd = torch.full((1,), ctx, dtype=torch.int32, device="cuda")
    out = {}
    for fmt in ("int8", "int8a", "bf16"):
        log(f"bench: {fmt} weights")
        w = synth.make_layer(cfg, fmt=fmt)
        ncp = 2
        layers = [binding.Layer(cfg, w) for _ in range(ncp)]
        del w
        caches = [(torch.from_numpy(kb.view(np.int16)).cuda(), torch.from_numpy(vb.view(np.int16)).cuda())
                  for _ in range(ncp)]
        h0 = layers[0].handle
        ws_bytes = max(binding.layer_workspace_size(h0, 0, 1, Tp, 0), binding.layer_workspace_size(h0, 1, 1, Tk, Lk),
                       binding.layer_workspace_size(h0, 2, 1, 1, ctx))
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

        def pre(i):
            k, v = caches[i % ncp]
            binding.check(binding.layer_prefill(layers[i % ncp].handle, xp, pp, Tp, k, v, yp, ws, ws_bytes, sp))

        def pkv(i):
            k, v = caches[i % ncp]
            binding.check(binding.layer_prefill_kv(layers[i % ncp].handle, xk, pk, Tk, Lk, k, v, yk, ws, ws_bytes, sp))

        def dec(i):
            k, v = caches[i % ncp]
            binding.check(binding.layer_decode(layers[i % ncp].handle, xd, cd, cd, ctx, None, 1, k, v, yd, ws,
                                               ws_bytes, sp))
        res = {"weight_mbytes": round(weight_bytes(cfg, fmt=fmt) / 1e6, 1)}
        for name, call, M, T, L in (("prefill", pre, Tp, Tp, 0), ("prefill_kv", pkv, Tk, Tk, Lk)):
            us = median_us(call)
            fl = stage_flops(cfg, M, T, L, 1)
            res[name] = {"us": round(us, 2), "tflops": round(fl / (us * 1e-6) / 1e12, 1),
                         "frac_mfma": round(fl / (us * 1e-6) / 1e12 / PEAK_MFMA_TFLOPS, 4)}
        us = median_us(dec)
        by = stage_bytes(cfg, 1, 1, ctx, 1, fmt=fmt)
        res["decode"] = {"us": round(us, 2), "layer_steps_per_s": round(1e6 / us, 1), "mbytes": round(by / 1e6, 2),
                         "gbps": round(by / (us * 1e-6) / 1e9, 1),
                         "frac_hbm": round(by / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
        torch.cuda.synchronize()
        for lay in layers:
            if lay.error():
                raise RuntimeError(f"{fmt}: a device error flag was raised")
            lay.close()
        del caches, ws, layers
        out[fmt] = res
    return out


# ---------------------------------------------------------------- CPU baseline

def cpu_baseline(cfg, w):
    """The oracle as it stands, timed on this host on a bounded sample of the
    workload: one decode layer-step (B = 1, context 2048) repeated for about
    5 s, one prefill of 512 tokens and one prefill_kv of 128 over 1024, in
    the oracle's fp64 and in its fp32 working precision (oracle.layer.
    working_precision, timing only).  The weights are dequantised once,
    outside the timed calls (the oracle's W argument).  Records the host's
    core count, this process's affinity and the BLAS thread count."""
    import numpy as np
    from oracle import layer as O
    from paper_2607_15865_amd import synth
    blas = None
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        blas = max([i.get("num_threads", 1) for i in info] or [1])
    except Exception:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except Exception:
        affinity = None
    Tp, Tk, Lk, ctx = WORKLOAD["prefill_T"], WORKLOAD["pkv_T"], WORKLOAD["pkv_L"], WORKLOAD["decode_ctx"]
    rng = np.random.default_rng(0)
    kb = synth.bf16_bits(rng.standard_normal((1, cfg.n_kv_heads, ctx + 1, cfg.head_dim)))
    vb = synth.bf16_bits(rng.standard_normal((1, cfg.n_kv_heads, ctx + 1, cfg.head_dim)))
    xd_b = synth.activations(cfg, synth.TID_X_DECODE, 1)
    xp_b = synth.activations(cfg, synth.TID_X_PREFILL, Tp)
    xk_b = synth.activations(cfg, synth.TID_X_PREFILL_KV, Tk)
    modes = {}
    for name, dt in (("fp64", np.float64), ("fp32", np.float32)):
        with O.working_precision(dt):
            W = O.dequant_layer(w, cfg)
            kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
            xd, xp, xk = O.bf16_to_f64(xd_b), O.bf16_to_f64(xp_b), O.bf16_to_f64(xk_b)
            n, t0 = 0, time.perf_counter()
            while n == 0 or time.perf_counter() - t0 < 5.0:
                O.decode(w, cfg, xd, [ctx], kc, vc, [ctx], W=W)
                n += 1
            dt_d = (time.perf_counter() - t0) / n
            t0 = time.perf_counter()
            O.prefill(w, cfg, xp, np.arange(Tp), W=W)
            dt_p = time.perf_counter() - t0
            t0 = time.perf_counter()
            O.prefill_kv(w, cfg, xk, np.arange(Lk, Lk + Tk), kc[0], vc[0], Lk, W=W)
            dt_k = time.perf_counter() - t0
        fl_p, fl_k = stage_flops(cfg, Tp, Tp, 0, 1), stage_flops(cfg, Tk, Tk, Lk, 1)
        modes[name] = {"decode_layer_steps_per_s": round(1.0 / dt_d, 3), "decode_calls": n,
                       "prefill_s": round(dt_p, 3), "prefill_gflops": round(fl_p / dt_p / 1e9, 1),
                       "prefill_kv_s": round(dt_k, 3), "prefill_kv_gflops": round(fl_k / dt_k / 1e9, 1)}
        del W
    return {"value": modes["fp64"]["decode_layer_steps_per_s"], "unit": "layer-steps/s",
            "cores": blas or affinity or os.cpu_count(), "kind": "oracle",
            "sample": f"decode layer-steps of the {WORKLOAD['name']}-shaped layer at context {ctx}, B=1, repeated "
                      f"for 5 s, fp64 numpy, weights dequantised outside the timing; also one prefill of {Tp} "
                      f"and one prefill_kv of {Tk} over {Lk}, and the same in the fp32 working precision",
            "os_cpu_count": os.cpu_count(), "affinity_cpus": affinity, "blas_threads": blas, "modes": modes}


# ---------------------------------------------------------------- ceilings

def ceilings(binding, stream, reps=5):
    """What the device sustains on the two bounding resources, measured with
    the library's ceiling kernels beside the published peaks: a pure streaming
    read of 2 GiB (best grid of 1024 / 2048 / 4096 blocks of 256 threads) and a
    pure fp16 MFMA loop (the GEMV's 16x16x32 and the GEMM's 32x32x16, 2 blocks
    of 4 waves per CU).  Median of `reps` launches, HIP events."""
    import numpy as np
    import torch
    nbytes = 2 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(7)
    sink = torch.empty(4096 * 256, dtype=torch.int32, device="cuda")
    cus = torch.cuda.get_device_properties(0).multi_processor_count

    def timed(call):
        ts = []
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return float(np.median(ts[1:]))

    best = None
    for blocks in (1024, 2048, 4096):
        t = timed(lambda: binding.check(binding.w4_ceiling_read(buf, nbytes, sink, blocks, stream)))
        gbs = nbytes / t / 1e9
        if best is None or gbs > best[0]:
            best = (gbs, blocks)
    out = {"hbm_read": {"gbps": round(best[0], 1), "frac_of_peak": round(best[0] / PEAK_HBM_GBS, 4),
                        "bytes": nbytes, "blocks": best[1]}}
    del buf
    fsink = torch.empty(2 * cus * 256, dtype=torch.float32, device="cuda")
    for key, big in (("mfma_f16_16x16x32", False), ("mfma_f16_32x32x16", True)):
        iters = 20000 if big else 40000
        rc, fl = binding.w4_ceiling_mfma(fsink, 2 * cus, iters, big, stream)
        binding.check(rc)
        t = timed(lambda: binding.check(binding.w4_ceiling_mfma(fsink, 2 * cus, iters, big, stream)[0]))
        out[key] = {"tflops": round(fl / t / 1e12, 1), "frac_of_peak": round(fl / t / 1e12 / PEAK_MFMA_TFLOPS, 4)}
    return out


# The paper's own decode figures (Table 2, Sec. 5.2): whole-model decode of
# W4BF16 Qwen3.5 models at 2K context on a Sophgo BM1684X (64 GB/s DDR),
# bandwidth utilisation = tokens/s x model size / peak bandwidth (Sec. 5.1).
# Another device and whole models: context for the per-layer figures here,
# not a baseline.
PAPER_TABLE2 = [{"model": "Qwen3.5-2B", "size_gb": 1.67, "tokens_per_s": 30.00, "bw_util": 0.780},
                {"model": "Qwen3.5-4B", "size_gb": 3.00, "tokens_per_s": 16.77, "bw_util": 0.786},
                {"model": "Qwen3.5-9B", "size_gb": 5.39, "tokens_per_s": 9.84, "bw_util": 0.830}]


# ---------------------------------------------------------------- main

STACK = dict(name="llama8b", prompt=1024, steps=256)


def run_stack(args):
    """The layer stack (one model's decoder layers, each with its own seeded
    weights and KV cache): prefill the prompt through all layers, then decode
    token by token with a growing cache.  Each decode step's layer-0 input is
    a seeded N(0, 1) row standing in for an embedded sampled token.  Prints
    one JSON line: end-to-end decode tokens/s."""
    import numpy as np
    import torch
    from paper_2607_15865_amd import binding, synth

    cfg = synth.CONFIGS[STACK["name"]]
    nl, P, S = args.stack_layers, STACK["prompt"], STACK["steps"]
    log(f"stack: building {nl} {cfg.name} layers")
    t0 = time.time()
    layers = [binding.Layer(cfg, synth.make_layer_words(cfg, l)) for l in range(nl)]
    log(f"stack: layers built in {time.time() - t0:.1f} s")
    st = binding.Stack(layers)
    caches = [l.new_cache(1) for l in layers]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]

    def rows_f32(bits):
        return torch.from_numpy((bits.astype(np.uint32) << 16).view(np.float32)).cuda()

    xp = rows_f32(synth.activations(cfg, synth.TID_X_PREFILL, P))
    yp = torch.empty_like(xp)
    xd = rows_f32(np.concatenate([synth.activations(cfg, synth.TID_X_DECODE + 1000 * s, 1) for s in range(S)]))
    yd = torch.empty_like(xd)
    slots = torch.arange(P, P + S, dtype=torch.int32, device="cuda")
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    torch.cuda.synchronize()
    e0.record()
    st.prefill(xp, torch.arange(P, dtype=torch.int32, device="cuda"), 0, kcs, vcs, yp)
    e1.record()
    for s in range(S):
        st.decode(xd[s:s + 1], slots[s:s + 1], slots[s:s + 1], P + s, kcs, vcs, yd[s:s + 1])
    e2.record()
    torch.cuda.synchronize()
    prefill_ms = e0.elapsed_time(e1)
    decode_ms = e1.elapsed_time(e2)
    assert torch.isfinite(yd).all() and torch.isfinite(yp).all()
    assert all(l.error() == 0 for l in layers), "a device error flag was raised"
    tok_s = S / (decode_ms * 1e-3)
    # bytes a decode step reads: all weights plus the K/V of every layer (ctx P..P+S-1)
    wbytes = weight_bytes(cfg) * nl
    kv = 2 * cfg.n_kv_heads * cfg.head_dim * 2 * nl * (P + S / 2)
    gbps = (wbytes + kv) * tok_s / 1e9
    pf = stage_flops(cfg, P, P, 0, 1) * nl
    line = {
        "metric": "end-to-end decode tokens/s of a 32-layer W4A16 Llama-3-8B-shaped stack",
        "value": round(tok_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": S, "warmup": 0,
        "ms_per_step": round(decode_ms / S, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16 activations, int4 weights, fp32 accumulate",
        "data": "synthetic: seeded int4 weights per layer, N(0,1) inputs",
        "config": {"workload": f"{nl}-layer {cfg.name}-shaped stack: prefill {P} tokens, then {S} decode steps "
                               f"at B=1 (context {P} -> {P + S - 1})"},
        "decode": {"layer_step_us": round(decode_ms * 1e3 / (S * nl), 2), "gbps": round(gbps, 1),
                   "frac_hbm": round(gbps / PEAK_HBM_GBS, 4)},
        "prefill": {"ms": round(prefill_ms, 3), "tflops": round(pf / (prefill_ms * 1e-3) / 1e12, 1),
                    "frac_mfma": round(pf / (prefill_ms * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4)},
    }
    line["model"] = run_model_loop(cfg, st, kcs, vcs, P, S, decode_ms, binding, synth)
    if args.stack_batch > 1:
        del caches, kcs, vcs
        line["model_batch"] = run_model_loop_batch(cfg, layers, st, args.stack_batch, binding, synth)
    print(json.dumps(line), flush=True)
    torch.cuda.synchronize()
    for l in layers:
        l.close()
    return 0


def run_model_loop(cfg, st, kcs, vcs, P, S, layers_ms, binding, synth, vocab=128256, reps=30):
    """The whole-model greedy loop on the stack: embed the prompt, prefill it
    through every layer, LM head + greedy pick on its last row, then S steps
    of the native loop step (model_decode_greedy: embed(picked token) ->
    every layer's decode -> LM head + pick), with no host round trip inside
    the timed region.  The ends use a Llama-3-8B
    vocabulary of 128256 tokens (seeded int4 head, bf16 embedding rows).
    Also the LM head + pick alone at B=1 (median of reps, HIP events)."""
    import numpy as np
    import torch
    lw = synth.make_lm(cfg, vocab, words=True)
    lm = binding.LM(cfg, lw, max_batch=1)
    del lw
    H = cfg.hidden
    prompt = torch.from_numpy(synth.tokens(cfg, vocab, P)).cuda()
    xp = torch.empty(P, H, device="cuda")
    yp = torch.empty_like(xp)
    x1 = torch.empty(1, H, device="cuda")
    y1 = torch.empty_like(x1)
    logits = torch.empty(1, vocab, device="cuda")
    picks = torch.empty(S + 1, dtype=torch.int32, device="cuda")
    slots = torch.arange(P, P + S, dtype=torch.int32, device="cuda")
    lm.head(y1, logits, picks[:1])               # workspace allocation outside the timed region
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    torch.cuda.synchronize()
    e0.record()
    lm.embed(prompt, xp)
    st.prefill(xp, torch.arange(P, dtype=torch.int32, device="cuda"), 0, kcs, vcs, yp)
    lm.head(yp[P - 1:P], logits, picks[0:1])
    handles = [l for l in st.handles]
    max_ctx = P + S
    n = binding.model_decode_workspace_size(handles, lm.handle, 1, max_ctx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    e1.record()
    for s in range(S):
        binding.check(binding.model_decode_greedy(handles, lm.handle, picks[s:s + 1], slots[s:s + 1], slots[s:s + 1],
                                                  P + s, 1, kcs, vcs, logits, picks[s + 1:s + 2], ws, n))
    e2.record()
    torch.cuda.synchronize()
    assert lm.error() == 0 and all(binding.layer_error(h) == (0, 0) for h in handles)
    toks = picks.cpu().numpy()
    assert ((toks >= 0) & (toks < vocab)).all()
    loop_ms = e1.elapsed_time(e2)
    ts = []
    for i in range(reps + 2):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        lm.head(y1, logits, picks[:1])
        b.record()
        b.synchronize()
        if i >= 2:
            ts.append(a.elapsed_time(b) * 1e3)
    head_us = float(np.median(ts))
    G = cfg.group_size
    hbytes = H * vocab // 2 + (H // G) * vocab * 2 + 4 * vocab + 4 * H
    lm.close()
    return {"workload": f"embed -> {len(kcs)} layers -> LM head (vocab {vocab}) -> greedy pick, "
                        f"prompt {P}, {S} generated tokens at B=1",
            "tokens_per_s": round(S / (loop_ms * 1e-3), 1), "ms_per_token": round(loop_ms / S, 4),
            "ends_ms_per_token": round((loop_ms - layers_ms) / S, 4),
            "prefill_to_first_token_ms": round(e0.elapsed_time(e1), 3),
            "lm_head_pick_us": round(head_us, 2),
            "lm_head_gbps": round(hbytes / (head_us * 1e-6) / 1e9, 1),
            "lm_head_frac_hbm": round(hbytes / (head_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}


def run_model_loop_batch(cfg, layers, st, B, binding, synth, vocab=128256, P=256, S=64):
    """The whole-model greedy loop for B sequences decoded together: each
    prompt of P tokens prefilled into its own cache row, then S steps of
    embed(B picked tokens) -> every layer's decode at B -> LM head + pick
    for the B rows, no host round trip inside the timed region.  Reports
    the aggregate generated tokens/s."""
    import torch
    lw = synth.make_lm(cfg, vocab, words=True)
    lm = binding.LM(cfg, lw, max_batch=B)
    del lw
    H = cfg.hidden
    caches = [l.new_cache(B) for l in layers]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    x1 = torch.empty(B, H, device="cuda")
    y1 = torch.empty_like(x1)
    logits = torch.empty(B, vocab, device="cuda")
    picks = torch.empty(S + 1, B, dtype=torch.int32, device="cuda")
    lm.head(y1, logits, picks[0])                # workspace allocation outside the timed region
    xp = torch.empty(P, H, device="cuda")
    yp = torch.empty_like(xp)
    ylast = torch.empty(B, H, device="cuda")
    pos = torch.arange(P, dtype=torch.int32, device="cuda")
    ctxs = (torch.arange(S, dtype=torch.int32, device="cuda")[:, None] + P).repeat(1, B).contiguous()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    torch.cuda.synchronize()
    e0.record()
    for b in range(B):
        prompt = torch.from_numpy(synth.tokens(cfg, vocab, P, seed=100 + b)).cuda()
        lm.embed(prompt, xp)
        st.prefill(xp, pos, 0, [k[b:b + 1] for k in kcs], [v[b:b + 1] for v in vcs], yp)
        ylast[b] = yp[P - 1]
    lm.head(ylast, logits, picks[0])
    handles = [l for l in st.handles]
    n = binding.model_decode_workspace_size(handles, lm.handle, B, P + S)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    e1.record()
    for s in range(S):
        binding.check(binding.model_decode_greedy(handles, lm.handle, picks[s], ctxs[s], ctxs[s], P + s, B, kcs, vcs,
                                                  logits, picks[s + 1], ws, n))
    e2.record()
    torch.cuda.synchronize()
    assert lm.error() == 0 and all(binding.layer_error(h) == (0, 0) for h in handles)
    toks = picks.cpu().numpy()
    assert ((toks >= 0) & (toks < vocab)).all()
    loop_ms = e1.elapsed_time(e2)
    lm.close()
    return {"workload": f"{B} sequences: prompts of {P} prefilled, then {S} greedy steps at B={B} through "
                        f"embed -> {len(layers)} layers -> LM head (vocab {vocab}) -> pick",
            "tokens_per_s": round(B * S / (loop_ms * 1e-3), 1), "ms_per_step": round(loop_ms / S, 4),
            "prefill_ms": round(e0.elapsed_time(e1), 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--copies", type=int, default=8, help="device copies of the layer (rotation)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the verification and long-prompt timings done after the steps")
    ap.add_argument("--no-reports", action="store_true",
                    help="skip the other workloads (Qwen-7B- and Qwen-0.5B-shaped layers) timed after the steps")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the streaming-read and MFMA-loop ceiling kernels timed after the steps")
    ap.add_argument("--no-formats", action="store_true",
                    help="skip the INT8 / BF16 weight layers timed after the steps")
    ap.add_argument("--stack", action="store_true",
                    help="instead: the 32-layer stack, 1024-token prefill then 256 decode steps")
    ap.add_argument("--stack-layers", type=int, default=32)
    ap.add_argument("--stack-batch", type=int, default=1,
                    help="with --stack: also run the whole-model greedy loop for this many sequences at once")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="instead: a plain 512 MiB device copy, the reference kernel for the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the layer's single-GPU kernels; --gpus {args.gpus} is not supported "
              "(the path runs on one GPU; sharding it over several is not built)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        return copy_calibration()
    if args.stack:
        return run_stack(args)

    import numpy as np
    import torch
    from paper_2607_15865_amd import binding, synth

    cfg = synth.CONFIGS[WORKLOAD["name"]]
    Tp, Tk, Lk = WORKLOAD["prefill_T"], WORKLOAD["pkv_T"], WORKLOAD["pkv_L"]
    Bd, ctx = WORKLOAD["decode_B"], WORKLOAD["decode_ctx"]
    log(f"bench: generating the {cfg.name} layer")
    w = synth.make_layer(cfg)
    layers, caches = [], []
    kb, vb = synth.kv_fill(cfg, 1)
    for i in range(args.copies):
        layers.append(binding.Layer(cfg, w))
        k = torch.from_numpy(kb.view(np.int16)).cuda()
        v = torch.from_numpy(vb.view(np.int16)).cuda()
        caches.append((k, v))
    log(f"bench: {args.copies} device copies created")

    def f32(bits):
        u = bits.astype(np.uint32) << 16
        return torch.from_numpy(u.view(np.float32).copy()).cuda()

    xp = f32(synth.activations(cfg, synth.TID_X_PREFILL, Tp))
    xk = f32(synth.activations(cfg, synth.TID_X_PREFILL_KV, Tk))
    xd = f32(synth.activations(cfg, synth.TID_X_DECODE, Bd))
    yp, yk, yd = torch.empty_like(xp), torch.empty_like(xk), torch.empty_like(xd)
    pp = torch.arange(Tp, dtype=torch.int32, device="cuda")
    pk = torch.arange(Lk, Lk + Tk, dtype=torch.int32, device="cuda")
    pd = torch.full((Bd,), ctx, dtype=torch.int32, device="cuda")
    cd = torch.full((Bd,), ctx, dtype=torch.int32, device="cuda")
    ws_bytes = max(binding.layer_workspace_size(layers[0].handle, 0, 1, Tp, 0),
                   binding.layer_workspace_size(layers[0].handle, 1, 1, Tk, Lk),
                   binding.layer_workspace_size(layers[0].handle, 2, Bd, 1, ctx))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    PREFILL_GU, DECODE_FUSED = 5, 6

    def step(i, ev=None):
        lay = layers[i % len(layers)].handle
        k, v = caches[i % len(layers)]
        if ev: ev[0].record(stream)
        binding.check(binding.layer_prefill(lay, xp, pp, Tp, k, v, yp, ws, ws_bytes, sp))
        if ev: ev[1].record(stream)
        binding.check(binding.layer_prefill_kv(lay, xk, pk, Tk, Lk, k, v, yk, ws, ws_bytes, sp))
        if ev: ev[2].record(stream)
        binding.check(binding.layer_decode(lay, xd, pd, cd, ctx, None, Bd, k, v, yd, ws, ws_bytes, sp))
        if ev: ev[3].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"bench: {args.warmup} warmup steps done")

    # The rooflined kernels are timed on the odd steps only (the library's
    # event pair around a launch lengthens the stage it sits in); the stage
    # times come from the even steps.
    prof_steps = set(range(1, args.steps, 2)) if args.steps >= 2 else {0}
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        on = i in prof_steps
        for lay in layers:
            binding.check(binding.layer_profile_kernel(lay.handle, 0, PREFILL_GU if on else -1))
            binding.check(binding.layer_profile_kernel(lay.handle, 2, DECODE_FUSED if on else -1))
        step(i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log(f"bench: {args.steps} timed steps in {wall:.3f} s")

    stage_steps = [i for i in range(args.steps) if i not in prof_steps] or list(range(args.steps))
    st_ms = np.zeros(3)
    for i in stage_steps:
        for j in range(3):
            st_ms[j] += evs[i][j].elapsed_time(evs[i][j + 1])
    st_ms /= len(stage_steps)
    gu_ms, gu_n, dgu_ms, dgu_n = 0.0, 0, 0.0, 0
    for lay in layers:
        rc, ms, n = binding.layer_profile_read(lay.handle, 0)
        binding.check(rc)
        gu_ms += ms; gu_n += n
        rc, ms, n = binding.layer_profile_read(lay.handle, 2)
        binding.check(rc)
        dgu_ms += ms; dgu_n += n
        binding.layer_profile_kernel(lay.handle, 0, -1)
        binding.layer_profile_kernel(lay.handle, 2, -1)

    # device error flags of the timed steps (a timed-out persistent-decode
    # wait, an activation beyond the fp16 operand range): any raised flag
    # makes the measurement invalid
    flags = 0
    for lay in layers:
        flags |= lay.error()

    fl_p = stage_flops(cfg, Tp, Tp, 0, 1)
    fl_k = stage_flops(cfg, Tk, Tk, Lk, 1)
    by_d = stage_bytes(cfg, Bd, 1, ctx, Bd)
    dec_s = st_ms[2] * 1e-3
    stages = {
        "prefill": {"T": Tp, "ms": round(st_ms[0], 4), "gflop": round(fl_p / 1e9, 2),
                    "tflops": round(fl_p / (st_ms[0] * 1e-3) / 1e12, 1),
                    "frac_mfma": round(fl_p / (st_ms[0] * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4)},
        "prefill_kv": {"T": Tk, "hist": Lk, "ms": round(st_ms[1], 4), "gflop": round(fl_k / 1e9, 2),
                       "tflops": round(fl_k / (st_ms[1] * 1e-3) / 1e12, 1),
                       "frac_mfma": round(fl_k / (st_ms[1] * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4)},
        "decode": {"B": Bd, "ctx": ctx, "us": round(st_ms[2] * 1e3, 2), "mbytes": round(by_d / 1e6, 2),
                   "layer_steps_per_s": round(1.0 / dec_s, 1),
                   "gbps": round(by_d / dec_s / 1e9, 1),
                   "frac_hbm": round(by_d / dec_s / 1e9 / PEAK_HBM_GBS, 4)},
    }
    # the same decode step run back to back over the rotating layer copies
    # (as a stack's layers run): one event pair around the whole run, so no
    # per-launch event or dispatch gap is counted; outside the timed steps
    nb2b = 8 * len(layers)
    torch.cuda.synchronize()
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b0.record(stream)
    for i in range(nb2b):
        k, v = caches[i % len(layers)]
        binding.check(binding.layer_decode(layers[i % len(layers)].handle, xd, pd, cd, ctx, None, Bd, k, v, yd,
                                           ws, ws_bytes, sp))
    b1.record(stream)
    torch.cuda.synchronize()
    b2b_us = b0.elapsed_time(b1) * 1e3 / nb2b
    for lay in layers:
        flags |= lay.error()
    stages["decode"]["back_to_back"] = {"us": round(b2b_us, 2), "layer_steps_per_s": round(1e6 / b2b_us, 1),
                                        "frac_hbm": round(by_d / (b2b_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                                        "calls": nb2b}
    gu_flop = 2.0 * Tp * cfg.hidden * 2 * cfg.ffn
    gu_avg = gu_ms / max(gu_n, 1)
    roofline = {"kernel": "prefill gate/up W4 GEMM (512 x 28672 x 4096, SwiGLU epilogue)",
                "bound": "mfma", "achieved": round(gu_flop / (gu_avg * 1e-3) / 1e12, 1),
                "peak": PEAK_MFMA_TFLOPS, "unit": "TFLOP/s",
                "frac": round(gu_flop / (gu_avg * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4),
                "avg_us": round(gu_avg * 1e3, 2), "launches": gu_n,
                "traffic": traffic("prefill_gate_up"),
                "algorithmic_unit": "2 flop per weight per token (512 tokens x 4096 x 28672 weights)"}
    dgu_avg = dgu_ms / max(dgu_n, 1)
    roofline_decode = {"kernel": "persistent decode kernel (whole decode step, B=1, ctx 2048)",
                       "bound": "hbm", "achieved": round(by_d / (dgu_avg * 1e-3) / 1e9, 1),
                       "peak": PEAK_HBM_GBS, "unit": "GB/s",
                       "frac": round(by_d / (dgu_avg * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                       "avg_us": round(dgu_avg * 1e3, 2), "launches": dgu_n,
                       "traffic": traffic("decode_fused")}
    out = {
        "metric": "decode layer-steps/s (+ prefill/prefill_kv TFLOP/s) of a W4A16 Llama-3-8B-shaped layer",
        "value": round(1.0 / dec_s, 1),
        "unit": "layer-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama8b-shaped W4A16 layer: prefill T=512; prefill_kv T=128 over 1024; "
                               "decode B=1 at ctx 2048",
                   "hidden": cfg.hidden, "heads": f"{cfg.n_heads}/{cfg.n_kv_heads}", "head_dim": cfg.head_dim,
                   "ffn": cfg.ffn, "group": cfg.group_size, "rotation_copies": args.copies},
        "stages": stages,
        "roofline": roofline,
        "roofline_decode": roofline_decode,
        "device_error_flags": flags,
        "decode_wait_timeouts": int(bool(flags & binding.W4_FLAG_WAIT_TIMEOUT)),
    }
    if not args.no_extras:
        out["extras"] = extras(cfg, layers, caches, binding, synth, stream)
    if not args.no_reports:
        out["reports"] = reports(binding, synth, stream)
    if not args.no_formats:
        out["weight_formats"] = formats(binding, synth, stream)
    if not args.no_ceilings:
        out["ceilings"] = ceilings(binding, stream)
    out["paper_context"] = {"table2": PAPER_TABLE2,
                            "note": "Sec. 5.2 Table 2: whole-model W4BF16 decode at 2K context on a Sophgo BM1684X "
                                    "(64 GB/s DDR), bandwidth utilisation 0.78-0.83 of peak; per-layer decode here "
                                    "is reported as a fraction of MI355X HBM (stages.decode.frac_hbm)"}
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle (decode, prefill, prefill_kv; fp64 and fp32)")
        out["cpu_baseline"] = cpu_baseline(cfg, w)
    for lay in layers:
        flags |= lay.error()
    out["device_error_flags"] = flags
    out["decode_wait_timeouts"] = int(bool(flags & binding.W4_FLAG_WAIT_TIMEOUT))
    print(json.dumps(out), flush=True)
    torch.cuda.synchronize()
    for lay in layers:
        lay.close()
    if flags:
        log(f"bench: device error flags raised ({flags}): the measurement is not valid")
        return 3
    return 0


if __name__ == "__main__":
    sys.exit(main())
