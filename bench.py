#!/usr/bin/env python3
"""Benchmark of the Fairy2i widely-linear hot path on one MI355X.

Workload (one "step"): the full LLaMA-2-7B linear stack for one decode token
-- 32 layers x {q, k, v, o: 4096x4096; gate, up: 11008x4096; down: 4096x11008}
as widely-linear T = 2 layers (complex U, W of half size, 2-bit codes, about
1.62 GB packed) -- each projection with its own bf16 activation token, all
decoded by one grouped call (activation-operand kernel and the
block-cooperative fp8 x fp4 MFMA product kernel; every layer is one full-K
work item per row block, so no split-K reduction runs) on one stream.  Weights are seeded synthetic
Student-t(4) draws with LLaMA-like outliers, quantised on the GPU by the
library itself during setup (not timed).

Printed: ONE JSON line.  `value` is packed-weight GB/s of the whole step
(packed code bytes / step time, inputs already resident in HBM).  Extra
objects: `roofline` (the product kernel, timed live with HIP events on its
stream), `cpu_baseline` (the CPU oracle on a bounded sample), `prefill`
(2048-token int8 GEMMs, effective dense int8 TOPS), `stack_T3`, `stack_B*`
(more tokens per layer), `stack_group256` (per-group scales), `per_layer`
(one layer per call over rotated copies), `decoder_block`, `qat_step`
(one training step of a q-shaped layer), `cpu_lut` (the host table-lookup
kernel over the whole stack), `quantizer`.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5000.0        # MI355X dense int8 MFMA, TOPS
FP8_PEAK_TOPS = 5000.0         # MI355X dense fp8 MFMA, TFLOP/s (the e4m3 x e2m1 product is counted against it)
PROFILES = os.path.join(ROOT, "profiles")
PRODUCT_KERNEL_SRC = os.path.join(ROOT, "paper_2512_02901_amd", "csrc", "decode_f4.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


stack_codes = []   # (N, K, tiled codes_U, scales_U, tiled codes_W, scales_W) of the last stack built


def batch_stack(f2, torch, dev, T, B, steps, warmup, seed=3000):
    """The last stack's codes decoding B bf16 tokens per layer; returns
    time_group's (ms per step, prep ms, product ms, reduce ms)."""
    g = torch.Generator(device=dev)
    g.manual_seed(seed + B)
    layers = []
    for (N, K, cu, su, cw, sw) in stack_codes:
        x = torch.randn(B, K, 2, generator=g, device=dev).to(torch.bfloat16)
        y = torch.empty(B, N, dtype=torch.complex64, device=dev)
        layers.append((cu, su, cw, sw, x, None, y))
    grp = f2.WlGroup(layers, T=T, B=B, tiled=True)
    return time_group(grp, torch, steps, warmup, label=f"stack_B{B}_int8")


def batch_stack_fp4(f2, torch, dev, T, fp4_layers, B, steps, warmup, seed=4000):
    """The stack's fp4 tiled codes decoding B <= 4 bf16 tokens per layer."""
    g = torch.Generator(device=dev)
    g.manual_seed(seed + B)
    grp_layers = []
    for (cu4, su, cw4, sw, x1, _, y1) in fp4_layers:
        N, K = y1.shape[1], x1.shape[1]
        x = torch.randn(B, K, 2, generator=g, device=dev).to(torch.bfloat16)
        y = torch.empty(B, N, dtype=torch.complex64, device=dev)
        grp_layers.append((cu4, su, cw4, sw, x, None, y))
    grp = f2.WlGroup(grp_layers, T=T, B=B, layout=f2.LAYOUT_TILED_FP4)
    return time_group(grp, torch, steps, warmup, label=f"stack_B{B}")


def build_stack(f2, synth, torch, dev, T, B=1, seed_base=1000, random_codes=False, with_tiled=False):
    """32 x 7 widely-linear layers with T-stage codes, each with its own
    bf16 activation token.  Returns (group, packed_bytes, algorithmic_bytes,
    layers, tiled_group, fp4_layers): the group decodes the fp4 tiled copies
    of the codes (made once by fairy2i_repack_tiled_fp4, like the
    quantisation, outside any timing); with_tiled also makes the tiled copies
    and a group over them (the int8 matrix-core path); `layers` holds the D3
    codes, `fp4_layers` the fp4 tiled copies."""
    layers, fp4_layers, tiled_layers, packed, algo = [], [], [], 0, 0
    stack_codes.clear()
    for layer in range(32):
        for p in synth.PROJ_ORDER:
            rows, cols = synth.LLAMA2_7B_PROJ[p]
            N, K = rows // 2, cols // 2
            g = torch.Generator(device=dev)
            g.manual_seed(seed_base * 31 + len(layers))
            if random_codes:
                # counter collection only: uniform random 2-bit codes and unit-range scales of the
                # same shapes (the product kernel's memory traffic does not depend on code values)
                cu = torch.randint(0, 256, (T, N, K // 4), dtype=torch.uint8, device=dev, generator=g)
                cw = torch.randint(0, 256, (T, N, K // 4), dtype=torch.uint8, device=dev, generator=g)
                su = torch.rand(T, 2, device=dev, generator=g) + 0.5
                sw = torch.rand(T, 2, device=dev, generator=g) + 0.5
            else:
                A = synth.torch_llama_weight(rows, cols, seed_base + 7 * layer + synth.PROJ_ORDER.index(p), dev)
                U, W = f2.to_widely_linear(A)
                del A
                cu, su = f2.quantize(U, T)
                cw, sw = f2.quantize(W, T)
                del U, W
            x = torch.randn(B, K, 2, generator=g, device=dev).to(torch.bfloat16)
            y = torch.empty(B, N, dtype=torch.complex64, device=dev)
            layers.append((cu, su, cw, sw, x, None, y))
            fp4_layers.append((f2.repack_tiled_fp4(cu), su, f2.repack_tiled_fp4(cw), sw, x, None, y))
            if with_tiled:
                tiled_layers.append((f2.repack_tiled(cu), su, f2.repack_tiled(cw), sw, x, None, y))
                stack_codes.append((N, K) + tiled_layers[-1][:4])
            codes = 2 * T * N * K // 4
            packed += codes
            # codes + bf16 activations + complex64 outputs + scales
            algo += codes + B * K * 2 * 2 + B * N * 8 + 2 * T * 2 * 4
    torch.cuda.synchronize()
    grp = f2.WlGroup(fp4_layers, T=T, B=B, layout=f2.LAYOUT_TILED_FP4)
    grp_tiled = f2.WlGroup(tiled_layers, T=T, B=B, tiled=True) if with_tiled else None
    return grp, packed, algo, layers, grp_tiled, fp4_layers


WARMUP_MIN_S = 0.5   # the GPU clocks take about 0.3 s of back-to-back launches to settle


def warm_up(fn, torch, count, min_s=WARMUP_MIN_S):
    """At least `count` calls and at least `min_s` seconds of calls, in
    batches of 10; returns (calls, seconds)."""
    n, t0 = 0, time.time()
    while n < count or time.time() - t0 < min_s:
        for _ in range(10):
            fn()
        n += 10
        torch.cuda.synchronize()
    return n, time.time() - t0


warmup_log = []      # (label, calls, seconds) of every warm-up phase


def time_group(grp, torch, steps, warmup, label="group"):
    """(ms per step, prep ms, product ms, reduce ms): the step time from a
    loop of plain calls; the per-kernel split from a second loop in which
    the library records events around its three launches.  Warm-up: at least
    `warmup` calls and WARMUP_MIN_S seconds."""
    n, sec = warm_up(grp.run, torch, warmup)
    warmup_log.append((label, n, round(sec, 3)))
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        grp.run()
    t1.record()
    torch.cuda.synchronize()
    step_ms = t0.elapsed_time(t1) / steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for es in ev:
        for e in es:
            e.record()        # create the events before handing them to the library
    torch.cuda.synchronize()
    for es in ev:
        grp.run(events=es)
    torch.cuda.synchronize()
    prep = sum(es[0].elapsed_time(es[1]) for es in ev) / steps
    prod = sum(es[1].elapsed_time(es[2]) for es in ev) / steps
    red = sum(es[2].elapsed_time(es[3]) for es in ev) / steps
    return step_ms, prep, prod, red


def quantizer_bench(f2, synth, torch, dev, T=2, reps=5):
    """Offline preparation wall time (real -> widely-linear, then the T-stage
    quantiser on U and W) for the q and gate shapes, on the GPU."""
    out = {}
    for name in ("q", "gate"):
        rows, cols = synth.LLAMA2_7B_PROJ[name]
        A = synth.torch_llama_weight(rows, cols, 5000 + len(out), dev)
        for _ in range(2):
            U, W = f2.to_widely_linear(A)
            f2.quantize(U, T)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        t_wl = t_q = 0.0
        for _ in range(reps):
            e[0].record()
            U, W = f2.to_widely_linear(A)
            e[1].record()
            f2.quantize(U, T)
            f2.quantize(W, T)
            e[2].record()
            torch.cuda.synchronize()
            t_wl += e[0].elapsed_time(e[1])
            t_q += e[1].elapsed_time(e[2])
        out[name] = {"real_shape": [rows, cols], "T": T, "to_widely_linear_us": round(t_wl / reps * 1e3, 1),
                     "quantize_U_and_W_us": round(t_q / reps * 1e3, 1)}
        del A, U, W
    torch.cuda.empty_cache()
    return out


def grouped_stack_bench(f2, synth, torch, dev, T, G, steps, warmup, seed_base=1000):
    """The decode stack with per-group axis scales (groups of G input columns
    per row, fairy2i_quantize_grouped) on the fp4 path: the same weights as
    the headline stack, the scale arrays read alongside the codes."""
    layers, packed, scale_bytes = [], 0, 0
    for layer in range(32):
        for p in synth.PROJ_ORDER:
            rows, cols = synth.LLAMA2_7B_PROJ[p]
            N, K = rows // 2, cols // 2
            g = torch.Generator(device=dev)
            g.manual_seed(seed_base * 31 + len(layers))
            A = synth.torch_llama_weight(rows, cols, seed_base + 7 * layer + synth.PROJ_ORDER.index(p), dev)
            U, W = f2.to_widely_linear(A)
            del A
            cu, su = f2.quantize_grouped(U, T, G)
            cw, sw = f2.quantize_grouped(W, T, G)
            del U, W
            x = torch.randn(1, K, 2, generator=g, device=dev).to(torch.bfloat16)
            y = torch.empty(1, N, dtype=torch.complex64, device=dev)
            layers.append((f2.repack_tiled_fp4(cu), su, f2.repack_tiled_fp4(cw), sw, x, None, y))
            del cu, cw
            packed += 2 * T * N * K // 4
            scale_bytes += su.numel() * 4 + sw.numel() * 4
    torch.cuda.synchronize()
    grp = f2.WlGroup(layers, T=T, B=1, layout=f2.LAYOUT_TILED_FP4, group_size=G)
    ms, _, prod, _ = time_group(grp, torch, steps, warmup, label=f"stack_group{G}")
    out = {"group_size": G, "ms_per_step": round(ms, 4), "product_us": round(prod * 1e3, 1),
           "packed_bytes": packed, "scale_bytes": scale_bytes,
           "GBs": round(packed / (ms * 1e-3) / 1e9, 1),
           "GBs_codes_and_scales": round((packed + scale_bytes) / (ms * 1e-3) / 1e9, 1)}
    del grp, layers
    torch.cuda.empty_cache()
    return out


def qat_bench(f2, synth, torch, dev, T=2, tokens=4096, reps=10):
    """One quantisation-aware training step of a q-shaped widely-linear layer
    (masters U, W complex 2048 x 2048, T stages) on `tokens` bf16 tokens:
    fake-quant forward of both masters, Y = X U^T + conj(X) W^T, the input
    gradient and both weight gradients, and the straight-through gradients
    of the masters.  The products run in the layer's real form (R from
    W^ once per step, three plain bf16 GEMMs, the weight gradients read off
    G_R); the same step with Gauss's complex GEMMs (planar path, and the
    single-kernel path for the GEMMs alone) is reported next to it.
    Synthetic LLaMA-shaped masters, N(0,1) tokens and output gradients."""
    rows, cols = synth.LLAMA2_7B_PROJ["q"]
    N, K = rows // 2, cols // 2
    A = synth.torch_llama_weight(rows, cols, 6000, dev)
    U, W = f2.to_widely_linear(A)
    del A
    g = torch.Generator(device=dev)
    g.manual_seed(6001)
    X = torch.randn(tokens, K, 2, generator=g, device=dev).to(torch.bfloat16)
    GY = torch.randn(tokens, N, 2, generator=g, device=dev).to(torch.bfloat16)
    Y = torch.empty(tokens, N, dtype=torch.complex64, device=dev)
    GX = torch.empty(tokens, K, dtype=torch.complex64, device=dev)
    GU = torch.empty(N, K, dtype=torch.complex64, device=dev)
    GW = torch.empty(N, K, dtype=torch.complex64, device=dev)
    R = torch.empty(2 * N, 2 * K, dtype=torch.bfloat16, device=dev)
    GR = torch.empty(2 * N, 2 * K, dtype=torch.float32, device=dev)
    Xr, GYr = X.view(tokens, 2 * K), GY.view(tokens, 2 * N)
    Yr, GXr = torch.view_as_real(Y).view(tokens, 2 * N), torch.view_as_real(GX).view(tokens, 2 * K)
    lt_ws = torch.empty(f2.load().fairy2i_gemm_bf16_workspace_bytes(), dtype=torch.uint8, device=dev)
    state = {}
    # the Gauss GEMMs on the planar path (bf16 planes, one batched library GEMM); one workspace for all
    ws = torch.empty(max(f2.cgemm_gauss_planar_workspace_bytes(kk, m, n)
                         for kk, m, n in (([K, K], tokens, N), ([N, N], tokens, K), ([tokens], N, K))),
                     dtype=torch.uint8, device=dev)
    mode = {"planar": True}

    def gemm(segs, m, n, out):
        f2.cgemm_gauss(segs, m, n, out=out, planar=mode["planar"], workspace=ws if mode["planar"] else None)

    def fq():
        state["u"] = f2.qat_fake_quant(U, T)
        state["w"] = f2.qat_fake_quant(W, T)

    def ste():
        f2.qat_ste_backward(state["u"][1], state["u"][2], GU)
        f2.qat_ste_backward(state["w"][1], state["w"][2], GW)

    # real form: the quantiser's codes and scales are all the step needs (R is formed from them directly, W^
    # is not written); the straight-through backward takes the same codes and scales
    def r_quant():
        state["u"] = (None, *f2.quantize(U, T))
        state["w"] = (None, *f2.quantize(W, T))

    def r_fwd():
        f2.wl_realify_codes(state["u"][1], state["u"][2], state["w"][1], state["w"][2], out=R)
        f2.gemm_bf16(Xr, R, transB=True, out=Yr, workspace=lt_ws)

    def r_bwd_x():
        f2.gemm_bf16(GYr, R, out=GXr, workspace=lt_ws)

    def r_bwd_w():
        f2.gemm_bf16(GYr, Xr, transA=True, out=GR, workspace=lt_ws)
        f2.wl_unrealify_grad(GR, N, K, out=(GU, GW))

    # Gauss's complex GEMMs
    def g_fwd():
        gemm([(X, 0, 0, state["u"][0], 0, 0, K), (X, 0, 1, state["w"][0], 0, 0, K)], tokens, N, Y)

    def g_bwd_x():
        gemm([(GY, 0, 0, state["u"][0], 1, 1, N), (GY, 0, 1, state["w"][0], 1, 0, N)], tokens, K, GX)

    def g_bwd_w():
        gemm([(GY, 1, 0, X, 1, 1, tokens)], N, K, GU)
        gemm([(GY, 1, 0, X, 1, 0, tokens)], N, K, GW)

    def timed(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    # the library's algorithm for each real-form GEMM chosen once by timing its candidates (a setup step)
    r_quant()
    f2.wl_realify_codes(state["u"][1], state["u"][2], state["w"][1], state["w"][2], out=R)
    f2.gemm_bf16(Xr, R, transB=True, out=Yr, workspace=lt_ws, tune=True)
    f2.gemm_bf16(GYr, R, out=GXr, workspace=lt_ws, tune=True)
    f2.gemm_bf16(GYr, Xr, transA=True, out=GR, workspace=lt_ws, tune=True)

    def run(phases):
        phases[0][1]()
        for _, fn in phases:
            fn()
        warm_up(lambda: [fn() for _, fn in phases], torch, 3)
        res = {}
        for name, fn in phases:
            res[name + "_us"] = round(timed(fn), 1)
        res["step_us"] = round(sum(res.values()), 1)
        return res

    out = {"workload": f"one QAT step of a q-shaped layer (complex {N}x{K}, T={T}), {tokens} bf16 tokens",
           "gemm_path": "real form: the masters quantised (codes and scales), R (bf16 2N x 2K) formed from them "
                        "each step, Y = X R^T, G_X = G_Y R, G_R = G_Y^T X as plain bf16 hipBLASLt GEMMs (algorithms "
                        "tuned once per shape), G_U and G_W read off G_R"}
    out.update(run([("fake_quant", r_quant), ("forward_gemm", r_fwd), ("input_grad_gemm", r_bwd_x),
                    ("weight_grad_gemms", r_bwd_w), ("ste_backward", ste)]))
    # per GEMM phase (M N K = tokens x 2048 x 2048): the real form executes one real product of
    # 2 M (2N) (2K) = 8 M N K flops; the layer's two complex products are 16 M N K flops counted as 8 per
    # complex MAC ("effective"); Gauss executes 3 real products of 2 M N (2K) = 12 M N K flops
    macs = {"forward_gemm": tokens * N * K, "input_grad_gemm": tokens * N * K, "weight_grad_gemms": N * K * tokens}
    gemm_us = sum(out[k + "_us"] for k in macs)
    out["gemm_exec_TFLOPs"] = round(8 * sum(macs.values()) / gemm_us / 1e6, 1)
    out["gemm_effective_TFLOPs"] = round(16 * sum(macs.values()) / gemm_us / 1e6, 1)
    out["gemm_frac_bf16_peak"] = round(out["gemm_exec_TFLOPs"] / 2500.0, 4)
    gauss = run([("fake_quant", fq), ("forward_gemm", g_fwd), ("input_grad_gemm", g_bwd_x),
                 ("weight_grad_gemms", g_bwd_w), ("ste_backward", ste)])
    g_us = sum(gauss[k + "_us"] for k in macs)
    gauss["gemm_exec_TFLOPs"] = round(12 * sum(macs.values()) / g_us / 1e6, 1)
    gauss["gemm_effective_TFLOPs"] = round(16 * sum(macs.values()) / g_us / 1e6, 1)
    out["gauss_planar"] = gauss
    # the same three GEMM phases on the single-kernel Gauss path, for comparison
    mode["planar"] = False
    warm_up(lambda: [fn() for fn in (g_fwd, g_bwd_x, g_bwd_w)], torch, 3)
    out["gauss_single_kernel_gemms_us"] = round(sum(timed(fn) for fn in (g_fwd, g_bwd_x, g_bwd_w)), 1)
    del U, W, X, GY, Y, GX, GU, GW, R, GR, state, ws, lt_ws
    torch.cuda.empty_cache()
    return out


def cpu_lut_bench(f2, torch, layers, T, passes=3):
    """The CPU table-lookup kernel over the whole stack on the host cores:
    the stack's canonical codes and scales copied to host memory, each
    layer's bf16 token quantised to int8 (fairy2i_quantize_act_int8), then
    whole passes over the 224 layers, one library call per layer."""
    import numpy as np
    host = []
    for (cu, su, cw, sw, x, _, y) in layers:
        q, f = f2.quantize_act_int8(x)
        host.append((cu.cpu().numpy(), su.cpu().numpy(), cw.cpu().numpy(), sw.cpu().numpy(),
                     q.cpu().numpy(), f.cpu().numpy()))
    kmax = max(h[0].shape[2] * 4 for h in host)
    ws = np.empty(f2.cpu_lut_workspace_bytes(T, kmax, 1), dtype=np.uint8)
    packed = sum(h[0].nbytes + h[2].nbytes for h in host)

    def one_pass():
        for (cu, su, cw, sw, q, f) in host:
            f2.cpu_lut_wl_matmul(cu, su, cw, sw, q, f, workspace=ws)

    one_pass()
    t0 = time.perf_counter()
    for _ in range(passes):
        one_pass()
    sec = (time.perf_counter() - t0) / passes
    del host
    return {"workload": f"LLaMA-2-7B linear stack, {len(layers)} layers, T={T}, one int8 token per layer, "
                        "host cores", "ms_per_step": round(sec * 1e3, 2), "GBs": round(packed / sec / 1e9, 2),
            "threads": len(os.sched_getaffinity(0)), "passes": passes,
            "kernel": "fairy2i_cpu_lut_wl_matmul (8-bit index of four codes, int16 tables, SSE2)"}


def code_hash(path):
    """First 16 hex digits of the sha256 of a C++/HIP source with its
    comments and white space removed: edits to comments leave it unchanged,
    edits to code do not."""
    import re
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()[:16]


def traffic_record():
    """HBM bytes per launch of the product kernel from committed rocprofv3
    --pmc summaries, or None when absent or when the kernel's code changed
    since the counters were taken."""
    path = os.path.join(PROFILES, "dec_coop_f4_stack_T2_bf16_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    if rec.get("kernel_code_sha256_16") != code_hash(PRODUCT_KERNEL_SRC):
        return None
    try:
        return float(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def mfma_probe(f2, torch, dev, kind, iters, reps=10):
    """Sustained rate of one MFMA instruction on this GPU (back-to-back
    independent MFMAs, four waves per SIMD, no memory traffic), in TOPS:
    the measured counterpart of the nominal peak, at the clock the chip
    holds under matrix-core load."""
    blocks = 4 * torch.cuda.get_device_properties(dev).multi_processor_count  # 16 waves per CU
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
    ops = f2.probe_mfma(kind, blocks, iters, sink)
    warm_up(lambda: f2.probe_mfma(kind, blocks, iters, sink), torch, 3, min_s=0.3)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        f2.probe_mfma(kind, blocks, iters, sink)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    return {"tops": round(ops / (us * 1e-6) / 1e12, 1), "us_per_launch": round(us, 1), "blocks": blocks,
            "iters": iters}


def prefill_bench(f2, synth, torch, dev, T=2, tokens=2048, reps=20):
    out = {}
    for name, (rows, cols) in (("q", synth.LLAMA2_7B_PROJ["q"]), ("gate", synth.LLAMA2_7B_PROJ["gate"])):
        N, K = rows // 2, cols // 2
        A = synth.torch_llama_weight(rows, cols, 4000 + len(out), dev)
        U, W = f2.to_widely_linear(A)
        del A
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        del U, W
        g = torch.Generator(device=dev)
        g.manual_seed(4100 + len(out))
        x = torch.randn(tokens, K, dtype=torch.complex64, device=dev, generator=g)
        q, xs = f2.quantize_act_int8(x)
        y = torch.empty(tokens, N, dtype=torch.complex64, device=dev)
        wsb = f2.wl_matmul_workspace_bytes(N, K, T, tokens, f2.ACT_I8)
        ws = torch.empty(max(1, wsb), dtype=torch.uint8, device=dev)
        # warm-up until the clocks are steady (at least 0.3 s of launches)
        t_w = time.time()
        while True:
            for _ in range(20):
                f2.wl_matmul(cu, su, cw, sw, q, xs, out=y, workspace=ws)
            torch.cuda.synchronize()
            if time.time() - t_w >= 0.3:
                break
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f2.wl_matmul(cu, su, cw, sw, q, xs, out=y, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        ops = 2 * (4 * T * N) * K * (2 * tokens)      # dense int8 ops of the (4TN) x K x (2 tokens) GEMM
        tops = ops / (ms * 1e-3) / 1e12
        out[name] = {"N": N, "K": K, "tokens": tokens, "us": round(ms * 1e3, 2), "tops": round(tops, 1),
                     "frac_int8_peak": round(tops / INT8_PEAK_TOPS, 4)}
        del cu, cw, q, y, ws
        # context, not the product: the same dense int8 op count as one plain library GEMM
        # ((2 tokens) x K x (4TN), torch._int_mm), timed the same way
        out[name]["library_int8_gemm"] = library_int8_gemm(torch, dev, 2 * tokens, K, 4 * T * N, reps)
    probe = mfma_probe(f2, torch, dev, f2.PROBE_MFMA_I8, 4096)
    probe["frac_nominal_peak"] = round(probe["tops"] / INT8_PEAK_TOPS, 4)
    probe["instruction"] = "v_mfma_i32_16x16x64_i8 (the GEMM's)"
    out["mfma_i8_probe"] = probe
    p32 = mfma_probe(f2, torch, dev, f2.PROBE_MFMA_I8_32X32, 4096)
    p32["frac_nominal_peak"] = round(p32["tops"] / INT8_PEAK_TOPS, 4)
    p32["instruction"] = "v_mfma_i32_32x32x32_i8"
    out["mfma_i8_32x32_probe"] = p32
    for name in ("q", "gate"):
        out[name]["frac_measured_i8_peak"] = round(out[name]["tops"] / probe["tops"], 4)
    return out


def library_int8_gemm(torch, dev, M, K, N, reps):
    """A plain int8 x int8 -> int32 GEMM of the given shape through torch's
    library path (hipBLASLt on ROCm): TOPS and fraction of the int8 peak."""
    g = torch.Generator(device=dev)
    g.manual_seed(4200 + M + N)
    a = torch.randint(-127, 128, (M, K), dtype=torch.int8, device=dev, generator=g)
    b = torch.randint(-127, 128, (K, N), dtype=torch.int8, device=dev, generator=g)
    try:
        t_w = time.time()
        while time.time() - t_w < 0.3:
            for _ in range(5):
                torch._int_mm(a, b)
            torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch._int_mm(a, b)
        e1.record()
        torch.cuda.synchronize()
    except RuntimeError as ex:  # no int8 GEMM in this torch build
        return {"error": str(ex)[:120]}
    ms = e0.elapsed_time(e1) / reps
    tops = 2 * M * K * N / (ms * 1e-3) / 1e12
    return {"shape_MxKxN": [M, K, N], "us": round(ms * 1e3, 2), "tops": round(tops, 1),
            "frac_int8_peak": round(tops / INT8_PEAK_TOPS, 4)}


def cpu_baseline(f2, synth, torch, dev, layers, T, budget_s=12.0):
    """The CPU oracle on a bounded sample: the stack's first q-projection,
    from packed codes to y (unpack + dequantise + complex128 product),
    repeated until ~budget_s; next to it the dense float64 product alone
    (the dequantised matrices applied to the token), all with the BLAS
    thread count set to the cores this process may run on."""
    import numpy as np
    import oracle
    cores = len(os.sched_getaffinity(0))
    blas = "unknown"
    limiter = None
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        info = [d for d in threadpool_info() if d.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
        limiter = threadpool_limits(limits=cores, user_api="blas")
    except Exception:
        pass
    cu, su, cw, sw, x, _, _ = layers[0]
    cu_p, cw_p = cu.cpu().numpy(), cw.cpu().numpy()
    K = 4 * cu.shape[2]
    su_h, sw_h = su.cpu().numpy(), sw.cpu().numpy()
    xb = x.float().cpu().numpy()
    xh = xb[..., 0].astype(np.complex128) + 1j * xb[..., 1]
    packed = 2 * T * cu.shape[1] * cu.shape[2]
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.wl_matmul(oracle.unpack(cu_p, K), su_h, oracle.unpack(cw_p, K), sw_h, xh)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 400:
            break
    Uh = oracle.dequantize(oracle.unpack(cu_p, K), su_h)
    Wh = oracle.dequantize(oracle.unpack(cw_p, K), sw_h)
    dreps, t1 = 0, time.perf_counter()
    while True:
        xv = xh.reshape(-1)
        _ = Uh @ xv + Wh @ np.conj(xv)
        dreps += 1
        del_ = time.perf_counter() - t1
        if del_ >= 2.0 or dreps >= 2000:
            break
    if limiter is not None:
        limiter.restore_original_limits()
    gbs = packed * reps / el / 1e9
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "blas": blas,
            "sample": f"{reps} oracle products (unpack + dequantise + complex128 product) of one 4096x4096 "
                      f"q-projection (complex 2048x2048, T={T}, {packed} packed bytes, bf16 token) in "
                      f"{el:.1f} s; unit as the metric",
            "oracle_us_per_layer": round(el / reps * 1e6, 1),
            "dense_f64_matvec_us": round(del_ / dreps * 1e6, 1)}


def per_layer_bench(f2, synth, torch, dev, T=2, min_bytes=512e6, reps=5):
    """One layer per call at bs = 1: q (4096x4096), gate (11008x4096) and down
    (4096x11008), each call on a different copy of the codes (at least
    min_bytes of copies, so no call finds its codes in the 256 MB
    last-level cache), launched from a HIP graph so host launch overhead does
    not count.  Two routes: a one-layer grouped call over fp4 tiled codes, and
    fairy2i_wl_matmul on the canonical codes."""
    out = {}
    for name in ("q", "gate", "down"):
        rows, cols = synth.LLAMA2_7B_PROJ[name]
        N, K = rows // 2, cols // 2
        A = synth.torch_llama_weight(rows, cols, 6000 + len(out), dev)
        U, W = f2.to_widely_linear(A)
        del A
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        del U, W
        nbytes = 2 * T * N * K // 4
        R = max(2, int(-(-min_bytes // nbytes)))
        g = torch.Generator(device=dev)
        g.manual_seed(6100 + len(out))
        x = torch.randn(1, K, 2, generator=g, device=dev).to(torch.bfloat16)
        y = torch.empty(1, N, dtype=torch.complex64, device=dev)
        res = {"N": N, "K": K, "T": T, "packed_bytes": nbytes, "copies": R,
               "rotated_MB": round(R * nbytes / 1e6, 1)}
        cu4, cw4 = f2.repack_tiled_fp4(cu), f2.repack_tiled_fp4(cw)
        groups = [f2.WlGroup([(cu4.clone(), su, cw4.clone(), sw, x, None, y)], T=T, B=1,
                             layout=f2.LAYOUT_TILED_FP4) for _ in range(R)]
        del cu4, cw4
        d3 = [(cu.clone(), cw.clone()) for _ in range(R)]
        ws = torch.empty(max(1, f2.wl_matmul_workspace_bytes(N, K, T, 1, f2.ACT_BF16)), dtype=torch.uint8,
                         device=dev)
        for label, calls in (("fp4_group", [grp.run for grp in groups]),
                             ("d3_wl_matmul", [(lambda c=c: f2.wl_matmul(c[0], su, c[1], sw, x, out=y, workspace=ws))
                                               for c in d3])):
            for c in calls:
                c()
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for c in calls:
                    c()
            warm_up(graph.replay, torch, 3, min_s=0.3)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                graph.replay()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (reps * R)
            res[f"{label}_us"] = round(us, 2)
            res[f"{label}_GBs"] = round(nbytes / (us * 1e-6) / 1e9, 1)
            del graph
        res["us_at_hbm_peak"] = round(nbytes / (HBM_PEAK_GBS * 1e9) * 1e6, 2)
        out[name] = res
        del groups, d3, cu, cw
        torch.cuda.empty_cache()
    return out


def block_bench(f2, synth, torch, dev, T=2, ctx=2048, reps=50):
    """One decode token through one widely-linear LLaMA-2-7B decoder block
    (fairy2i_block_decode: n = 2048 complex, 32 heads, FFN 5504 complex,
    T = 2 seeded synthetic weights) attending over `ctx` cached positions:
    time per token from plain calls and from a HIP graph of the calls, and
    the bytes a token reads (packed codes of the seven projections and the
    key/value caches)."""
    n, f, H = 2048, 5504, 32
    shapes = {"q": (n, n), "k": (n, n), "v": (n, n), "o": (n, n), "gate": (f, n), "up": (f, n), "down": (n, f)}
    layers, code_bytes = {}, 0
    for i, (name, (N, K)) in enumerate(shapes.items()):
        A = synth.torch_llama_weight(2 * N, 2 * K, 9000 + i, dev)
        U, W = f2.to_widely_linear(A)
        del A
        cu, su = f2.quantize(U, T)
        cw, sw = f2.quantize(W, T)
        del U, W
        layers[name] = (f2.repack_tiled_fp4(cu), su, f2.repack_tiled_fp4(cw), sw)
        code_bytes += 2 * T * N * K // 4
    g = torch.Generator(device=dev)
    g.manual_seed(9100)
    norm_a = 1.0 + 0.1 * torch.randn(2 * n, generator=g, device=dev)
    norm_m = 1.0 + 0.1 * torch.randn(2 * n, generator=g, device=dev)
    blk = f2.WlBlock(layers, norm_a, norm_m, n=n, n_ff=f, n_heads=H, T=T, max_ctx=ctx)
    kc = torch.randn(H, ctx, n // H, generator=g, device=dev, dtype=torch.complex64)
    vc = torch.randn(H, ctx, n // H, generator=g, device=dev, dtype=torch.complex64)
    x = torch.randn(1, n, generator=g, device=dev, dtype=torch.complex64)
    y = torch.empty(1, n, dtype=torch.complex64, device=dev)
    pos = ctx - 1

    def call():
        blk.decode(x, kc, vc, pos, out=y)
    warm_up(call, torch, 10, min_s=0.3)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(10):
            call()
    warm_up(graph.replay, torch, 3, min_s=0.3)
    e0.record()
    for _ in range(reps // 10):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    us_graph = e0.elapsed_time(e1) * 1e3 / (10 * (reps // 10))
    kv_bytes = 2 * H * ctx * (n // H) * 8
    return {"workload": f"one decode token, LLaMA-2-7B block shape (4096 hidden, 32 heads, 11008 FFN), T={T}, "
                        f"context {ctx}", "us_per_token": round(us, 2), "us_per_token_graph": round(us_graph, 2),
            "code_bytes": code_bytes, "kv_cache_bytes": kv_bytes,
            "GBs_graph": round((code_bytes + kv_bytes) / (us_graph * 1e-6) / 1e9, 1)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="skip prefill, T=3 and D3-layout measurements")
    ap.add_argument("--random-codes", action="store_true",
                    help="random codes instead of quantised weights (for hardware-counter runs only; "
                         "the JSON line then says so in `data`)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only run the two 2048-token prefill GEMMs (for hardware-counter runs)")
    ap.add_argument("--qat-only", action="store_true",
                    help="only run the QAT training-step leg (for profiler runs)")
    ap.add_argument("--grouped-only", action="store_true",
                    help="only run the per-group-scale stack leg, G = 256 (for profiler runs)")
    ap.add_argument("--block-only", action="store_true",
                    help="only run the decoder-block leg (for profiler runs)")
    ap.add_argument("--quantizer-only", action="store_true",
                    help="only run the offline quantisation leg, q and gate shapes (for profiler runs)")
    ap.add_argument("--batch-only", type=int, default=0, metavar="B",
                    help="only run the fp4 stack with B tokens per layer, 2..16 (for profiler runs)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run 5 plain 256 MiB device copies (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(a layer would shard by output rows, with one all-gather of y per layer)",
              file=sys.stderr)
        sys.exit(2)

    if args.batch_only and not 2 <= args.batch_only <= 16:
        print("--batch-only takes 2..16 tokens per layer", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel(), "copies": 5}), flush=True)
        return
    import paper_2512_02901_amd as f2
    import synth

    dev = torch.device("cuda:0")
    f2.load()
    if args.prefill_only:
        print(json.dumps({"prefill": prefill_bench(f2, synth, torch, dev)}), flush=True)
        return
    if args.qat_only:
        print(json.dumps({"qat_step": qat_bench(f2, synth, torch, dev)}), flush=True)
        return
    if args.quantizer_only:
        print(json.dumps({"quantizer": quantizer_bench(f2, synth, torch, dev)}), flush=True)
        return
    if args.block_only:
        print(json.dumps({"decoder_block": block_bench(f2, synth, torch, dev)}), flush=True)
        return
    if args.grouped_only:
        print(json.dumps({"stack_group256": grouped_stack_bench(f2, synth, torch, dev, 2, 256, args.steps,
                                                                args.warmup)}), flush=True)
        return
    T = 2
    t0 = time.time()
    if args.batch_only:
        _, packed, _, _, _, fp4_layers = build_stack(f2, synth, torch, dev, T, random_codes=args.random_codes)
        msb, _, prodb, _ = batch_stack_fp4(f2, torch, dev, T, fp4_layers, args.batch_only, args.steps, args.warmup)
        print(json.dumps({f"stack_B{args.batch_only}": {
            "ms_per_step": round(msb, 4), "GBs": round(packed / (msb * 1e-3) / 1e9, 1),
            "product_us": round(prodb * 1e3, 1), "random_codes": args.random_codes}}), flush=True)
        return
    grp, packed, algo, layers, grp_tiled, fp4_layers = build_stack(f2, synth, torch, dev, T,
                                                                   random_codes=args.random_codes,
                                                                   with_tiled=not args.no_extras)
    log(f"stack T={T}: {len(layers)} layers, {packed / 1e9:.3f} GB packed, setup {time.time() - t0:.1f} s")

    ms, prep_ms, prod_ms, red_ms = time_group(grp, torch, args.steps, args.warmup, label="headline")
    gbs = packed / (ms * 1e-3) / 1e9
    log(f"step {ms * 1e3:.1f} us: prep {prep_ms * 1e3:.1f} us, product {prod_ms * 1e3:.1f} us, "
        f"reduce {red_ms * 1e3:.1f} us -> {gbs:.1f} GB/s packed")

    achieved = algo / (prod_ms * 1e-3) / 1e9
    traffic = traffic_record()
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                # calibrated rocprofv3 FETCH_SIZE + WRITE_SIZE bytes per launch (null when the
                # committed counters were taken for another kernel source)
                "traffic": None if traffic is None else int(traffic),
                "traffic_over_algorithmic": None if traffic is None else round(traffic / algo, 3),
                "kernel": "dec_coop_f4_kernel<T=2> (fp8 x fp4 MFMA product over fp4-tiled codes, four waves "
                          "per block sharing one activation ring; one launch per step)",
                "algorithmic_bytes_per_launch": algo, "avg_launch_us": round(prod_ms * 1e3, 2)}

    result = {
        "metric": "packed-weight GB/s (%HBM peak) at bs=1; int8-MFMA TOPS at 2048 tokens",
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 activations as two e4m3 digits per value, fp8 x fp4 MFMA, float32 accumulation",
        "data": ("synthetic: seeded uniform random 2-bit codes (counter run), N(0,1) bf16 tokens"
                 if args.random_codes else
                 "synthetic: seeded Student-t(4) weights with 1% outlier input channels, N(0,1) bf16 tokens"),
        "config": {"workload": "LLaMA-2-7B linear stack, 32 layers x 7 projections, widely-linear T=2, "
                               "one decode token (bs=1) per projection, bf16 activations",
                   "layers": len(layers), "T": T, "batch": 1, "packed_bytes": packed,
                   "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                   "step_breakdown_us": {"prep": round(prep_ms * 1e3, 1), "product": round(prod_ms * 1e3, 1),
                                         "reduce": round(red_ms * 1e3, 1)}},
        "roofline": roofline,
    }
    if not args.no_extras:
        # the same stack on the int8 matrix cores over the tiled copies
        ms_t, _, prod_t, _ = time_group(grp_tiled, torch, args.steps, args.warmup, label="stack_tiled_int8")
        result["stack_tiled_int8"] = {"ms_per_step": round(ms_t, 4), "GBs": round(packed / (ms_t * 1e-3) / 1e9, 1),
                                      "product_us": round(prod_t * 1e3, 1)}
        del grp_tiled
        # 2, 4, 8 and 16 tokens per layer on the fp4 path (one two-band tile of 2 tokens, one, two or
        # four one-band tiles of 4)
        for Bb in (2, 4, 8, 16):
            msb, _, prodb, _ = batch_stack_fp4(f2, torch, dev, T, fp4_layers, Bb, args.steps, args.warmup)
            result[f"stack_B{Bb}"] = {"ms_per_step": round(msb, 4), "GBs": round(packed / (msb * 1e-3) / 1e9, 1),
                                      "product_us": round(prodb * 1e3, 1)}
        # 4, 8 and 16 tokens per layer on the int8 matrix cores (tiled copies)
        for Bb in (4, 8, 16):
            msb, _, prodb, _ = batch_stack(f2, torch, dev, T, Bb, max(10, args.steps // 2), args.warmup)
            result[f"stack_B{Bb}_int8"] = {"ms_per_step": round(msb, 4),
                                           "GBs": round(packed / (msb * 1e-3) / 1e9, 1),
                                           "product_us": round(prodb * 1e3, 1)}
        # the same stack decoded straight from the canonical D3 codes
        grp_d3 = f2.WlGroup(layers, T=T, B=1)
        ms_d3, _, prod_d3, _ = time_group(grp_d3, torch, args.steps, args.warmup, label="stack_d3_layout")
        result["stack_d3_layout"] = {"ms_per_step": round(ms_d3, 4), "GBs": round(packed / (ms_d3 * 1e-3) / 1e9, 1),
                                     "product_us": round(prod_d3 * 1e3, 1)}
        del grp_d3
        result["cpu_lut"] = cpu_lut_bench(f2, torch, layers, T)
    del grp, layers, fp4_layers
    stack_codes.clear()
    torch.cuda.empty_cache()

    if not args.no_extras:
        grp3, packed3, _, layers3, _, f3 = build_stack(f2, synth, torch, dev, 3, seed_base=2000)
        ms3, _, _, _ = time_group(grp3, torch, max(5, args.steps // 2), args.warmup, label="stack_T3")
        result["stack_T3"] = {"ms_per_step": round(ms3, 4), "packed_bytes": packed3,
                              "GBs": round(packed3 / (ms3 * 1e-3) / 1e9, 1),
                              "time_ratio_T3_over_T2": round(ms3 / ms, 3)}
        del grp3, layers3, f3
        torch.cuda.empty_cache()
        result["stack_group256"] = grouped_stack_bench(f2, synth, torch, dev, T, 256, args.steps, args.warmup)
        result["stack_group256"]["time_ratio_over_per_tensor"] = round(result["stack_group256"]["ms_per_step"] / ms, 3)
        result["per_layer"] = per_layer_bench(f2, synth, torch, dev, T)
        result["decoder_block"] = block_bench(f2, synth, torch, dev, T)
        result["qat_step"] = qat_bench(f2, synth, torch, dev, T)
        pf = prefill_bench(f2, synth, torch, dev)
        g = pf["gate"]
        # headline: the 11008x4096 (gate/up) shape; half of the dense MACs multiply structural zeros
        result["prefill"] = {"tops": g["tops"], "frac_int8_peak": g["frac_int8_peak"], "useful_frac": 0.5,
                             "useful_tops": round(g["tops"] * 0.5, 1), "us": g["us"],
                             "workload": "2048 tokens x gate/up shape (real 11008x4096, complex 5504x2048), "
                                         "T=2, int8 activations",
                             "frac_measured_i8_peak": g["frac_measured_i8_peak"],
                             "mfma_i8_probe": pf["mfma_i8_probe"], "mfma_i8_32x32_probe": pf["mfma_i8_32x32_probe"],
                             "q": pf["q"], "gate": pf["gate"]}
        probe = mfma_probe(f2, torch, dev, f2.PROBE_MFMA_F8F4, 4096)
        probe["frac_nominal_peak"] = round(probe["tops"] / FP8_PEAK_TOPS, 4)
        result["mfma_f8f4_probe"] = probe
        result["quantizer"] = quantizer_bench(f2, synth, torch, dev)

    if not args.no_cpu_baseline:
        # a fresh single-layer copy of the stack's first projection
        g1, _, _, l1 = build_stack_first(f2, synth, torch, dev, T)
        result["cpu_baseline"] = cpu_baseline(f2, synth, torch, dev, l1, T)
    result["warmup_phases"] = [{"label": lab, "calls": n, "s": sec} for (lab, n, sec) in warmup_log]
    print(json.dumps(result), flush=True)


def build_stack_first(f2, synth, torch, dev, T):
    """Only the first projection of the stack (same seeds), for the CPU leg."""
    rows, cols = synth.LLAMA2_7B_PROJ["q"]
    N, K = rows // 2, cols // 2
    A = synth.torch_llama_weight(rows, cols, 1000, dev)
    U, W = f2.to_widely_linear(A)
    cu, su = f2.quantize(U, T)
    cw, sw = f2.quantize(W, T)
    g = torch.Generator(device=dev)
    g.manual_seed(1000 * 31)
    x = torch.randn(1, K, 2, generator=g, device=dev).to(torch.bfloat16)
    y = torch.empty(1, N, dtype=torch.complex64, device=dev)
    torch.cuda.synchronize()
    return None, 0, 0, [(cu, su, cw, sw, x, None, y)]


if __name__ == "__main__":
    main()
