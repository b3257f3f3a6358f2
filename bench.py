"""Benchmark of the W4A8 linear layer on one MI355X.

A step is one full pass of the hot path, y = dequant(quant8(x) . int4(W)^T):
activation quantize, packed-int4 weight stream and int8 MFMA contraction,
dequant epilogue, bf16 out, with every input already resident in HBM.

Primary line: draft-block verification of the fused gate+up projection,
M=16 tokens, K=4096, N=24576 (bandwidth bound, reported in GB/s of
algorithmic bytes: packed weights + weight scales + bf16 x + bf16 y).
Sixteen copies of the packed weight (805 MB, three times the 256 MB
Infinity Cache) are cycled so every step streams its weights from HBM.

Secondary object: streaming prefill of new-frame tokens through the fused
QKV projection, M=1024, K=4096, N=6144 (MFMA bound, reported in INT8 TOPS,
2*M*N*K ops per step), cycling 24 weight copies.

Sweep object: the down projection at verification sizes (M = 1, 4, 16,
K=12288, N=4096, GB/s) and one decoder layer's four linears with group-128
fp16 scales (M = 1, 16, 256, 2048; GB/s and TOPS per layer).

Timing: W untimed warmup steps, then exactly K steps between HIP events on
the launch stream, bracketed by device synchronization.  The dominant
kernel's average duration for the roofline is timed the same way over its
own back-to-back launches.  The CPU baseline times the oracle (test
infrastructure, plain scalar C) on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4A8 linear: HBM GB/s at M=16, INT8 TOPS at M=1024 (% of roofline)"
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0      # MI355X dense INT8 MFMA (5.0 POPS)
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA (2.5 PFLOP/s)
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["device.h", "kernels.h", "gemm_smallm.hip", "largem_kernel.h", "gemm_largem.hip",
                  "gemm_largem_group.hip", "quantize.hip", "api.cpp"]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_12932_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def file_hash(name: str) -> str:
    """Short hash of one kernel source file."""
    with open(os.path.join(ROOT, "paper_2608_12932_amd", "csrc", name), "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def profile_summary(name: str):
    """The key: value lines of a committed rocprofv3 summary
    (profiles/<name>.txt), or None if there is none or the kernel sources
    changed since it was taken."""
    path = os.path.join(PROFILES, f"{name}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_hash") != kernel_source_hash():
        return None
    return vals


def counter_traffic(name: str):
    """HBM bytes per dispatch of the profiled kernel (FETCH_SIZE + WRITE_SIZE,
    calibrated), or None."""
    vals = profile_summary(name)
    try:
        return float(vals["hbm_bytes_per_dispatch"]) if vals else None
    except (KeyError, ValueError):
        return None


def trace_roofline(name: str, work: float, peak: float, unit_scale: float):
    """The dominant kernel's roofline from the committed kernel trace: its
    average duration over the profiled run and the fraction of `peak` that
    `work` (bytes or ops per launch) in that time gives.  unit_scale turns
    work per second into the peak's unit."""
    vals = profile_summary(name)
    if not vals or "avg_us" not in vals:
        return None
    us = float(vals["avg_us"])
    achieved = work / (us * 1e-6) / unit_scale
    return {"file": f"profiles/{name}.txt", "kernel": vals.get("kernel"), "avg_us": us,
            "achieved": round(achieved, 2), "frac": round(achieved / peak, 4)}


class DirectCall:
    """w4a8_linear with every argument resolved once (device pointers and
    sizes), so a step costs one C call: the binding's per-call tensor checks
    would otherwise dominate a ~10 us kernel."""

    def __init__(self, x, wps, w_scale, N, y, x_scale=None, workspace=None, out_kind=0, scale_mode=0,
                 entry="w4a8_linear"):
        import ctypes
        import paper_2608_12932_amd as w

        self.L = w.lib()
        self.fn = getattr(self.L, entry)
        self.entry = entry
        self.M, self.K = x.shape
        self.in_kind = w.IN_I8 if x.dtype.is_floating_point is False else w.IN_BF16
        self.x = x.data_ptr()
        self.xs = None if x_scale is None else x_scale.data_ptr()
        self.wps = [t.data_ptr() for t in wps]
        self.ws = w_scale.data_ptr()
        self.N = N
        self.y = y.data_ptr()
        self.out_kind = out_kind
        self.scale_mode = scale_mode
        need = int(getattr(self.L, entry + "_workspace_bytes")(self.M, N, self.K, scale_mode, self.in_kind))
        self.wk = None
        self.wk_bytes = 0
        buf = None
        if need:
            buf = workspace.get(need)
            self.wk, self.wk_bytes = buf.data_ptr(), buf.numel()
        self.keep = (x, wps, w_scale, y, x_scale, buf)
        self.c_size = ctypes.c_size_t

    def __call__(self, i, stream):
        rc = self.fn(self.x, self.in_kind, self.xs, self.M, self.K, self.wps[i % len(self.wps)],
                     self.ws, self.scale_mode, self.N, self.y, self.out_kind,
                     self.wk, self.wk_bytes, stream)
        if rc:
            raise RuntimeError(f"{self.entry} failed: {rc}")


def graph_ms(call, steps: int, reps: int = 20):
    """ms per call of call(i, stream) captured reps times into one graph
    (the calls cycle their weight copies as in eager timing) and replayed."""
    import torch

    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        call(0, cap.cuda_stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=cap):
            for i in range(reps):
                call(i, cap.cuda_stream)
    torch.cuda.current_stream().wait_stream(cap)
    ms = time_steps(lambda i: g.replay(), max(2, steps // reps), 2) / reps
    del g
    return ms


def time_direct(call, steps: int, warmup: int):
    import torch

    stream = torch.cuda.current_stream().cuda_stream
    return time_steps(lambda i: call(i, stream), steps, warmup)


def time_steps(fn, steps: int, warmup: int):
    import torch

    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps  # ms per step


def gate_up_setup(copies=16):
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    x, W, s, K, N = I.workload_inputs("gate_up_verify", 16)
    dev = torch.device("cuda:0")
    xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    wp0 = w.w4a8_pack_weights(torch.from_numpy(W).to(dev))
    wps = [wp0] + [wp0.clone() for _ in range(copies - 1)]
    sd = torch.from_numpy(s).to(dev)
    y = torch.empty((16, N), dtype=torch.bfloat16, device=dev)
    ws = w.Workspace(dev)
    return dict(x=x, W=W, s=s, xd=xd, wps=wps, sd=sd, y=y, ws=ws, M=16, K=K, N=N)


def bench_gate_up(steps, warmup):
    """Whole step (bf16 x in, quantize + GEMM + dequant, bf16 y out) and the
    GEMM kernel alone on int8 codes (the dominant kernel)."""
    import torch
    import paper_2608_12932_amd as w

    d = gate_up_setup()
    M, K, N = d["M"], d["K"], d["N"]
    step = DirectCall(d["xd"], d["wps"], d["sd"], N, d["y"], workspace=d["ws"])
    ms_step = time_direct(step, steps, warmup)
    q, sx = w.w4a8_quantize_act(d["xd"])
    gemm = DirectCall(q, d["wps"], d["sd"], N, d["y"], x_scale=sx)
    ms_gemm = time_direct(gemm, steps, warmup)
    torch.cuda.synchronize()
    step_bytes = N * K // 2 + N * 4 + M * K * 2 + M * N * 2        # bf16 x in
    gemm_bytes = N * K // 2 + N * 4 + M * K + M * 4 + M * N * 2    # int8 codes + scales in
    return d, ms_step, step_bytes, ms_gemm, gemm_bytes


def qkv_setup(copies=24):
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    x, W, s, K, N = I.workload_inputs("qkv_prefill", 1024)
    dev = torch.device("cuda:0")
    xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    wp0 = w.w4a8_pack_weights(torch.from_numpy(W).to(dev))
    wps = [wp0] + [wp0.clone() for _ in range(copies - 1)]
    sd = torch.from_numpy(s).to(dev)
    y = torch.empty((1024, N), dtype=torch.bfloat16, device=dev)
    return dict(xd=xd, wps=wps, sd=sd, y=y, ws=w.Workspace(dev), M=1024, K=K, N=N)


def bench_qkv(steps, warmup):
    import paper_2608_12932_amd as w

    d = qkv_setup()
    M, K, N = d["M"], d["K"], d["N"]
    step = DirectCall(d["xd"], d["wps"], d["sd"], N, d["y"], workspace=d["ws"])
    ms_step = time_direct(step, steps, warmup)
    q, sx = w.w4a8_quantize_act(d["xd"])
    gemm = DirectCall(q, d["wps"], d["sd"], N, d["y"], x_scale=sx)
    ms_gemm = time_direct(gemm, steps, warmup)
    L = w.lib()
    xp, qp, sp = d["xd"].data_ptr(), q.data_ptr(), sx.data_ptr()
    import torch

    # The quantize launch alone is shorter than a ctypes call from Python, so
    # it is timed as 50 launches captured in a graph.
    reps = 50
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        L.w4a8_quantize_act(xp, M, K, qp, sp, cap.cuda_stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=cap):
            for _ in range(reps):
                L.w4a8_quantize_act(xp, M, K, qp, sp, cap.cuda_stream)
    torch.cuda.current_stream().wait_stream(cap)
    ms_quant = time_steps(lambda i: g.replay(), max(2, steps // reps), 2) / reps
    del g
    ops = 2 * M * N * K
    return dict(M=M, K=K, N=N, ms_step=ms_step, ms_gemm=ms_gemm, ms_quant=ms_quant, ops=ops)


def _dev_inputs(key, M, mat_index, copies, cache):
    """bf16 x, packed weight copies (device clones of one seeded weight, so
    each step streams distinct addresses), scales and a bf16 y.  The weights
    are made once per matrix and kept in `cache`."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    wl = I.WORKLOADS[key]
    name, K, N = wl.mats[mat_index]
    dev = torch.device("cuda:0")
    if mat_index not in cache:
        W, s = I.weights(N, K, I.seed_w(wl.number, 0, name), wl.group)
        wp0 = w.w4a8_pack_weights(torch.from_numpy(W).to(dev))
        cache[mat_index] = ([wp0] + [wp0.clone() for _ in range(copies - 1)], torch.from_numpy(s).to(dev))
    wps, sd = cache[mat_index]
    x = I.activations(M, K, I.seed_x(wl.number, M), wl.outliers)
    xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    return xd, wps, sd, y, K, N, sd.numel() * sd.element_size()


def bench_down_verify(steps, warmup, copies=16):
    """Down projection at draft-block verification sizes, K=12288 N=4096,
    per-channel fp32 scales; 16 weight copies (403 MB) cycled."""
    import torch
    import paper_2608_12932_amd as w

    rows, cache = [], {}
    for M in (1, 4, 16):
        xd, wps, sd, y, K, N, sbytes = _dev_inputs("down_verify", M, 0, copies, cache)
        call = DirectCall(xd, wps, sd, N, y, workspace=w.Workspace(xd.device))
        ms = time_direct(call, steps, warmup)
        nbytes = N * K // 2 + sbytes + M * K * 2 + M * N * 2
        rows.append({"M": M, "us_per_step": round(ms * 1e3, 3), "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes": nbytes, "kernel": w.w4a8_linear_describe(M, N, K)})
        del xd, wps, sd, y, call
    cache.clear()
    torch.cuda.empty_cache()
    return {"workload": "down verify (down projection, draft-block verification)", "K": 12288, "N": 4096,
            "scales": "per-channel fp32", "x": "bf16 in, quantized in the step", "weight_copies": copies,
            "rows": rows}


def bench_gate_up_swiglu(steps, warmup, copies=16):
    """The gated gate+up projection (gate rows then up rows, N = 24576, K =
    4096, per-channel scales) at M = 1 and 16 (verify / decode) and 1024
    (prefill): w4a8_linear_swiglu writes silu(g) * u [M][12288] from the
    epilogue; the unfused form is w4a8_linear to [M][24576] bf16 followed by
    torch's silu and multiply."""
    import torch
    import paper_2608_12932_amd as w

    rows, cache = [], {}
    for M in (1, 16, 1024):
        xd, wps, sd, y, K, N, sbytes = _dev_inputs("gate_up_verify", M, 0, copies, cache)
        F = N // 2
        yg = torch.empty((M, F), dtype=torch.bfloat16, device=xd.device)
        fused = DirectCall(xd, wps, sd, N, yg, workspace=w.Workspace(xd.device), entry="w4a8_linear_swiglu")
        ms_fused = time_direct(fused, steps, warmup)
        plain = DirectCall(xd, wps, sd, N, y, workspace=w.Workspace(xd.device))

        def unfused(i, stream):
            plain(i, stream)
            torch.mul(torch.nn.functional.silu(y[:, :F]), y[:, F:], out=yg)

        ms_unfused = time_direct(unfused, steps, warmup)
        # the same two forms replayed from a graph (no host launch cost)
        g_fused, g_unfused = graph_ms(fused, steps), graph_ms(unfused, steps)
        nbytes = N * K // 2 + sbytes + M * K * 2 + M * F * 2
        rows.append({"M": M, "us_fused": round(ms_fused * 1e3, 3), "us_unfused": round(ms_unfused * 1e3, 3),
                     "us_fused_graph": round(g_fused * 1e3, 3), "us_unfused_graph": round(g_unfused * 1e3, 3),
                     "TOPS_fused": round(2 * M * N * K / (ms_fused * 1e-3) / 1e12, 1),
                     "GB/s_fused": round(nbytes / (ms_fused * 1e-3) / 1e9, 1),
                     "frac_hbm_fused": round(nbytes / (ms_fused * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes": nbytes, "kernel": w.w4a8_linear_swiglu_describe(M, N, K)})
        del xd, wps, sd, y, yg, fused, plain
    cache.clear()
    torch.cuda.empty_cache()
    return {"workload": "gated gate+up (silu(gate) * up merged into the projection's epilogue)", "K": 4096,
            "N": 24576, "F": 12288, "scales": "per-channel fp32", "x": "bf16 in, quantized in the step",
            "weight_copies": copies, "unfused": "w4a8_linear bf16 [M][N], then torch silu and mul", "rows": rows}


def bench_rmsnorm_prologue(steps):
    """The normalization prologue of the gate+up projection (K = 4096) at M =
    16 and 1024, graph-replayed: w4a8_rmsnorm_quantize_act (one kernel)
    against torch's RMSNorm in fp32 rounded to bf16, then
    w4a8_quantize_act; and each prologue followed by the gate+up GEMM on
    its int8 codes (N = 24576, per-channel scales)."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    L = w.lib()
    rows, cache = [], {}
    for M in (16, 1024):
        xd, wps, sd, y, K, N, sbytes = _dev_inputs("gate_up_verify", M, 0, 8, cache)
        gamma = torch.from_numpy(I.activations(1, K, 77, outliers=False)[0].view(np.int16)).to(xd.device).view(torch.bfloat16)
        q = torch.empty((M, K), dtype=torch.int8, device=xd.device)
        sx = torch.empty((M,), dtype=torch.float32, device=xd.device)
        xp, gp, qp, sp = xd.data_ptr(), gamma.data_ptr(), q.data_ptr(), sx.data_ptr()
        gf = gamma.float()
        hb = torch.empty_like(xd)
        hp = hb.data_ptr()

        def fused(i, stream):
            L.w4a8_rmsnorm_quantize_act(xp, gp, 1e-6, M, K, qp, sp, stream)

        def unfused(i, stream):
            xf = xd.float()
            hb.copy_(xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + 1e-6) * gf)
            L.w4a8_quantize_act(hp, M, K, qp, sp, stream)

        gemm = DirectCall(q, wps, sd, N, y, x_scale=sx)

        def fused_gemm(i, stream):
            fused(i, stream)
            gemm(i, stream)

        def unfused_gemm(i, stream):
            unfused(i, stream)
            gemm(i, stream)

        t = {k: graph_ms(f, steps) * 1e3 for k, f in (("fused", fused), ("unfused", unfused),
                                                       ("fused_gemm", fused_gemm), ("unfused_gemm", unfused_gemm))}
        nbytes = M * K * 2 + K * 2 + M * K + M * 4
        rows.append({"M": M, "us_fused": round(t["fused"], 3), "us_unfused": round(t["unfused"], 3),
                     "GB/s_fused": round(nbytes / (t["fused"] * 1e-6) / 1e9, 1),
                     "us_fused_with_gemm": round(t["fused_gemm"], 3), "us_unfused_with_gemm": round(t["unfused_gemm"], 3),
                     "algorithmic_bytes": nbytes})
        del xd, wps, sd, y, q, sx, gemm
    cache.clear()
    torch.cuda.empty_cache()
    return {"workload": "RMSNorm + int8 quantize prologue of the gate+up projection (K = 4096), graph-replayed",
            "unfused": "torch RMSNorm (fp32, rounded to bf16) then w4a8_quantize_act",
            "gemm": "gate+up N = 24576 on the int8 codes, per-channel scales", "rows": rows}


def bench_stream_attention(steps):
    """Streaming prefill attention of one layer: 4 views x 4 frames x 192
    tokens in a ring-ordered view-major cache (3072 keys), the newest frame's
    768 queries, 32 query heads on 8 kv heads, D = 128, graph-replayed.
    Algorithmic flops count the visible (query, key) pairs only: 4 D per
    pair (QK^T and PV); the kernel's work covers every pair."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    V, F, T, H, Hkv, D = 4, 4, 192, 32, 8, 128
    pos_k = np.empty(V * F * T, np.int32)
    for v in range(V):
        for f in range(F):
            slot = (f + 1) % F
            pos_k[(v * F + slot) * T:(v * F + slot + 1) * T] = v * F * T + f * T + np.arange(T)
    pos_q = np.concatenate([v * F * T + (F - 1) * T + np.arange(T) for v in range(V)]).astype(np.int32)
    Nq, Nk = len(pos_q), len(pos_k)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    q = t(I.activations(H * Nq, D, 90).reshape(H, Nq, D))
    k = t(I.activations(Hkv * Nk, D, 91).reshape(Hkv, Nk, D))
    v = t(I.activations(Hkv * Nk, D, 92).reshape(Hkv, Nk, D))
    n_pos = V * F * T
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * 1e6 ** (-2.0 * np.arange(D // 2) / D)[None, :]
    cos_t = torch.from_numpy(np.cos(ang).astype(np.float32)).to(dev)
    sin_t = torch.from_numpy(np.sin(ang).astype(np.float32)).to(dev)
    pq, pk = torch.from_numpy(pos_q).to(dev), torch.from_numpy(pos_k).to(dev)
    o = torch.empty((H, Nq, D), dtype=torch.bfloat16, device=dev)
    L = w.lib()
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), pq.data_ptr(), pk.data_ptr(), cos_t.data_ptr(), sin_t.data_ptr())

    need = int(L.w4a8_stream_attention_workspace_bytes(H, Nq, Nk))
    ws = torch.zeros(max(need, 1), dtype=torch.uint8, device=dev)

    def call(i, stream):
        rc = L.w4a8_stream_attention(*ptrs, n_pos, H, Hkv, Nq, Nk, D, 1.0 / np.sqrt(D), o.data_ptr(),
                                     ws.data_ptr() if need else None, need, stream)
        if rc:
            raise RuntimeError(f"w4a8_stream_attention failed: {rc}")

    ms = graph_ms(call, steps)
    visible = int((pos_k[None, :] <= pos_q[:, None]).sum())
    flops = 4 * H * D * visible
    tflops = flops / (ms * 1e-3) / 1e12
    return {"workload": f"streaming prefill attention, {V} views x {F} frames x {T} tokens, H={H}, Hkv={Hkv}, D={D}",
            "Nq": Nq, "Nk": Nk, "us": round(ms * 1e3, 3), "visible_pairs": visible,
            "algorithmic_flops": flops, "TFLOP/s": round(tflops, 1), "peak": BF16_PEAK_TFLOPS,
            "frac_bf16": round(tflops / BF16_PEAK_TFLOPS, 4)}


def bench_flow(steps):
    """The flow-matching Euler step with the velocity cache (w4a8_flow_step),
    graph-replayed.  The paper's shape: 6 trajectory samples x 64 waypoints
    x 2 values, launch-bound; per step and for the 8-step solve with 4
    steps reused (4 evaluated steps with their row sums, 4 reused; the
    action network itself is not part of this library).  The bandwidth
    shape, 16384 x 2048: algorithmic bytes 14 per element on an evaluated
    step (x read and written, v read, cache read and written), 10 on a
    reused one (x read and written, cache read)."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    L = w.lib()
    dev = torch.device("cuda:0")
    out = {}
    for label, B, n in (("paper", 6, 128), ("bandwidth", 16384, 2048)):
        x = torch.from_numpy(I.flow_state(B, n, 61)).to(dev)
        bf = lambda bits: torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)
        v = bf(I.flow_velocity(B, n, 62))
        c = bf(I.flow_velocity(B, n, 63))
        st = torch.empty((B, 4), dtype=torch.float64, device=dev)
        # a device copy of known size (B n 2 bytes read and written), the
        # calibration of the HBM byte counters in a profiled run
        calib = v.clone()
        xp, vp, cp, sp = x.data_ptr(), v.data_ptr(), c.data_ptr(), st.data_ptr()
        dt = 0.125

        def fresh(i, stream, repeat=1):
            if L.w4a8_flow_step(xp, vp, cp, B, n, dt, repeat, sp, stream):
                raise RuntimeError("w4a8_flow_step failed")

        def reuse(i, stream):
            if L.w4a8_flow_step(xp, None, cp, B, n, dt, 1, None, stream):
                raise RuntimeError("w4a8_flow_step failed")

        sched = w.w4a8_flow_schedule(8, 4)
        # one call per evaluated step, the reused steps after it folded in
        runs = []
        for f in sched:
            if f:
                runs.append(1)
            else:
                runs[-1] += 1

        def solve(i, stream):
            for f in sched:
                (fresh if f else reuse)(i, stream)

        def solve_runs(i, stream):
            for r in runs:
                fresh(i, stream, r)

        t_f = graph_ms(fresh, steps) * 1e3
        t_r = graph_ms(reuse, steps) * 1e3
        row = {"B": B, "n": n, "us_evaluated_step": round(t_f, 3), "us_reused_step": round(t_r, 3)}
        if label == "paper":
            row["us_solve_8_steps_4_reused"] = round(graph_ms(solve, max(10, steps // 8), reps=5) * 1e3, 3)
            row["us_solve_folded_runs"] = round(graph_ms(solve_runs, max(10, steps // 8), reps=5) * 1e3, 3)
            row["calls_folded"] = len(runs)
            row["network_evaluations"] = {"cached": sum(sched), "uncached": len(sched)}
        else:
            # the folded run of an evaluated step with its 4 reused steps: 14 bytes per element, one pass
            t_5 = graph_ms(lambda i, st_: fresh(i, st_, 5), steps) * 1e3
            row["us_evaluated_plus_4_reused_folded"] = round(t_5, 3)
            row["us_evaluated_plus_4_reused_separate"] = round(t_f + 4 * t_r, 3)
            ef, er = 14 * B * n, 10 * B * n
            row.update({"GB/s_evaluated": round(ef / (t_f * 1e-6) / 1e9, 1),
                        "GB/s_reused": round(er / (t_r * 1e-6) / 1e9, 1),
                        "frac_hbm_evaluated": round(ef / (t_f * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                        "algorithmic_bytes_evaluated": ef, "algorithmic_bytes_reused": er})
        out[label] = row
        del x, v, c, st, calib
    torch.cuda.empty_cache()
    return {"workload": "flow-matching Euler step with the velocity cache, graph-replayed", **out}


def bench_layer_group(steps, warmup, copies=6):
    """One decoder layer's four linears (QKV, O, gate+up, down) with group-128
    fp16 scales; a step is the four calls, each on its own bf16 x.  Six copies
    of the layer's weights (580 MB) are cycled."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    rows, cache = [], {}
    for M in (1, 16, 256, 2048):
        calls, nbytes, ops, kinds = [], 0, 0, []
        for mi, (name, K, N) in enumerate(I.LAYER_MATS):
            xd, wps, sd, y, K, N, sbytes = _dev_inputs("layer_group", M, mi, copies, cache)
            calls.append(DirectCall(xd, wps, sd, N, y, workspace=w.Workspace(xd.device),
                                    scale_mode=w.SCALE_GROUP_F16))
            nbytes += N * K // 2 + sbytes + M * K * 2 + M * N * 2
            ops += 2 * M * N * K
            kinds.append(f"{name}: " + w.w4a8_linear_describe(M, N, K, w.SCALE_GROUP_F16))
        stream = torch.cuda.current_stream().cuda_stream

        def layer(i):
            for c in calls:
                c(i, stream)

        n = max(20, steps // (1 if M < 256 else 4 if M == 256 else 16))
        ms = time_steps(layer, n, max(5, warmup // 4))
        rows.append({"M": M, "us_per_layer": round(ms * 1e3, 3),
                     "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "TOPS": round(ops / (ms * 1e-3) / 1e12, 2),
                     "frac_int8": round(ops / (ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
                     "steps": n, "algorithmic_bytes": nbytes, "ops": ops, "kernels": kinds})
        del calls
    cache.clear()
    torch.cuda.empty_cache()
    return {"workload": "decoder layer (QKV, O, gate+up, down) with group-128 fp16 scales",
            "scales": "fp16 per 128 k per channel", "x": "bf16 in, quantized in the step",
            "layer_copies": copies, "rows": rows}


def bench_stack(steps, layers=36):
    """The backbone's W4A8 linears for one decode/verify step: 36 decoder
    layers x (QKV, O, gate+up, down) with group-128 fp16 scales, each call on
    its own bf16 x, at M = 1 and 16 tokens.  Weights are device clones of
    one seeded layer (3.5 GB of distinct addresses, far past the 256 MB
    Infinity Cache).  Timed as eager calls on torch's stream and as the
    replay of one captured HIP graph of the whole stack."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    dev = torch.device("cuda:0")
    base = []
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        W, sc = I.weights(N, K, I.seed_w(5, 0, name), group=True)
        base.append((name, K, N, w.w4a8_pack_weights(torch.from_numpy(W).to(dev)), torch.from_numpy(sc).to(dev)))
    weights = [[(name, K, N, wp if l == 0 else wp.clone(), sc) for (name, K, N, wp, sc) in base] for l in range(layers)]
    rows = []
    for M in (1, 16):
        calls, nbytes = [], 0
        for l in range(layers):
            for mi, (name, K, N, wp, sc) in enumerate(weights[l]):
                x = I.activations(M, K, I.seed_x(5, M) + 7 * l + mi)
                xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
                y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
                calls.append(DirectCall(xd, [wp], sc, N, y, workspace=w.Workspace(dev), scale_mode=w.SCALE_GROUP_F16))
                nbytes += N * K // 2 + sc.numel() * 2 + M * K * 2 + M * N * 2

        def run_all(stream):
            for c in calls:
                c(0, stream)

        stream = torch.cuda.current_stream().cuda_stream
        ms_eager = time_steps(lambda i: run_all(stream), steps, 3)
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            run_all(cap.cuda_stream)  # warm the capture stream
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=cap):
                run_all(cap.cuda_stream)
        torch.cuda.current_stream().wait_stream(cap)
        ms_graph = time_steps(lambda i: g.replay(), steps, 3)
        rows.append({"M": M, "linears": len(calls), "us_eager": round(ms_eager * 1e3, 1),
                     "us_graph": round(ms_graph * 1e3, 1), "us_per_token_graph": round(ms_graph * 1e3 / M, 2),
                     "GB/s_graph": round(nbytes / (ms_graph * 1e-3) / 1e9, 1),
                     "frac_hbm_graph": round(nbytes / (ms_graph * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes": nbytes})
        del calls, g
    del weights, base
    torch.cuda.empty_cache()
    return {"workload": f"{layers}-layer backbone linears per decode/verify step (QKV, O, gate+up, down; "
                        "group-128 fp16 scales)", "rows": rows}


def profile_workload(spec: str, steps: int, warmup: int):
    """One workload alone, for a rocprofv3 run: `steps` timed steps after
    `warmup`, each step as in the JSON line (bf16 x in, bf16 y out).  spec:
      gate_up        gate+up verify step, M=16 (and the GEMM on int8 codes)
      qkv            qkv prefill step, M=1024 (and the GEMM on int8 codes)
      down:M         down verify, K=12288 N=4096, M in 1, 4, 16
      layer:M        one decoder layer with group-128 scales, M in 1, 16, 256, 2048
    Prints one JSON object with the event-timed us per step."""
    import torch
    import paper_2608_12932_amd as w
    from paper_2608_12932_amd import inputs as I

    name, _, arg = spec.partition(":")
    if name == "gate_up":
        d, ms, nbytes, ms_gemm, gemm_bytes = bench_gate_up(steps, warmup)
        return {"profile": spec, "us_step": round(ms * 1e3, 3), "us_gemm": round(ms_gemm * 1e3, 3),
                "step_bytes": nbytes, "gemm_bytes": gemm_bytes, "kernel": w.w4a8_linear_describe(16, d["N"], d["K"])}
    if name == "qkv":
        r = bench_qkv(steps, warmup)
        return {"profile": spec, "us_step": round(r["ms_step"] * 1e3, 3), "us_gemm": round(r["ms_gemm"] * 1e3, 3),
                "ops": r["ops"], "kernel": w.w4a8_linear_describe(r["M"], r["N"], r["K"])}
    M = int(arg)
    cache = {}
    if name == "down":
        xd, wps, sd, y, K, N, sbytes = _dev_inputs("down_verify", M, 0, 16, cache)
        calls = [DirectCall(xd, wps, sd, N, y, workspace=w.Workspace(xd.device))]
        nbytes = N * K // 2 + sbytes + M * K * 2 + M * N * 2
        kinds = [w.w4a8_linear_describe(M, N, K)]
    elif name == "layer":
        calls, nbytes, kinds = [], 0, []
        for mi, (mname, K, N) in enumerate(I.LAYER_MATS):
            xd, wps, sd, y, K, N, sbytes = _dev_inputs("layer_group", M, mi, 6, cache)
            calls.append(DirectCall(xd, wps, sd, N, y, workspace=w.Workspace(xd.device), scale_mode=w.SCALE_GROUP_F16))
            nbytes += N * K // 2 + sbytes + M * K * 2 + M * N * 2
            kinds.append(f"{mname}: " + w.w4a8_linear_describe(M, N, K, w.SCALE_GROUP_F16))
    else:
        raise SystemExit(f"unknown profile workload {spec!r}")
    stream = torch.cuda.current_stream().cuda_stream

    def step(i):
        for c in calls:
            c(i, stream)

    ms = time_steps(step, steps, warmup)
    return {"profile": spec, "us_step": round(ms * 1e3, 3), "algorithmic_bytes": nbytes,
            "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1), "kernels": kinds}


# ---- rocprofv3 summaries (profiles/<name>.txt) -------------------------------
# Each summary comes from separate rocprofv3 runs of `bench.py --profile SPEC`
# (a kernel trace, then FETCH_SIZE, then WRITE_SIZE, and at large M one pass
# of MFMA / VALU counters; counters are never combined with tracing), and
# `bench.py --summarize-profile NAME --prof-dir DIR` turns their CSV files
# into the summary.  `--profile-commands NAME --prof-dir DIR` prints the
# rocprofv3 commands, one per line.

PROFILE_SPECS = {
    "smallm_gate_up_verify": ("gate_up", "gate+up verify, M=16 K=4096 N=24576, per-channel scales; GEMM on int8 codes"),
    "largem_qkv_prefill": ("qkv", "qkv prefill, M=1024 K=4096 N=6144, per-channel scales; GEMM on int8 codes"),
    "smallm_down_verify_m1": ("down:1", "down verify, M=1 K=12288 N=4096, per-channel scales; GEMM on int8 codes"),
    "smallm_down_verify_m4": ("down:4", "down verify, M=4 K=12288 N=4096, per-channel scales; GEMM on int8 codes"),
    "smallm_down_verify_m16": ("down:16", "down verify, M=16 K=12288 N=4096, per-channel scales; GEMM on int8 codes"),
    "smallm_group_layer_m1": ("layer:1", "decoder layer with group-128 fp16 scales, M=1: small-M GEMMs"),
    "smallm_group_layer_m16": ("layer:16", "decoder layer with group-128 fp16 scales, M=16: small-M GEMMs"),
    "largem_group_layer_m256": ("layer:256", "decoder layer with group-128 fp16 scales, M=256: large-M GEMMs"),
    "largem_group_layer_m2048": ("layer:2048", "decoder layer with group-128 fp16 scales, M=2048: large-M GEMMs"),
}
MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_I8 SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU SQ_BUSY_CYCLES "
                 "SQ_ACTIVE_INST_VALU SQ_WAIT_INST_LDS SQ_INSTS_MFMA GRBM_GUI_ACTIVE")
N_SIMDS, N_XCDS = 1024, 8  # MI355X: 256 CUs x 4 SIMDs, 8 XCDs


def _profile_gemms(spec: str):
    """The GEMMs one profiled step launches, in order: (label, M, N, K, group),
    and the packed-weight bytes of the matrix whose device clones calibrate
    the counters (the largest one the run clones)."""
    from paper_2608_12932_amd import inputs as I

    kind, _, arg = spec.partition(":")
    if kind == "gate_up":
        g = [("", 16, 24576, 4096, False)]
    elif kind == "qkv":
        g = [("", 1024, 6144, 4096, False)]
    elif kind == "down":
        g = [("", int(arg), 4096, 12288, False)]
    elif kind == "layer":
        g = [(name, int(arg), N, K, True) for name, K, N in I.LAYER_MATS]
    else:
        raise SystemExit(f"unknown profile workload {spec!r}")
    return g, max(N * K // 2 for _, _, N, K, _ in g)


def profile_commands(name: str, out_dir: str):
    spec = PROFILE_SPECS[name][0]
    large = any(M > 64 for _, M, _, _, _ in _profile_gemms(spec)[0])
    run = f"-o p --output-format csv -- python3 bench.py --profile {spec}"
    cmds = [f"rocprofv3 --kernel-trace --stats -d {out_dir}/{name}_trace {run} --steps 100 --warmup 10",
            f"rocprofv3 --pmc FETCH_SIZE -d {out_dir}/{name}_fetch {run} --steps 20 --warmup 3",
            f"rocprofv3 --pmc WRITE_SIZE -d {out_dir}/{name}_write {run} --steps 20 --warmup 3"]
    if large:
        cmds.append(f"rocprofv3 --pmc {MFMA_COUNTERS} -d {out_dir}/{name}_mfma {run} --steps 20 --warmup 3")
    return cmds


def _csv_rows(run_dir: str, suffix: str):
    import csv
    import glob

    files = sorted(glob.glob(os.path.join(run_dir, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no {suffix} under {run_dir}")
    with open(files[0], newline="") as f:
        return list(csv.DictReader(f))


def _short_kernel(full: str) -> str:
    """'void w4a8::(anonymous namespace)::smallm<1, 6, ...>(args)' -> 'smallm<1, 6, ...>':
    the name up to its argument list, without return type and namespaces."""
    name = full.replace("(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    depth, out = 0, []
    for ch in name:
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    name, depth, cut = "".join(out), 0, 0
    for i, ch in enumerate(name):  # the last "::" outside template arguments
        depth += ch == "<"
        depth -= ch == ">"
        if depth == 0 and name.startswith("::", i):
            cut = i + 2
    return name[cut:]


def _is_gemm(kernel: str) -> bool:
    k = _short_kernel(kernel)
    return k.startswith("smallm<") or k.startswith("largem<")


def _per_dispatch(rows, counter: str):
    """{dispatch id: (kernel name, value)} for one counter of a --pmc run."""
    out = {}
    for r in rows:
        if r["Counter_Name"] == counter:
            out[int(r["Dispatch_Id"])] = (r["Kernel_Name"], float(r["Counter_Value"]))
    return [out[d] for d in sorted(out)]


def _calibration(rows, counter: str, nbytes: int):
    """The factor that turns `counter` (KiB per dispatch) into bytes, from the
    run's own device copies (__amd_rocclr_copyBuffer) of its largest weight,
    nbytes: the copies whose count is within 10 % of the largest one (the
    weights of one run differ by 1.5x or more)."""
    import statistics

    copies = [v for k, v in _per_dispatch(rows, counter) if "copyBuffer" in k]
    if not copies:
        raise SystemExit(f"no device copies to calibrate {counter}")
    vals = [v for v in copies if v >= 0.9 * max(copies)]
    return nbytes / (statistics.median(vals) * 1024), len(vals)


def summarize_profile(name: str, out_dir: str) -> str:
    import statistics

    spec, desc = PROFILE_SPECS[name]
    gemms, cal_bytes = _profile_gemms(spec)
    ng = len(gemms)
    cmds = profile_commands(name, out_dir)
    trace = sorted(_csv_rows(os.path.join(out_dir, f"{name}_trace"), "kernel_trace.csv"),
                   key=lambda r: int(r["Start_Timestamp"]))
    durs = [(r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3) for r in trace]
    gemm_durs = [(k, d) for k, d in durs if _is_gemm(k)]
    quant = [(k, d) for k, d in durs if "quantize_rows" in k]
    fetch_rows = _csv_rows(os.path.join(out_dir, f"{name}_fetch"), "counter_collection.csv")
    write_rows = _csv_rows(os.path.join(out_dir, f"{name}_write"), "counter_collection.csv")
    ff, nf = _calibration(fetch_rows, "FETCH_SIZE", cal_bytes)
    wf, nw = _calibration(write_rows, "WRITE_SIZE", cal_bytes)
    fetch = [v for k, v in _per_dispatch(fetch_rows, "FETCH_SIZE") if _is_gemm(k)]
    write = [v for k, v in _per_dispatch(write_rows, "WRITE_SIZE") if _is_gemm(k)]
    mfma = None
    if len(cmds) == 4:
        mrows = _csv_rows(os.path.join(out_dir, f"{name}_mfma"), "counter_collection.csv")
        mfma = {c: [v for k, v in _per_dispatch(mrows, c) if _is_gemm(k)] for c in MFMA_COUNTERS.split()}

    lines = [f"# rocprofv3 summary: {desc}",
             "# commands (each a separate run; counters never combined with tracing), from the repository root after",
             "#   cd /tmp && export TMPDIR=/tmp:"]
    lines += [f"#   {c}" for c in cmds]
    if ng == 1 and spec.split(":")[0] in ("gate_up", "qkv"):
        lines.append("# the profiled run times the bf16-in step (quantize launch + GEMM) and then the GEMM alone on "
                     f"int8 codes;\n#   the GEMM kernel's durations below cover both ({len(gemm_durs)} dispatches "
                     "incl. warmup)")
    elif ng == 1:
        lines.append("# the profiled run times the bf16-in step (quantize launch + GEMM on its codes); "
                     f"{len(gemm_durs)} GEMM dispatches incl. warmup")
    else:
        qa = statistics.mean(d for _, d in quant) if quant else 0.0
        lines.append("# a step is the four linears in order, each a quantize launch + GEMM on bf16 x; GEMM "
                     "dispatches are\n#   assigned to the matrices by their order; "
                     f"{len(quant)} quantize dispatches average {qa:.3f} us")
    lines.append("# HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) calibrated on __amd_rocclr_copyBuffer "
                 f"copying a\n#   {cal_bytes} B packed weight in the same runs: FETCH factor {ff:.4f} ({nf} copies), "
                 f"WRITE factor {wf:.4f} ({nw} copies)")

    def stats_for(i):
        sel = lambda seq: [x for j, x in enumerate(seq) if j % ng == i]
        d = sel(gemm_durs)
        us = [x for _, x in d]
        label, M, N, K, group = gemms[i]
        scale_bytes = (K // 128) * N * 2 if group else N * 4
        algo = N * K // 2 + scale_bytes + M * K + 4 * M + 2 * M * N
        ops = 2 * M * N * K
        avg = statistics.mean(us)
        fb = statistics.median(sel(fetch)) * 1024 * ff
        wb = statistics.median(sel(write)) * 1024 * wf
        out = [("kernel", _short_kernel(d[0][0])), ("avg_us", f"{avg:.3f}")]
        if ng == 1:
            out += [("median_us", f"{statistics.median(us):.3f}"), ("min_us", f"{min(us):.3f}")]
        out.append(("calls", str(len(us))))
        if ng == 1 and quant:
            out += [("quantize_kernel", _short_kernel(quant[0][0])),
                    ("quantize_avg_us", f"{statistics.mean(x for _, x in quant):.3f}")]
        out.append(("algorithmic_bytes_per_dispatch", str(algo)))
        if ng == 1:
            out.append(("achieved_GBps_from_avg", f"{algo / avg / 1e3:.1f}"))
        out.append(("frac_of_8TBps_from_avg", f"{algo / avg / 1e3 / HBM_PEAK_GBS:.4f}"))
        if ng == 1:
            out += [("int8_ops_per_dispatch", str(ops)), ("achieved_TOPS_from_avg", f"{ops / avg / 1e6:.1f}")]
        out.append(("frac_of_5POPS_from_avg", f"{ops / avg / 1e6 / INT8_PEAK_TOPS:.4f}"))
        if ng == 1:
            out += [("fetch_bytes_per_dispatch", f"{fb:.0f}"), ("write_bytes_per_dispatch", f"{wb:.0f}")]
        out += [("hbm_bytes_per_dispatch", f"{fb + wb:.0f}"), ("traffic_over_algorithmic", f"{(fb + wb) / algo:.3f}")]
        if mfma:
            med = {c: statistics.median(sel(v)) for c, v in mfma.items()}
            gui = med["GRBM_GUI_ACTIVE"] / N_XCDS
            out += [("mfma_int8_ops_per_dispatch",
                     f"{med['SQ_INSTS_VALU_MFMA_MOPS_I8'] * 512:.0f}   (SQ_INSTS_VALU_MFMA_MOPS_I8 x 512; 2*M*N*K = {ops}; "
                     f"median over {len(sel(mfma['SQ_INSTS_MFMA']))} dispatches)"),
                    ("mfma_busy_over_gui_active_per_simd",
                     f"{med['SQ_VALU_MFMA_BUSY_CYCLES'] / N_SIMDS / gui:.3f}   (SQ_VALU_MFMA_BUSY_CYCLES per SIMD over "
                     "GRBM_GUI_ACTIVE per XCD)"),
                    ("valu_insts_per_mfma",
                     f"{med['SQ_INSTS_VALU'] / med['SQ_INSTS_MFMA']:.2f}   (SQ_INSTS_VALU, which counts the MFMAs, over "
                     "the 32x32x32 MFMA count)"),
                    ("valu_active_over_gui_active_per_simd",
                     f"{med['SQ_ACTIVE_INST_VALU'] * 4 / N_SIMDS / gui:.3f}   (SQ_ACTIVE_INST_VALU, quad-cycles, x 4 per "
                     "SIMD over GRBM_GUI_ACTIVE per XCD)"),
                    ("lds_wait_over_gui_active_per_simd",
                     f"{med['SQ_WAIT_INST_LDS'] / N_SIMDS / gui:.3f}   (SQ_WAIT_INST_LDS per SIMD over GRBM_GUI_ACTIVE "
                     "per XCD)"),
                    ("raw", " ".join(f"{c}={med[c]:.0f}" for c in sorted(med))),
                    ("sq_insts_mfma", f"{med['SQ_INSTS_MFMA']:.0f}")]
        return label, avg, out

    total = 0.0
    for i in range(ng):
        label, avg, out = stats_for(i)
        total += avg
        prefix = f"{label}." if label else ""
        lines += [f"{prefix}{k}: {v}" for k, v in out]
    if ng > 1:
        lines.append(f"gemm_sum_avg_us: {total:.3f}")
        if quant:
            lines.append(f"quantize_avg_us: {statistics.mean(x for _, x in quant):.3f}")
    lines.append(f"source_hash: {kernel_source_hash()}")
    return "\n".join(lines) + "\n"


def measure_ceilings():
    """Measured HBM-read and INT8-MFMA ceilings (libw4a8_ceiling.so): a plain
    16-byte streaming read of 1 GiB, and independent 32x32x32 int8 MFMA
    chains with register operands."""
    import ctypes
    import torch

    L = ctypes.CDLL(os.path.join(ROOT, "paper_2608_12932_amd", "libw4a8_ceiling.so"))
    L.w4a8_ceiling_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    L.w4a8_ceiling_mfma_i8.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    st = torch.cuda.current_stream().cuda_stream
    nbytes = 1 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(7)
    sink = torch.empty(256 * 512, dtype=torch.int32, device="cuda")

    def read(i):
        if L.w4a8_ceiling_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(), st):
            raise RuntimeError("ceiling read launch failed")

    ms_read = time_steps(read, 10, 2)
    iters = 2048
    msink = torch.empty(1024 * 256, dtype=torch.int32, device="cuda")

    def mfma(i):
        if L.w4a8_ceiling_mfma_i8(iters, msink.data_ptr(), st):
            raise RuntimeError("ceiling mfma launch failed")

    ms_mfma = time_steps(mfma, 5, 1)
    ops = 1024 * 4 * 4 * iters * 65536
    del buf
    torch.cuda.empty_cache()
    gbs = nbytes / (ms_read * 1e-3) / 1e9
    tops = ops / (ms_mfma * 1e-3) / 1e12
    return {"hbm_read": {"value": round(gbs, 1), "unit": "GB/s", "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
                         "what": "16-byte non-temporal streaming read of 1 GiB, 256 workgroups x 512 threads, "
                                 "one contiguous range each"},
            "int8_mfma": {"value": round(tops, 1), "unit": "TOPS", "frac_of_peak": round(tops / INT8_PEAK_TOPS, 4),
                          "what": "4 independent v_mfma_i32_32x32x32_i8 chains per wave, 4096 waves"}}


def library_int8_gemm(M=1024, N=6144, K=4096, steps=50, warmup=10):
    """The vendor library's plain int8 GEMM at the qkv prefill shape, for
    context: torch._int_mm (hipBLASLt) on int8 activations [M][K] and 8-bit
    weights stored [N][K] (passed as the transposed view), int32 out.  It
    reads twice the weight bytes of the 4-bit path and applies no scales."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(2608)
    a = torch.randint(-127, 128, (M, K), dtype=torch.int8, device="cuda", generator=g)
    b = torch.randint(-8, 8, (N, K), dtype=torch.int8, device="cuda", generator=g)
    bt = b.t()
    ms = time_steps(lambda i: torch._int_mm(a, bt), steps, warmup)
    tops = 2.0 * M * N * K / (ms * 1e-3) / 1e12
    return {"value": round(tops, 1), "unit": "TOPS", "us": round(ms * 1e3, 3),
            "frac_of_peak": round(tops / INT8_PEAK_TOPS, 4),
            "what": f"torch._int_mm (hipBLASLt) int8 x int8 -> int32, M={M} N={N} K={K}, 8-bit weights, no scales"}


def host_cpu():
    """The host's logical CPU count, the CPUs this process may run on, and
    the CPU model name (from /proc/cpuinfo, as lscpu reports it)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)), "model": model}


def cpu_baseline(d, algo_bytes, budget_s=10.0, budget_1t_s=8.0):
    """The oracle on the full gate+up verify layer: with one thread per token
    row (the oracle splits the rows over threads, so at most M = 16), up to
    the CPUs this process may use, repeated for about budget_s seconds of
    CPU work; and on one thread for about budget_1t_s.  The rates are the
    median run's.  The oracle is plain scalar C (int64 dot products), a
    correctness reference, not a tuned CPU GEMM."""
    import oracle

    cpu = host_cpu()

    def timed(threads, budget):
        times = []
        t_start = time.perf_counter()
        while not times or (time.perf_counter() - t_start < budget and len(times) < 1000):
            t0 = time.perf_counter()
            oracle.linear(d["x"], d["W"], s_w=d["s"], nthreads=threads)
            times.append(time.perf_counter() - t0)
        return statistics.median(times), times

    threads = min(d["M"], cpu["affinity"])
    t, times = timed(threads, budget_s)
    t1, times1 = timed(1, budget_1t_s)
    return {"value": round(algo_bytes / t / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "host": cpu,
            "one_thread": {"value": round(algo_bytes / t1 / 1e9, 4), "unit": "GB/s", "ms_per_run": round(t1 * 1e3, 1),
                           "runs": len(times1)},
            "sample": f"the full gate+up verify layer (M=16 K=4096 N=24576: quantize, int64 contraction, "
                      f"dequant) run {len(times)} times on {threads} threads ({sum(times):.1f} s), median "
                      f"{t*1e3:.1f} ms per run; and {len(times1)} times on 1 thread ({sum(times1):.1f} s), median "
                      f"{t1*1e3:.1f} ms; host {cpu['model']}, {cpu['nproc']} logical CPUs, {cpu['affinity']} "
                      f"available to this process"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the down-projection verify and group-scale layer sweeps")
    ap.add_argument("--sweep-only", action="store_true",
                    help="run only the sweeps (for profiling their kernels); prints the sweep object")
    ap.add_argument("--attention-only", action="store_true",
                    help="run only the streaming attention workload (for profiling its kernels)")
    ap.add_argument("--flow-only", action="store_true",
                    help="run only the flow-matching step workloads (for profiling their kernel)")
    ap.add_argument("--profile", default=None, metavar="WORKLOAD",
                    help="run one workload only, for rocprofv3: gate_up, qkv, down:M, layer:M")
    ap.add_argument("--profile-commands", default=None, metavar="NAME",
                    help="print the rocprofv3 commands of summary NAME (see --prof-dir)")
    ap.add_argument("--summarize-profile", default=None, metavar="NAME",
                    help="print summary NAME from the rocprofv3 CSV files under --prof-dir")
    ap.add_argument("--prof-dir", default="prof", help="rocprofv3 output root of the two options above (default: ./prof)")
    args = ap.parse_args()
    if args.profile_commands:
        print("\n".join(profile_commands(args.profile_commands, args.prof_dir)))
        return
    if args.summarize_profile:
        sys.stdout.write(summarize_profile(args.summarize_profile, args.prof_dir))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the layer would shard by output columns or by K).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_12932_amd as w

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w.lib()
    if args.profile:
        print(json.dumps(profile_workload(args.profile, args.steps, args.warmup)), flush=True)
        return
    if args.attention_only:
        print(json.dumps(bench_stream_attention(max(50, args.steps // 4))), flush=True)
        return
    if args.flow_only:
        print(json.dumps(bench_flow(max(50, args.steps // 4))), flush=True)
        return
    if args.sweep_only:
        ss, sw = max(50, args.steps // 4), max(10, args.warmup // 4)
        print(json.dumps({"sweep": {"down_verify": bench_down_verify(ss, sw),
                                    "gate_up_swiglu": bench_gate_up_swiglu(ss, sw),
                                    "rmsnorm_prologue": bench_rmsnorm_prologue(ss),
                                    "stream_attention": bench_stream_attention(ss),
                                    "flow_step": bench_flow(ss),
                                    "layer_group": bench_layer_group(ss, sw),
                                    "stack": bench_stack(max(10, args.steps // 50))}}), flush=True)
        return
    d, ms, algo_bytes, ms_gemm, gemm_bytes = bench_gate_up(args.steps, args.warmup)
    gbs = algo_bytes / (ms * 1e-3) / 1e9
    gemm_gbs = gemm_bytes / (ms_gemm * 1e-3) / 1e9
    M, K, N = d["M"], d["K"], d["N"]
    traffic = counter_traffic("smallm_gate_up_verify")
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "gate+up verify (fused gate+up projection, draft-block verification)",
                   "M": M, "K": K, "N": N, "scales": "per-channel fp32", "x": "bf16 in, quantized in the step",
                   "y": "bf16", "weight_copies": len(d["wps"]), "algorithmic_bytes": algo_bytes},
        "kernel": w.w4a8_linear_describe(M, N, K),
        "roofline": {"bound": "hbm", "achieved": round(gemm_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gemm_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": w.w4a8_linear_describe(M, N, K, 0, 1), "kernel_ms": round(ms_gemm, 6),
                     "algorithmic_bytes": gemm_bytes,
                     "timing": "HIP events on the launch stream over back-to-back launches (launch to launch)",
                     "from_trace": trace_roofline("smallm_gate_up_verify", gemm_bytes, HBM_PEAK_GBS, 1e9)},
    }
    if not args.no_secondary:
        r = bench_qkv(max(50, args.steps // 4), max(10, args.warmup // 4))
        tops_step = r["ops"] / (r["ms_step"] * 1e-3) / 1e12
        tops_gemm = r["ops"] / (r["ms_gemm"] * 1e-3) / 1e12
        out["secondary"] = {
            "metric": "INT8 TOPS at M=1024 (qkv prefill)",
            "value": round(tops_step, 2),
            "unit": "TOPS",
            "ms_per_step": round(r["ms_step"], 6),
            "config": {"workload": "qkv prefill (fused QKV projection, streaming prefill of new-frame tokens)",
                       "M": r["M"], "K": r["K"], "N": r["N"], "scales": "per-channel fp32",
                       "x": "bf16 in, quantized by its own kernel", "y": "bf16", "weight_copies": 24},
            "kernel": w.w4a8_linear_describe(r["M"], r["N"], r["K"]),
            "quantize_ms": round(r["ms_quant"], 6),
            "roofline": {"bound": "mfma", "achieved": round(tops_gemm, 2), "peak": INT8_PEAK_TOPS, "unit": "TOPS",
                         "frac": round(tops_gemm / INT8_PEAK_TOPS, 4), "kernel_ms": round(r["ms_gemm"], 6),
                         "kernel": w.w4a8_linear_describe(r["M"], r["N"], r["K"], 0, 1),
                         "traffic": counter_traffic("largem_qkv_prefill"),
                         "from_trace": trace_roofline("largem_qkv_prefill", r["ops"], INT8_PEAK_TOPS, 1e12)},
        }
    out["ceilings"] = measure_ceilings()
    try:
        out["ceilings"]["library_int8_gemm"] = library_int8_gemm()
        if "secondary" in out:
            out["secondary"]["roofline"]["speedup_vs_library_int8_gemm"] = round(
                out["ceilings"]["library_int8_gemm"]["us"] / (out["secondary"]["roofline"]["kernel_ms"] * 1e3), 3)
    except RuntimeError as e:  # torch built without the int8 GEMM
        out["ceilings"]["library_int8_gemm"] = {"error": str(e)[:200]}
    if not args.no_sweep:
        ss, sw = max(50, args.steps // 4), max(10, args.warmup // 4)
        out["sweep"] = {"down_verify": bench_down_verify(ss, sw), "gate_up_swiglu": bench_gate_up_swiglu(ss, sw),
                        "rmsnorm_prologue": bench_rmsnorm_prologue(ss),
                        "stream_attention": bench_stream_attention(ss),
                        "flow_step": bench_flow(ss),
                        "layer_group": bench_layer_group(ss, sw),
                        "stack": bench_stack(max(10, args.steps // 50))}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(d, algo_bytes)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
