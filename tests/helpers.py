"""Shared plumbing for the GPU parity tests: move seeded inputs to the
device, call the HIP path through the binding, and compare with the oracle."""
from __future__ import annotations

import os

import numpy as np
import torch

import oracle
import paper_2608_12932_amd as w

NTHREADS = min(16, len(os.sched_getaffinity(0)))

# bf16 output tolerance of the group-scale path: |y - y64| <= REL |y64| + FLOOR B
# (B = s_x sum_g |p_g| s_g).  bf16 rounding contributes <= 2^-8 |y|; fp32
# accumulation over <= 512 groups contributes <= 512 * 2^-24 B < 3.1e-5 B.
REL = 1e-2
GROUP_FLOOR = 1e-4


# (label, shape, scales, max elementwise and normwise relative error of the
# bf16 output against the oracle's fp64 value); printed in the terminal
# summary by conftest.py
ERROR_REPORT = []


def record_errors(label, shape, group, y, y64):
    """Max elementwise relative error over nonzero reference values, and
    the normwise ||y - y64|| / ||y64||."""
    y = y.astype(np.float64)
    nz = y64 != 0
    max_rel = float(np.max(np.abs(y[nz] - y64[nz]) / np.abs(y64[nz]))) if nz.any() else 0.0
    den = float(np.linalg.norm(y64))
    norm_rel = float(np.linalg.norm(y - y64)) / den if den > 0 else float(np.linalg.norm(y - y64))
    ERROR_REPORT.append((label, shape, "group" if group else "channel", max_rel, norm_rel))


def dev():
    return torch.device("cuda:0")


def bf16_dev(x_bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(dev()).view(torch.bfloat16)


def to_np_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def pack(W: np.ndarray) -> torch.Tensor:
    return w.w4a8_pack_weights(torch.from_numpy(np.ascontiguousarray(W)).to(dev()))


def scales_dev(s: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(s)).to(dev())


def run_linear(x_bits, wp, s, N, *, group, out_kind, codes=None, workspace=None):
    """HIP path.  codes=(q, s_x) feeds pre-quantized int8 input."""
    mode = w.SCALE_GROUP_F16 if group else w.SCALE_CHANNEL_F32
    sd = None if out_kind == w.OUT_I32_ACC else scales_dev(s)
    if codes is None:
        x = bf16_dev(x_bits)
        y = w.w4a8_linear(x, wp, sd, N, scale_mode=mode, out_kind=out_kind, workspace=workspace)
    else:
        q, sx = codes
        y = w.w4a8_linear(torch.from_numpy(q).to(dev()), wp, sd, N, x_scale=torch.from_numpy(sx).to(dev()),
                          scale_mode=mode, out_kind=out_kind, workspace=workspace)
    torch.cuda.synchronize()
    if out_kind == w.OUT_BF16:
        return to_np_bits(y)
    return y.cpu().numpy()


def check_all_outputs(x_bits, W, s, *, group, codes=False, ref=None, rows=None, label="", wp=None):
    """Run I32 / F32 / BF16 outputs and compare with the oracle.
    rows: optional index array; only those token rows are compared (the
    oracle computes just them, rows being independent).  wp: W already
    packed on the device (packed here otherwise)."""
    M, K = x_bits.shape
    N = W.shape[0]
    print(f"[case] {label} M={M} K={K} N={N} group={group} codes={codes} "
          f"plan={w.w4a8_linear_describe(M, N, K, int(group), int(codes))}", flush=True)
    if ref is None:
        xs = x_bits if rows is None else x_bits[rows]
        ref = oracle.linear(xs, W, s_w=None if group else s, s_g=s if group else None, nthreads=NTHREADS)
    if wp is None:
        wp = pack(W)
    cq = None
    if codes:
        qq, ss = oracle.quantize_act(x_bits)
        cq = (qq, ss)
    sel = slice(None) if rows is None else rows
    acc = run_linear(x_bits, wp, s, N, group=group, out_kind=w.OUT_I32_ACC, codes=cq)
    np.testing.assert_array_equal(acc[sel], ref["acc"], err_msg=f"{label}: int32 accumulator")
    y32 = run_linear(x_bits, wp, s, N, group=group, out_kind=w.OUT_F32, codes=cq)
    yb = run_linear(x_bits, wp, s, N, group=group, out_kind=w.OUT_BF16, codes=cq)
    y32, yb = y32[sel], yb[sel]
    record_errors(label, (M, K, N), group, (yb.astype(np.uint32) << 16).view(np.float32), ref["y64"])
    if not group:
        np.testing.assert_array_equal(y32.view(np.uint32), ref["y32"].view(np.uint32),
                                      err_msg=f"{label}: fp32 dequant")
        np.testing.assert_array_equal(yb, ref["y"], err_msg=f"{label}: bf16 output")
        ybf = (yb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        assert np.all(np.abs(ybf - ref["y64"]) <= REL * np.abs(ref["y64"])), label
    else:
        ybf = (yb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        err = np.abs(ybf - ref["y64"])
        bound = REL * np.abs(ref["y64"]) + GROUP_FLOOR * ref["bound"]
        bad = err > bound
        assert not bad.any(), f"{label}: {bad.sum()} bf16 outputs outside tolerance, max err {err.max()}"
        err32 = np.abs(y32.astype(np.float64) - ref["y64"])
        assert np.all(err32 <= 1e-5 * np.abs(ref["y64"]) + GROUP_FLOOR * ref["bound"]), label
    return ref
