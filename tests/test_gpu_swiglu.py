"""Parity of the gated gate+up projection (w4a8_linear_swiglu) with the
oracle's gated output, silu(g) * u, of its gate and up halves.

Per-channel scales: the kernel's fp32 gate and up values are the oracle's
y32 bit for bit (the same op order as w4a8_linear), so the output is
compared with silu_mul of those fp32 values.  Its own error comes from the
fast e^-g, computed as 2^(-g log2 e): the rounded product (and constant)
shift the exponent by up to 2 |g| 2^-24 log2 e, a relative error of
|g| 2^-23 in e^-g, plus about one ulp (2^-23) from the 2^t instruction;
then one add, one divide and one multiply in fp32 (2^-24 each), and the
final bf16 rounding (2^-8).  In all, relative 2^-23 (|g| + 4) before the
bf16 rounding.  Below 2^-110 (|u| + 1) differences are absolute: for
g < -88, e^-g leaves the fp32 range and the kernel's silu(g) is exactly 0,
while the true value is under 10^-36 |u|.  Group scales: the fp32
gate and up values carry the linear layer's group tolerance, which is
propagated through silu(g) * u (|silu'| <= 1.1) against the fp64 values.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I
from helpers import GROUP_FLOOR, NTHREADS, REL, bf16_dev, dev, pack, record_errors, scales_dev, to_np_bits

pytestmark = pytest.mark.gpu

BF16_REL = 2.0 ** -8


def floor(u):
    return 2.0 ** -110 * (np.abs(u) + 1.0)


def f32_rel(g):
    return 2.0 ** -23 * (np.abs(g) + 4.0)


def run(x_bits, wp, s, N, *, group, out_kind, codes=None, workspace=None):
    mode = w.SCALE_GROUP_F16 if group else w.SCALE_CHANNEL_F32
    if codes is None:
        y = w.w4a8_linear_swiglu(bf16_dev(x_bits), wp, scales_dev(s), N, scale_mode=mode, out_kind=out_kind,
                                 workspace=workspace)
    else:
        q, sx = codes
        y = w.w4a8_linear_swiglu(torch.from_numpy(q).to(dev()), wp, scales_dev(s), N,
                                 x_scale=torch.from_numpy(sx).to(dev()), scale_mode=mode, out_kind=out_kind,
                                 workspace=workspace)
    torch.cuda.synchronize()
    if out_kind == w.OUT_BF16:
        return (to_np_bits(y).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return y.cpu().numpy().astype(np.float64)


def check(M, F, K, group, codes, seed, label, rows=None):
    """rows: optional token rows to compare (the oracle computes only those;
    rows are independent)."""
    N = 2 * F
    x = I.activations(M, K, seed)
    W, s = I.weights(N, K, seed + 1, group)
    print(f"[case] swiglu {label} M={M} K={K} N={N} group={group} codes={codes} "
          f"plan={w.w4a8_linear_swiglu_describe(M, N, K, int(group), int(codes))}", flush=True)
    xs = x if rows is None else x[rows]
    ref = oracle.linear(xs, W, s_w=None if group else s, s_g=s if group else None, nthreads=NTHREADS)
    gt = oracle.gated(ref)
    wp = pack(W)
    cq = oracle.quantize_act(x) if codes else None
    y32 = run(x, wp, s, N, group=group, out_kind=w.OUT_F32, codes=cq)
    yb = run(x, wp, s, N, group=group, out_kind=w.OUT_BF16, codes=cq)
    assert y32.shape == (M, F) and yb.shape == (M, F)
    if rows is not None:
        y32, yb = y32[rows], yb[rows]
    # (the relative-error report leaves out outputs under the absolute floor)
    big = np.abs(gt["y64"]) > floor(gt["u64"])
    record_errors(f"swiglu {label}", (M, K, N), group, yb[big], gt["y64"][big])
    if not group:
        ref32 = gt["y_of32"]
        r32 = f32_rel(ref["y32"][:, :F].astype(np.float64))
        fl = floor(ref["y32"][:, F:].astype(np.float64))
        e32 = np.abs(y32 - ref32)
        bad = e32 > r32 * np.abs(ref32) + fl
        assert not bad.any(), f"{label}: {bad.sum()} fp32 outputs, e.g. {y32[bad][:3]} against {ref32[bad][:3]}"
        eb = np.abs(yb - ref32)
        assert np.all(eb <= (BF16_REL + r32) * np.abs(ref32) + fl), f"{label}: bf16 output"
    else:
        sil = np.abs(oracle.silu_mul(gt["g64"], 1.0))
        au = np.abs(gt["u64"])
        for y, rel, what in ((yb, REL, "bf16"), (y32, 1e-5, "fp32")):
            tg = rel * np.abs(gt["g64"]) + GROUP_FLOOR * gt["g_bound"]
            tu = rel * au + GROUP_FLOOR * gt["u_bound"]
            bound = (1.1 * au * tg + sil * tu + 1.1 * tg * tu +
                     (BF16_REL + f32_rel(gt["g64"])) * np.abs(gt["y64"]) + floor(au))
            err = np.abs(y - gt["y64"])
            bad = err > bound
            assert not bad.any(), f"{label}: {bad.sum()} {what} outputs outside tolerance"


@pytest.mark.parametrize("group", [False, True])
@pytest.mark.parametrize("M", [1, 16])
def test_gate_up_verify(M, group):
    # the fused gate+up projection of the verify / decode step: 2 x 12288 x 4096
    check(M, 12288, 4096, group, False, 300 + M, "gate+up")


@pytest.mark.parametrize("group", [False, True])
def test_gate_up_prefill(group):
    # the same projection at prefill size (large-M kernel), 64 sampled rows
    rows = np.sort(np.random.Generator(np.random.PCG64(330)).choice(1024, 64, replace=False))
    check(1024, 12288, 4096, group, False, 331, "gate+up prefill", rows=rows)


def test_wide_gated_tile_ragged():
    # the 128 x 256 gated tile (128 output columns) with a ragged last row
    # tile (1000 = 7 x 128 + 104) and a half-full last column tile (12224 =
    # 95 x 128 + 64); sampled rows include the last row tile
    M, F, K = 1000, 12224, 4096
    assert "largem<128x256,channel,swiglu>" in w.w4a8_linear_swiglu_describe(M, 2 * F, K)
    r = np.random.Generator(np.random.PCG64(344))
    rows = np.sort(np.concatenate([r.choice(896, 24, replace=False), r.choice(np.arange(896, 1000), 24, replace=False)]))
    check(M, F, K, False, False, 345, "wide gated tile", rows=rows)


@pytest.mark.parametrize("group", [False, True])
@pytest.mark.parametrize("M,F,K,codes,seed", [
    (65, 48, 256, False, 340),     # just past the small-M path; one ragged 64-column tile
    (200, 80, 640, False, 341),    # ragged rows and a 16-column last tile
    (300, 192, 1024, True, 342),   # int8 codes in
    (129, 1024, 12288, False, 343),
])
def test_large_m_shapes(M, F, K, codes, seed, group):
    check(M, F, K, group, codes, seed, f"M={M} F={F} K={K}")


@pytest.mark.parametrize("group", [False, True])
@pytest.mark.parametrize("M,F,K,codes,seed", [
    (3, 48, 256, False, 310),      # NT=2, ragged rows
    (17, 96, 640, False, 311),     # two 16-row tiles
    (33, 64, 384, True, 312),      # four 16-row tiles, int8 codes in
    (64, 48, 1024, False, 313),    # the largest M
    (2, 6144, 4096, True, 314),    # NT=4
    (1, 2048, 12288, False, 315),  # the down projection's K, quantize launch first
    (4, 2048, 12288, False, 316),
    (1, 16, 32768, False, 320),    # quantize fused into the GEMM (very long K)
    (16, 16, 65536, False, 317),   # split K (S=8), separate quantize
    (1, 16, 65536, False, 318),    # split K with the fused quantize
    (16, 16, 65536, True, 319),
])
def test_shapes(M, F, K, codes, seed, group):
    check(M, F, K, group, codes, seed, f"M={M} F={F} K={K}")


def test_gate_half_zero_gives_zero_and_sign_of_up_half():
    # gate weights zero: silu(0) = 0 for every output, exactly
    M, F, K = 5, 64, 512
    x = I.activations(M, K, 320)
    W, s = I.weights(2 * F, K, 321)
    W[:F] = 0
    y = run(x, pack(W), s, 2 * F, group=False, out_kind=w.OUT_F32)
    assert not y.any()


def test_swiglu_repeated_calls_share_a_workspace():
    # split-K counters are left at zero: two calls on one workspace agree
    M, F, K = 16, 16, 65536
    x = I.activations(M, K, 322)
    W, s = I.weights(2 * F, K, 323)
    wp = pack(W)
    ws = w.Workspace(dev())
    a = run(x, wp, s, 2 * F, group=False, out_kind=w.OUT_F32, workspace=ws)
    b = run(x, wp, s, 2 * F, group=False, out_kind=w.OUT_F32, workspace=ws)
    np.testing.assert_array_equal(a, b)


def test_empty_and_rejected_calls():
    x = torch.empty((0, 256), dtype=torch.bfloat16, device=dev())
    W, s = I.weights(64, 256, 324)
    wp = pack(W)
    y = w.w4a8_linear_swiglu(x, wp, scales_dev(s), 64)
    assert y.shape == (0, 32)
    xb = bf16_dev(I.activations(65, 256, 325))
    W48, s48 = I.weights(48, 256, 326)
    with pytest.raises(w.W4A8Error) as e:
        w.w4a8_linear_swiglu(xb[:4], pack(W48), scales_dev(s48), 48)   # N % 32 != 0
    assert e.value.status == w.W4A8_EINVAL
