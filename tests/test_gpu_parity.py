"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer results (activation codes, scales, int32 accumulators) and the
per-channel fp32/bf16 outputs must be bit-identical; the group-scale path,
whose fp32 summation order is unspecified, must lie within the tolerance in
helpers.py.  Shapes span several tiles with ragged tails on every axis, the
workload sizes, and the degenerate cases of the method.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I

from helpers import (GROUP_FLOOR, NTHREADS, REL, bf16_dev, check_all_outputs, pack, run_linear,
                     to_np_bits)

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def quant_gpu(x_bits):
    q, s = w.w4a8_quantize_act(bf16_dev(x_bits))
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


# ------------------------------------------------------------ quantize

@pytest.mark.parametrize("M,K,seed", [(4, 256, 1), (16, 4096, 2), (16, 12288, 3), (1024, 4096, 4),
                                      (3, 128, 5), (17, 640, 6), (1000, 384, 7), (2, 65536, 8),
                                      (65, 65536, 9), (301, 12288, 10), (66, 4224, 11),
                                      # every threads-per-row / chunks-per-thread choice of the launcher
                                      (200, 1024, 12), (130, 2048, 13), (8, 8192, 14), (100, 8192, 15),
                                      (5, 2048, 16)])
def test_quantize_bit_exact(M, K, seed):
    print(f"[case] quantize M={M} K={K} seed={seed}", flush=True)
    x = I.activations(M, K, seed)
    q, s = quant_gpu(x)
    qo, so = oracle.quantize_act(x)
    np.testing.assert_array_equal(s.view(np.uint32), so.view(np.uint32))
    np.testing.assert_array_equal(q, qo)


def test_quantize_special_rows():
    print("[case] quantize special rows", flush=True)
    K = 256
    rows = []
    ties = I.to_bf16_bits(np.array([127.0, 0.5, 1.5, 2.5, -2.5, 126.5, -126.5, 3.5] * (K // 8), np.float32))
    rows.append(ties)
    rows.append(np.zeros(K, np.uint16))                         # +0 row
    rows.append(np.full(K, 0x8000, np.uint16))                  # -0 row
    r = rng(9)
    tiny = I.to_bf16_bits(r.standard_normal(K).astype(np.float32) * np.float32(1e-33))
    rows.append(tiny)                                           # absmax below 2^-96: IEEE division path
    denorm = r.integers(1, 0x80, K).astype(np.uint16) | (r.integers(0, 2, K).astype(np.uint16) << 15)
    rows.append(denorm)                                         # bf16 subnormals only
    mixed = I.activations(1, K, 10)[0].copy()
    mixed[::7] = denorm[::7]
    rows.append(mixed)
    big = I.to_bf16_bits(r.standard_normal(K).astype(np.float32) * np.float32(1e30))
    rows.append(big)
    x = np.stack(rows)
    q, s = quant_gpu(x)
    qo, so = oracle.quantize_act(x)
    np.testing.assert_array_equal(s.view(np.uint32), so.view(np.uint32))
    np.testing.assert_array_equal(q, qo)
    assert q[0, :8].tolist() == [127, 0, 2, 2, -2, 126, -126, 4]
    assert not q[1].any() and not q[2].any() and s[1] == 0 and s[2] == 0


def test_quantize_empty():
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    q, s = w.w4a8_quantize_act(x)
    assert q.shape == (0, 256) and s.shape == (0,)


# ------------------------------------------------------------ packing

@pytest.mark.parametrize("v", [1, 7, -8])
@pytest.mark.parametrize("M", [4, 200])
def test_one_hot_rows_select_columns(v, M):
    # pins nibble order, sign extension of -8 and the operand lane maps of
    # both GEMM paths
    print(f"[case] one-hot v={v} M={M}", flush=True)
    K, N = 512, 64
    x = I.activations(M, K, 11)
    r = rng(12)
    W = np.zeros((N, K), np.int8)
    cols = r.integers(0, K, size=N)
    W[np.arange(N), cols] = v
    acc = run_linear(x, pack(W), None, N, group=False, out_kind=w.OUT_I32_ACC)
    q, _ = oracle.quantize_act(x)
    np.testing.assert_array_equal(acc, v * q[:, cols].astype(np.int32))


def test_pack_range_errors():
    W = np.zeros((16, 128), np.int8)
    W[3, 5] = 8
    with pytest.raises(w.W4A8Error) as e:
        pack(W)
    assert e.value.status == w.W4A8_ERANGE
    W[3, 5] = -9
    with pytest.raises(w.W4A8Error):
        pack(W)
    W[3, 5] = -8
    pack(W)  # in range again: the error word was cleared


# ------------------------------------------------------------ linear, per channel

SMALL_SHAPES = [(1, 256, 256), (3, 384, 64), (4, 256, 256), (16, 4096, 1024), (17, 1024, 320),
                (33, 640, 96), (64, 512, 128), (7, 12288, 512), (16, 12288, 256)]


@pytest.mark.parametrize("M,K,N", SMALL_SHAPES)
@pytest.mark.parametrize("codes", [False, True])
def test_small_m_per_channel(M, K, N, codes):
    x = I.activations(M, K, 100 + M)
    W, s = I.weights(N, K, 200 + N)
    check_all_outputs(x, W, s, group=False, codes=codes, label="small-M")


LARGE_SHAPES = [(65, 256, 320), (128, 1024, 192), (300, 640, 1040), (1024, 512, 6144), (257, 4096, 256)]


@pytest.mark.parametrize("M,K,N", LARGE_SHAPES)
@pytest.mark.parametrize("codes", [False, True])
def test_large_m_per_channel(M, K, N, codes):
    x = I.activations(M, K, 300 + M)
    W, s = I.weights(N, K, 400 + N)
    check_all_outputs(x, W, s, group=False, codes=codes, label="large-M")


# ------------------------------------------------------------ linear, group scales

# small-M kernels, then the large-M tiles 64x64 (two accumulator sets) and
# 128x128 (one set, rescale wrapping into the next step), with ragged row
# and column tails and odd step counts
@pytest.mark.parametrize("M,K,N", [(1, 4096, 256), (16, 1024, 384), (5, 12288, 128), (48, 512, 64),
                                   (100, 1024, 192), (256, 1024, 1024), (513, 256, 80),
                                   (1000, 384, 4080), (1500, 256, 2032), (1000, 640, 6128)])
def test_group_scales(M, K, N):
    x = I.activations(M, K, 500 + M)
    W, s = I.weights(N, K, 600 + N, group=True)
    check_all_outputs(x, W, s, group=True, label="group")


# The large-M step loop runs over a 4-stage LDS ring, four steps per
# iteration: every remainder of the step count (K / 128 mod 4), and counts
# below and above one iteration, with each tile size the planner picks
# (64x64 at few tiles, 128x128, 128x192) and ragged row and column tails.
@pytest.mark.parametrize("M,K,N", [(70, 128, 96), (130, 256, 160), (200, 384, 64), (129, 640, 128),
                                   (257, 768, 96), (300, 896, 1040), (65, 1280, 48),
                                   (2048, 128, 4096), (2048, 256, 4096), (2048, 384, 4096), (2048, 640, 4096),
                                   (2000, 768, 4080), (2048, 896, 4096),
                                   (1024, 256, 6144), (1024, 384, 6144), (1024, 1152, 6144)])
@pytest.mark.parametrize("group", [False, True])
def test_large_m_every_ring_remainder(M, K, N, group):
    x = I.activations(M, K, 800 + M)
    W, s = I.weights(N, K, 900 + N, group=group)
    assert "largem" in w.w4a8_linear_describe(M, N, K, int(group))
    check_all_outputs(x, W, s, group=group, label="large-M ring remainder")


@pytest.mark.parametrize("M,K,N", [(70, 65536, 96), (130, 12288, 4096)])
def test_large_m_k_split_long_k(M, K, N):
    # group tiles that fill at most one round run with two k groups of waves
    # merged at the end: the longest K (256 steps per group) and a down
    # projection at a ragged M (sampled rows)
    assert "ksplit" in w.w4a8_linear_describe(M, N, K, 1)
    x = I.activations(M, K, 820 + M)
    W, s = I.weights(N, K, 821 + N, group=True)
    rows = None if N < 1024 else np.arange(0, M, 7)
    check_all_outputs(x, W, s, group=True, rows=rows, label="large-M k split")


# ------------------------------------------------------------ split-K, determinism, workspace reuse

@pytest.mark.parametrize("M,N", [(16, 32), (1, 16)])
def test_split_k_paths_and_reuse(M, N):
    # one or two output tiles over the longest supported K make the planner
    # split K across workgroups (with the quantize separate at M = 16 and
    # fused at M = 1)
    for group in (False, True):
        K = 65536
        desc = w.w4a8_linear_describe(M, N, K, int(group))
        assert "S=1 " not in desc, desc
        assert ("fused-quant" in desc) == (M == 1), desc
        x = I.activations(M, K, 700 + M)
        W, s = I.weights(N, K, 701 + N, group=group)
        ref = check_all_outputs(x, W, s, group=group, label="split-K")
        ws = w.Workspace()
        wp = pack(W)
        outs = [run_linear(x, wp, s, N, group=group, out_kind=w.OUT_BF16, workspace=ws) for _ in range(20)]
        for o in outs[1:]:
            np.testing.assert_array_equal(o, outs[0])
        if not group:
            np.testing.assert_array_equal(outs[0], ref["y"])


def test_repeat_runs_are_identical():
    M, K, N = 1024, 4096, 6144
    x = I.activations(M, K, 702)
    W, s = I.weights(N, K, 703, group=True)
    wp = pack(W)
    first = run_linear(x, wp, s, N, group=True, out_kind=w.OUT_F32)
    for _ in range(5):
        np.testing.assert_array_equal(run_linear(x, wp, s, N, group=True, out_kind=w.OUT_F32).view(np.uint32),
                                      first.view(np.uint32))


# ------------------------------------------------------------ degenerate cases

def test_zero_weights_and_zero_tokens():
    for M in (4, 200):
        K, N = 256, 64
        x = I.activations(M, K, 800)
        x[1] = 0
        W = np.zeros((N, K), np.int8)
        s = np.full(N, 0.01, np.float32)
        yb = run_linear(x, pack(W), s, N, group=False, out_kind=w.OUT_BF16)
        assert not yb.any()
        W2, s2 = I.weights(N, K, 801)
        yb2 = run_linear(x, pack(W2), s2, N, group=False, out_kind=w.OUT_BF16)
        assert not yb2[1].any()


def test_empty_batch():
    wp = pack(np.zeros((64, 256), np.int8))
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    y = w.w4a8_linear(x, wp, torch.ones(64, device="cuda"), 64)
    assert y.shape == (0, 64)


def test_minimum_and_extreme_shapes():
    # smallest legal layer, and the closed-form extreme: x = +-1, W = -8
    for M, K, N in ((1, 128, 16), (2, 12288, 16)):
        xs = np.stack([I.to_bf16_bits(np.ones(K, np.float32)), I.to_bf16_bits(-np.ones(K, np.float32))])[:M]
        W = np.full((N, K), -8, np.int8)
        acc = run_linear(xs, pack(W), None, N, group=False, out_kind=w.OUT_I32_ACC)
        assert (acc[0] == -1016 * K).all()
        if M > 1:
            assert (acc[1] == 1016 * K).all()


def test_nan_and_inf_scales():
    # Non-finite scales propagate as in the reference arithmetic: inf x 0 and
    # NaN inputs give NaN, which the bf16 output writes as 0x7FC0 whatever
    # the input NaN's payload; +-inf scales give +-inf or NaN.
    for M in (8, 300):
        K, N = 256, 96
        x = I.activations(M, K, 901)
        W, s = I.weights(N, K, 902)
        W = W.copy()
        W[5] = 0  # an all-zero channel under an infinite scale: inf x 0
        s = s.copy()
        s_bits = s.view(np.uint32)
        s_bits[3] = 0x7FA12345   # signalling NaN with a payload
        s_bits[7] = 0xFFC00001   # negative quiet NaN with a payload
        s[5] = np.inf
        s[11] = -np.inf
        s[13] = 0.0
        q, sx = oracle.quantize_act(x)
        sx = sx.copy()
        sx.view(np.uint32)[2] = 0x7FC0BEEF
        sx[4] = np.inf
        ref = oracle.linear_q(q, sx, W, s_w=s, nthreads=NTHREADS)
        wp = pack(W)
        yb = run_linear(x, wp, s, N, group=False, out_kind=w.OUT_BF16, codes=(q, sx))
        np.testing.assert_array_equal(yb, ref["y"], err_msg=f"M={M}: bf16 with non-finite scales")
        y32 = run_linear(x, wp, s, N, group=False, out_kind=w.OUT_F32, codes=(q, sx))
        np.testing.assert_array_equal(y32, ref["y32"], err_msg=f"M={M}: fp32 with non-finite scales")
        assert np.isnan(y32[:, 3]).all() and np.isnan(y32[2]).all() and np.isnan(y32[:, 5]).all()


@pytest.mark.parametrize("M", [8, 300, 1024])
def test_token_scales_at_the_epilogue_bounds(M):
    # Token scales on both sides of every bound the large-M epilogue's fast
    # path checks (0, subnormal, 2^-123 / 2^-122, 2^100 / 2^101, negative,
    # near the fp32 maximum) must give the reference bits in every output
    # mode; rows are arranged so that some waves see only in-range scales.
    K, N = 512, 320
    x = I.activations(M, K, 903)
    W, s = I.weights(N, K, 904)
    q, sx = oracle.quantize_act(x)
    sx = sx.copy()
    special = np.array([0.0, 2.0**-130, 2.0**-123, 2.0**-122, 2.0**100, 2.0**101, -2.0**-122, -0.75,
                        3.0e38, 1.5e-30], np.float32)
    rows = np.arange(0, M, max(1, M // 40))[: special.size]
    sx[rows] = special[: rows.size]
    ref = oracle.linear_q(q, sx, W, s_w=s, nthreads=NTHREADS)
    wp = pack(W)
    yb = run_linear(x, wp, s, N, group=False, out_kind=w.OUT_BF16, codes=(q, sx))
    np.testing.assert_array_equal(yb, ref["y"], err_msg=f"M={M}: bf16 at the scale bounds")
    y32 = run_linear(x, wp, s, N, group=False, out_kind=w.OUT_F32, codes=(q, sx))
    np.testing.assert_array_equal(y32.view(np.uint32), ref["y32"].view(np.uint32), err_msg=f"M={M}: fp32")


@pytest.mark.parametrize("group", [False, True])
def test_large_m_longest_k(group):
    # K = 65536 (512 scale groups) on the large-M path: the closed-form
    # extreme x = +-1, W = -8 gives acc = -+1016 K (16 acc stays below 2^31),
    # and random rows match the oracle.
    M, K, N = 80, 65536, 64
    xs = np.stack([I.to_bf16_bits(np.ones(K, np.float32)), I.to_bf16_bits(-np.ones(K, np.float32))])
    x = I.activations(M, K, 905)
    x[:2] = xs
    W, s = I.weights(N, K, 906, group=group)
    W = W.copy()
    W[:8] = -8
    assert "largem" in w.w4a8_linear_describe(M, N, K, int(group))
    ref = check_all_outputs(x, W, s, group=group, label="large-M K=65536")
    assert (ref["acc"][0, :8] == -1016 * K).all() and (ref["acc"][1, :8] == 1016 * K).all()
