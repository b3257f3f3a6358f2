"""Parity of the fused RMSNorm + int8 quantize prologue
(w4a8_rmsnorm_quantize_act) with the oracle: codes and scales bit for bit.

The oracle sums the exact squares with math.fsum; the kernel sums them in
fp64 in its own fixed order.  Both round the mean square to fp32 from fp64,
so they agree unless ss / K lies within a few fp64 ulps of an fp32
rounding boundary (about 2^-26 of rows); every other step is the same IEEE
fp32 operation on both sides."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I
from helpers import bf16_dev, dev, pack, scales_dev

pytestmark = pytest.mark.gpu


def norm_gpu(x_bits, g_bits, eps):
    q, s = w.w4a8_rmsnorm_quantize_act(bf16_dev(x_bits), bf16_dev(g_bits), eps)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def check(x, g, eps, label):
    M, K = x.shape
    print(f"[case] rmsnorm+quantize {label} M={M} K={K} eps={eps}", flush=True)
    q, s = norm_gpu(x, g, eps)
    qo, so, _, _ = oracle.rmsnorm_quantize(x, g, eps)
    np.testing.assert_array_equal(s.view(np.uint32), so.view(np.uint32), err_msg=f"{label}: scales")
    np.testing.assert_array_equal(q, qo, err_msg=f"{label}: codes")


# every threads-per-row / chunks-per-thread choice of the launcher, the
# re-read of rows longer than the register cache, ragged row counts
@pytest.mark.parametrize("M,K,seed", [(1, 4096, 1), (16, 4096, 2), (16, 12288, 3), (1024, 4096, 4), (3, 128, 5),
                                      (200, 1024, 6), (130, 2048, 7), (8, 8192, 8), (100, 8192, 9), (2, 65536, 10),
                                      (65, 65536, 11), (301, 12288, 12), (5, 640, 13)])
@pytest.mark.parametrize("eps", [1e-6, 1e-5])
def test_rmsnorm_quantize_bit_exact(M, K, seed, eps):
    x = I.activations(M, K, 500 + seed)
    g = I.activations(1, K, 600 + seed, outliers=False)[0]
    check(x, g, eps, "random gain")


def test_unit_gain_and_special_rows():
    K = 1024
    r = np.random.Generator(np.random.PCG64(700))
    rows = [np.zeros(K, np.float32),                                   # all zero: s = 0, q = 0
            r.standard_normal(K).astype(np.float32) * np.float32(1e-20),  # mean square far below eps
            r.standard_normal(K).astype(np.float32) * np.float32(1e18),   # mean square near 1e36
            np.full(K, 2.0 ** -7, np.float32),                         # constant row
            np.where(r.random(K) < 0.25, 2.0, 0.0).astype(np.float32)]  # mean square exactly 1
    x = I.to_bf16_bits(np.stack(rows))
    for g in (I.to_bf16_bits(np.ones(K, np.float32)), I.activations(1, K, 701, outliers=False)[0]):
        check(x, g, 1e-6, "special rows")
    q, s = norm_gpu(x, I.to_bf16_bits(np.ones(K, np.float32)), 1e-6)
    assert s[0] == 0 and not q[0].any()


def test_feeds_the_linear_as_int8_input():
    # the prologue's codes and scales through the GEMM equal the oracle's
    # linear on the oracle's codes, bit for bit (per-channel scales)
    M, K, N = 16, 4096, 512
    x = I.activations(M, K, 702)
    g = I.activations(1, K, 703, outliers=False)[0]
    W, sw = I.weights(N, K, 704)
    qo, so, _, _ = oracle.rmsnorm_quantize(x, g, 1e-6)
    ref = oracle.linear_q(qo, so, W, s_w=sw)
    q, s = w.w4a8_rmsnorm_quantize_act(bf16_dev(x), bf16_dev(g), 1e-6)
    y = w.w4a8_linear(q, pack(W), scales_dev(sw), N, x_scale=s)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.view(torch.int16).cpu().numpy().view(np.uint16), ref["y"])


def test_rejected_calls():
    x = bf16_dev(I.activations(4, 256, 705))
    g = bf16_dev(I.activations(1, 256, 706)[0])
    for eps in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(w.W4A8Error) as e:
            w.w4a8_rmsnorm_quantize_act(x, g, eps)
        assert e.value.status == w.W4A8_EINVAL
    q, s = w.w4a8_rmsnorm_quantize_act(x[:0], g, 1e-6)
    assert q.shape == (0, 256)
