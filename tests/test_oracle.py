"""Pins of the CPU oracle against facts fixed by the mathematics (no GPU).

The paper prints no worked W4A8 example, so each oracle function is pinned
by closed forms, special cases that reduce to a library routine (numpy's
integer matmul, numpy's fp16 decode, torch's bf16 rounding), brute force on
tiny inputs, and invariants chosen so that a dropped term, a wrong sign or
index, or a transposed operand fails at least one test.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2608_12932_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed=0):
    return np.random.Generator(np.random.PCG64(seed))


def bits_of(vals):
    return I.to_bf16_bits(np.asarray(vals, np.float32))


def f32_of_bits(b):
    return (np.asarray(b, np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- formats

def test_bf16_decode_exhaustive():
    b = np.arange(65536, dtype=np.uint32)
    want = (b << 16).view(np.float32)
    L = oracle.lib()
    sel = b[::7]
    got = np.array([L.oracle_bf16_to_f32(int(v)) for v in sel], np.float32)
    w = want[::7]
    fin = ~np.isnan(w)   # a NaN may come back quieted through the C return path
    np.testing.assert_array_equal(got[fin].view(np.uint32), w[fin].view(np.uint32))
    assert np.all(np.isnan(got[~fin]))


def test_bf16_rne_matches_torch_and_ties():
    r = rng(1)
    vals = r.standard_normal(20000).astype(np.float32) * np.float32(1e3)
    vals = np.concatenate([vals, np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0,
                                           3.0e38, 1e-40], np.float32)])
    want = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.f32_to_bf16(float(v)) for v in vals], np.uint16)
    np.testing.assert_array_equal(got, want)
    # 1 + 2^-8 is a tie between 1.0 (even) and 1 + 2^-7: must go to 0x3F80.
    assert oracle.f32_to_bf16(1.00390625) == 0x3F80
    # 1 + 3*2^-8 is a tie between 1+2^-7 (odd) and 1+2^-6 (even): 0x3F82.
    assert oracle.f32_to_bf16(1.01171875) == 0x3F82
    assert oracle.f32_to_bf16(float("nan")) == 0x7FC0


def test_f16_decode_exhaustive():
    b = np.arange(65536, dtype=np.uint16)
    want = b.view(np.float16).astype(np.float32)
    got = np.array([oracle.f16_to_f32(int(v)) for v in b], np.float32)
    fin = np.isfinite(want)
    np.testing.assert_array_equal(got[fin].view(np.uint32), want[fin].view(np.uint32))
    assert np.all(np.isnan(got[np.isnan(want)]))
    assert np.all(got[np.isinf(want)] == want[np.isinf(want)])


# ---------------------------------------------------------------- quantize

def load_ties():
    rows = []
    with open(os.path.join(GOLDEN, "quant_ties.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b = line.split()
            rows.append((float(a), int(b)))
    return rows


def test_quantize_round_half_even_golden():
    rows = load_ties()
    x = bits_of([[v for v, _ in rows]])
    q, s = oracle.quantize_act(x)
    assert s[0] == np.float32(1.0)
    assert q[0].tolist() == [e for _, e in rows]


def test_quantize_zero_row_and_argmax():
    x = I.activations(6, 512, 11)
    x[2] = 0                                 # +0.0 row
    x[4] = 0x8000                            # -0.0 row
    q, s = oracle.quantize_act(x)
    assert s[2] == 0 and s[4] == 0 and not q[2].any() and not q[4].any()
    xf = f32_of_bits(x)
    for m in (0, 1, 3, 5):
        j = int(np.argmax(np.abs(xf[m])))
        assert abs(int(q[m, j])) == 127
        assert np.sign(q[m, j]) == np.sign(xf[m, j])
        assert s[m] == np.float32(np.abs(xf[m]).max()) / np.float32(127.0)


def test_quantize_properties():
    x = I.activations(8, 1024, 12)
    q, s = oracle.quantize_act(x)
    xf = f32_of_bits(x).astype(np.float64)
    assert np.abs(q).max() <= 127
    # nearest-integer property of the code: |x/s - q| <= 1/2 (+ fp32 slack)
    r = xf / s[:, None].astype(np.float64)
    assert np.all(np.abs(r - q) <= 0.5 + 1e-5)
    # negation symmetry
    qn, sn = oracle.quantize_act(x ^ np.uint16(0x8000))
    np.testing.assert_array_equal(sn, s)
    np.testing.assert_array_equal(qn, -q)
    # scaling a row by a power of two leaves the codes unchanged and scales s exactly
    x4 = bits_of(f32_of_bits(x) * np.float32(4.0))
    q4, s4 = oracle.quantize_act(x4)
    np.testing.assert_array_equal(q4, q)
    np.testing.assert_array_equal(s4, s * np.float32(4.0))


def test_quantize_matches_numpy_ieee():
    # numpy's fp32 division and rint implement the same IEEE operations as
    # the oracle's C code, by an independent implementation.
    x = I.activations(16, 4096, 13)
    q, s = oracle.quantize_act(x)
    xf = f32_of_bits(x)
    a = np.abs(xf).max(axis=1)
    s_np = (a / np.float32(127.0)).astype(np.float32)
    q_np = np.clip(np.rint(xf / s_np[:, None]), -127, 127).astype(np.int8)
    np.testing.assert_array_equal(s, s_np)
    np.testing.assert_array_equal(q, q_np)


def test_quantize_rejects_nonfinite():
    x = I.activations(2, 256, 14)
    x[1, 5] = 0x7F80  # +inf
    with pytest.raises(ValueError):
        oracle.quantize_act(x)


# ---------------------------------------------------------------- contraction

def brute_acc(q, w):
    M, K = q.shape
    N = w.shape[0]
    return [[sum(int(q[m][k]) * int(w[n][k]) for k in range(K)) for n in range(N)] for m in range(M)]


@pytest.mark.parametrize("M,N,K", [(1, 1, 128), (3, 5, 128), (8, 8, 256), (2, 7, 384)])
def test_acc_brute_force(M, N, K):
    r = rng(M * 100 + N)
    x = I.activations(M, K, 20 + M)
    W = r.integers(-8, 8, size=(N, K), dtype=np.int8)
    out = oracle.linear(x, W, s_w=np.ones(N, np.float32))
    assert out["acc"].tolist() == brute_acc(out["q"], W)


@pytest.mark.parametrize("M,N,K", [(4, 256, 256), (33, 96, 1024), (16, 64, 12288)])
def test_acc_matches_numpy_matmul(M, N, K):
    x = I.activations(M, K, 30 + M)
    W, sw = I.weights(N, K, 40 + N)
    out = oracle.linear(x, W, s_w=sw, nthreads=3)
    ref = out["q"].astype(np.int64) @ W.astype(np.int64).T
    np.testing.assert_array_equal(out["acc"].astype(np.int64), ref)


def test_zero_weights_give_positive_zero():
    x = I.activations(5, 256, 50)
    W = np.zeros((64, 256), np.int8)
    out = oracle.linear(x, W, s_w=np.full(64, 0.01, np.float32))
    assert not out["acc"].any()
    assert not out["y"].any()                     # +0.0 bf16 pattern
    assert not out["y32"].view(np.uint32).any()
    _, sg = I.weights(64, 256, 51, group=True)
    outg = oracle.linear(x, W, s_g=sg)
    assert not outg["y"].any() and not outg["y32"].view(np.uint32).any()


@pytest.mark.parametrize("v", [1, 7, -8])
def test_one_hot_row_selects_column(v):
    K, N = 384, 16
    x = I.activations(6, K, 60)
    r = rng(61)
    W = np.zeros((N, K), np.int8)
    cols = r.integers(0, K, size=N)
    W[np.arange(N), cols] = v
    out = oracle.linear(x, W, s_w=np.ones(N, np.float32))
    for n in range(N):
        np.testing.assert_array_equal(out["acc"][:, n], v * out["q"][:, cols[n]].astype(np.int32))


@pytest.mark.parametrize("K", [128, 4096, 12288])
def test_closed_form_extremes(K):
    x = np.stack([bits_of(np.ones(K)), bits_of(-np.ones(K))])
    W = np.full((64, K), -8, np.int8)
    out = oracle.linear(x, W, s_w=np.ones(64, np.float32))
    assert (out["q"][0] == 127).all() and (out["q"][1] == -127).all()
    assert (out["acc"][0] == -1016 * K).all()
    assert (out["acc"][1] == 1016 * K).all()


def test_additivity_in_weights():
    K, N = 512, 32
    x = I.activations(4, K, 70)
    r = rng(71)
    W1 = r.integers(-4, 4, size=(N, K), dtype=np.int8)
    W2 = r.integers(-4, 4, size=(N, K), dtype=np.int8)
    one = np.ones(N, np.float32)
    a1 = oracle.linear(x, W1, s_w=one)["acc"].astype(np.int64)
    a2 = oracle.linear(x, W2, s_w=one)["acc"].astype(np.int64)
    a12 = oracle.linear(x, (W1 + W2).astype(np.int8), s_w=one)["acc"].astype(np.int64)
    np.testing.assert_array_equal(a12, a1 + a2)


def test_rejects_out_of_range_weights():
    x = I.activations(1, 128, 72)
    W = np.zeros((4, 128), np.int8)
    W[2, 3] = 8
    with pytest.raises(ValueError):
        oracle.linear(x, W, s_w=np.ones(4, np.float32))


# ---------------------------------------------------------------- dequant

def test_per_channel_y64_exact_rational():
    x = I.activations(3, 256, 80)
    W, sw = I.weights(8, 256, 81)
    out = oracle.linear(x, W, s_w=sw)
    for m in range(3):
        for n in range(8):
            exact = Fraction(int(out["acc"][m, n])) * Fraction(float(out["s_x"][m])) * Fraction(float(sw[n]))
            got = out["y64"][m, n]
            assert abs(Fraction(got) - exact) <= abs(exact) * Fraction(1, 2**52)


def test_bf16_output_is_rne_of_y32():
    x = I.activations(8, 1024, 82)
    W, sw = I.weights(128, 1024, 83)
    out = oracle.linear(x, W, s_w=sw)
    want = torch.from_numpy(out["y32"]).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(out["y"], want)
    rel = np.abs(out["y32"].astype(np.float64) - out["y64"]) / np.maximum(np.abs(out["y64"]), 1e-30)
    assert rel.max() < 2.0 ** -22


def test_scale_linearity_power_of_two():
    x = I.activations(8, 512, 84)
    W, sw = I.weights(64, 512, 85)
    a = oracle.linear(x, W, s_w=sw)
    b = oracle.linear(x, W, s_w=sw * np.float32(2.0))
    np.testing.assert_array_equal(b["y32"], a["y32"] * np.float32(2.0))
    np.testing.assert_array_equal(b["y64"], a["y64"] * 2.0)
    nz = a["y"] & 0x7FFF != 0
    np.testing.assert_array_equal(b["y"][nz], a["y"][nz] + np.uint16(0x80))   # exponent + 1
    # activation scale: doubling x doubles s_x and so y, codes unchanged
    x2 = bits_of(f32_of_bits(x) * np.float32(2.0))
    c = oracle.linear(x2, W, s_w=sw)
    np.testing.assert_array_equal(c["q"], a["q"])
    np.testing.assert_array_equal(c["y32"], a["y32"] * np.float32(2.0))


def test_scale_linearity_general():
    x = I.activations(4, 512, 86)
    W, sw = I.weights(64, 512, 87)
    a = oracle.linear(x, W, s_w=sw)
    b = oracle.linear(x, W, s_w=(sw * np.float32(1.37)).astype(np.float32))
    np.testing.assert_allclose(b["y64"], a["y64"] * 1.37, rtol=1e-6, atol=0)


def test_group_k128_equals_per_channel():
    x = I.activations(6, 128, 88)
    W, sg = I.weights(64, 128, 89, group=True)
    g = oracle.linear(x, W, s_g=sg)
    c = oracle.linear(x, W, s_w=sg[0].astype(np.float32))
    np.testing.assert_array_equal(g["acc"], c["acc"])
    np.testing.assert_array_equal(g["y64"], c["y64"])


def test_group_constant_along_k_equals_per_channel():
    K, N = 1024, 64
    x = I.activations(5, K, 90)
    W, sw16 = I.weights(N, K, 91, group=True)
    per_n = sw16[0]
    sg = np.tile(per_n, (K // 128, 1))
    g = oracle.linear(x, W, s_g=sg)
    c = oracle.linear(x, W, s_w=per_n.astype(np.float32))
    np.testing.assert_allclose(g["y64"], c["y64"], rtol=1e-12, atol=0)


def test_group_indicator_selects_one_group():
    # s_g = 1 on group g0 and 0 elsewhere reduces the group layer to a
    # per-channel layer (unit scales) over the 128 columns of that group.
    K, N = 768, 32
    x = I.activations(4, K, 92)
    W, _ = I.weights(N, K, 93)
    full = oracle.linear(x, W, s_w=np.ones(N, np.float32))
    for g0 in (0, 2, 5):
        sg = np.zeros((K // 128, N), np.float16)
        sg[g0] = 1.0
        g = oracle.linear_q(full["q"], full["s_x"], W, s_g=sg)
        sub = oracle.linear_q(full["q"][:, 128 * g0:128 * (g0 + 1)], np.ones(4, np.float32),
                              W[:, 128 * g0:128 * (g0 + 1)], s_w=np.ones(N, np.float32))
        np.testing.assert_array_equal(g["y64"], sub["acc"].astype(np.float64) * full["s_x"][:, None].astype(np.float64))
    # and the group sum adds up: sum over indicators equals all-ones group scales
    ones = oracle.linear_q(full["q"], full["s_x"], W, s_g=np.ones((K // 128, N), np.float16))
    np.testing.assert_array_equal(ones["acc"], full["acc"])
    np.testing.assert_allclose(ones["y64"], full["acc"] * full["s_x"][:, None].astype(np.float64), rtol=1e-15)


def test_group_bound_dominates():
    x = I.activations(4, 1024, 94)
    W, sg = I.weights(64, 1024, 95, group=True)
    g = oracle.linear(x, W, s_g=sg)
    assert np.all(g["bound"] >= np.abs(g["y64"]) * (1 - 1e-12))
    # a weight row of constant sign against a positive row makes all partials one-signed
    xp = bits_of(np.abs(f32_of_bits(x)) + np.float32(0.5))
    Wp = np.minimum(np.abs(W.astype(np.int16)), 7).astype(np.int8)
    gp = oracle.linear(xp, Wp, s_g=sg)
    np.testing.assert_allclose(gp["bound"], np.abs(gp["y64"]), rtol=1e-12)


def test_threads_do_not_change_results():
    x = I.activations(13, 512, 96)
    W, sg = I.weights(64, 512, 97, group=True)
    a = oracle.linear(x, W, s_g=sg, nthreads=1)
    b = oracle.linear(x, W, s_g=sg, nthreads=5)
    for k in ("acc", "y32", "y", "y64"):
        np.testing.assert_array_equal(a[k], b[k])


# ---------------------------------------------------------------- gated output

def test_silu_mul_special_values():
    g = np.array([0.0, -0.0, 1.0, -3.0, 50.0, -50.0, -800.0, 800.0])
    u = np.array([5.0, 5.0, 0.0, 2.0, 3.0, 3.0, 7.0, 0.5])
    y = oracle.silu_mul(g, u)
    assert y[0] == 0.0 and y[1] == 0.0 and y[2] == 0.0
    assert y[3] == pytest.approx(-3.0 / (1.0 + math.exp(3.0)) * 2.0, rel=1e-15)
    assert y[4] == pytest.approx(150.0, rel=1e-15)              # silu(g) -> g for large g
    assert abs(y[5]) < 1e-18 and y[5] < 0                       # silu(g) -> 0- for very negative g
    assert y[6] == 0.0 and not np.isnan(y[6])                   # e^800 overflows: still exactly 0
    assert y[7] == 400.0


def test_silu_mul_matches_scipy_sigmoid():
    # silu(g) = g * sigmoid(g); scipy's expit is an independent sigmoid
    import scipy.special
    r = rng(90)
    g = np.concatenate([r.standard_normal(2000) * 4, np.linspace(-40, 40, 161)])
    u = r.standard_normal(g.size)
    np.testing.assert_allclose(oracle.silu_mul(g, u), g * scipy.special.expit(g) * u, rtol=2e-15, atol=1e-300)


def test_silu_odd_part_is_identity():
    # silu(g) - silu(-g) = g exactly in the reals: a dropped 1 in the
    # denominator, or a missing factor g, breaks it (a sign slip in e^-g
    # keeps it and is caught by the sigmoid and large-g pins above)
    g = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(oracle.silu_mul(g, 1.0) - oracle.silu_mul(-g, 1.0), g, rtol=1e-14, atol=1e-14)


def test_gated_output_halves_and_composition():
    K, F = 384, 32
    x = I.activations(5, K, 91)
    r = rng(92)
    Wg = r.integers(-7, 8, size=(F, K), dtype=np.int8)    # symmetric range: -Wg is valid too
    Wu = r.integers(-8, 8, size=(F, K), dtype=np.int8)
    sg = (r.random(F) * 0.02 + 0.001).astype(np.float32)
    su = (r.random(F) * 0.02 + 0.001).astype(np.float32)
    s = np.concatenate([sg, su])
    pos = oracle.gated(oracle.linear(x, np.concatenate([Wg, Wu]), s_w=s))
    neg = oracle.gated(oracle.linear(x, np.concatenate([-Wg, Wu]).astype(np.int8), s_w=s))
    g = oracle.linear(x, Wg, s_w=sg)["y64"]
    u = oracle.linear(x, Wu, s_w=su)["y64"]
    # the halves are the separate projections (gate first, then up)
    np.testing.assert_array_equal(pos["g64"], g)
    np.testing.assert_array_equal(pos["u64"], u)
    # odd part of silu: y(Wg) - y(-Wg) = g * u
    np.testing.assert_allclose(pos["y64"] - neg["y64"], g * u, rtol=1e-12, atol=1e-12 * np.abs(g * u).max())
    # a zero gate gives an exactly zero output whatever the up projection
    zero = oracle.gated(oracle.linear(x, np.concatenate([np.zeros_like(Wg), Wu]), s_w=s))
    assert not zero["y64"].any() and not zero["y_of32"].any()


# ---------------------------------------------------------------- norm + quantize prologue

def test_rmsnorm_power_of_two_rows_reduce_to_the_quantize_of_gamma():
    # x_k = c = +-2^j, eps tiny: ss = K c^2, v = c^2, r = 1/|c| (every step
    # exact), so h = sign(c) gamma and the codes are quantize_act(gamma)'s
    K = 384
    g = I.activations(1, K, 95)[0]
    for c in (1.0, -4.0, 2.0 ** -10, 2.0 ** 12):
        x = bits_of(np.full((1, K), c))
        q, s, h, r = oracle.rmsnorm_quantize(x, g, 2.0 ** -126)
        qg, sg = oracle.quantize_act(g[None, :])
        assert r[0] == np.float32(1.0 / abs(c))
        np.testing.assert_array_equal(h[0], np.sign(c) * f32_of_bits(g))
        np.testing.assert_array_equal(q[0], np.sign(c).astype(np.int8) * qg[0])
        assert s[0] == sg[0]


def test_rmsnorm_known_mean_square_and_eps():
    # a quarter of the entries +-2, the rest 0: mean square exactly 1.  With
    # gamma = 1 and eps tiny, r = 1 and the codes are quantize_act(x)'s; with
    # eps = 3, r = 1/2 exactly and the scale halves (eps goes with the mean,
    # under the root)
    K = 512
    r_ = rng(96)
    vals = np.zeros((3, K), np.float32)
    for m in range(3):
        idx = r_.permutation(K)[: K // 4]
        vals[m, idx] = r_.choice([-2.0, 2.0], size=K // 4)
    x = bits_of(vals)
    one = bits_of(np.ones(K))
    q0, s0 = oracle.quantize_act(x)
    q, s, h, r = oracle.rmsnorm_quantize(x, one, 2.0 ** -126)
    assert (r == 1.0).all()
    np.testing.assert_array_equal(q, q0)
    np.testing.assert_array_equal(s, s0)
    q, s, h, r = oracle.rmsnorm_quantize(x, one, 3.0)
    assert (r == 0.5).all()
    np.testing.assert_array_equal(q, q0)
    np.testing.assert_array_equal(s, s0 * np.float32(0.5))


def test_rmsnorm_scale_invariance():
    # x -> 2^j x leaves h unchanged when eps is negligible against the mean
    # square (a wrong power in the root, or a missing one, would not)
    K = 1024
    x = I.activations(4, K, 97)
    g = I.activations(1, K, 98)[0]
    xf = f32_of_bits(x)
    q1, s1, h1, _ = oracle.rmsnorm_quantize(x, g, 2.0 ** -126)
    for j in (-3, 5):
        q2, s2, h2, _ = oracle.rmsnorm_quantize(bits_of(xf * np.float32(2.0 ** j)), g, 2.0 ** -126)
        np.testing.assert_array_equal(h1, h2)
        np.testing.assert_array_equal(q1, q2)
        np.testing.assert_array_equal(s1, s2)


def test_rmsnorm_matches_float64_definition():
    # fp64 reference of the same formula: r within 2 ulp (fp32), codes within
    # one step where the fp32 quotient sits next to a half
    K = 2048
    x = I.activations(8, K, 99)
    g = I.activations(1, K, 100)[0]
    q, s, h, r = oracle.rmsnorm_quantize(x, g, 1e-6)
    xf = f32_of_bits(x).astype(np.float64)
    r64 = 1.0 / np.sqrt((xf * xf).mean(axis=1) + np.float64(np.float32(1e-6)))
    np.testing.assert_allclose(r, r64, rtol=2.5e-7)
    h64 = xf * r64[:, None] * f32_of_bits(g).astype(np.float64)
    np.testing.assert_allclose(h, h64, rtol=5e-7, atol=1e-30)
    q64 = h64 / (np.abs(h64).max(axis=1, keepdims=True) / 127.0)
    assert np.abs(q.astype(np.float64) - q64).max() <= 0.5 + 1e-4


def test_rmsnorm_zero_row_and_rejections():
    K = 256
    x = np.zeros((2, K), np.uint16)
    x[1] = I.activations(1, K, 101)[0]
    g = bits_of(np.ones(K))
    q, s, h, r = oracle.rmsnorm_quantize(x, g, 1e-6)
    assert s[0] == 0 and not q[0].any() and not h[0].any()
    with pytest.raises(ValueError):
        oracle.rmsnorm_quantize(x, g, 0.0)
    bad = x.copy()
    bad[1, 3] = 0x7F80  # +inf
    with pytest.raises(ValueError):
        oracle.rmsnorm_quantize(bad, g, 1e-6)


# ---------------------------------------------------------------- streaming attention

def _attn_inputs(H, Hkv, Nq, Nk, D, seed):
    q = I.activations(H * Nq, D, seed).reshape(H, Nq, D)
    k = I.activations(Hkv * Nk, D, seed + 1).reshape(Hkv, Nk, D)
    v = I.activations(Hkv * Nk, D, seed + 2).reshape(Hkv, Nk, D)
    return q, k, v


def test_rope_rotation_pair_formula_and_norm():
    # rotate-half pairs (i, i + D/2) by the table's angle: a 90 degree turn
    # maps (a, b) to (-b, a); any angle keeps the pair's norm (fp32 + bf16)
    D = 128
    x = I.activations(6, D, 110)
    cos_t = np.zeros((3, D // 2), np.float32)
    sin_t = np.zeros((3, D // 2), np.float32)
    cos_t[0], sin_t[1] = 1.0, 1.0           # position 0: identity; 1: +90 degrees
    cos_t[2], sin_t[2] = np.cos(0.7), np.sin(0.7)
    xf = f32_of_bits(x)
    y0 = f32_of_bits(oracle.rope_rotate(x, np.zeros(6, int), cos_t, sin_t))
    y1 = f32_of_bits(oracle.rope_rotate(x, np.ones(6, int), cos_t, sin_t))
    np.testing.assert_array_equal(y0, xf)
    np.testing.assert_array_equal(y1[:, : D // 2], -xf[:, D // 2:])
    np.testing.assert_array_equal(y1[:, D // 2:], xf[:, : D // 2])
    y2 = f32_of_bits(oracle.rope_rotate(x, np.full(6, 2), cos_t, sin_t)).astype(np.float64)
    n_in = np.hypot(xf[:, : D // 2], xf[:, D // 2:])
    n_out = np.hypot(y2[:, : D // 2], y2[:, D // 2:])
    np.testing.assert_allclose(n_out, n_in, rtol=2 ** -7)


def test_rope_scores_depend_on_relative_position():
    # with exact angles, q(p + d) . k(p' + d) = q(p) . k(p'): shifting every
    # position by the same amount (the streaming window's shift) keeps the
    # scores up to the bf16 rounding of the rotated operands
    D = 128
    cos_t, sin_t = oracle.rope_tables(4096, D)
    q = I.activations(1, D, 111, outliers=False)
    k = I.activations(1, D, 112, outliers=False)
    def score(pq, pk):
        a = f32_of_bits(oracle.rope_rotate(q, np.array([pq]), cos_t, sin_t)).astype(np.float64)
        b = f32_of_bits(oracle.rope_rotate(k, np.array([pk]), cos_t, sin_t)).astype(np.float64)
        return float((a @ b.T)[0, 0])
    mag = float((np.abs(f32_of_bits(q)).astype(np.float64) @ np.abs(f32_of_bits(k)).astype(np.float64).T)[0, 0])
    for pq, pk, d in [(100, 37, 1000), (7, 7, 3000), (500, 0, 64)]:
        assert abs(score(pq, pk) - score(pq + d, pk + d)) <= 2 ** -6 * mag
    assert abs(score(100, 37) - score(100, 38)) > 2 ** -6 * mag  # and it does depend on the offset


def test_attention_without_rotation_or_mask_is_plain_softmax():
    # identity tables and equal positions: every key visible, no rotation ->
    # softmax(q k^T s) v with scipy's softmax
    import scipy.special
    H, Hkv, Nq, Nk, D = 4, 2, 5, 24, 128
    q, k, v = _attn_inputs(H, Hkv, Nq, Nk, D, 113)
    cos_t = np.ones((1, D // 2), np.float32)
    sin_t = np.zeros((1, D // 2), np.float32)
    o, _ = oracle.streaming_attention(q, k, v, np.zeros(Nq, int), np.zeros(Nk, int), cos_t, sin_t, 0.125)
    for h in range(H):
        qf = f32_of_bits(q[h]).astype(np.float64)
        kf = f32_of_bits(k[h // 2]).astype(np.float64)
        vf = f32_of_bits(v[h // 2]).astype(np.float64)
        ref = scipy.special.softmax(qf @ kf.T * 0.125, axis=1) @ vf
        np.testing.assert_allclose(o[h], ref, rtol=1e-12, atol=1e-12)


def test_streaming_mask_hides_later_keys():
    # query i sees key j iff pos_k[j] <= pos_q[i]: values of hidden keys do
    # not matter; one visible key gives exactly its value; permuting key
    # slots together with their positions changes nothing
    H, Hkv, Nq, Nk, D = 2, 1, 4, 16, 128
    q, k, v = _attn_inputs(H, Hkv, Nq, Nk, D, 114)
    cos_t, sin_t = oracle.rope_tables(64, D)
    pos_k = np.arange(Nk) + 10
    pos_q = np.array([10, 13, 20, 25])
    o, _ = oracle.streaming_attention(q, k, v, pos_q, pos_k, cos_t, sin_t, 0.1)
    v2 = v.copy()
    v2[:, pos_k > 20] = I.activations(int((pos_k > 20).sum()), D, 115)
    o2, _ = oracle.streaming_attention(q, k, v2, pos_q, pos_k, cos_t, sin_t, 0.1)
    np.testing.assert_array_equal(o2[:, :3], o[:, :3])   # queries at 10, 13, 20 see none of them
    assert not np.array_equal(o2[:, 3], o[:, 3])
    np.testing.assert_array_equal(o[:, 0], np.broadcast_to(f32_of_bits(v[0, 0]).astype(np.float64), (H, D)))
    perm = rng(116).permutation(Nk)
    o3, _ = oracle.streaming_attention(q, k[:, perm], v[:, perm], pos_q, pos_k[perm], cos_t, sin_t, 0.1)
    np.testing.assert_allclose(o3, o, rtol=1e-12, atol=1e-12)


def test_attention_of_constant_values_is_that_value():
    H, Hkv, Nq, Nk, D = 2, 2, 3, 20, 128
    q, k, _ = _attn_inputs(H, Hkv, Nq, Nk, D, 117)
    row = I.activations(1, D, 118)[0]
    v = np.broadcast_to(row, (Hkv, Nk, D)).copy()
    cos_t, sin_t = oracle.rope_tables(64, D)
    o, bnd = oracle.streaming_attention(q, k, v, np.array([5, 12, 19]), np.arange(Nk), cos_t, sin_t, 0.3)
    np.testing.assert_allclose(o, np.broadcast_to(f32_of_bits(row).astype(np.float64), o.shape), rtol=1e-13)
    np.testing.assert_allclose(bnd, np.abs(o), rtol=1e-13)


# ---- adaptive-step flow matching with the velocity cache (Sec. 3.3)

def test_flow_schedule_paper_case_and_shapes():
    T, F = True, False
    # 8 steps, 4 reused: the first two and the last two evaluated, the middle four reused
    assert oracle.flow_schedule(8, 4) == [T, T, F, F, F, F, T, T]
    assert oracle.flow_schedule(8, 0) == [T] * 8
    assert oracle.flow_schedule(1, 0) == [T]
    assert oracle.flow_schedule(5, 4) == [T, F, F, F, F]
    assert oracle.flow_schedule(8, 3) == [T, T, T, F, F, F, T, T]
    for n in range(1, 13):
        for r in range(n):
            s = oracle.flow_schedule(n, r)
            assert len(s) == n and s[0] and s.count(False) == r
            idx = [i for i, f in enumerate(s) if not f]
            assert idx == list(range(idx[0], idx[0] + r)) if r else True  # one contiguous run
            assert abs(s.index(False) - (n - 1 - idx[-1])) <= 1 if r else True  # centred
    for bad in ((0, 0), (4, 4), (4, -1)):
        with pytest.raises(ValueError):
            oracle.flow_schedule(*bad)


def test_flow_constant_field_integrates_exactly_under_any_schedule():
    # dx/dt = c from t = 0 to 1 gives x0 + c; Euler is exact for a constant
    # field, and a reused velocity equals the fresh one
    x0 = np.full((2, 3), 0.5, np.float32)
    for r in range(8):
        x, _, _ = oracle.flow_solve(x0, lambda x, t: bits_of(np.full(x.shape, 0.75)), 8, r)
        assert (x == np.float32(1.25)).all()


def test_flow_time_field_closed_forms():
    # dx/dt = 2t: fresh Euler sums 2 t_i dt = 1 - 1/n (all values dyadic, so exact)
    vel = lambda x, t: bits_of(np.full(x.shape, 2.0 * t))
    for n in (4, 8, 16):
        x, _, _ = oracle.flow_solve(np.zeros((1, 2), np.float32), vel, n, 0)
        assert (x == np.float32(1 - 1 / n)).all()
    # 8 steps with 2-5 reused: the velocities taken are those of t = 0, 1/8
    # (five times), 6/8 and 7/8 -> (0 + 5 * 0.25 + 1.5 + 1.75) / 8 = 0.5625
    x, states, stats = oracle.flow_solve(np.zeros((1, 2), np.float32), vel, 8, 4)
    assert (x == np.float32(0.5625)).all()
    assert len(stats) == 4 and len(states) == 8
    # a distinct constant per evaluation: 1 + 8t at t = 0, 1/8, 6/8, 7/8 -> (1 + 5 * 2 + 7 + 8) / 8
    x, _, _ = oracle.flow_solve(np.zeros((1, 1), np.float32), lambda x, t: bits_of(np.full(x.shape, 1 + 8 * t)), 8, 4)
    assert x[0, 0] == np.float32(3.25)


def test_flow_step_stats_special_cases():
    c = np.array([[3.0, 4.0]] * 5, np.float32)
    v = np.array([[3.0, 4.0], [6.0, 8.0], [-3.0, -4.0], [4.0, -3.0], [0.0, 0.0]], np.float32)
    x = np.zeros((5, 2), np.float32)
    _, cache, st = oracle.flow_step(x, bits_of(v), bits_of(c), 0.125)
    assert (cache == bits_of(v)).all()
    # (v.c, v.v, c.c, |v - c|^2) by hand
    assert st.tolist() == [[25, 25, 25, 0], [50, 100, 25, 25], [-25, 25, 25, 100], [0, 25, 25, 50], [0, 0, 25, 25]]
    rel, cos = oracle.flow_measures(st)
    assert rel[:4].tolist() == [0.0, 1.0, 2.0, math.sqrt(2.0)] and rel[4] == 1.0
    assert cos[:4].tolist() == [1.0, 1.0, -1.0, 0.0] and np.isnan(cos[4])
    # a reused step leaves the cache and returns no stats
    x2, cache2, st2 = oracle.flow_step(x, None, bits_of(c), 0.5)
    assert st2 is None and (cache2 == bits_of(c)).all() and (x2 == 0.5 * c).all()


def test_flow_stats_match_exact_rational_sums():
    r = rng(41)
    v = bits_of(r.uniform(-4, 4, (3, 37)))
    c = bits_of(r.uniform(-4, 4, (3, 37)))
    _, _, st = oracle.flow_step(np.zeros((3, 37), np.float32), v, c, 0.25)
    vf, cf = oracle._f32(v), oracle._f32(c)
    for b in range(3):
        V = [Fraction(float(a)) for a in vf[b]]
        C = [Fraction(float(a)) for a in cf[b]]
        want = (sum(a * e for a, e in zip(V, C)), sum(a * a for a in V), sum(e * e for e in C),
                sum((a - e) ** 2 for a, e in zip(V, C)))
        assert st[b].tolist() == [float(w) for w in want]


def _round_f32(q: Fraction) -> float:
    """Exact round-to-nearest-even of a rational to fp32 (normal range)."""
    if q == 0:
        return 0.0
    s = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    m = a / Fraction(2) ** (e - 23)                 # in [2^23, 2^24)
    fl = m.numerator // m.denominator
    rem = m - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2):
        fl += 1
    return s * float(Fraction(fl) * Fraction(2) ** (e - 23))


def test_flow_update_rounds_the_product_then_the_sum():
    # x' = fl32(x + fl32(dt v)): checked with exact rational arithmetic; the
    # fused form fl32(x + dt v) differs on some of these inputs
    r = rng(42)
    x = r.uniform(-2, 2, (1, 400)).astype(np.float32)
    v = bits_of(r.uniform(-4, 4, (1, 400)))
    dt = np.float32(0.1)
    out, _, _ = oracle.flow_step(x, v, v, dt)
    vf = oracle._f32(v)
    differ = 0
    for i in range(400):
        p = _round_f32(Fraction(float(dt)) * Fraction(float(vf[0, i])))
        want = _round_f32(Fraction(float(x[0, i])) + Fraction(p))
        fused = _round_f32(Fraction(float(x[0, i])) + Fraction(float(dt)) * Fraction(float(vf[0, i])))
        assert float(out[0, i]) == want
        differ += fused != want
    assert differ > 0
