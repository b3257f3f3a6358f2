"""ctypes front end of the CPU oracle (oracle/oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the package smoke check and
by the CPU-baseline leg of bench.py, never by the product path.  It shares no
code with the HIP sources.  The linear-layer functions follow FlashDrive
Sec. 3.4 (4-bit weights, 8-bit activations, integer contraction) with the
readings stated in oracle.c's header; silu_mul / gated follow Sec. 3.5
(Kernel Fusion) with the SiLU reading stated in silu_mul; rmsnorm_quantize
follows Sec. 3.5 too, streaming_attention Sec. 3.1, and the flow_* functions
(adaptive-step flow matching with its velocity cache) Sec. 3.3.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
GCC_FLAGS = ["-O2", "-ffp-contract=off", "-std=c11", "-fPIC", "-shared", "-pthread"]

OK, EINVAL, ENONFINITE, EOVERFLOW = 0, 1, 2, 3


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (no HIP involved)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(["gcc", *GCC_FLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        L.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_f32.restype = ctypes.c_float
        L.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        L.oracle_f32_to_bf16.restype = ctypes.c_uint16
        L.oracle_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.oracle_f16_to_f32.restype = ctypes.c_float
        L.oracle_quantize_act.argtypes = [P, I64, I64, P, P]
        L.oracle_quantize_act.restype = ctypes.c_int
        L.oracle_linear_q.argtypes = [P, P, I64, I64, P, I64, P, P, ctypes.c_int, P, P, P, P, P]
        L.oracle_linear_q.restype = ctypes.c_int
        L.oracle_linear.argtypes = [P, I64, I64, P, I64, P, P, ctypes.c_int, P, P, P, P, P, P, P]
        L.oracle_linear.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != OK:
        raise ValueError(f"oracle {what} failed with code {rc}")


def bf16_to_f32(bits: int) -> float:
    return lib().oracle_bf16_to_f32(int(bits))


def f32_to_bf16(v: float) -> int:
    return lib().oracle_f32_to_bf16(float(v))


def f16_to_f32(bits: int) -> float:
    return lib().oracle_f16_to_f32(int(bits))


def quantize_act(x_bits: np.ndarray):
    """x_bits: uint16 bf16 patterns [M][K] -> (q int8 [M][K], s fp32 [M])."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    M, K = x.shape
    q = np.empty((M, K), np.int8)
    s = np.empty((M,), np.float32)
    _check(lib().oracle_quantize_act(_ptr(x), M, K, _ptr(q), _ptr(s)), "quantize_act")
    return q, s


def linear_q(q, s_x, w, s_w=None, s_g=None, nthreads=1):
    """Linear layer on pre-quantized activations.  Returns a dict with
    acc (int32), y32 (fp32), y (bf16 bits), y64 (fp64), bound (fp64)."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    s_x = np.ascontiguousarray(s_x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.int8)
    M, K = q.shape
    N = w.shape[0]
    assert w.shape == (N, K)
    sw = None if s_w is None else np.ascontiguousarray(s_w, dtype=np.float32)
    sg = None if s_g is None else np.ascontiguousarray(s_g).view(np.uint16)
    out = dict(acc=np.empty((M, N), np.int32), y32=np.empty((M, N), np.float32),
               y=np.empty((M, N), np.uint16), y64=np.empty((M, N), np.float64),
               bound=np.empty((M, N), np.float64))
    rc = lib().oracle_linear_q(_ptr(q), _ptr(s_x), M, K, _ptr(w), N, _ptr(sw), _ptr(sg),
                               int(nthreads), _ptr(out["acc"]), _ptr(out["y32"]), _ptr(out["y"]),
                               _ptr(out["y64"]), _ptr(out["bound"]))
    _check(rc, "linear_q")
    return out


def linear(x_bits, w, s_w=None, s_g=None, nthreads=1):
    """The whole path from bf16 activations.  Returns linear_q's dict plus
    q (int8 [M][K]) and s_x (fp32 [M])."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    w = np.ascontiguousarray(w, dtype=np.int8)
    M, K = x.shape
    N = w.shape[0]
    assert w.shape == (N, K)
    sw = None if s_w is None else np.ascontiguousarray(s_w, dtype=np.float32)
    sg = None if s_g is None else np.ascontiguousarray(s_g).view(np.uint16)
    out = dict(q=np.empty((M, K), np.int8), s_x=np.empty((M,), np.float32),
               acc=np.empty((M, N), np.int32), y32=np.empty((M, N), np.float32),
               y=np.empty((M, N), np.uint16), y64=np.empty((M, N), np.float64),
               bound=np.empty((M, N), np.float64))
    rc = lib().oracle_linear(_ptr(x), M, K, _ptr(w), N, _ptr(sw), _ptr(sg), int(nthreads),
                             _ptr(out["q"]), _ptr(out["s_x"]), _ptr(out["acc"]), _ptr(out["y32"]),
                             _ptr(out["y"]), _ptr(out["y64"]), _ptr(out["bound"]))
    _check(rc, "linear")
    return out


def silu_mul(g, u):
    """silu(g) * u in fp64, with silu(g) = g / (1 + e^-g).

    The gated activation merged into the fused gate+up projection.
    FlashDrive Sec. 3.5 (Kernel Fusion) fuses the MLP's gate and up
    projections into one GEMM and merges the element-wise operations after
    it, without naming the activation; SiLU gating is this oracle's reading.
    """
    g = np.asarray(g, np.float64)
    u = np.asarray(u, np.float64)
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g)) * u


def gated(out):
    """The gated output of a linear() / linear_q() result whose weight holds
    the gate rows [0, N/2) followed by the up rows [N/2, N).

    Returns y64 (silu_mul of the fp64 gate and up values), y_of32 (silu_mul
    of their fp32 values y32, the values the per-channel kernel holds before
    its fp32 activation), and the halves' fp64 values and error bounds."""
    F = out["y64"].shape[1] // 2
    g64, u64 = out["y64"][:, :F], out["y64"][:, F:]
    g32, u32 = out["y32"][:, :F], out["y32"][:, F:]
    return dict(y64=silu_mul(g64, u64), y_of32=silu_mul(g32, u32), g64=g64, u64=u64,
                g_bound=out["bound"][:, :F], u_bound=out["bound"][:, F:])


def rmsnorm_quantize(x_bits, gamma_bits, eps):
    """RMSNorm of each token row followed by the per-token int8 quantize,
    the normalization prologue of a backbone linear.

    FlashDrive Sec. 3.5 (Kernel Fusion) folds the pointwise and row-reduction
    work around its GEMMs into them, without saying which ops those are;
    RMSNorm with a learned bf16 gain is this oracle's reading of the
    normalization.  Per
    row (fp32 IEEE operations unless stated):
        ss = sum_k x_k^2               (exact squares; math.fsum, fp64)
        v  = fl32(ss / K)              (fp64 division, then rounded to fp32)
        r  = 1 / sqrt(v + eps)
        h_k = (x_k * r) * gamma_k
    then the quantize of quantize_act on the fp32 h: a = max_k |h_k|,
    s = a / 127, q_k = round_half_even(h_k / s) clamped to [-127, 127]; an
    all-zero h has s = 0 and q = 0.  Inputs must be finite, eps > 0 (so r is
    finite) and fl32(ss / K) finite; |h_k| <= sqrt(K) |gamma_k| then holds.
    Returns (q int8 [M][K], s fp32 [M], h fp32 [M][K], r fp32 [M]).
    """
    import math

    x = (np.ascontiguousarray(x_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    g = (np.ascontiguousarray(gamma_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    if not (np.isfinite(x).all() and np.isfinite(g).all() and math.isfinite(eps) and np.float32(eps) > 0):
        raise ValueError("rmsnorm_quantize takes finite inputs and eps > 0")
    M, K = x.shape
    assert g.shape == (K,)
    e32 = np.float32(eps)
    q = np.zeros((M, K), np.int8)
    s = np.zeros(M, np.float32)
    h = np.empty((M, K), np.float32)
    r = np.empty(M, np.float32)
    for m in range(M):
        x64 = x[m].astype(np.float64)
        ss = math.fsum(x64 * x64)              # each square is exact in fp64
        v = np.float32(ss / K)
        if not np.isfinite(v):
            raise ValueError("rmsnorm_quantize: mean square beyond the fp32 range")
        rr = np.float32(1.0) / np.sqrt(np.float32(v + e32))
        r[m] = rr
        h[m] = (x[m] * rr) * g
        a = np.float32(np.max(np.abs(h[m])))
        if a == 0:
            continue
        s[m] = a / np.float32(127.0)
        q[m] = np.clip(np.rint(h[m] / s[m]), -127, 127).astype(np.int8)
    return q, s, h, r


def _bf16_round(x32):
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _f32(bits):
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rope_rotate(x_bits, pos, cos_t, sin_t):
    """Rotary embedding of bf16 rows x [N][D] at integer positions pos [N],
    rotate-half pairing (d, d + D/2), angles given by the caller's fp32
    tables cos_t, sin_t [P][D/2]; fp32 IEEE operations, result rounded to
    bf16 (the rotated operands of a bf16 model):
        y_i       = x_i cos - x_{i+D/2} sin
        y_{i+D/2} = x_{i+D/2} cos + x_i sin
    Returns bf16 bit patterns [N][D]."""
    x = _f32(x_bits)
    D = x.shape[1]
    h = D // 2
    c = cos_t[pos].astype(np.float32)
    s = sin_t[pos].astype(np.float32)
    a, b = x[:, :h], x[:, h:]
    y = np.empty_like(x)
    y[:, :h] = (a * c) - (b * s)
    y[:, h:] = (b * c) + (a * s)
    return _bf16_round(y)


def streaming_attention(q_bits, k_bits, v_bits, pos_q, pos_k, cos_t, sin_t, scale):
    """Streaming prefill attention (FlashDrive Sec. 3.1, streaming design):
    queries are the newest frame's tokens, keys and values the whole
    window's cache, keys stored before their rotary embedding and rotated
    here at their current window positions; the streaming mask lets query
    i see key j iff pos_k[j] <= pos_q[i] (causal order of the view-major
    window).

    q [H][Nq][D], k and v [Hkv][Nk][D] bf16 bit patterns (query head h reads
    kv head h // (H / Hkv)); pos_q [Nq], pos_k [Nk] int; tables [P][D/2]
    fp32.  Rotated q and k are rounded to bf16 (rope_rotate); scores,
    softmax and the weighted sum are fp64.  Returns (o64 [H][Nq][D] fp64,
    bnd [H][Nq][D] fp64 = sum_j P_ij |v_jd|, the cancellation-free size of
    each output)."""
    H, Nq, D = q_bits.shape
    Hkv, Nk, _ = k_bits.shape
    G = H // Hkv
    pos_q = np.asarray(pos_q)
    pos_k = np.asarray(pos_k)
    vis = pos_k[None, :] <= pos_q[:, None]                     # [Nq][Nk]
    if not vis.any(axis=1).all():
        raise ValueError("every query must see at least one key")
    o64 = np.empty((H, Nq, D))
    bnd = np.empty((H, Nq, D))
    kr = [_f32(rope_rotate(k_bits[g], pos_k, cos_t, sin_t)).astype(np.float64) for g in range(Hkv)]
    vv = [_f32(v_bits[g]).astype(np.float64) for g in range(Hkv)]
    for h in range(H):
        qr = _f32(rope_rotate(q_bits[h], pos_q, cos_t, sin_t)).astype(np.float64)
        s = (qr @ kr[h // G].T) * float(scale)
        s = np.where(vis, s, -np.inf)
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        o64[h] = p @ vv[h // G]
        bnd[h] = p @ np.abs(vv[h // G])
    return o64, bnd


def rope_tables(P, D, base=10000.0):
    """fp32 cos / sin tables [P][D/2] for angle p * base^(-2i/D), from fp64."""
    i = np.arange(D // 2, dtype=np.float64)
    ang = np.arange(P, dtype=np.float64)[:, None] * base ** (-2.0 * i / D)[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def flow_schedule(n_steps, n_reuse):
    """Which steps of an n_steps flow-matching solve evaluate the velocity
    network (True) and which reuse the cached velocity (False).

    FlashDrive Sec. 3.3 (adaptive caching): the first few and the last few
    steps are evaluated fresh, and n_reuse steps between them take the
    velocity of the step before them, i.e. the last fresh one.  The paper
    does not say how the fresh steps split between the two ends; this
    oracle's reading splits them evenly, the odd one at the start: the first
    ceil((n_steps - n_reuse) / 2) steps and the last floor((n_steps -
    n_reuse) / 2) are fresh.  Step 0 is always fresh (1 <= n_steps, 0 <=
    n_reuse < n_steps).  For the paper's 8 steps with 4 reused: steps 0, 1,
    6 and 7 are fresh, 2 to 5 reuse step 1's velocity."""
    if not (1 <= n_steps and 0 <= n_reuse < n_steps):
        raise ValueError("flow_schedule needs 1 <= n_steps and 0 <= n_reuse < n_steps")
    head = (n_steps - n_reuse + 1) // 2
    return [i < head or i >= head + n_reuse for i in range(n_steps)]


def flow_step(x, v_bits, cache_bits, dt):
    """One explicit Euler step of the flow-matching ODE dx/dt = v (FlashDrive
    Sec. 3.3), with the velocity cache.

    x fp32 [B][n] (the trajectory state), v_bits the fresh velocity as bf16
    bit patterns [B][n] (the action network's output) or None on a step
    that reuses the cache, cache_bits bf16 [B][n] the cached velocity.
    The update is x' = fl32(x + fl32(dt * v)), two fp32 IEEE operations
    (no fused multiply-add), v being the fresh velocity or, on a reused
    step, the cache.  A fresh step also replaces the cache by v and
    returns, per row b, the four sums that give the consecutive-velocity
    measures the paper plots for this section (relative difference and
    cosine similarity, see flow_measures), taken against the cache before
    the step:
        stats[b] = (sum v c, sum v v, sum c c, sum (v - c)^2)
    each term formed in fp64 from the bf16 values and the sum rounded once
    (math.fsum).  Returns (x' fp32, cache' bf16 bits, stats fp64 [B][4] or
    None)."""
    import math

    x = np.ascontiguousarray(x, dtype=np.float32)
    c_bits = np.ascontiguousarray(cache_bits, dtype=np.uint16)
    dt32 = np.float32(dt)
    if v_bits is None:
        vel = _f32(c_bits)
        return (x + dt32 * vel).astype(np.float32), c_bits.copy(), None
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    vel = _f32(v_bits)
    B = x.shape[0]
    v64 = vel.astype(np.float64).reshape(B, -1)
    c64 = _f32(c_bits).astype(np.float64).reshape(B, -1)
    stats = np.empty((B, 4))
    for b in range(B):
        d = v64[b] - c64[b]
        stats[b] = (math.fsum(v64[b] * c64[b]), math.fsum(v64[b] * v64[b]),
                    math.fsum(c64[b] * c64[b]), math.fsum(d * d))
    return (x + dt32 * vel).astype(np.float32), v_bits.copy(), stats


def flow_measures(stats):
    """(relative difference ||v - c|| / ||c||, cosine similarity v.c / (||v|| ||c||))
    per row of flow_step's stats; nan where a norm is zero."""
    s = np.asarray(stats, dtype=np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.sqrt(s[:, 3]) / np.sqrt(s[:, 2])
        cos = s[:, 0] / np.sqrt(s[:, 1] * s[:, 2])
    return rel, cos


def flow_solve(x0, velocity, n_steps, n_reuse):
    """The adaptive-step solve of FlashDrive Sec. 3.3 over t in [0, 1] with
    uniform steps dt = 1 / n_steps: at step i (time t_i = i dt), a fresh
    step calls velocity(x, t_i) -> bf16 bits [B][n] and updates the cache,
    a reused one takes the cache (flow_schedule).  Returns (x after the last
    step, list of per-step states, list of stats per fresh step)."""
    fresh = flow_schedule(n_steps, n_reuse)
    dt = np.float32(1.0) / np.float32(n_steps)
    x = np.ascontiguousarray(x0, dtype=np.float32)
    cache = np.zeros(x.shape, np.uint16)
    states, stats = [], []
    for i in range(n_steps):
        v = velocity(x, i / n_steps) if fresh[i] else None
        x, cache, st = flow_step(x, v, cache, dt)
        states.append(x)
        if st is not None:
            stats.append(st)
    return x, states, stats
