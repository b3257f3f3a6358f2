"""Parity of the flow-matching Euler step with the velocity cache
(w4a8_flow_step) with the oracle.

The state update and the cache are bit-exact (the same two fp32 IEEE
operations on both sides).  The four row sums are fp64 on both sides over
the same fp64 terms, in a different order; the rounding of a sum of n terms
is bounded by (n - 1) 2^-53 times the sum of their magnitudes, so the test
allows (n + 8) 2^-52 sum |term|."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I

pytestmark = pytest.mark.gpu


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda:0").view(torch.bfloat16)


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def stat_bound(v_bits, c_bits):
    v = oracle._f32(v_bits).astype(np.float64)
    c = oracle._f32(c_bits).astype(np.float64)
    n = v.shape[1]
    mags = np.stack([np.abs(v * c).sum(1), (v * v).sum(1), (c * c).sum(1), ((v - c) ** 2).sum(1)], axis=1)
    return (n + 8) * 2.0 ** -52 * mags


def check_step(x0, v_bits, c_bits, dt, stats, label, rows=None):
    B, n = x0.shape
    print(f"[case] flow step {label} B={B} n={n} fresh={v_bits is not None} stats={stats}", flush=True)
    x = torch.from_numpy(x0).to("cuda:0")
    c = dev_bf16(c_bits)
    v = None if v_bits is None else dev_bf16(v_bits)
    st = w.w4a8_flow_step(x, v, c, dt, stats=stats)
    torch.cuda.synchronize()
    xg, cg = x.cpu().numpy(), host_bits(c)
    sel = slice(None) if rows is None else rows
    xo, co, so = oracle.flow_step(x0[sel], None if v_bits is None else v_bits[sel], c_bits[sel], dt)
    np.testing.assert_array_equal(xg[sel].view(np.uint32), xo.view(np.uint32), err_msg=f"{label}: x")
    np.testing.assert_array_equal(cg[sel], co, err_msg=f"{label}: cache")
    if stats:
        sg = st.cpu().numpy()[sel]
        bound = stat_bound(v_bits[sel], c_bits[sel])
        assert (np.abs(sg - so) <= bound).all(), f"{label}: stats off by {np.max(np.abs(sg - so) - bound)}"
    else:
        assert st is None


# the paper's shape (6 samples x 64 waypoints x 2), the 16-byte path with
# one, several and a ragged last pass, the one-element path on ragged rows
SHAPES = [(6, 128, 1), (1, 1, 2), (1, 3, 3), (3, 1000, 4), (5, 8, 5), (4, 2056, 6), (2, 4104, 7), (257, 2048, 8),
          (7, 16383, 9), (64, 16384, 10), (1000, 129, 11), (16384, 8, 12)]


@pytest.mark.parametrize("B,n,seed", SHAPES)
@pytest.mark.parametrize("mode", ["fresh_stats", "fresh", "reuse"])
def test_flow_step_parity(B, n, seed, mode):
    x0 = I.flow_state(B, n, seed)
    c = I.flow_velocity(B, n, seed + 100)
    v = None if mode == "reuse" else I.flow_velocity(B, n, seed + 200)
    check_step(x0, v, c, 0.125, mode == "fresh_stats", f"{mode} seed={seed}")


def test_flow_step_odd_dt_and_equal_buffers():
    # dt = 0.1 (inexact products), and v_new aliasing the cache: stats of v against itself
    B, n = 6, 128
    x0 = I.flow_state(B, n, 31)
    c = I.flow_velocity(B, n, 32)
    check_step(x0, I.flow_velocity(B, n, 33), c, np.float32(0.1), True, "dt=0.1")
    x = torch.from_numpy(x0).to("cuda:0")
    cd = dev_bf16(c)
    st = w.w4a8_flow_step(x, cd, cd, 0.1, stats=True).cpu().numpy()
    xo, _, so = oracle.flow_step(x0, c, c, 0.1)
    np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), xo.view(np.uint32))
    assert (st[:, 3] == 0).all() and (np.abs(st - so) <= stat_bound(c, c)).all()


def test_flow_step_full_size_sampled_rows():
    # the bandwidth shape of the benchmark, 16384 x 2048, rows sampled for the oracle
    B, n = 16384, 2048
    x0 = I.flow_state(B, n, 41)
    c = I.flow_velocity(B, n, 42)
    v = I.flow_velocity(B, n, 43)
    rows = np.arange(0, B, 97)
    check_step(x0, v, c, 0.125, True, "full size", rows=rows)


@pytest.mark.parametrize("B,n,seed", [(6, 128, 71), (3, 1000, 72), (257, 2048, 73)])
@pytest.mark.parametrize("repeat", [2, 5])
@pytest.mark.parametrize("fresh", [True, False])
def test_flow_step_repeat_equals_separate_steps(B, n, seed, repeat, fresh):
    print(f"[case] flow step repeat={repeat} fresh={fresh} B={B} n={n}", flush=True)
    x0 = I.flow_state(B, n, seed)
    c = I.flow_velocity(B, n, seed + 100)
    v = I.flow_velocity(B, n, seed + 200) if fresh else None
    x = torch.from_numpy(x0).to("cuda:0")
    cd = dev_bf16(c)
    st = w.w4a8_flow_step(x, None if v is None else dev_bf16(v), cd, 0.125, stats=fresh, repeat=repeat)
    torch.cuda.synchronize()
    xo, co, so = oracle.flow_step(x0, v, c, 0.125)
    for _ in range(repeat - 1):
        xo, co, _ = oracle.flow_step(xo, None, co, 0.125)
    np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), xo.view(np.uint32))
    np.testing.assert_array_equal(host_bits(cd), co)
    if fresh:
        assert (np.abs(st.cpu().numpy() - so) <= stat_bound(v, c)).all()


def test_flow_step_empty_batch():
    c = torch.zeros((0, 8), dtype=torch.bfloat16, device="cuda:0")
    x = torch.zeros((0, 8), dtype=torch.float32, device="cuda:0")
    assert w.w4a8_flow_step(x, c, c, 0.125, stats=True).shape == (0, 4)


def _velocity(x, t):
    """A deterministic stand-in for the action network: bf16 of a smooth
    function of the state and time, evaluated on the host for both sides."""
    return I.to_bf16_bits(np.tanh(0.5 * x).astype(np.float32) * np.float32(1.0 + 2.0 * (t - 0.5) ** 2)
                          + np.float32(t))


def runs(fresh):
    """(step, repeat) per evaluated step: the step and the reused steps after it."""
    out = []
    for i, f in enumerate(fresh):
        if f:
            out.append([i, 1])
        else:
            out[-1][1] += 1
    return out


@pytest.mark.parametrize("B,n,n_reuse", [(6, 128, 4), (33, 1000, 4), (8, 4096, 3), (6, 128, 7)])
def test_flow_solve_fused_runs(B, n, n_reuse):
    # one call per evaluated step, its reused steps folded in with repeat
    print(f"[case] flow solve fused runs B={B} n={n} steps=8 reuse={n_reuse}", flush=True)
    n_steps = 8
    x0 = I.flow_state(B, n, 52)
    xo, _, stats_o = oracle.flow_solve(x0, _velocity, n_steps, n_reuse)
    x = torch.from_numpy(x0).to("cuda:0")
    cache = torch.zeros((B, n), dtype=torch.bfloat16, device="cuda:0")
    c_host = np.zeros((B, n), np.uint16)
    dt = np.float32(1.0) / np.float32(n_steps)
    rs = runs(w.w4a8_flow_schedule(n_steps, n_reuse))
    assert len(rs) == n_steps - n_reuse and sum(r for _, r in rs) == n_steps
    for k, (i, r) in enumerate(rs):
        vb = _velocity(x.cpu().numpy(), i / n_steps)
        st = w.w4a8_flow_step(x, dev_bf16(vb), cache, dt, stats=True, repeat=r).cpu().numpy()
        assert (np.abs(st - stats_o[k]) <= stat_bound(vb, c_host)).all(), f"run {k}: stats"
        c_host = vb
    np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), xo.view(np.uint32))
    np.testing.assert_array_equal(host_bits(cache), c_host)


@pytest.mark.parametrize("B,n,n_reuse", [(6, 128, 4), (6, 128, 0), (33, 1000, 4), (8, 4096, 3)])
def test_flow_solve_parity(B, n, n_reuse):
    print(f"[case] flow solve B={B} n={n} steps=8 reuse={n_reuse}", flush=True)
    n_steps = 8
    x0 = I.flow_state(B, n, 51)
    xo, states_o, stats_o = oracle.flow_solve(x0, _velocity, n_steps, n_reuse)
    fresh = w.w4a8_flow_schedule(n_steps, n_reuse)
    x = torch.from_numpy(x0).to("cuda:0")
    cache = torch.zeros((B, n), dtype=torch.bfloat16, device="cuda:0")
    c_host = np.zeros((B, n), np.uint16)
    dt = np.float32(1.0) / np.float32(n_steps)
    k = 0
    for i in range(n_steps):
        if fresh[i]:
            vb = _velocity(x.cpu().numpy(), i / n_steps)
            st = w.w4a8_flow_step(x, dev_bf16(vb), cache, dt, stats=True).cpu().numpy()
            assert (np.abs(st - stats_o[k]) <= stat_bound(vb, c_host)).all(), f"step {i}: stats"
            c_host = vb
            k += 1
        else:
            w.w4a8_flow_step(x, None, cache, dt)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), states_o[i].view(np.uint32),
                                      err_msg=f"step {i}")
    assert k == len(stats_o) == n_steps - n_reuse
    np.testing.assert_array_equal(host_bits(cache), c_host)
    np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32), xo.view(np.uint32))
