"""Seeded random shapes through every planner branch: M from 1 to ~2000
(small-M tiles, fused or separate quantize, K splits, every large-M tile),
N any multiple of 16, K any multiple of 128, both scale modes, bf16 or int8
input, each checked against the oracle like the fixed-shape parity tests."""
import numpy as np
import pytest

import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I

from helpers import check_all_outputs

pytestmark = pytest.mark.gpu

MAX_MACS = 2e9  # about 0.1 s of the oracle on 16 threads


def cases(seed=20260812):
    """Strata: small M with any N, K; the fused quantize (M = 1, 2 with
    bf16 input over K = 32768..65536 and few columns); K splits (one to four
    column tiles over a very long K); large M over few or many columns, so
    that every tile of the menu is drawn."""
    rng = np.random.Generator(np.random.PCG64(seed))
    any_codes = lambda: bool(rng.integers(0, 2))
    strata = [
        (12, lambda: (int(rng.integers(1, 65)), 128 * int(rng.integers(1, 97)), 16 * int(rng.integers(1, 1537))),
         any_codes),
        (4, lambda: (int(rng.choice([1, 2])), 8192 * int(rng.integers(4, 9)), 16 * int(rng.integers(1, 129))),
         lambda: False),
        (4, lambda: (int(rng.integers(1, 17)), 128 * int(rng.integers(256, 513)), 16 * int(rng.integers(1, 5))),
         any_codes),
        (10, lambda: (int(rng.integers(65, 2100)), 128 * int(rng.integers(1, 33)), 16 * int(rng.integers(8, 1537))),
         any_codes),
        (6, lambda: (int(rng.integers(512, 2049)), 128 * int(rng.integers(1, 5)), 16 * int(rng.integers(256, 1537))),
         any_codes),
    ]
    out = []
    for n, draw, codes in strata:
        got = 0
        while got < n:
            M, K, N = draw()
            if M * N * K > MAX_MACS:
                continue
            out.append((M, K, N, bool(rng.integers(0, 2)), codes(), int(rng.integers(1 << 30))))
            got += 1
    return out


@pytest.mark.parametrize("M,K,N,group,codes,seed", cases())
def test_random_shape(M, K, N, group, codes, seed):
    x = I.activations(M, K, seed)
    W, s = I.weights(N, K, seed + 1, group=group)
    check_all_outputs(x, W, s, group=group, codes=codes,
                      label=f"fuzz {w.w4a8_linear_describe(M, N, K, int(group), int(codes)).split(' workspace')[0][:40]}")


def gated_cases(seed=20260913):
    """Gated gate+up shapes: small M (any even tile count), K splits, and
    large M over both gated tiles (F = N / 2 any multiple of 16)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    any_codes = lambda: bool(rng.integers(0, 2))
    strata = [
        (8, lambda: (int(rng.integers(1, 65)), 128 * int(rng.integers(1, 97)), 16 * int(rng.integers(1, 769)))),
        (3, lambda: (int(rng.integers(1, 17)), 128 * int(rng.integers(256, 513)), 16 * int(rng.integers(1, 3)))),
        (7, lambda: (int(rng.integers(65, 2100)), 128 * int(rng.integers(1, 33)), 16 * int(rng.integers(4, 769)))),
    ]
    out = []
    for n, draw in strata:
        got = 0
        while got < n:
            M, K, F = draw()
            if M * 2 * F * K > MAX_MACS:
                continue
            out.append((M, K, F, bool(rng.integers(0, 2)), any_codes(), int(rng.integers(1 << 30))))
            got += 1
    return out


@pytest.mark.parametrize("M,K,F,group,codes,seed", gated_cases())
def test_random_gated_shape(M, K, F, group, codes, seed):
    from test_gpu_swiglu import check
    check(M, F, K, group, codes, seed,
          f"fuzz {w.w4a8_linear_swiglu_describe(M, 2 * F, K, int(group), int(codes)).split(' workspace')[0][:40]}")
