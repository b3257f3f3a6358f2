"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (bf16 activations in, bf16 out).

Rows of a linear layer are independent, so where the oracle cannot finish
the whole workload in seconds it computes a seeded sample of token rows and
those rows are compared exactly.  Coverage:
  - tiny, gate+up verify and qkv prefill: every output;
  - down verify: every output at M = 1, 4 and 16 on all 36 weight matrices;
  - the group-scale layer, all four matrices: every output at M = 1, 16 and
    256 on all 36 layers, 128 seeded token rows at M = 2048 on all 36
    layers, and every output at M = 2048 on layers 0, 1, 17 and 35.
"""
import numpy as np
import pytest

from paper_2608_12932_amd import inputs as I

from helpers import check_all_outputs, pack

pytestmark = pytest.mark.gpu


def test_tiny():
    x, W, s, K, N = I.workload_inputs("tiny", 4)
    check_all_outputs(x, W, s, group=False, label="tiny M=4 K=256 N=256")


def test_gate_up_verify():
    x, W, s, K, N = I.workload_inputs("gate_up_verify", 16)
    check_all_outputs(x, W, s, group=False, label="gate+up verify M=16 K=4096 N=24576")


def test_qkv_prefill():
    x, W, s, K, N = I.workload_inputs("qkv_prefill", 1024)
    check_all_outputs(x, W, s, group=False, label="qkv prefill M=1024 K=4096 N=6144")


@pytest.mark.parametrize("layer", range(36))
def test_down_verify_every_matrix(layer):
    # each matrix made and packed once, then every output at the three
    # verification batch sizes
    wl = I.WORKLOADS["down_verify"]
    x0, W, s, K, N = I.workload_inputs("down_verify", 1, layer=layer)
    wp = pack(W)
    for M in (1, 4, 16):
        x = x0 if M == 1 else I.activations(M, K, I.seed_x(wl.number, M), wl.outliers)
        check_all_outputs(x, W, s, group=False, wp=wp, label=f"down verify layer {layer}")


def _sampled_rows(M, n, layer):
    return np.sort(np.random.Generator(np.random.PCG64(2608 + 100 * layer + M)).choice(M, n, replace=False))


@pytest.mark.parametrize("layer", range(36))
def test_layer_group_every_layer(layer):
    # the layer's weights made and packed once; every output of the decode,
    # verify and short-prefill sizes (M = 1, 16, 256) and 128 seeded token
    # rows of the long prefill (M = 2048)
    wl = I.WORKLOADS["layer_group"]
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        W, s = I.weights(N, K, I.seed_w(wl.number, layer, name), group=True)
        wp = pack(W)
        for M in (1, 16, 256, 2048):
            x = I.activations(M, K, I.seed_x(wl.number, M), wl.outliers)
            rows = _sampled_rows(M, 128, layer) if M == 2048 else None
            check_all_outputs(x, W, s, group=True, rows=rows, wp=wp,
                              label=f"layer {layer} {name}" + ("" if rows is None else " (128 sampled rows)"))


@pytest.mark.parametrize("layer", [0, 1, 17, 35])
def test_layer_group_2048_every_row(layer):
    M = 2048
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        x, W, s, K, N = I.workload_inputs("layer_group", M, layer=layer, mat_index=mi)
        check_all_outputs(x, W, s, group=True, label=f"layer {layer} {name}")
