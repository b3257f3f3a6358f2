"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (bf16 activations in, bf16 out).

Rows of a linear layer are independent, so where the oracle cannot finish
the whole workload in seconds it computes a seeded sample of token rows and
those rows are compared exactly.  Coverage:
  - tiny, gate+up verify and qkv prefill: every output;
  - down verify: every output at M = 1, 4, 16 on layers 0 and 35, and at
    M = 1 on all 36 weight matrices;
  - the group-scale layer: every output at M = 1 and 16 on all 36 layers,
    16 seeded token rows at M = 256 and 2048 on all 36 layers, every output
    at M = 256 on layer 0 and 48 seeded rows at M = 2048 on layer 17.
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


@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("layer", [0, 35])
def test_down_verify(M, layer):
    x, W, s, K, N = I.workload_inputs("down_verify", M, layer=layer)
    check_all_outputs(x, W, s, group=False, label=f"down verify layer {layer}")


def test_qkv_prefill():
    x, W, s, K, N = I.workload_inputs("qkv_prefill", 1024)
    check_all_outputs(x, W, s, group=False, label="qkv prefill M=1024 K=4096 N=6144")


@pytest.mark.parametrize("layer", range(36))
def test_down_verify_every_matrix_one_token(layer):
    x, W, s, K, N = I.workload_inputs("down_verify", 1, layer=layer)
    check_all_outputs(x, W, s, group=False, label=f"down verify layer {layer}")


def test_layer_group_256_every_row():
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        x, W, s, K, N = I.workload_inputs("layer_group", 256, layer=0, mat_index=mi)
        check_all_outputs(x, W, s, group=True, label=f"layer 0 {name}")


@pytest.mark.parametrize("layer", range(36))
def test_layer_group_every_layer(layer):
    # the layer's weights made and packed once, then every decode / verify
    # row (M = 1, 16) and 16 seeded rows of the prefill sizes (M = 256, 2048)
    wl = I.WORKLOADS["layer_group"]
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        W, s = I.weights(N, K, I.seed_w(wl.number, layer, name), group=True)
        wp = pack(W)
        for M in (1, 16, 256, 2048):
            x = I.activations(M, K, I.seed_x(wl.number, M), wl.outliers)
            rows = None
            if M > 16:
                rows = np.sort(np.random.Generator(np.random.PCG64(2608 + 100 * layer + M)).choice(M, 16, replace=False))
            check_all_outputs(x, W, s, group=True, rows=rows, wp=wp,
                              label=f"layer {layer} {name}" + ("" if rows is None else " (16 sampled rows)"))


def test_layer_group_2048_sampled_rows():
    M = 2048
    rows = np.sort(np.random.Generator(np.random.PCG64(2608)).choice(M, 48, replace=False))
    for mi, (name, K, N) in enumerate(I.LAYER_MATS):
        x, W, s, K, N = I.workload_inputs("layer_group", M, layer=17, mat_index=mi)
        check_all_outputs(x, W, s, group=True, rows=rows, label=f"layer 17 {name} (48 sampled rows)")
