"""HIP-graph capture of the layer's calls: a captured stack of W4A8 linears
(quantize + GEMM launches on the capturing stream, preallocated workspaces)
replays to the same bits as the eager calls, replay after replay, with eager
work and synchronizations in between."""
import numpy as np
import pytest
import torch

import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I

pytestmark = pytest.mark.gpu


def build_calls(M, group, layers=2):
    dev = torch.device("cuda:0")
    mode = w.SCALE_GROUP_F16 if group else w.SCALE_CHANNEL_F32
    calls = []
    for l in range(layers):
        for mi, (name, K, N) in enumerate(I.LAYER_MATS):
            W, s = I.weights(N, K, 1000 + 10 * l + mi, group=group)
            wp = w.w4a8_pack_weights(torch.from_numpy(W).to(dev))
            x = torch.from_numpy(I.activations(M, K, 2000 + 10 * l + mi).view(np.int16)).to(dev).view(torch.bfloat16)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            ws = w.Workspace(dev)
            ws.get(w.w4a8_linear_workspace_bytes(M, N, K, mode))  # allocated before any capture
            calls.append((x, wp, torch.from_numpy(s).to(dev), N, y, ws, mode))
    return calls


def run(calls, stream=None):
    for x, wp, s, N, y, ws, mode in calls:
        w.w4a8_linear(x, wp, s, N, scale_mode=mode, out=y, workspace=ws, stream=stream)


@pytest.mark.parametrize("M,group", [(16, True), (16, False), (300, True), (1, False)])
def test_graph_replays_match_eager(M, group):
    calls = build_calls(M, group)
    run(calls)
    torch.cuda.synchronize()
    ref = [c[4].clone() for c in calls]
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            run(calls, stream=cap)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()
    for rep in range(4):
        for c in calls:
            c[4].zero_()
        g.replay()
        torch.cuda.synchronize()
        for i, c in enumerate(calls):
            assert torch.equal(c[4].view(torch.int16), ref[i].view(torch.int16)), (rep, i)
        # eager work between the replays: the same calls on the default stream
        run(calls)
        torch.cuda.synchronize()
        for i, c in enumerate(calls):
            assert torch.equal(c[4].view(torch.int16), ref[i].view(torch.int16)), ("eager", rep, i)
