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


@pytest.mark.parametrize("M,F,K,group", [(16, 12288, 4096, False), (16, 16, 65536, True), (1024, 12288, 4096, False)])
def test_gated_graph_replays_match_eager(M, F, K, group):
    # the gated gate+up call: small M, small M with K split (its arrival
    # counters are reset by every call), and the large-M gated tile
    dev = torch.device("cuda:0")
    mode = w.SCALE_GROUP_F16 if group else w.SCALE_CHANNEL_F32
    print(f"[case] gated graph M={M} F={F} K={K} group={group} "
          f"plan={w.w4a8_linear_swiglu_describe(M, 2 * F, K, mode, 0)}", flush=True)
    W, s = I.weights(2 * F, K, 3000 + M, group=group)
    wp = w.w4a8_pack_weights(torch.from_numpy(W).to(dev))
    sd = torch.from_numpy(s).to(dev)
    x = torch.from_numpy(I.activations(M, K, 3001 + M).view(np.int16)).to(dev).view(torch.bfloat16)
    y = torch.empty((M, F), dtype=torch.bfloat16, device=dev)
    ws = w.Workspace(dev)
    ws.get(w.w4a8_linear_swiglu_workspace_bytes(M, 2 * F, K, mode))

    def call(stream=None):
        w.w4a8_linear_swiglu(x, wp, sd, 2 * F, scale_mode=mode, out=y, workspace=ws, stream=stream)

    call()
    torch.cuda.synchronize()
    ref = y.clone()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            call(stream=cap)
            call(stream=cap)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()
    for rep in range(4):
        y.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), rep
        call()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), ("eager", rep)


@pytest.mark.parametrize("M,group", [(1, False), (16, False), (1, True), (16, True)])
def test_replayed_decoder_stack_matches_oracle(M, group):
    """The backbone's linears of a decode / verify step as one captured HIP
    graph (the per-stage graph capture of FlashDrive Sec. 3.5): four decoder
    layers x (QKV, O, gate+up, down) with distinct seeded weights, each call
    on its own bf16 input.  Every replay, with eager calls between replays,
    is compared with the oracle linear by linear: per-channel outputs bit for
    bit, group-scale outputs within the derived tolerance."""
    import oracle
    from helpers import GROUP_FLOOR, NTHREADS, REL, to_np_bits

    layers = 4
    calls = build_calls(M, group, layers=layers)
    print(f"[case] replayed stack M={M} group={group} linears={len(calls)}", flush=True)
    refs = []
    for l in range(layers):
        for mi, (name, K, N) in enumerate(I.LAYER_MATS):
            W, s = I.weights(N, K, 1000 + 10 * l + mi, group=group)
            x = I.activations(M, K, 2000 + 10 * l + mi)
            refs.append(oracle.linear(x, W, s_w=None if group else s, s_g=s if group else None, nthreads=NTHREADS))
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    run(calls)  # warm the binding's lazy state before capture
    torch.cuda.synchronize()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            run(calls, stream=cap)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()

    def check(tag):
        for i, c in enumerate(calls):
            got = to_np_bits(c[4])
            ref = refs[i]
            if not group:
                np.testing.assert_array_equal(got, ref["y"], err_msg=f"{tag} linear {i}")
            else:
                yf = (got.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
                bound = REL * np.abs(ref["y64"]) + GROUP_FLOOR * ref["bound"]
                assert np.all(np.abs(yf - ref["y64"]) <= bound), f"{tag} linear {i}"

    for rep in range(3):
        for c in calls:
            c[4].fill_(1.0)
        g.replay()
        torch.cuda.synchronize()
        check(f"replay {rep}")
        run(calls)
        torch.cuda.synchronize()
        check(f"eager {rep}")
