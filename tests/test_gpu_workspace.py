"""One zero-filled workspace shared by calls of different shapes: a K-split
call (arrival counters), a call whose bf16 input is quantized into the
workspace, a split streaming attention, then the K-split call again.  Every
call's counters sit in the workspace's first 64 KiB, which nothing else
writes, so the repeated call must still give the oracle's bits."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I
from helpers import bf16_dev, dev, pack, run_linear, scales_dev, to_np_bits

pytestmark = pytest.mark.gpu


def test_workspace_shared_across_shapes():
    ws = w.Workspace(dev())
    shapes = [(1, 16, 65536, 11), (16, 4096, 4096, 12)]
    assert "S=8 " in w.w4a8_linear_describe(1, 16, 65536, 0, 0)
    assert "quantize_rows" in w.w4a8_linear_describe(16, 4096, 4096, 0, 0)
    cases = []
    for M, N, K, seed in shapes:
        x = I.activations(M, K, seed)
        W, s = I.weights(N, K, seed + 1)
        cases.append((x, pack(W), s, N, oracle.linear(x, W, s_w=s, nthreads=8)["y"]))
    H, Nq, Nk = 2, 64, 2048
    assert w.w4a8_stream_attention_workspace_bytes(H, Nq, Nk) > 64 * 1024
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)
    q = t(I.activations(H * Nq, 128, 20).reshape(H, Nq, 128))
    k = t(I.activations(H * Nk, 128, 21).reshape(H, Nk, 128))
    v = t(I.activations(H * Nk, 128, 22).reshape(H, Nk, 128))
    cos_t, sin_t = (torch.from_numpy(a).to(dev()) for a in oracle.rope_tables(Nk, 128))
    pq = torch.arange(Nk - Nq, Nk, dtype=torch.int32, device=dev())
    pk = torch.arange(Nk, dtype=torch.int32, device=dev())
    for order in ([0, 1, 0], [1, 0, 1, 0]):
        for i in order:
            x, wp, s, N, want = cases[i]
            print(f"[case] shared workspace shape {shapes[i][:3]}", flush=True)
            got = run_linear(x, wp, s, N, group=False, out_kind=w.OUT_BF16, workspace=ws)
            np.testing.assert_array_equal(got, want, err_msg=f"shape {shapes[i][:3]}")
            w.w4a8_stream_attention(q, k, v, pq, pk, cos_t, sin_t, 128 ** -0.5, workspace=ws)
            torch.cuda.synchronize()


def test_calls_on_a_side_stream():
    """Calls enqueued on a stream other than torch's current one: the
    binding's temporary workspace and a Workspace's growth are zero-filled on
    that stream, before the K-split call's arrival counters are read, and the
    outputs are allocated there.  Checked against the oracle."""
    side = torch.cuda.Stream(dev())
    M, N, K = 1, 16, 65536
    assert "S=8 " in w.w4a8_linear_describe(M, N, K, 0, 0)
    x = I.activations(M, K, 31)
    W, s = I.weights(N, K, 32)
    want = oracle.linear(x, W, s_w=s, nthreads=8)["y"]
    wp, xd, sd = pack(W), bf16_dev(x), scales_dev(s)
    H, Nq, Nk = 2, 64, 2048
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)
    q = t(I.activations(H * Nq, 128, 33).reshape(H, Nq, 128))
    k = t(I.activations(H * Nk, 128, 34).reshape(H, Nk, 128))
    v = t(I.activations(H * Nk, 128, 35).reshape(H, Nk, 128))
    cos_t, sin_t = (torch.from_numpy(a).to(dev()) for a in oracle.rope_tables(Nk, 128))
    pq = torch.arange(Nk - Nq, Nk, dtype=torch.int32, device=dev())
    pk = torch.arange(Nk, dtype=torch.int32, device=dev())
    torch.cuda.synchronize()  # inputs made on the current stream are ready for the side stream
    print("[case] side stream: split-K linear (temporary and grown workspace), split attention", flush=True)
    ws = w.Workspace(dev())
    ys = [w.w4a8_linear(xd, wp, sd, N, stream=side),
          w.w4a8_linear(xd, wp, sd, N, workspace=ws, stream=side),
          w.w4a8_linear(xd, wp, sd, N, workspace=ws, stream=side)]
    o_side = w.w4a8_stream_attention(q, k, v, pq, pk, cos_t, sin_t, 128 ** -0.5, stream=side)
    side.synchronize()
    for i, y in enumerate(ys):
        np.testing.assert_array_equal(to_np_bits(y), want, err_msg=f"side-stream call {i}")
    o_cur = w.w4a8_stream_attention(q, k, v, pq, pk, cos_t, sin_t, 128 ** -0.5)
    torch.cuda.synchronize()
    assert torch.equal(o_side.view(torch.int16), o_cur.view(torch.int16))
