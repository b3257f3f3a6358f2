"""w4a8_linear_noalloc (the library-owned scratch variant of w4a8_linear)
against w4a8_linear itself, called through the C ABI.

Each case is two calls in a row of the no-allocation entry point, the
second on a smaller problem, so the second finds the first one's contents
in the shared scratch array: split-K arrival counters and partial sums, or
the codes and scales of a separately quantized bf16 input.  The outputs
must equal w4a8_linear's bit for bit (the same kernels run on the same
inputs; the group-scale outputs are deterministic too).  Two calls of the
same split-K problem follow each other, so a counter left behind would show.
"""
import ctypes

import numpy as np
import pytest
import torch

import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I
from helpers import bf16_dev, dev, pack, scales_dev

pytestmark = pytest.mark.gpu

# (M, N, K, scale mode, int8 input): first the larger problem, then a smaller one
PAIRS = [
    [(16, 24576, 4096, 0, False), (3, 4096, 4096, 0, False)],     # separate quantize into the scratch
    [(2, 16, 65536, 0, False), (1, 16, 65536, 0, False)],         # split K: counters + partials
    [(1, 16, 65536, 0, False), (1, 16, 65536, 0, False)],         # the same split twice
    [(1024, 6144, 4096, 0, False), (300, 256, 4096, 0, False)],   # large M, codes in the scratch
    [(16, 4096, 12288, 1, False), (5, 4096, 4096, 1, False)],     # group scales
    [(1, 16, 65536, 1, False), (40, 512, 2048, 1, True)],         # group split, then int8 input
]


def _problem(M, N, K, mode, i8, seed):
    x = I.activations(M, K, seed)
    W, s = I.weights(N, K, seed + 1, group=bool(mode))
    xd = bf16_dev(x)
    xs = None
    if i8:
        xd, xs = w.w4a8_quantize_act(xd)
    return xd, xs, pack(W), scales_dev(s)


def _call(entry, xd, xs, wp, sd, M, N, K, mode, y, ws=None):
    L = w.lib()
    st = torch.cuda.current_stream().cuda_stream
    in_kind = w.IN_I8 if xs is not None else w.IN_BF16
    args = (xd.data_ptr(), in_kind, None if xs is None else xs.data_ptr(), M, K, wp.data_ptr(), sd.data_ptr(),
            mode, N, y.data_ptr(), w.OUT_BF16)
    if entry == "noalloc":
        rc = L.w4a8_linear_noalloc(*args, st)
    else:
        rc = L.w4a8_linear(*args, None if ws is None else ws.data_ptr(), 0 if ws is None else ws.numel(), st)
    assert rc == w.W4A8_OK, (entry, M, N, K, rc)


@pytest.mark.parametrize("pair", range(len(PAIRS)))
def test_noalloc_matches_linear(pair):
    for j, (M, N, K, mode, i8) in enumerate(PAIRS[pair]):
        need = w.w4a8_linear_workspace_bytes(M, N, K, mode, int(i8))
        print(f"[case] noalloc pair {pair} call {j}: M={M} N={N} K={K} mode={mode} int8={i8} "
              f"workspace={need} plan={w.w4a8_linear_describe(M, N, K, mode, int(i8))}", flush=True)
        assert need <= w.NOALLOC_SCRATCH_BYTES
        xd, xs, wp, sd = _problem(M, N, K, mode, i8, 7000 + 10 * pair + j)
        y_ref = torch.empty((M, N), dtype=torch.bfloat16, device=dev())
        y_na = torch.full((M, N), 7.0, dtype=torch.bfloat16, device=dev())
        ws = torch.zeros(max(need, 1), dtype=torch.uint8, device=dev()) if need else None
        _call("linear", xd, xs, wp, sd, M, N, K, mode, y_ref, ws)
        _call("noalloc", xd, xs, wp, sd, M, N, K, mode, y_na)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y_na.view(torch.int16).cpu().numpy(), y_ref.view(torch.int16).cpu().numpy(),
                                      err_msg=f"pair {pair} call {j}")
