"""The ceiling probes (libw4a8_ceiling.so) read and multiply what they
claim: the streaming read's per-thread XOR matches numpy over the same bytes,
and the MFMA chains give the closed-form sum 2048 * iters."""
import ctypes
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
READ_BLOCKS, READ_THREADS = 256, 512


def lib():
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2608_12932_amd", "libw4a8_ceiling.so"))
    L.w4a8_ceiling_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    L.w4a8_ceiling_mfma_i8.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    return L


def expected_read_sink(host_words, nbytes):
    """Workgroup b XORs the 16-byte chunks of [b P, (b + 1) P) that lie in
    the buffer, thread i those at i * 16 + j * 8192 of the range."""
    per = 16 * (-(-nbytes // (16 * READ_BLOCKS)))
    chunks = host_words.reshape(-1, 4)
    out = np.zeros(READ_BLOCKS * READ_THREADS, np.uint32)
    for b in range(READ_BLOCKS):
        lo, hi = b * per // 16, min(nbytes, (b + 1) * per) // 16
        if lo >= hi:
            continue
        blk = chunks[lo:hi]
        n = blk.shape[0]
        rows = -(-n // READ_THREADS)
        pad = np.zeros((rows * READ_THREADS, 4), np.uint32)
        pad[:n] = blk
        x = np.bitwise_xor.reduce(pad.reshape(rows, READ_THREADS, 4), axis=0)
        out[b * READ_THREADS:(b + 1) * READ_THREADS] = np.bitwise_xor.reduce(x, axis=1)
    return out


@pytest.mark.parametrize("mib,tail", [(64, 0), (9, 48)])
def test_stream_read_covers_every_byte(mib, tail):
    nbytes = mib * 2**20 + tail
    host = np.random.Generator(np.random.PCG64(mib)).integers(0, 2**32, nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(READ_BLOCKS * READ_THREADS, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    assert lib().w4a8_ceiling_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(), st) == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sink.cpu().numpy().view(np.uint32), expected_read_sink(host, nbytes))


def test_stream_read_rejects_bad_sizes():
    st = torch.cuda.current_stream().cuda_stream
    sink = torch.zeros(READ_BLOCKS * READ_THREADS, dtype=torch.int32, device="cuda")
    assert lib().w4a8_ceiling_stream_read(sink.data_ptr(), 24, sink.data_ptr(), st) != 0
    assert lib().w4a8_ceiling_stream_read(sink.data_ptr(), 1 << 31, sink.data_ptr(), st) != 0


def test_mfma_chain_closed_form():
    sink = torch.zeros(1024 * 256, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    assert lib().w4a8_ceiling_mfma_i8(100, sink.data_ptr(), st) == 0
    torch.cuda.synchronize()
    assert (sink == 2048 * 100).all()
