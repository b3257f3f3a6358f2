"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/w4a8.h declares, and rejects malformed calls before
launching anything."""
import ctypes
import os
import re

import pytest

import paper_2608_12932_amd as w

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions(header="w4a8.h"):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(w4a8_[a-z0-9_]+)\s*\(", text)))


def test_ceiling_library_exports_every_declared_symbol():
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2608_12932_amd", "libw4a8_ceiling.so"))
    names = declared_functions("w4a8_ceiling.h")
    assert names == ["w4a8_ceiling_mfma_i8", "w4a8_ceiling_stream_read"]
    for name in names:
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(w.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = w.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_status_strings():
    for s in range(5):
        assert w.status_string(s)
    assert "unknown" in w.status_string(99)


@pytest.mark.parametrize("N,K,want", [(24576, 4096, 24576 * 4096 // 2), (16, 128, 1024),
                                      (4096, 12288, 4096 * 12288 // 2), (8, 128, 0), (16, 100, 0),
                                      (16, 0, 0), (-16, 128, 0), (16, 65536 + 128, 0)])
def test_packed_weight_bytes(N, K, want):
    assert w.w4a8_packed_weight_bytes(N, K) == want


def test_workspace_bytes_plans():
    # gate+up verify: codes from the quantize kernel live in the workspace
    assert w.w4a8_linear_workspace_bytes(16, 24576, 4096) >= 16 * 4096 + 16 * 4
    assert w.w4a8_linear_workspace_bytes(16, 24576, 4096, in_kind=w.IN_I8) == 0
    # down verify at M=1: a quantize launch first, its codes in the workspace
    assert w.w4a8_linear_workspace_bytes(1, 4096, 12288) >= 64 * 1024 + 12288 + 4
    assert "quantize_rows + " in w.w4a8_linear_describe(1, 4096, 12288)
    # very long K over one or two column tiles: quantize fused, no workspace
    assert w.w4a8_linear_workspace_bytes(1, 32, 32768) == 0
    assert "fused-quant" in w.w4a8_linear_describe(1, 32, 32768)
    # large M with bf16 input: codes + scales in the workspace
    ws = w.w4a8_linear_workspace_bytes(1024, 6144, 4096)
    assert ws >= 1024 * 4096 + 1024 * 4
    assert w.w4a8_linear_workspace_bytes(1024, 6144, 4096, in_kind=w.IN_I8) == 0
    # invalid shapes
    assert w.w4a8_linear_workspace_bytes(16, 24575, 4096) == 0
    assert w.w4a8_linear_workspace_bytes(0, 256, 256) == 0
    assert "smallm" in w.w4a8_linear_describe(16, 24576, 4096)
    assert "largem" in w.w4a8_linear_describe(1024, 6144, 4096)
    assert w.w4a8_linear_describe(16, 24575, 4096) == "invalid shape"


def test_plans_fill_the_chip():
    # The tilings chosen for the benchmark shapes fill the 256 CUs in whole waves.
    assert "NT=6" in w.w4a8_linear_describe(16, 24576, 4096) and "S=1 groups=256" in w.w4a8_linear_describe(16, 24576, 4096)
    assert "tiles=8x32" in w.w4a8_linear_describe(1024, 6144, 4096)
    d = w.w4a8_linear_describe(16, 4096, 12288)
    assert "groups=256" in d


def test_split_and_fusion_choices():
    # K is split across workgroups only where one workgroup's weight stream
    # would be long (one or two column tiles over K = 65536), never at the
    # decoder-layer shapes; the quantize is fused only for narrow column
    # groups over a very long K (never at the layer shapes).
    for K, N in ((4096, 6144), (4096, 4096), (4096, 24576), (12288, 4096)):
        for M in (1, 4, 16, 64):
            for mode in (0, 1):
                assert "S=1 " in w.w4a8_linear_describe(M, N, K, mode), (M, N, K, mode)
    for M in (1, 16):
        assert "S=8 " in w.w4a8_linear_describe(M, 16, 65536)
    for K, N in ((4096, 6144), (4096, 4096), (4096, 24576), (12288, 4096)):
        for M in (1, 4, 16):
            assert "fused-quant" not in w.w4a8_linear_describe(M, N, K), (M, N, K)
    assert "fused-quant" in w.w4a8_linear_describe(1, 16, 65536)
    assert "fused-quant" in w.w4a8_linear_describe(2, 32, 32768, 1)
    # group scales use the same column groups as per-channel scales
    assert "NT=6" in w.w4a8_linear_describe(16, 24576, 4096, 1)


def test_malformed_calls_are_rejected_without_launch():
    L = w.lib()
    P = ctypes.c_void_p
    fake = P(1 << 20)  # never dereferenced: validation fails first
    # negative M
    assert L.w4a8_linear(fake, 0, None, -1, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # K not a multiple of 128
    assert L.w4a8_linear(fake, 0, None, 4, 200, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # N not a multiple of 16
    assert L.w4a8_linear(fake, 0, None, 4, 256, fake, fake, 0, 250, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # bad modes
    assert L.w4a8_linear(fake, 7, None, 4, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    assert L.w4a8_linear(fake, 0, None, 4, 256, fake, fake, 5, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    assert L.w4a8_linear(fake, 0, None, 4, 256, fake, fake, 0, 256, fake, 9, None, 0, None) == w.W4A8_EINVAL
    # null / misaligned pointers
    assert L.w4a8_linear(None, 0, None, 4, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    assert L.w4a8_linear(P((1 << 20) + 8), 0, None, 4, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # int8 input without scales
    assert L.w4a8_linear(fake, 1, None, 4, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # missing weight scales for a scaled output
    assert L.w4a8_linear(fake, 0, None, 4, 256, fake, None, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # workspace too small (large M with bf16 input needs one)
    assert L.w4a8_linear(fake, 0, None, 1024, 4096, fake, fake, 0, 6144, fake, 0, None, 0, None) == w.W4A8_EINVAL
    # M == 0 is a no-op even with null pointers
    assert L.w4a8_linear(None, 0, None, 0, 256, None, None, 0, 256, None, 0, None, 0, None) == w.W4A8_OK
    assert L.w4a8_quantize_act(None, 0, 256, None, None, None) == w.W4A8_OK
    assert L.w4a8_quantize_act(fake, 4, 100, fake, fake, None) == w.W4A8_EINVAL
    assert L.w4a8_quantize_act(None, 4, 256, fake, fake, None) == w.W4A8_EINVAL
    assert L.w4a8_pack_weights(fake, 250, 256, fake, None) == w.W4A8_EINVAL
    assert L.w4a8_pack_weights(None, 256, 256, fake, None) == w.W4A8_EINVAL


def test_swiglu_plans_and_rejections():
    # gate+up verify: the same column groups as the plain projection, gate
    # and up tiles paired (NT even)
    d = w.w4a8_linear_swiglu_describe(16, 24576, 4096)
    assert "swiglu" in d and "NT=6" in d and "S=1" in d
    assert w.w4a8_linear_swiglu_workspace_bytes(16, 24576, 4096) == w.w4a8_linear_workspace_bytes(16, 24576, 4096)
    # odd tile counts per half are never paired across halves
    for M, F, K in [(3, 48, 256), (1, 2048, 12288), (16, 16, 65536), (64, 80, 512)]:
        d = w.w4a8_linear_swiglu_describe(M, 2 * F, K)
        nt = int(d.split("NT=")[1].split(",")[0])
        assert nt % 2 == 0 and (F // 16) % (nt // 2) == 0, d
    # large M: the 128 x 128 tile, 64 output columns per tile
    d = w.w4a8_linear_swiglu_describe(1024, 24576, 4096)
    assert "largem<128x256,channel,swiglu>" in d and "tiles=8x96" in d, d
    d = w.w4a8_linear_swiglu_describe(1024, 24576, 4096, 1)
    assert "largem<128x128,group,swiglu>" in d and "tiles=8x192" in d, d
    assert "largem<128x128,group,swiglu> tiles=1x2" in w.w4a8_linear_swiglu_describe(65, 160, 256, 1)
    assert w.w4a8_linear_swiglu_workspace_bytes(1024, 24576, 4096) == w.w4a8_linear_workspace_bytes(1024, 24576, 4096)
    # shapes the gated call rejects
    assert w.w4a8_linear_swiglu_describe(4, 48, 256) == "invalid shape"
    assert w.w4a8_linear_swiglu_workspace_bytes(4, 48, 256) == 0
    L = w.lib()
    P = ctypes.c_void_p
    fake = P(1 << 20)
    f = L.w4a8_linear_swiglu
    assert f(fake, 0, None, 1024, 4096, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL  # no workspace
    assert f(fake, 0, None, 4, 256, fake, fake, 0, 48, fake, 0, None, 0, None) == w.W4A8_EINVAL
    assert f(fake, 0, None, 4, 256, fake, fake, 0, 256, fake, w.OUT_I32_ACC, None, 0, None) == w.W4A8_EINVAL
    assert f(None, 0, None, 0, 256, None, None, 0, 256, None, 0, None, 0, None) == w.W4A8_OK
    assert f(None, 0, None, 4, 256, fake, fake, 0, 256, fake, 0, None, 0, None) == w.W4A8_EINVAL


def test_rmsnorm_quantize_rejections():
    L = w.lib()
    P = ctypes.c_void_p
    fake = P(1 << 20)
    f = L.w4a8_rmsnorm_quantize_act
    assert f(fake, fake, 0.0, 4, 256, fake, fake, None) == w.W4A8_EINVAL       # eps must be > 0
    assert f(fake, fake, float("nan"), 4, 256, fake, fake, None) == w.W4A8_EINVAL
    assert f(fake, fake, 1e-6, 4, 200, fake, fake, None) == w.W4A8_EINVAL      # K % 128
    assert f(None, fake, 1e-6, 4, 256, fake, fake, None) == w.W4A8_EINVAL
    assert f(fake, P((1 << 20) + 8), 1e-6, 4, 256, fake, fake, None) == w.W4A8_EINVAL  # misaligned gamma
    assert f(None, None, 1e-6, 0, 256, None, None, None) == w.W4A8_OK          # M == 0 is a no-op


def test_stream_attention_rejections():
    L = w.lib()
    P = ctypes.c_void_p
    fake = P(1 << 20)
    f = L.w4a8_stream_attention
    args = lambda H=4, Hkv=2, Nq=8, Nk=16, D=128, ws=None, wsb=0: (fake, fake, fake, fake, fake, fake, fake, 64, H, Hkv,
                                                                   Nq, Nk, D, 0.1, fake, ws, wsb, None)
    assert f(*args(D=64)) == w.W4A8_EUNSUPPORTED
    assert f(*args(H=4, Hkv=3)) == w.W4A8_EINVAL          # H % Hkv
    assert f(*args(Nk=0)) == w.W4A8_EINVAL
    assert f(*args(Nq=1 << 23)) == w.W4A8_EINVAL          # beyond 32-bit row offsets
    assert f(*args(Nq=0)) == w.W4A8_OK
    # the workspace: counter region, the rotated keys (room for H kv heads),
    # the tiles' position bounds (8 bytes per 32 keys), the dispatch schedule
    # (4 bytes per work item: 12 query blocks x 2 splits x 32 heads) and the
    # per-block solo-split table (4 bytes per block), each region in 256-byte
    # units, then, for a shape that splits its key range, the partials
    need = w.w4a8_stream_attention_workspace_bytes(32, 768, 3072)
    assert need == 64 * 1024 + 32 * 3072 * 128 * 2 + 768 + 3328 + 2 * 32 * 768 * (128 + 2) * 4
    assert f(*args(H=32, Hkv=8, Nq=768, Nk=3072)) == w.W4A8_EINVAL
    assert f(*args(H=32, Hkv=8, Nq=768, Nk=3072, ws=P((1 << 20) + 16), wsb=need)) == w.W4A8_EINVAL  # misaligned
    assert w.w4a8_stream_attention_workspace_bytes(4, 64, 256) == 64 * 1024 + 4 * 256 * 128 * 2 + 256 + 256  # no split
    assert f(*args(H=4, Hkv=2, Nq=64, Nk=256)) == w.W4A8_EINVAL  # the rotated keys need the workspace


def test_flow_schedule_matches_the_oracle_reading():
    import oracle

    assert w.w4a8_flow_schedule(8, 4) == [True, True, False, False, False, False, True, True]
    for n in range(1, 17):
        for r in range(n):
            assert w.w4a8_flow_schedule(n, r) == oracle.flow_schedule(n, r), (n, r)
    L = w.lib()
    buf = (ctypes.c_int32 * 8)()
    for bad in ((0, 0), (8, 8), (8, -1), (4097, 0)):
        assert L.w4a8_flow_schedule(*bad, buf) == w.W4A8_EINVAL
    assert L.w4a8_flow_schedule(8, 4, None) == w.W4A8_EINVAL


def test_flow_step_rejections():
    L = w.lib()
    P = ctypes.c_void_p
    X, V, C, S = P(1 << 24), P(2 << 24), P(3 << 24), P(4 << 24)  # disjoint fake addresses
    f = L.w4a8_flow_step
    assert f(X, None, C, 6, 128, 0.125, 1, S, None) == w.W4A8_EINVAL      # stats on a reused step
    assert f(X, V, C, 6, 0, 0.125, 1, None, None) == w.W4A8_EINVAL        # n >= 1
    assert f(X, V, C, -1, 8, 0.125, 1, None, None) == w.W4A8_EINVAL
    assert f(X, V, C, (1 << 24) + 1, 8, 0.125, 1, None, None) == w.W4A8_EINVAL
    assert f(X, V, C, 6, 128, float("inf"), 1, None, None) == w.W4A8_EINVAL
    assert f(X, V, C, 6, 128, float("nan"), 1, None, None) == w.W4A8_EINVAL
    assert f(P((1 << 24) + 4), V, C, 6, 128, 0.125, 1, None, None) == w.W4A8_EINVAL   # misaligned x
    assert f(X, V, C, 6, 128, 0.125, 1, P((4 << 24) + 4), None) == w.W4A8_EINVAL      # misaligned stats
    assert f(X, V, P((1 << 24) + 1024), 6, 128, 0.125, 1, None, None) == w.W4A8_EINVAL  # cache inside x
    assert f(X, P((3 << 24) + 16), C, 6, 128, 0.125, 1, None, None) == w.W4A8_EINVAL   # v_new straddles the cache
    assert f(X, V, C, 6, 128, 0.125, 1, P((2 << 24) + 64), None) == w.W4A8_EINVAL      # stats inside v_new
    assert f(X, V, C, 6, 128, 0.125, 0, None, None) == w.W4A8_EINVAL                # repeat >= 1
    assert f(X, V, C, 6, 128, 0.125, 4097, None, None) == w.W4A8_EINVAL
    assert f(None, None, None, 0, 128, 0.125, 1, None, None) == w.W4A8_OK               # B == 0 is a no-op


@pytest.mark.parametrize("scale_mode", [w.SCALE_CHANNEL_F32, w.SCALE_GROUP_F16])
def test_largest_shapes_plan_a_grid_that_fits_one_launch(scale_mode):
    # M = 2^20 rows over N = 2^24 columns: the tile count is formed in 64
    # bits and the planned grid stays below 2^31 workgroups
    M, N, K = 1 << 20, 1 << 24, 128
    d = w.w4a8_linear_describe(M, N, K, scale_mode)
    m = re.search(r"tiles=(\d+)x(\d+)", d)
    assert m, d
    assert int(m.group(1)) * int(m.group(2)) < 2 ** 31
    assert w.w4a8_linear_workspace_bytes(M, N, K, scale_mode) >= M * K


def test_noalloc_rejects_problems_past_its_scratch_before_any_launch():
    # bf16 input at M = 4096, K = 65536 needs 256 MiB of codes, more than the
    # 32 MiB scratch: rejected on the host (the dummy pointers are never used)
    L = w.lib()
    p = ctypes.c_void_p(0x10000)
    M, K, N = 4096, 65536, 16
    assert w.w4a8_linear_workspace_bytes(M, N, K) > w.NOALLOC_SCRATCH_BYTES
    rc = L.w4a8_linear_noalloc(p, w.IN_BF16, None, M, K, p, p, w.SCALE_CHANNEL_F32, N, p, w.OUT_BF16, None)
    assert rc == w.W4A8_EUNSUPPORTED
    # argument errors come first, as for w4a8_linear; M == 0 is a no-op
    assert L.w4a8_linear_noalloc(p, w.IN_BF16, None, 16, 100, p, p, 0, N, p, 0, None) == w.W4A8_EINVAL
    assert L.w4a8_linear_noalloc(p, w.IN_BF16, None, 0, K, p, p, 0, N, p, 0, None) == w.W4A8_OK


# The small-M plan's time estimate (the "model=" field of the description)
# against the committed rocprofv3 kernel-trace averages of the layer shapes
# (int8 codes in).  A summary taken before the kernel sources last changed
# is skipped.
SMALLM_PROFILES = [
    ("smallm_gate_up_verify", "avg_us", (16, 24576, 4096, 0)),
    ("smallm_down_verify_m1", "avg_us", (1, 4096, 12288, 0)),
    ("smallm_down_verify_m4", "avg_us", (4, 4096, 12288, 0)),
    ("smallm_down_verify_m16", "avg_us", (16, 4096, 12288, 0)),
] + [(f"smallm_group_layer_m{M}", f"{name}.avg_us", (M, N, K, 1))
     for M in (1, 16)
     for name, N, K in (("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 24576, 4096), ("down", 4096, 12288))]


@pytest.mark.parametrize("profile,key,shape", SMALLM_PROFILES)
def test_smallm_time_estimate_matches_profile(profile, key, shape):
    import sys
    sys.path.insert(0, ROOT)
    import bench

    vals = bench.profile_summary(profile)
    if vals is None:
        pytest.skip(f"profiles/{profile}.txt was taken with other kernel sources")
    measured = float(vals[key])
    M, N, K, mode = shape
    d = w.w4a8_linear_describe(M, N, K, mode, 1)
    est = float(re.search(r"model=([0-9.]+)us", d).group(1))
    assert abs(est - measured) <= 0.2 * measured, (d, measured)
