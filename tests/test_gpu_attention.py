"""Parity of the streaming prefill attention (w4a8_stream_attention) with
the oracle (fp64 scores, softmax and sum over the same bf16-rounded rotated
operands).

Tolerance, derived: the kernel rounds the softmax weights to bf16 for the
P V product (relative 2^-9 each, so at most 2^-9 sum_j P_ij |v_jd| per
output), sums in fp32, and rounds the output to bf16 (2^-8 relative); its
fp32 scores from exact bf16 products and its base-2 exponentials add
errors far below those.  Written as |o - o64| <= 2^-8 |o64| + 2^-8 B with
B = sum_j P_ij |v_jd| from the oracle (twice the weight term)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_12932_amd as w
from paper_2608_12932_amd import inputs as I
from helpers import dev

pytestmark = pytest.mark.gpu

D = 128


def window(V, F, T, shift):
    """A view-major window of V views x F frames x T tokens.  The cache
    keeps each view's frames in a ring, slot (f + shift) % F holding frame f,
    so slot order is not window order; the queries are the newest frame of
    every view.  Returns (pos_k per cache slot, pos_q per query)."""
    pos_k = np.empty(V * F * T, np.int32)
    for v in range(V):
        for f in range(F):
            slot = (f + shift) % F
            pos_k[(v * F + slot) * T:(v * F + slot + 1) * T] = v * F * T + f * T + np.arange(T)
    pos_q = np.concatenate([v * F * T + (F - 1) * T + np.arange(T) for v in range(V)]).astype(np.int32)
    return pos_k, pos_q


def run(q, k, v, pos_q, pos_k, cos_t, sin_t, scale):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)
    o = w.w4a8_stream_attention(t(q), t(k), t(v), torch.from_numpy(pos_q).to(dev()), torch.from_numpy(pos_k).to(dev()),
                                torch.from_numpy(cos_t).to(dev()), torch.from_numpy(sin_t).to(dev()), scale)
    torch.cuda.synchronize()
    return (o.view(torch.int16).cpu().numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def check(H, Hkv, pos_q, pos_k, seed, label, rows=None):
    Nq, Nk = len(pos_q), len(pos_k)
    print(f"[case] stream attention {label} H={H} Hkv={Hkv} Nq={Nq} Nk={Nk}", flush=True)
    q = I.activations(H * Nq, D, seed).reshape(H, Nq, D)
    k = I.activations(Hkv * Nk, D, seed + 1).reshape(Hkv, Nk, D)
    v = I.activations(Hkv * Nk, D, seed + 2).reshape(Hkv, Nk, D)
    n_pos = int(max(pos_q.max(), pos_k.max())) + 1
    cos_t, sin_t = oracle.rope_tables(n_pos, D, base=1e6)
    scale = 1.0 / np.sqrt(D)
    o = run(q, k, v, pos_q, pos_k, cos_t, sin_t, scale)
    sel = np.arange(Nq) if rows is None else rows
    o64, bnd = oracle.streaming_attention(q[:, sel], k, v, pos_q[sel], pos_k, cos_t, sin_t, np.float32(scale))
    err = np.abs(o[:, sel] - o64)
    bound = 2.0 ** -8 * np.abs(o64) + 2.0 ** -8 * bnd + 1e-30
    bad = err > bound
    assert not bad.any(), f"{label}: {bad.sum()} outputs outside tolerance, worst ratio {np.max(err / bound):.2f}"
    return float(np.max(err / bound))


@pytest.mark.parametrize("V,F,T,shift,H,Hkv", [(4, 4, 16, 0, 4, 2), (4, 4, 16, 3, 4, 4), (2, 3, 40, 1, 8, 2),
                                               (4, 4, 23, 2, 2, 1)])
def test_streaming_window(V, F, T, shift, H, Hkv):
    # ragged query and key counts (not multiples of 64 and 32), ring-ordered slots
    pos_k, pos_q = window(V, F, T, shift)
    check(H, Hkv, pos_q, pos_k, 800 + T, f"window {V}x{F}x{T} shift {shift}")


def test_streaming_window_realistic_size():
    # 4 views x 4 frames x 192 tokens, 32 query heads on 8 kv heads (128 sampled queries)
    pos_k, pos_q = window(4, 4, 192, 1)
    rows = np.sort(np.random.Generator(np.random.PCG64(801)).choice(len(pos_q), 128, replace=False))
    check(32, 8, pos_q, pos_k, 802, "4x4x192", rows=rows)


def test_key_range_splits():
    # few query blocks over a long cache: the key range is split over
    # workgroups and merged (8 splits here; early queries see no key of the
    # later splits), with a ragged last tile
    pos_k, pos_q = window(4, 4, 125, 2)
    assert w.w4a8_stream_attention_workspace_bytes(2, len(pos_q), len(pos_k)) > 0
    check(2, 1, pos_q, pos_k, 804, "splits 4x4x125")


def test_queries_seeing_one_key_and_all_keys():
    # query positions below all but one key, and above every key
    pos_k = np.arange(10, 110, dtype=np.int32)
    pos_q = np.array([10, 11, 50, 109, 500, 10], np.int32)
    check(2, 1, pos_q, pos_k, 803, "edge visibility")


def test_cache_shorter_than_one_tile():
    # 14 keys: one partial key tile; 7 queries: one partial query block
    pos_k, pos_q = window(1, 2, 7, 1)
    check(2, 2, pos_q, pos_k, 805, "window 1x2x7")


def test_lone_split_past_the_first():
    # keys in descending position order, so the earliest positions sit in
    # the last key split: the first query block (positions 0..63) sees keys
    # of the last of 8 splits only and writes its output from that split;
    # the second block (the largest positions) sees every split and goes
    # through the merge
    Nk = 4096
    pos_k = (Nk - 1 - np.arange(Nk)).astype(np.int32)
    pos_q = np.concatenate([np.arange(64), Nk - 64 + np.arange(64)]).astype(np.int32)
    check(2, 1, pos_q, pos_k, 813, "lone split 7 of 8")


@pytest.mark.parametrize("H,Hkv,Nq", [(4, 2, 4096), (2, 1, 10240)])
def test_schedule_limit(H, Hkv, Nq):
    # 4096 keys in position order under Nq queries spread over them: 4 query
    # heads x 4096 queries give 64 query blocks x 4 splits = 256 (block,
    # split) pairs, the most the dispatch schedule deals (1024 workgroups);
    # 2 heads x 10240 queries give 160 x 2 = 320 pairs, past it, so the plain
    # grid with a merge runs (64 sampled queries each)
    Nk = 4096
    pos_k = np.arange(Nk, dtype=np.int32)
    pos_q = np.sort(np.random.Generator(np.random.PCG64(814)).integers(0, Nk, Nq)).astype(np.int32)
    rows = np.sort(np.random.Generator(np.random.PCG64(815)).choice(Nq, 64, replace=False))
    check(H, Hkv, pos_q, pos_k, 816, f"schedule limit H={H} Nq={Nq}", rows=rows)


def test_query_seeing_no_key_gets_zero():
    pos_k = np.arange(10, 110, dtype=np.int32)
    pos_q = np.array([5, 50, 3, 109], np.int32)
    H, Hkv = 2, 1
    q = I.activations(H * 4, D, 806).reshape(H, 4, D)
    k = I.activations(Hkv * 100, D, 807).reshape(Hkv, 100, D)
    v = I.activations(Hkv * 100, D, 808).reshape(Hkv, 100, D)
    cos_t, sin_t = oracle.rope_tables(110, D, base=1e6)
    o = run(q, k, v, pos_q, pos_k, cos_t, sin_t, 1.0 / np.sqrt(D))
    assert (o[:, [0, 2]] == 0).all()
    sel = np.array([1, 3])
    o64, bnd = oracle.streaming_attention(q[:, sel], k, v, pos_q[sel], pos_k, cos_t, sin_t, np.float32(1.0 / np.sqrt(D)))
    assert (np.abs(o[:, sel] - o64) <= 2.0 ** -8 * np.abs(o64) + 2.0 ** -8 * bnd + 1e-30).all()


def test_long_cache_without_tile_skipping():
    # 10 frames x 4096 tokens of one view (40960 keys) under 4096 queries: so
    # many query blocks that the key range splits in 2 only, with more tiles
    # per split than the skip table holds, so every tile is computed and
    # masked (the path without tile skipping); 64 sampled queries
    pos_k, pos_q = window(1, 10, 4096, 3)
    H, Hkv, Nq, Nk = 8, 2, len(pos_q), len(pos_k)
    # workspace: 64 KiB, the rotated keys (H * Nk * 128 bf16), the partials
    rot = (H * Nk * 128 * 2 + 255) // 256 * 256
    bounds = ((Nk + 31) // 32 * 8 + 255) // 256 * 256
    assert (Nk + 31) // 32 > 1024  # past the dispatch schedule's limit: no schedule bytes
    S = (w.w4a8_stream_attention_workspace_bytes(H, Nq, Nk) - 64 * 1024 - rot - bounds) // (H * Nq * 130 * 4)
    assert S >= 1 and (Nk // 32) / S > 512
    rows = np.sort(np.random.Generator(np.random.PCG64(809)).choice(Nq, 64, replace=False))
    check(H, Hkv, pos_q, pos_k, 810, "long cache 1x10x4096", rows=rows)


def test_dispatch_schedule():
    # The key pre-pass deals the work items (query block, split, head) to
    # workgroup ids: ranked by visible key tiles, heaviest first, dealt in
    # rounds of one id per CU, every second full round reversed.  Read the
    # schedule back from a caller workspace and compare it with that rule
    # computed here from the positions; it must be a permutation, and the
    # per-CU tile sums of the 4x4x192 window must stay within 10 % of the
    # mean (94 against 87; the plain order gives up to 140).
    V, F, T, H, Hkv = 4, 4, 192, 32, 8
    pos_k, pos_q = window(V, F, T, 1)
    Nq, Nk = len(pos_q), len(pos_k)
    need = w.w4a8_stream_attention_workspace_bytes(H, Nq, Nk)
    ws = torch.zeros(need, dtype=torch.uint8, device=dev())
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)
    q = I.activations(H * Nq, D, 811).reshape(H, Nq, D)
    k = I.activations(Hkv * Nk, D, 812).reshape(Hkv, Nk, D)
    cos_t, sin_t = oracle.rope_tables(Nk, D, base=1e6)
    w.w4a8_stream_attention(t(q), t(k), t(k), torch.from_numpy(pos_q).to(dev()), torch.from_numpy(pos_k).to(dev()),
                            torch.from_numpy(cos_t).to(dev()), torch.from_numpy(sin_t).to(dev()), 0.1, workspace=ws)
    torch.cuda.synchronize()
    X, ntiles = (Nq + 63) // 64, (Nk + 31) // 32
    S = 2  # the split rule's choice here: 384 blocks x 2 fill one resident round
    tps = (ntiles + S - 1) // S
    G = X * S * H
    off = 64 * 1024 + (H * Nk * 128 * 2 + 255) // 256 * 256 + (ntiles * 8 + 255) // 256 * 256
    sched = ws[off:off + 4 * G].cpu().numpy().view(np.int32)
    assert sorted(sched.tolist()) == list(range(G))
    qmax = [pos_q[x * 64:(x + 1) * 64].max() for x in range(X)]
    tmin = [pos_k[u * 32:(u + 1) * 32].min() for u in range(ntiles)]
    vis = [sum(tmin[u] <= qmax[c // S] for u in range((c % S) * tps, min(ntiles, (c % S + 1) * tps)))
           for c in range(X * S)]
    order = sorted(range(X * S), key=lambda c: (-vis[c], c))
    C = torch.cuda.get_device_properties(0).multi_processor_count
    want = np.empty(G, np.int32)
    for kk in range(G):
        r, h = divmod(kk, H)
        rnd, pp = divmod(kk, C)
        rev = rnd % 2 == 1 and (rnd + 1) * C <= G
        want[rnd * C + (C - 1 - pp if rev else pp)] = order[r] * H + h
    assert np.array_equal(sched, want)
    # the solo table after it: the one split that sees keys of a block, else -1
    solo = ws[off + 4 * G:off + 4 * G + 4 * X].cpu().numpy().view(np.int32)
    nonempty = [[z for z in range(S) if vis[x * S + z] > 0] for x in range(X)]
    assert solo.tolist() == [ne[0] if len(ne) == 1 else -1 for ne in nonempty]
    assert (solo >= 0).any() and (solo < 0).any()  # both paths occur in this window
    if C == 256:
        cu = np.zeros(C)
        for i, code in enumerate(sched):
            cu[i % C] += vis[code // H]
        assert cu.max() <= 1.10 * cu.mean(), (cu.min(), cu.mean(), cu.max())


def test_rejected_calls():
    L = w.lib()
    import ctypes
    P = ctypes.c_void_p
    fake = P(1 << 20)
    f = L.w4a8_stream_attention
    args = lambda H=4, Hkv=2, Nq=8, Nk=16, Dd=128: (fake, fake, fake, fake, fake, fake, fake, 64, H, Hkv, Nq, Nk, Dd,
                                                    0.1, fake, None, 0, None)
    assert f(*args(Dd=64)) == w.W4A8_EUNSUPPORTED
    assert f(*args(H=4, Hkv=3)) == w.W4A8_EINVAL
    assert f(*args(Nk=0)) == w.W4A8_EINVAL
    assert f(*args(Nq=0)) == w.W4A8_OK
    # a split shape without its workspace
    assert w.w4a8_stream_attention_workspace_bytes(32, 768, 3072) > 0
    assert f(*args(H=32, Hkv=8, Nq=768, Nk=3072)) == w.W4A8_EINVAL
