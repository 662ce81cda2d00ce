"""GPU parity of pkv_mixed_decode_attention against the oracle (Eq. (1) over
the rebuilt cache), through the C ABI.

Both sides read the same stored pages: dense pages from the seeded generator
and factor pages from the oracle's Eq. (2) decomposition of those pages,
rounded to the storage type and written into the GPU cache by
pkv_import_pages. Bar: max-abs <= 1e-2 and normwise mean-relative <= 1e-3
(bf16 storage, fp32 accumulation); fp32 storage is held to 1e-5."""
import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, build_head_pages, errors, import_head, oracle_head

pytestmark = pytest.mark.gpu


def _workload(B, Hkv, g, d, P, T, S, W, r0, dtype, rope=None, outliers=0, wid=90):
    return synth.Workload("case", wid, B, Hkv, Hkv * g, d, P, T, S, W, r0, (r0,), dtype, rope, outliers)


def run_case(B, Hkv, g, d, P, seq_lens, S, W, ranks, dense_dtype="bf16", factor_dtype="bf16",
             seed=0, r0=None, rope=None, outliers=0, wid=90):
    """ranks: int, or callable (b, h, j) -> (rk, rv)."""
    import torch
    import paper_2608_23843_amd as pk
    Tmax = max(seq_lens)
    max_pages = max(1, -(-Tmax // P))
    max_rank = 1
    rank_of = ranks if callable(ranks) else (lambda b, h, j: (ranks, ranks))
    for b in range(B):
        for h in range(Hkv):
            for j in range(max_pages):
                max_rank = max(max_rank, *rank_of(b, h, j))
    wl = _workload(B, Hkv, g, d, P, Tmax, S, W, r0 or 8, dense_dtype, rope, outliers, wid)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, d, P, max_pages, max_rank, S, W, dense_dtype,
                             factor_dtype)
    heads = {}
    for b in range(B):
        T = seq_lens[b]
        if T == 0:
            continue
        for h in range(Hkv):
            K, V = synth.kv_head(wl, seed, 0, b, h, max_pages * P)
            rk = [rank_of(b, h, j) for j in range(max_pages)]
            pages = build_head_pages(K.astype(np.float64), V.astype(np.float64), T, P, S, W, rk,
                                     factor_dtype)
            import_head(cache, 0, b, h, pages)
            heads[(b, h)] = oracle_head(T, P, d, pages)
    q = synth.queries(wl, seed)
    qt = torch.from_numpy(q).to(device="cuda", dtype=cache.qdtype).contiguous()
    out, lse = cache.attention(0, qt, seq_lens)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    ref = np.zeros_like(out)
    ref_lse = np.full_like(lse, -np.inf)
    for (b, h), head in heads.items():
        o, l = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ref[b, h * g:(h + 1) * g] = o
        ref_lse[b, h * g:(h + 1) * g] = l
    return out, ref, lse, ref_lse


def _assert_close(out, ref, lse, ref_lse, tight=False):
    ma, mr = errors(out, ref)
    if tight:
        assert ma <= 1e-5 * max(1.0, np.abs(ref).max()) and mr <= 1e-5, (ma, mr)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (ma, mr)
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isfinite(lse), fin)
    assert np.abs(lse[fin] - ref_lse[fin]).max(initial=0.0) <= (1e-5 if tight else 1e-3)


def test_tiny_workload_fp32():
    """Tiny workload: 1 KV head, 1 query head, d=64, P=16, T=256, 16 sink and
    32 window tokens, 13 middle pages at rank 4, fp32."""
    wl = synth.WORKLOADS["tiny"]
    out, ref, lse, rl = run_case(1, 1, 1, wl.head_dim, wl.page, [wl.tokens], wl.sink, wl.window, 4,
                                 "f32", "f32", r0=4, wid=wl.wid)
    _assert_close(out, ref, lse, rl, tight=True)


def test_llama_shape_subset_bf16():
    """Llama-3-8B head geometry (g=4, d=128, P=64, r=24, RoPE keys with outlier
    channels), 2 KV heads, ragged tail."""
    out, ref, lse, rl = run_case(1, 2, 4, 128, 64, [1024 + 37], 64, 256, 24, r0=24, rope=5e5,
                                 outliers=4)
    _assert_close(out, ref, lse, rl)


def test_qwen_shape_variable_ranks_bf16():
    """Qwen3-32B head geometry (g=8, 512-token window) with per-page ranks drawn
    from {16, 24, 32}; two sequences of different length."""
    rng = np.random.default_rng(3)
    table = rng.choice([16, 24, 32], size=(2, 2, 64))
    out, ref, lse, rl = run_case(2, 2, 8, 128, 64, [2048 + 5, 1536], 64, 512,
                                 lambda b, h, j: (int(table[b, h, j]), int(table[b, h, j])),
                                 r0=24, rope=1e6, outliers=4)
    _assert_close(out, ref, lse, rl)


@pytest.mark.parametrize("P", [16, 32])
def test_small_pages_asymmetric_ranks(P):
    """Paper-default style geometry: sink one page, window one page, and
    different key / value ranks (r_K, r_V) = (P/2, P/2 - 2)."""
    out, ref, lse, rl = run_case(2, 2, 4, 128, P, [P * 20 + 3, P * 7], P, P,
                                 lambda b, h, j: (P // 2, P // 2 - 2), r0=P // 2)
    _assert_close(out, ref, lse, rl)


def test_edge_lengths():
    """T=1, a single partial page, an empty sequence and a long one in one batch."""
    out, ref, lse, rl = run_case(4, 1, 2, 64, 16, [1, 15, 0, 16 * 9 + 1], 16, 32, 4)
    assert np.all(out[2] == 0) and np.all(np.isneginf(lse[2]))
    _assert_close(out, ref, lse, rl)


def test_no_sink_no_window_and_rank_one():
    out, ref, lse, rl = run_case(1, 2, 2, 64, 16, [16 * 6 + 9], 0, 0, 1)
    _assert_close(out, ref, lse, rl)


def test_full_rank_factors_match_dense_fp32():
    """Factor pages at r = P reproduce the page exactly (Eq. (2) at full rank):
    the GPU result over full-rank factors equals the oracle's dense attention."""
    import torch
    import paper_2608_23843_amd as pk
    P, d, T, g = 16, 64, 16 * 5, 2
    wl = _workload(1, 1, g, d, P, T, 0, 0, 8, "f32")
    K, V = synth.kv_head(wl, 1, 0, 0, 0, T)
    pages = build_head_pages(K.astype(np.float64), V.astype(np.float64), T, P, 0, 0, P, "f32")
    cache = pk.PuzzleKVCache(1, 1, 1, g, d, P, 5, P, 0, 0, "f32", "f32")
    import_head(cache, 0, 0, 0, pages)
    q = synth.queries(wl, 1)
    out, lse = cache.attention(0, torch.from_numpy(q).cuda().contiguous(), [T])
    dense = oracle.HeadCache(T, P, d, [("dense", K[j * P:(j + 1) * P].astype(np.float64),
                                        V[j * P:(j + 1) * P].astype(np.float64)) for j in range(5)])
    ref, _ = oracle.attention(dense, q[0].astype(np.float64))
    ma, mr = errors(out.cpu().numpy()[0], ref)
    assert ma < 1e-4 and mr < 1e-5, (ma, mr)


def test_repeated_calls_share_workspace():
    """The merge and page counters return to zero after every call, so calls
    that reuse one workspace give the same results, for both kernels (bf16
    pages use the matrix-core kernel, fp32 pages the generic one). The generic
    kernel's chunks are fixed, so it repeats bit for bit; the matrix-core
    kernel hands pages to waves dynamically, so its summation order (and the
    last bits) may change between calls."""
    import torch
    import paper_2608_23843_amd as pk
    for dt, P in (("bf16", 64), ("f32", 16)):
        wl = _workload(2, 2, 4, 128, P, P * 40, P, P * 2, 8, dt)
        cache = pk.PuzzleKVCache(1, 2, 2, 8, 128, P, 40, 8, P, 2 * P, dt, dt)
        for b in range(2):
            for h in range(2):
                K, V = synth.kv_head(wl, 0, 0, b, h, P * 40)
                pages = build_head_pages(K.astype(np.float64), V.astype(np.float64), P * 40, P, P, 2 * P,
                                         8, dt)
                import_head(cache, 0, b, h, pages)
        q = torch.from_numpy(synth.queries(wl, 0)).to("cuda", cache.qdtype).contiguous()
        ws = cache.workspace(pk.PKV_OP_ATTENTION, P * 40)
        first, lse0 = cache.attention(0, q, [P * 40, P * 33], workspace=ws)
        first, lse0 = first.clone(), lse0.clone()
        for _ in range(3):
            out, lse = cache.attention(0, q, [P * 40, P * 33], workspace=ws)
            if dt == "f32":
                assert torch.equal(out, first) and torch.equal(lse, lse0)
            else:
                scale = float(first.abs().max())
                assert float((out - first).abs().max()) <= 1e-5 * scale
                assert float((lse - lse0).abs().max()) <= 1e-5
        assert np.all(ws[-16:].cpu().numpy() == 0)


@pytest.mark.parametrize("g", [1, 16])
def test_query_group_extremes_bf16(g):
    """One query head per KV head (g = 1, 15 of the 16 MFMA columns unused)
    and the largest supported group (g = 16), d = 128, P = 64."""
    out, ref, lse, rl = run_case(2, 2, g, 128, 64, [64 * 11 + 20, 64 * 6], 64, 128,
                                 lambda b, h, j: (24 - (j % 3) * 4, 20), r0=24, wid=91)
    _assert_close(out, ref, lse, rl)


def test_ragged_lengths_around_unit_boundaries():
    """P = 64 dense pages are streamed as two 32-token units: lengths just
    below, at and above 32, 64 and the window edge, in one batch, with heads
    too short to fill one round of page claims."""
    lens = [1, 31, 32, 33, 63, 64, 65, 127, 129, 64 * 9 + 31, 64 * 9 + 32, 64 * 9 + 33]
    out, ref, lse, rl = run_case(len(lens), 1, 4, 128, 64, lens, 64, 128,
                                 lambda b, h, j: (16 + 4 * (j % 4), 32 - 4 * (j % 3)), r0=24, wid=92)
    _assert_close(out, ref, lse, rl)


def test_largest_batch():
    """255 sequences (the batch limit) of lengths 0 .. 260 in one call."""
    rng = np.random.default_rng(8)
    lens = [int(x) for x in rng.integers(0, 261, 255)]
    lens[0], lens[1] = 0, 260
    out, ref, lse, rl = run_case(255, 1, 2, 64, 32, lens, 32, 32, 8, r0=8, wid=93)
    for b, T in enumerate(lens):
        if T == 0:
            assert np.all(out[b] == 0) and np.all(np.isneginf(lse[b]))
    _assert_close(out, ref, lse, rl)


def test_many_chunks_per_head_16byte_merge():
    """Heads of 8 queries x 128 dims (more outputs than one pass of the
    workgroup's threads, so the last workgroup folds with 16-byte loads) and
    301 pages per sequence in a batch of two: 101 chunks per head (several
    groups of 32, an odd count against two lanes per output group), the
    shorter sequence leaving its last chunks empty."""
    rng = np.random.default_rng(5)
    T0 = 301 * 64 - 10
    table = rng.choice([16, 24, 32], size=(2, 1, 301))
    out, ref, lse, rl = run_case(2, 1, 8, 128, 64, [T0, 3000], 64, 512,
                                 lambda b, h, j: (int(table[b, h, j]), int(table[b, h, j])),
                                 r0=24, rope=1e6, outliers=4)
    _assert_close(out, ref, lse, rl)


@pytest.mark.parametrize("case", range(12))
def test_random_geometries(case):
    """Seeded draws over the bf16 matrix-core kernel's geometry: (d, P)
    cycling over {64, 128} x {16, 32, 64}, query group 1..16, sink and window of 0..3
    pages (in tokens, not always page multiples), ranks 1..min(P, 32) drawn
    per page for K and V separately, 1..4 sequences of ragged lengths (one
    possibly empty)."""
    rng = np.random.default_rng(1000 + case)
    d = (64, 128)[(case // 3) % 2]
    P = (16, 32, 64)[case % 3]
    g = int(rng.integers(1, 17))
    Hkv = int(rng.integers(1, 4))
    B = int(rng.integers(1, 5))
    S = int(rng.integers(0, 3 * P + 1))
    W = int(rng.integers(0, 3 * P + 1))
    rmax = min(P, 32)
    lens = [int(rng.integers(1, 40 * P)) for _ in range(B)]
    if B > 1 and rng.random() < 0.3:
        lens[int(rng.integers(0, B))] = 0
    rk = rng.integers(1, rmax + 1, (B, Hkv, 64))
    rv = rng.integers(1, rmax + 1, (B, Hkv, 64))
    out, ref, lse, rl = run_case(B, Hkv, g, d, P, lens, S, W,
                                 lambda b, h, j: (int(rk[b, h, j % 64]), int(rv[b, h, j % 64])),
                                 r0=int(rng.integers(2, rmax + 1)), wid=100 + case)
    print("case %d: B=%d Hkv=%d g=%d d=%d P=%d S=%d W=%d lens=%s" % (case, B, Hkv, g, d, P, S, W, lens))
    for b, T in enumerate(lens):
        if T == 0:
            assert np.all(out[b] == 0) and np.all(np.isneginf(lse[b]))
    _assert_close(out, ref, lse, rl)


def test_workspace_reuse_across_chunk_counts():
    """One workspace serves calls whose lengths give different chunk counts
    (at B = 1, 8 KV heads, P = 32 a head of 1,000 tokens splits into 32
    chunks, one of 1,100 tokens into 18): the counters sit at a fixed offset,
    so every call matches a call on a fresh workspace and the oracle, and the
    counters read zero afterwards."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, g, d, P, S, W, r = 1, 8, 4, 128, 32, 32, 32, 16
    lens = (1000, 1100)
    wl = _workload(B, Hkv, g, d, P, max(lens), S, W, 8, "bf16", wid=93)
    caches, refs = [], []
    q = synth.queries(wl, 0)
    qt = torch.from_numpy(q).to(device="cuda", dtype=torch.bfloat16).contiguous()
    for T in lens:
        max_pages = -(-max(lens) // P)
        cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, d, P, max_pages, r, S, W, "bf16", "bf16")
        ref = np.zeros((B, Hkv * g, d))
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, 0, h, max_pages * P)
            pages = build_head_pages(K.astype(np.float64), V.astype(np.float64), T, P, S, W, r, "bf16")
            import_head(cache, 0, 0, h, pages)
            ref[0, h * g:(h + 1) * g], _ = oracle.attention(oracle_head(T, P, d, pages),
                                                            q[0, h * g:(h + 1) * g].astype(np.float64))
        caches.append(cache)
        refs.append(ref)
    sizes = [caches[0].workspace_bytes(pk.PKV_OP_ATTENTION, T) for T in lens]
    assert sizes[0] != sizes[1], "the two lengths must give different partial layouts"
    ws = caches[0].workspace(pk.PKV_OP_ATTENTION, 4096)
    for rep in range(2):
        for cache, T, ref in zip(caches, lens, refs):
            out, lse = cache.attention(0, qt, [T], workspace=ws)
            fresh, lse_f = cache.attention(0, qt, [T], workspace=cache.workspace(pk.PKV_OP_ATTENTION, T))
            torch.cuda.synchronize()
            assert cache.device_status() == 0
            o = out.cpu().numpy().astype(np.float64)
            assert float((out - fresh).abs().max()) <= 1e-5 * float(fresh.abs().max())
            assert float((lse - lse_f).abs().max()) <= 1e-5
            ma, mr = errors(o, ref)
            assert ma <= MAX_ABS and mr <= MEAN_REL, (T, rep, ma, mr)
    heads = B * Hkv
    counters = (4 * heads + 255) // 256 * 256 + 256 * heads
    assert int(ws[:counters].count_nonzero()) == 0
