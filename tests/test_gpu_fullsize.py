"""Parity at the full benchmark sizes, in the launch configuration bench.py
times: the 128K Qwen3-32B-shaped layer with bf16 factors (batch 4) and the
same heads with INT4 factors (batch 8).

As in bench.py, the seeded generator draws the prompt K/V, the GPU
decomposition builds the cache (per-page ranks drawn from {16, 24, 32}), and
one attention call covers the whole batch. Checked on what the oracle can
compute one head at a time:
* attention: for every (sequence, KV head) of the 128K bf16, INT4, adaptive
  and pre-RoPE layers, the paper-default layer and the Llama-3-8B layer, the
  oracle attends over that head's exported pages (dense pages as stored,
  factor pages as the GPU stored them -- for INT4 the dequantized balanced
  factors) with the same queries; bar max-abs <= 1e-2, normwise
  mean-relative <= 1e-3;
* decomposition: sampled factor pages against the oracle's SVD of the stored
  page (sign-invariant checks, as in test_gpu_compress);
* the page table: every entry's kind and ranks against the oracle's plan and
  the rank table, bit for bit."""
import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, errors
from test_gpu_compress import _adaptive_ok, _check_factor

pytestmark = pytest.mark.gpu


def _build(name):
    import torch
    import paper_2608_23843_amd as pk
    wl = synth.WORKLOADS[name]
    B, Hkv, Hq, d, P, T, S, W = (wl.batch, wl.kv_heads, wl.q_heads, wl.head_dim, wl.page, wl.tokens, wl.sink,
                                 wl.window)
    max_pages = -(-T // P)
    K, V = synth.kv_layer(wl, 0, 0, T, workers=16)
    ranks = synth.page_ranks(wl, 0, 0, max_pages)
    ranks_v = synth.page_ranks(wl, 0, 0, max_pages, "v")
    if wl.rank_error > 0:          # rank 0: the decomposition chooses
        ranks[:] = 0
        ranks_v[:] = 0
    cache = pk.PuzzleKVCache(1, B, Hkv, Hq, d, P, max_pages, max(wl.ranks + wl.ranks_v), S, W, wl.dtype,
                             wl.factors, adaptive_rank_error=wl.rank_error,
                             key_rope_base=wl.rope_base if wl.key_rope else 0.0)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    rt = torch.from_numpy(ranks).cuda().contiguous()
    rtv = torch.from_numpy(ranks_v).cuda().contiguous()
    cache.prefill(0, kt, vt, [T] * B, rank_k=rt, rank_v=rtv)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    del kt, vt
    return wl, cache, K, V, ranks, ranks_v


def _head_pages(cache, wl, b, h):
    n = -(-wl.tokens // wl.page)
    return cache.export_pages(0, [b] * n, [h] * n, list(range(n))).cpu().numpy().astype(np.float64)


def _run(name, heads, n_pages_checked, deep=None):
    """Attention of every head in `heads`; the chosen ranks (adaptive caches)
    and sampled decompositions of the heads in `deep` (default: all of them)."""
    import torch
    deep = set(heads if deep is None else deep)
    wl, cache, K, V, ranks, ranks_v = _build(name)
    B, Hkv, d, P, T = wl.batch, wl.kv_heads, wl.head_dim, wl.page, wl.tokens
    g, R = wl.group, max(wl.ranks + wl.ranks_v)
    n = -(-T // P)
    kinds = oracle.plan_pages(T, P, wl.sink, wl.window, n)
    # page table: kinds and ranks of every entry
    _, kind, rk, rv = cache.page_table_host(0)
    assert np.array_equal(kind[:, :, :n], np.broadcast_to(kinds, (B, Hkv, n)))
    fac = kinds == oracle.FACTOR
    if wl.rank_error > 0:
        # chosen ranks: within [1, cap] everywhere, checked against the
        # oracle's singular values on the sampled heads below
        for t in (rk, rv):
            assert t[:, :, :n][:, :, fac].min() >= 1 and t[:, :, :n][:, :, fac].max() <= R
        ranks, ranks_v = rk.astype(np.uint8), rv.astype(np.uint8)
    assert np.array_equal(rk[:, :, :n][:, :, fac], ranks[:, :, :n][:, :, fac])
    assert np.array_equal(rv[:, :, :n][:, :, fac], ranks_v[:, :, :n][:, :, fac])
    # one attention call over the whole batch, as bench.py makes it
    q = synth.queries(wl, 0, 0)
    qt = torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous()
    import paper_2608_23843_amd as pk
    ws = cache.workspace(pk.PKV_OP_ATTENTION, T)
    out, lse = cache.attention(0, qt, [T] * B, workspace=ws)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    rng = np.random.default_rng(11)
    checked = 0
    worst = [0.0, 0.0]
    for (b, h) in heads:
        blk = _head_pages(cache, wl, b, h)
        pages = []
        for j in range(n):
            o = blk[j]
            if kinds[j] == oracle.FACTOR:
                r, r_v = int(ranks[b, h, j]), int(ranks_v[b, h, j])
                Lk = o[:P * R].reshape(P, R)[:, :r]
                Rk = o[P * R:P * R + R * d].reshape(R, d)[:r]
                Lv = o[P * R + R * d:2 * P * R + R * d].reshape(P, R)[:, :r_v]
                Rv = o[2 * P * R + R * d:2 * P * R + 2 * R * d].reshape(R, d)[:r_v]
                pages.append(("factor", Lk, Rk, Lv, Rv))
            else:
                pages.append(("dense", o[:P * d].reshape(P, d), o[P * d:2 * P * d].reshape(P, d)))
        head = oracle.HeadCache(T, P, d, pages, key_rope_base=wl.rope_base if wl.key_rope else 0.0)
        ro, rl = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ma, mr = errors(out[b, h * g:(h + 1) * g], ro)
        print("%s head (%d, %d): max-abs %.3e, normwise mean-relative %.3e" % (name, b, h, ma, mr))
        assert ma <= MAX_ABS and mr <= MEAN_REL, (b, h, ma, mr)
        worst = [max(worst[0], ma), max(worst[1], mr)]
        assert np.abs(lse[b, h * g:(h + 1) * g] - rl).max() <= 1e-3
        if (b, h) not in deep:
            continue
        if wl.rank_error > 0:     # every factor page of this head: the chosen ranks
            for j in np.flatnonzero(fac):
                for X, rr in ((K[b, h, j * P:(j + 1) * P], rk[b, h, j]), (V[b, h, j * P:(j + 1) * P], rv[b, h, j])):
                    s = np.linalg.svd(synth.round_bf16(X).astype(np.float64), compute_uv=False)
                    assert _adaptive_ok(s, int(rr), wl.rank_error, R), (b, h, j, int(rr))
        # sampled decompositions of this head (bf16 factors; the INT4 path's
        # quantizer is checked against the oracle in test_gpu_int4)
        if wl.factors == "bf16":
            for j in rng.choice(np.flatnonzero(fac), n_pages_checked, replace=False):
                r, r_v = int(ranks[b, h, j]), int(ranks_v[b, h, j])
                Lk, Rk, Lv, Rv = pages[j][1:]
                for L, Rm, X, rr in ((Lk, Rk, K[b, h, j * P:(j + 1) * P], r),
                                     (Lv, Rv, V[b, h, j * P:(j + 1) * P], r_v)):
                    _check_factor(L, Rm, X.astype(np.float64), rr, 6e-3, 1e-2, 4e-3)
                    checked += 1
    print("%s: %d heads, worst max-abs %.3e, worst normwise mean-relative %.3e" % (name, len(heads), *worst))
    return checked


def test_fullsize_qwen32b_128k_bf16():
    """B=4, 64 q / 8 kv heads, d=128, P=64, T=131072, S=64, W=512, r in {16, 24, 32}:
    every (sequence, KV head) against the oracle."""
    checked = _run("qwen32b_128k", [(b, h) for b in range(4) for h in range(8)], 2)
    assert checked == 32 * 2 * 2


def test_fullsize_qwen32b_128k_tp8_share():
    """One GPU's share of the 128K layer under 8-way tensor parallelism by KV
    head (B=4, 1 kv head with 8 q heads): every sequence against the oracle."""
    checked = _run("qwen32b_128k_tp8", [(b, 0) for b in range(4)], 2)
    assert checked == 4 * 2 * 2


def test_fullsize_qwen32b_128k_adaptive_ranks():
    """The 128K layer with every page's ranks chosen by the decomposition for
    relative Frobenius error 0.2 (cap 32): attention of every (sequence, KV
    head); the chosen ranks of every factor page of three heads against the
    oracle's singular values, and sampled decompositions at those ranks."""
    heads = [(b, h) for b in range(4) for h in range(8)]
    checked = _run("qwen32b_128k_adaptive", heads, 4, deep=[(0, 0), (2, 3), (3, 7)])
    assert checked == 3 * 4 * 2


def test_fullsize_qwen32b_128k_pre_rope():
    """The 128K layer with keys cached before RoPE (rotated at access, base
    1e6): attention of every (sequence, KV head) against the oracle's fp64
    rotation, and sampled decompositions of the pre-RoPE pages of three."""
    heads = [(b, h) for b in range(4) for h in range(8)]
    checked = _run("qwen32b_128k_prerope", heads, 4, deep=[(0, 0), (1, 6), (3, 2)])
    assert checked == 3 * 4 * 2


def test_fullsize_qwen32b_int4():
    """B=8, same heads and length, INT4 factors with fp16 scales: every
    (sequence, KV head) against the oracle."""
    _run("qwen32b_int4", [(b, h) for b in range(8) for h in range(8)], 0)


def test_fullsize_paper_default_qwen8b_16k():
    """The paper's default configuration: Qwen3-8B heads (32 q / 8 kv, d=128),
    pages of 32 tokens, (r_K, r_V) = (16, 14), 32-token sink, dense region of
    the last completed page plus the partial page, T=16384: every KV head,
    three sampled decompositions each (two pages per wavefront at P = 32)."""
    checked = _run("qwen8b_paper_default", [(0, h) for h in range(8)], 3)
    assert checked == 8 * 3 * 2


def test_fullsize_llama8b_32k_all_heads():
    """B=1, 32 q / 8 kv heads, d=128, P=64, T=32768, S=64, W=256, r=24: every KV head."""
    checked = _run("llama8b_32k", [(0, h) for h in range(8)], 2)
    assert checked == 8 * 2 * 2


def _incr_head_pages(cache, b, h, n, kinds, P, d, r):
    blk = cache.export_pages(0, [b] * n, [h] * n, list(range(n))).cpu().numpy().astype(np.float64)
    pages = []
    for j in range(n):
        o = blk[j]
        if kinds[j] == oracle.FACTOR:
            pages.append(("factor", o[:P * r].reshape(P, r), o[P * r:P * r + r * d].reshape(r, d),
                          o[P * r + r * d:2 * P * r + r * d].reshape(P, r),
                          o[2 * P * r + r * d:2 * P * r + 2 * r * d].reshape(r, d)))
        else:
            pages.append(("dense", o[:P * d].reshape(P, d), o[P * d:2 * P * d].reshape(P, d)))
    return pages


def test_fullsize_incremental_512_steps():
    """Incremental decode at full size, the whole schedule: batch 32,
    Llama-3-8B heads, prefill 16K, then 512 decode steps. Each step appends
    one token per sequence; at each of the 8 window boundaries all 32 x 8
    newly eligible pages are compressed before that step's attention. After
    every boundary the page table (kinds, ranks, dense rows) is checked bit
    for bit against the oracle's plan, the new factor pages of sampled heads
    against the oracle's SVD of the stored page, and the boundary step's
    attention of sampled heads against the oracle; at the end the appended
    tokens are checked as stored."""
    import torch
    import paper_2608_23843_amd as pk
    wl = synth.WORKLOADS["llama8b_incremental"]
    B, Hkv, Hq, d, P, T, S, W = (wl.batch, wl.kv_heads, wl.q_heads, wl.head_dim, wl.page, wl.tokens, wl.sink,
                                 wl.window)
    steps = wl.decode_steps
    max_pages = -(-(T + steps + 1) // P) + 1
    K, V = synth.kv_layer(wl, 0, 0, T, workers=16)
    ranks = synth.page_ranks(wl, 0, 0, max_pages)
    r = int(wl.ranks[0])
    g = wl.group
    cache = pk.PuzzleKVCache(1, B, Hkv, Hq, d, P, max_pages, r, S, W, wl.dtype, wl.factors)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    rt = torch.from_numpy(ranks).cuda().contiguous()
    cache.prefill(0, kt, vt, [T] * B, rank_k=rt, rank_v=rt)
    del kt, vt
    ws = cache.workspace(pk.PKV_OP_ATTENTION, T + steps + 1)
    Kd, Vd = {}, {}
    boundaries = []
    sample = [(0, 0), (13, 4), (31, 7)]
    worst = [0.0, 0.0]
    for s in range(steps):
        pos = T + s
        kn, vn = synth.decode_kv(wl, 0, 0, pos)
        Kd[pos], Vd[pos] = kn, vn
        cache.append(0, torch.from_numpy(kn).to("cuda", torch.bfloat16).contiguous(),
                     torch.from_numpy(vn).to("cuda", torch.bfloat16).contiguous(), [pos] * B)
        el = pk.eligible_pages(pos, pos + 1, P, S, W)
        assert np.array_equal(el, oracle.eligible_pages(pos, pos + 1, P, S, W))
        if len(el):
            bb, hh, jj = zip(*[(b, h, int(j)) for b in range(B) for h in range(Hkv) for j in el])
            cache.compress_pages(0, bb, hh, jj, r, r)
        qs = synth.queries(wl, 0, s)
        out, lse = cache.attention(0, torch.from_numpy(qs).to("cuda", torch.bfloat16).contiguous(), [pos + 1] * B,
                                   workspace=ws)
        if not len(el):
            continue
        # a boundary step: table, new factor pages and attention of sampled heads
        torch.cuda.synchronize()
        assert cache.device_status() == 0, pos
        boundaries += list(el)
        Tn = pos + 1
        n = -(-Tn // P)
        kinds = oracle.plan_pages(Tn, P, S, W, max_pages)
        t = cache.page_table(0).cpu().numpy()
        assert np.array_equal(t[..., 4], np.broadcast_to(kinds, t[..., 4].shape)), Tn
        fac = kinds == oracle.FACTOR
        assert np.all(t[..., 5][:, :, fac] == r) and np.all(t[..., 6][:, :, fac] == r), Tn
        rows = np.array([min(P, Tn - j * P) if kinds[j] == oracle.DENSE else 0 for j in range(max_pages)])
        assert np.array_equal(t[..., 7], np.broadcast_to(rows, t[..., 7].shape)), Tn
        o_np, l_np = out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)
        for (b, h) in sample:
            pages = _incr_head_pages(cache, b, h, n, kinds[:n], P, d, r)
            for j in el:
                # the stored page: prompt rows, or rows appended while decoding (bf16)
                Xk = np.stack([K[b, h, t] if t < T else synth.round_storage(Kd[t][b, h], "bf16")
                               for t in range(j * P, (j + 1) * P)]).astype(np.float64)
                Xv = np.stack([V[b, h, t] if t < T else synth.round_storage(Vd[t][b, h], "bf16")
                               for t in range(j * P, (j + 1) * P)]).astype(np.float64)
                _check_factor(pages[j][1], pages[j][2], Xk, r, 6e-3, 1e-2, 4e-3)
                _check_factor(pages[j][3], pages[j][4], Xv, r, 6e-3, 1e-2, 4e-3)
            ro, rl = oracle.attention(oracle.HeadCache(Tn, P, d, pages), qs[b, h * g:(h + 1) * g].astype(np.float64))
            ma, mr = errors(o_np[b, h * g:(h + 1) * g], ro)
            assert ma <= MAX_ABS and mr <= MEAN_REL, (Tn, b, h, ma, mr)
            assert np.abs(l_np[b, h * g:(h + 1) * g] - rl).max() <= 1e-3
            worst = [max(worst[0], ma), max(worst[1], mr)]
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    assert len(boundaries) == 8 and boundaries == [(T - W) // P + i for i in range(8)]
    print("llama8b_incremental: 512 steps, 8 boundaries, worst max-abs %.3e, worst normwise mean-relative %.3e"
          % tuple(worst))
    # the appended tokens, as stored
    Tn = T + steps
    n = -(-Tn // P)
    kinds = oracle.plan_pages(Tn, P, S, W, n)
    for (b, h) in sample:
        pages = _incr_head_pages(cache, b, h, n, kinds, P, d, r)
        for pos in range(T, Tn):
            j, row = divmod(pos, P)
            if kinds[j] != oracle.DENSE:
                continue
            assert np.array_equal(pages[j][1][row], synth.round_storage(Kd[pos][b, h], "bf16").astype(np.float64))
            assert np.array_equal(pages[j][2][row], synth.round_storage(Vd[pos][b, h], "bf16").astype(np.float64))


def test_fullsize_qwen32b_128k_global():
    """The Global SVD baseline at the 128K layer (B = 4, rank 71, matched to
    PuzzleKV's whole-cache ratio there): the page table; for sampled heads the
    basis (orthonormal rows), the coefficients (the projection with the
    stored basis), the Eckart-Young error against LAPACK's spectral tail of
    the region (the oracle's Jacobi SVD of a 130K-row region is out of reach
    here; it is checked against the oracle at smaller sizes in
    test_gpu_global), and attention against the oracle over the exported
    factors."""
    import torch
    import paper_2608_23843_amd as pk
    wl = synth.WORKLOADS["qwen32b_128k_global"]
    B, Hkv, Hq, d, P, T, S, W = (wl.batch, wl.kv_heads, wl.q_heads, wl.head_dim, wl.page, wl.tokens, wl.sink,
                                 wl.window)
    g = wl.group
    kinds = oracle.plan_pages(T, P, S, W)
    fac = [j for j, k in enumerate(kinds) if k == oracle.FACTOR]
    rows = np.concatenate([np.arange(j * P, (j + 1) * P) for j in fac])
    r = pk.global_rank(T, P, S, W, d, wl.global_rho)
    assert r == 71
    K, V = synth.kv_layer(wl, 0, 0, T, workers=16)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hq, d, P, len(kinds), 1, S, W, "bf16", "bf16")
    gs = pk.GlobalSVD(cache, r, -(-len(rows) // 32) * 32)
    gs.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16), torch.from_numpy(V).to("cuda", torch.bfloat16),
               [T] * B)
    q = synth.queries(wl, 0, 0)
    out, lse = gs.attention(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous(), [T] * B)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    t = cache.page_table(0).cpu().numpy()
    want = np.where(kinds == oracle.FACTOR, 3, kinds)
    assert np.array_equal(t[..., 4], np.broadcast_to(want, t[..., 4].shape))
    out, lse = out.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)
    for (b, h) in [(0, 0), (2, 5), (3, 7)]:
        bk, bv, ak, av = (x.cpu().numpy().astype(np.float64) for x in gs.export(0, b, h, len(rows)))
        for X, Bm, Am in ((K[b, h][rows].astype(np.float64), bk, ak), (V[b, h][rows].astype(np.float64), bv, av)):
            assert np.abs(Bm @ Bm.T - np.eye(r)).max() < 1e-2
            Pj = X @ Bm.T
            assert np.abs(Am - Pj).sum() <= 2.0 ** -8 * np.abs(Pj).sum()
            sig = np.linalg.svd(X, compute_uv=False)
            err = np.sqrt(np.sum((X - Am @ Bm) ** 2))
            tail, fro = np.sqrt(np.sum(sig[r:] ** 2)), np.sqrt(np.sum(X * X))
            assert tail - 1e-3 * fro <= err <= tail * (1 + 1e-3) + 4 * 2.0 ** -9 * fro, (b, h, err, tail, fro)
        head = oracle.global_head(T, P, d, kinds, K[b, h], V[b, h], ak, bk, av, bv)
        ro, rl = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ma, mr = errors(out[b, h * g:(h + 1) * g], ro)
        print("qwen32b_128k_global head (%d, %d): max-abs %.3e, normwise mean-relative %.3e" % (b, h, ma, mr))
        assert ma <= MAX_ABS and mr <= MEAN_REL, (b, h, ma, mr)
        assert np.abs(lse[b, h * g:(h + 1) * g] - rl).max() <= 1e-3
