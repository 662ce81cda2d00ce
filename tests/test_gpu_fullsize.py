"""Parity at the full benchmark sizes, in the launch configuration bench.py
times: the 128K Qwen3-32B-shaped layer with bf16 factors (batch 4) and the
same heads with INT4 factors (batch 8).

As in bench.py, the seeded generator draws the prompt K/V, the GPU
decomposition builds the cache (per-page ranks drawn from {16, 24, 32}), and
one attention call covers the whole batch. Checked on samples the oracle can
compute one by one:
* attention: for sampled (sequence, KV head) pairs, the oracle attends over
  that head's exported pages (dense pages as stored, factor pages as the GPU
  stored them -- for INT4 the dequantized balanced factors) with the same
  queries; bar max-abs <= 1e-2, normwise mean-relative <= 1e-3;
* decomposition: sampled factor pages against the oracle's SVD of the stored
  page (sign-invariant checks, as in test_gpu_compress);
* the page table: every entry's kind and ranks against the oracle's plan and
  the rank table, bit for bit."""
import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, errors
from test_gpu_compress import _check_factor

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
    cache = pk.PuzzleKVCache(1, B, Hkv, Hq, d, P, max_pages, max(wl.ranks), S, W, wl.dtype, wl.factors)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    rt = torch.from_numpy(ranks).cuda().contiguous()
    cache.prefill(0, kt, vt, [T] * B, rank_k=rt, rank_v=rt)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    del kt, vt
    return wl, cache, K, V, ranks


def _head_pages(cache, wl, b, h):
    n = -(-wl.tokens // wl.page)
    return cache.export_pages(0, [b] * n, [h] * n, list(range(n))).cpu().numpy().astype(np.float64)


def _run(name, heads, n_pages_checked):
    import torch
    wl, cache, K, V, ranks = _build(name)
    B, Hkv, d, P, T = wl.batch, wl.kv_heads, wl.head_dim, wl.page, wl.tokens
    g, R = wl.group, max(wl.ranks)
    n = -(-T // P)
    kinds = oracle.plan_pages(T, P, wl.sink, wl.window, n)
    # page table: kinds and ranks of every entry
    _, kind, rk, rv = cache.page_table_host(0)
    assert np.array_equal(kind[:, :, :n], np.broadcast_to(kinds, (B, Hkv, n)))
    fac = kinds == oracle.FACTOR
    assert np.array_equal(rk[:, :, :n][:, :, fac], ranks[:, :, :n][:, :, fac])
    assert np.array_equal(rv[:, :, :n][:, :, fac], ranks[:, :, :n][:, :, fac])
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
    for (b, h) in heads:
        blk = _head_pages(cache, wl, b, h)
        pages = []
        for j in range(n):
            o = blk[j]
            if kinds[j] == oracle.FACTOR:
                r = int(ranks[b, h, j])
                Lk = o[:P * R].reshape(P, R)[:, :r]
                Rk = o[P * R:P * R + R * d].reshape(R, d)[:r]
                Lv = o[P * R + R * d:2 * P * R + R * d].reshape(P, R)[:, :r]
                Rv = o[2 * P * R + R * d:2 * P * R + 2 * R * d].reshape(R, d)[:r]
                pages.append(("factor", Lk, Rk, Lv, Rv))
            else:
                pages.append(("dense", o[:P * d].reshape(P, d), o[P * d:2 * P * d].reshape(P, d)))
        head = oracle.HeadCache(T, P, d, pages)
        ro, rl = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ma, mr = errors(out[b, h * g:(h + 1) * g], ro)
        print("%s head (%d, %d): max-abs %.3e, normwise mean-relative %.3e" % (name, b, h, ma, mr))
        assert ma <= MAX_ABS and mr <= MEAN_REL, (b, h, ma, mr)
        assert np.abs(lse[b, h * g:(h + 1) * g] - rl).max() <= 1e-3
        # sampled decompositions of this head (bf16 factors; the INT4 path's
        # quantizer is checked against the oracle in test_gpu_int4)
        if wl.factors == "bf16":
            for j in rng.choice(np.flatnonzero(fac), n_pages_checked, replace=False):
                r = int(ranks[b, h, j])
                Lk, Rk, Lv, Rv = pages[j][1:]
                for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
                    _check_factor(L, Rm, X.astype(np.float64), r, 6e-3, 1e-2, 4e-3)
                    checked += 1
    return checked


def test_fullsize_qwen32b_128k_bf16():
    """B=4, 64 q / 8 kv heads, d=128, P=64, T=131072, S=64, W=512, r in {16, 24, 32}."""
    checked = _run("qwen32b_128k", [(0, 0), (1, 5), (3, 7)], 4)
    assert checked == 3 * 4 * 2


def test_fullsize_qwen32b_int4():
    """B=8, same heads and length, INT4 factors with fp16 scales."""
    _run("qwen32b_int4", [(0, 0), (4, 3), (7, 7)], 0)
