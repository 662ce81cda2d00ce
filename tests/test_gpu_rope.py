"""Caches of pre-RoPE keys (Section 4.2 "Main Results"; Appendix "RoPE Key
Analysis"): the keys are cached and factorized before the rotation, and the
attention rotates every key to its position when it reads the cache.

Each test compares the GPU attention with the oracle's textbook attention
over the same stored pages (dense pages as stored, factor pages as the GPU
stored them or as the oracle decomposed them), the oracle rotating the
rebuilt keys in fp64. Bar: max-abs <= 1e-2, normwise mean-relative <= 1e-3.
Ranks include values that are not multiples of 4 (padding of R_K^T) and the
sequences end inside a page (masked dense tail)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, build_head_pages, errors, import_head

pytestmark = pytest.mark.gpu

BASE = 1.0e6


def _pages_from_export(cache, b, h, n, plan, rk, rv, P, d, R):
    # rows of the last dense page past the sequence hold whatever the slot
    # held before (any bit pattern); the oracle never reads them
    with np.errstate(invalid="ignore"):
        blk = cache.export_pages(0, [b] * n, [h] * n, list(range(n))).cpu().numpy().astype(np.float64)
    pages = []
    for j in range(n):
        o = blk[j]
        if plan[j] == oracle.FACTOR:
            a, c = int(rk[b, h, j]), int(rv[b, h, j])
            pages.append(("factor", o[:P * R].reshape(P, R)[:, :a], o[P * R:P * R + R * d].reshape(R, d)[:a],
                          o[P * R + R * d:2 * P * R + R * d].reshape(P, R)[:, :c],
                          o[2 * P * R + R * d:2 * P * R + 2 * R * d].reshape(R, d)[:c]))
        else:
            pages.append(("dense", o[:P * d].reshape(P, d), o[P * d:2 * P * d].reshape(P, d)))
    return pages


def _check(cache, q, seq, plan_of, rk, rv, P, d, R, G, label):
    import torch
    out, lse = cache.attention(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous(), seq)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    worst = 0.0
    for b, T in enumerate(seq):
        if T == 0:   # empty sequences are checked by the caller
            continue
        n = -(-T // P)
        for h in range(cache.c.n_kv_heads):
            pages = _pages_from_export(cache, b, h, n, plan_of(T, n), rk, rv, P, d, R)
            ro, rl = oracle.attention(oracle.HeadCache(T, P, d, pages, key_rope_base=BASE),
                                      q[b, h * G:(h + 1) * G].astype(np.float64))
            ma, mr = errors(out[b, h * G:(h + 1) * G], ro)
            assert ma <= MAX_ABS and mr <= MEAN_REL, (label, b, h, ma, mr)
            assert np.abs(lse[b, h * G:(h + 1) * G] - rl).max() <= 1e-3, (label, b, h)
            worst = max(worst, mr)
    print("%s: worst normwise mean-relative %.3e" % (label, worst))


@pytest.mark.parametrize("d,P,G", [(128, 64, 8), (128, 32, 4), (64, 64, 8), (64, 32, 16)])
def test_pre_rope_prefill_then_attention(d, P, G):
    """Pre-RoPE keys decomposed by the GPU at ranks drawn from {5, 13, 22,
    32} (K and V separately), then attended: two sequences ending inside a
    page, the shorter one partly outside the other's pages."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, S, W = 2, 2, P, 2 * P
    T = [P * 12 + 9, P * 7 + 30]
    npg = -(-max(T) // P)
    R = 32
    wl = synth.Workload("rope", 94, B, Hkv, Hkv * G, d, P, max(T), S, W, 24, (24,), "bf16", BASE, 4,
                        key_rope=True)
    K, V = synth.kv_layer(wl, 0, 0, npg * P)
    rng = np.random.default_rng(5)
    rk = rng.choice(np.array([5, 13, 22, 32], dtype=np.uint8), (B, Hkv, npg))
    rv = rng.choice(np.array([5, 13, 22, 32], dtype=np.uint8), (B, Hkv, npg))
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * G, d, P, npg, R, S, W, "bf16", "bf16", key_rope_base=BASE)
    cache.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), T,
                  rank_k=torch.from_numpy(rk).cuda().contiguous(), rank_v=torch.from_numpy(rv).cuda().contiguous())
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    q = synth.queries(wl, 0, 0)
    _check(cache, q, T, lambda Tb, n: oracle.plan_pages(Tb, P, S, W, n), rk, rv, P, d, R, G,
           "prefill d=%d P=%d" % (d, P))


def test_pre_rope_imported_oracle_factors():
    """Factor pages from the oracle's own decomposition of the pre-RoPE keys
    and dense pages, imported through the C ABI: no GPU decomposition
    involved, so this pins the attention side alone."""
    import torch
    import paper_2608_23843_amd as pk
    d, P, G, B, Hkv, S, W = 128, 64, 8, 1, 2, 64, 128
    T = P * 10 + 41
    n = -(-T // P)
    wl = synth.Workload("rope_imp", 95, B, Hkv, Hkv * G, d, P, T, S, W, 24, (24,), "bf16", BASE, 4,
                        key_rope=True)
    K, V = synth.kv_layer(wl, 0, 0, n * P)
    R = 24
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * G, d, P, n, R, S, W, "bf16", "bf16", key_rope_base=BASE)
    cache.reset()
    ranks = [(r, 23 - (j % 5)) for j, r in enumerate([24, 7, 18, 21, 24, 11, 24, 15, 24, 24, 24])][:n]
    q = synth.queries(wl, 0, 0)
    refs = []
    for h in range(Hkv):
        pages = build_head_pages(K[0, h], V[0, h], T, P, S, W, ranks, "bf16")
        import_head(cache, 0, 0, h, pages)
        refs.append(pages)
    out, _ = cache.attention(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous(), [T])
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    for h in range(Hkv):
        ro, _ = oracle.attention(oracle.HeadCache(T, P, d, refs[h], key_rope_base=BASE),
                                 q[0, h * G:(h + 1) * G].astype(np.float64))
        ma, mr = errors(out[0, h * G:(h + 1) * G], ro)
        print("imported head %d: max-abs %.3e, normwise mean-relative %.3e" % (h, ma, mr))
        assert ma <= MAX_ABS and mr <= MEAN_REL, (h, ma, mr)


def test_pre_rope_positions_up_to_128k():
    """One head of 131,055 tokens (2048 pages of 64, the last partial): the
    angles reach t theta_0 = 1.3e5 rad, so the reduction of the angle before
    the hardware sine and cosine is what is checked."""
    import torch
    import paper_2608_23843_amd as pk
    d, P, G, S, W = 128, 64, 8, 64, 512
    T = 131072 - 17
    npg = -(-T // P)
    wl = synth.Workload("rope_long", 96, 1, 1, G, d, P, T, S, W, 24, (24,), "bf16", BASE, 4, key_rope=True)
    K, V = synth.kv_layer(wl, 0, 0, npg * P)
    R = 32
    rng = np.random.default_rng(6)
    rk = rng.choice(np.array([16, 24, 32], dtype=np.uint8), (1, 1, npg))
    cache = pk.PuzzleKVCache(1, 1, 1, G, d, P, npg, R, S, W, "bf16", "bf16", key_rope_base=BASE)
    rt = torch.from_numpy(rk).cuda().contiguous()
    cache.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), [T], rank_k=rt, rank_v=rt)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    q = synth.queries(wl, 0, 0)
    _check(cache, q, [T], lambda Tb, n: oracle.plan_pages(Tb, P, S, W, n), rk, rk, P, d, R, G, "T=131055")


def test_pre_rope_decode_steps_with_compression():
    """Incremental decoding with pre-RoPE tokens: append, compress the page
    that leaves the window, attend; checked after the boundary step."""
    import torch
    import paper_2608_23843_amd as pk
    d, P, G, B, Hkv, S, W = 128, 64, 4, 3, 2, 64, 128
    T0 = P * 6 + 60
    steps = 8
    npg = -(-(T0 + steps) // P) + 1
    wl = synth.Workload("rope_dec", 97, B, Hkv, Hkv * G, d, P, T0, S, W, 24, (24,), "bf16", BASE, 4,
                        key_rope=True)
    K, V = synth.kv_layer(wl, 0, 0, -(-T0 // P) * P)
    r = 20
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * G, d, P, npg, 32, S, W, "bf16", "bf16", key_rope_base=BASE)
    cache.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), [T0] * B, default_rank=(r, r))
    compressed = 0
    for s in range(steps):
        pos = T0 + s
        kn, vn = synth.decode_kv(wl, 0, 0, pos)
        cache.append(0, torch.from_numpy(kn).to("cuda", torch.bfloat16).contiguous(),
                     torch.from_numpy(vn).to("cuda", torch.bfloat16).contiguous(), [pos] * B)
        el = pk.eligible_pages(pos, pos + 1, P, S, W)
        if len(el):
            bb, hh, jj = zip(*[(b, h, int(j)) for b in range(B) for h in range(Hkv) for j in el])
            cache.compress_pages(0, bb, hh, jj, r, r)
            compressed += len(el)
    torch.cuda.synchronize()
    assert cache.device_status() == 0 and compressed == 1
    T = T0 + steps
    _, _, rk, rv = cache.page_table_host(0)
    q = synth.queries(wl, 0, 3)
    _check(cache, q, [T] * B, lambda Tb, n: oracle.plan_pages(Tb, P, S, W, n), rk, rv, P, d, 32, G, "decode")


def test_pre_rope_with_adaptive_ranks():
    """Both variants at once: pre-RoPE keys whose ranks the decomposition
    chooses for relative error 0.2 (R_K^T stored at the chosen rank, padded to
    a multiple of 4), then attention with the rotation at access; also an
    empty sequence in the batch (output 0, lse -inf)."""
    import torch
    import paper_2608_23843_amd as pk
    from test_gpu_compress import _adaptive_ok
    d, P, G, B, Hkv, S, W = 128, 64, 8, 2, 2, 64, 128
    T = [P * 9 + 33, 0]
    npg = -(-T[0] // P)
    wl = synth.Workload("rope_ad", 98, B, Hkv, Hkv * G, d, P, T[0], S, W, 24, (24,), "bf16", BASE, 4,
                        key_rope=True)
    K, V = synth.kv_layer(wl, 0, 0, npg * P)
    R, eps = 32, 0.2
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * G, d, P, npg, R, S, W, "bf16", "bf16", adaptive_rank_error=eps,
                             key_rope_base=BASE)
    cache.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), T, default_rank=(0, 0))
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    _, kind, rk, rv = cache.page_table_host(0)
    plan = oracle.plan_pages(T[0], P, S, W, npg)
    for h in range(Hkv):
        for j in np.flatnonzero(plan == oracle.FACTOR):
            for X, r in ((K[0, h, j * P:(j + 1) * P], rk[0, h, j]), (V[0, h, j * P:(j + 1) * P], rv[0, h, j])):
                _, s, _, _ = oracle.svd_rows(X.astype(np.float64))
                assert _adaptive_ok(s, int(r), eps, R), (h, j, int(r))
    q = synth.queries(wl, 0, 0)
    out, lse = cache.attention(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous(), T)
    torch.cuda.synchronize()
    o1 = out[1].cpu().numpy()
    assert np.all(o1 == 0) and np.all(np.isneginf(lse[1].cpu().numpy()))
    _check(cache, q, T, lambda Tb, n: oracle.plan_pages(Tb, P, S, W, n), rk, rv, P, d, R, G,
           "pre-RoPE + adaptive")
    # the footprint counts the transposed, padded R_K of these slots
    f = cache.footprint(T)
    fac_pages = [(h, j) for h in range(Hkv) for j in np.flatnonzero(plan == oracle.FACTOR)]
    assert f["factor_pages"] == len(fac_pages)
    assert f["factor_slot_bytes"] == sum(cache.factor_page_bytes(int(rk[0, h, j]), int(rv[0, h, j]))
                                         for h, j in fac_pages)
    assert f["factor_bytes"] == sum((int(rk[0, h, j]) + int(rv[0, h, j])) * (P + d) * 2 for h, j in fac_pages)
