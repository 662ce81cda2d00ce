"""The library's footprint accounting (pkv_cache_bytes) read from real page
tables against the oracle's storage formulas (Eq. (3); the whole-cache ratio
of the paper's Memory Footprint paragraph; INT4 codes plus scales), which
tests/test_oracle_pins.py ties to the paper's printed numbers."""
import numpy as np
import pytest

import oracle
import synth
from oracle import accounting

pytestmark = pytest.mark.gpu


def _cache(B, Hkv, d, P, T, S, W, ranks, factors, max_pages=None, layers=1):
    import torch
    import paper_2608_23843_amd as pk
    npg = max_pages or -(-max(T) // P)
    wl = synth.Workload("acct", 120, B, Hkv, Hkv, d, P, max(T), S, W, 8, (ranks[0],), "bf16", None, 0)
    K, V = synth.kv_layer(wl, 0, 0, -(-max(T) // P) * P)
    cache = pk.PuzzleKVCache(layers, B, Hkv, Hkv, d, P, npg, max(ranks), S, W, "bf16", factors)
    for layer in range(layers):
        cache.prefill(layer, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                      torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), T, default_rank=ranks)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    return cache, wl


def test_paper_default_whole_cache_ratio():
    """The paper's default configuration at 16K (P = 32, (r_K, r_V) = (16, 14),
    one sink page and the last page dense): 510 factor pages and 2 dense pages
    per head, so the live footprint ratio is the oracle's whole-cache ratio,
    0.58755 (the paper prints 58.76%)."""
    P, d, T = 32, 128, 16384
    cache, _ = _cache(1, 2, d, P, [T], P, P, (16, 14), "bf16", layers=2)
    f = cache.footprint([T])
    assert f["dense_pages"] == 2 * 2 * 2 and f["factor_pages"] == 2 * 2 * 510
    assert f["raw_bytes"] == 2 * 2 * 2 * T * d * 2
    ratio = (f["dense_bytes"] + f["factor_bytes"]) / f["raw_bytes"]
    ref = accounting.cache_ratio(512, 2, P, 16, 14, d)
    assert abs(ratio - ref) < 1e-12, (ratio, ref)
    assert abs(ratio - 0.5876) < 5e-5
    assert f["factor_slot_bytes"] == f["factor_pages"] * cache.factor_page_bytes(16, 14)
    one = cache.footprint([T], layer=1)
    assert all(2 * one[k] == f[k] for k in f)


def test_ragged_int4_footprint():
    """INT4 factors at (24, 24), two sequences ending inside a page: dense
    pages count their live rows, factor pages the oracle's INT4 bytes."""
    P, d, S, W = 64, 128, 64, 128
    T = [64 * 30 + 17, 64 * 11]
    cache, _ = _cache(2, 2, d, P, T, S, W, (24, 24), "int4")
    f = cache.footprint(T)
    n_f = n_d = dense_rows = 0
    for Tb in T:
        n = -(-Tb // P)
        kinds = oracle.plan_pages(Tb, P, S, W, n)
        for j in range(n):
            if kinds[j] == oracle.FACTOR:
                n_f += 1
            else:
                n_d += 1
                dense_rows += min(P, Tb - j * P)
    Hkv = 2
    assert f["factor_pages"] == Hkv * n_f and f["dense_pages"] == Hkv * n_d
    assert f["dense_bytes"] == Hkv * dense_rows * 2 * d * 2
    assert f["factor_bytes"] == Hkv * n_f * accounting.int4_page_bytes(P, 24, 24, d)
    assert f["raw_bytes"] == Hkv * sum(T) * 2 * d * 2


def test_footprint_after_decode_steps():
    """Update complete: after appending tokens and compressing the page that
    left the window, the counts follow the plan of the new length."""
    import torch
    import paper_2608_23843_amd as pk
    P, d, S, W = 32, 128, 32, 32
    T0, steps = 32 * 20 + 31, 40
    cache, wl = _cache(1, 2, d, P, [T0], S, W, (16, 14), "bf16", max_pages=-(-(T0 + steps) // P))
    for s in range(steps):
        pos = T0 + s
        kn = torch.zeros((1, 2, d), dtype=torch.bfloat16, device="cuda")
        cache.append(0, kn, kn, [pos])
        el = pk.eligible_pages(pos, pos + 1, P, S, W)
        if len(el):
            cache.compress_pages(0, [0] * 2 * len(el), [0, 1] * len(el), [int(j) for j in el for _ in range(2)],
                                 16, 14)
    T = T0 + steps
    f = cache.footprint([T])
    n = -(-T // P)
    kinds = oracle.plan_pages(T, P, S, W, n)
    n_f = int((kinds == oracle.FACTOR).sum())
    assert f["factor_pages"] == 2 * n_f and f["dense_pages"] == 2 * (n - n_f)
    rows = sum(min(P, T - j * P) for j in range(n) if kinds[j] != oracle.FACTOR)
    assert f["dense_bytes"] + f["factor_bytes"] == 2 * (rows * 2 * d * 2 + n_f * (16 + 14) * (P + d) * 2)
