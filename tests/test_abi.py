"""CPU checks of the C ABI: the library loads without a GPU, exports every
symbol include/puzzlekv.h declares, its integer page planner matches the
oracle bit for bit, its sizing follows the documented layout, and argument
errors are reported before anything is enqueued (no device work here)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from oracle import accounting

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def pk():
    import paper_2608_23843_amd as pk
    pk.load_library()
    return pk


def _header_functions():
    src = open(os.path.join(ROOT, "include", "puzzlekv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pkv_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol(pk):
    from paper_2608_23843_amd import _lib
    declared = _header_functions()
    assert declared == sorted(_lib.EXPORTS)
    lib = pk.load_library()
    for name in declared:
        assert hasattr(lib, name), name
    assert b"gfx950" in lib.pkv_version()


@pytest.mark.parametrize("P,S,W", [(16, 16, 32), (16, 0, 0), (32, 32, 32), (64, 64, 256), (64, 64, 512),
                                   (16, 40, 20)])
def test_planner_bit_exact_vs_oracle(pk, P, S, W):
    for T in list(range(0, 6 * P + 3)) + [32768, 131072, 131073]:
        n = -(-T // P) + 2
        assert np.array_equal(pk.plan_pages(T, P, S, W, n), oracle.plan_pages(T, P, S, W, n)), T
    for T in range(1, 12 * P):
        assert np.array_equal(pk.eligible_pages(T - 1, T, P, S, W), oracle.eligible_pages(T - 1, T, P, S, W))
    assert np.array_equal(pk.eligible_pages(100, 5000, P, S, W), oracle.eligible_pages(100, 5000, P, S, W))


def test_workload_page_counts(pk):
    # Qwen3-32B shape at 128K: pages 1..2039 factorized, 0 and 2040..2047 dense
    kind = pk.plan_pages(131072, 64, 64, 512)
    assert int((kind == 2).sum()) == 2039 and list(np.nonzero(kind == 1)[0]) == [0] + list(range(2040, 2048))
    # Llama-3-8B shape at 32K with a 256-token window: 507 factor pages
    assert int((pk.plan_pages(32768, 64, 64, 256) == 2).sum()) == 507


def _cache(pk, **kw):
    from paper_2608_23843_amd import _lib
    c = _lib.PkvCache()
    geo = dict(n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8, head_dim=128, page_size=64, max_pages=8,
               max_rank=32, sink_tokens=64, window_tokens=256, dense_dtype=1, factor_dtype=1)
    geo.update(kw)
    for k, v in geo.items():
        setattr(c, k, v)
    return c


def test_sizing_follows_layout(pk):
    lib = pk.load_library()
    c = _cache(pk)
    P, d = 64, 128
    for rk, rv in [(16, 16), (24, 24), (32, 32), (14, 16), (1, 3)]:
        r4 = lambda r: (r + 3) // 4 * 4
        assert lib.pkv_factor_page_bytes(c, rk, rv) == 2 * (P * r4(rk) + rk * d + rv * P + d * r4(rv))
    # rank multiple of 4: exactly the Eq. (3) storage of the factor pair
    for r in (16, 24, 32):
        ratio = lib.pkv_factor_page_bytes(c, r, r) / (2 * P * d * 2)
        assert abs(ratio - accounting.page_storage_ratio(P, r, r, d)) < 1e-12
    assert lib.pkv_dense_slot_bytes(c) == 2 * P * d * 2
    assert lib.pkv_dense_slots_per_head(c) == 1 + 256 // 64 + 2
    assert lib.pkv_factor_slot_bytes(c) % 256 == 0
    assert lib.pkv_factor_slot_bytes(c) >= lib.pkv_factor_page_bytes(c, 32, 32)
    assert lib.pkv_page_table_bytes(c) == 2 * 2 * 2 * 8 * 8
    assert lib.pkv_dense_pool_bytes(c) == 2 * 2 * 2 * 7 * 2 * P * d * 2
    assert lib.pkv_export_block_elems(c) == max(2 * P * d, 2 * (P + d) * 32)
    assert lib.pkv_workspace_bytes(c, 0, 8 * 64) > 0


@pytest.mark.parametrize("kw,code", [(dict(page_size=48), 2), (dict(head_dim=100), 2), (dict(max_rank=0), 3),
                                     (dict(max_rank=65), 3), (dict(n_q_heads=7), 2), (dict(dense_dtype=5), 6),
                                     (dict(batch=0), 2), (dict(sink_tokens=-1), 2)])
def test_geometry_errors(pk, kw, code):
    lib = pk.load_library()
    c = _cache(pk, **kw)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    assert lib.pkv_cache_check(c) == code
    assert lib.pkv_last_error()


def test_call_errors_before_any_launch(pk):
    """Every call below fails host-side validation, so no kernel is launched on
    the fake (never dereferenced) pool pointers."""
    lib = pk.load_library()
    c = _cache(pk)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    vp = ctypes.c_void_p
    i32 = lambda *v: np.array(v, dtype=np.int32)
    u8 = lambda *v: np.array(v, dtype=np.uint8)
    P = lambda a: a.ctypes.data_as(vp)
    seq = i32(128, 128)
    # attention: no workspace / too small / length beyond the table / bad layer
    assert lib.pkv_mixed_decode_attention(c, 0, vp(0x2000), P(seq), vp(0x3000), None, None, 0, None) == 5
    assert lib.pkv_mixed_decode_attention(c, 0, vp(0x2000), P(seq), vp(0x3000), None, vp(0x4000), 1, None) == 5
    assert lib.pkv_mixed_decode_attention(c, 0, vp(0x2000), P(i32(8 * 64 + 1, 1)), vp(0x3000), None,
                                          vp(0x4000), 1 << 30, None) == 2
    assert lib.pkv_mixed_decode_attention(c, 2, vp(0x2000), P(seq), vp(0x3000), None, vp(0x4000), 1 << 30,
                                          None) == 1
    # compress: rank 0, rank above max, duplicate page, page out of range
    b, h, j = i32(0, 1), i32(0, 1), i32(2, 3)
    assert lib.pkv_compress_pages(c, 0, 2, P(b), P(h), P(j), P(u8(0, 4)), P(u8(4, 4)), None, 0, None) == 3
    assert lib.pkv_compress_pages(c, 0, 2, P(b), P(h), P(j), P(u8(33, 4)), P(u8(4, 4)), None, 0, None) == 3
    assert lib.pkv_compress_pages(c, 0, 2, P(i32(0, 0)), P(i32(1, 1)), P(i32(3, 3)), P(u8(4, 4)),
                                  P(u8(4, 4)), None, 0, None) == 1
    assert lib.pkv_compress_pages(c, 0, 2, P(b), P(h), P(i32(2, 8)), P(u8(4, 4)), P(u8(4, 4)), None, 0,
                                  None) == 1
    # compress a sink page: refused on the host, the sink stays dense
    assert lib.pkv_compress_pages(c, 0, 2, P(b), P(h), P(i32(0, 3)), P(u8(4, 4)), P(u8(4, 4)), None, 0,
                                  None) == 4
    # append beyond the table; prefill with a length beyond the source
    assert lib.pkv_append_kv(c, 0, vp(0x2000), vp(0x2000), P(i32(8 * 64, 0)), None) == 2
    assert lib.pkv_prefill(c, 0, vp(0x2000), vp(0x2000), 100, P(i32(101, 5)), None, None, 4, 4, None, 0,
                           None) == 2
    assert lib.pkv_prefill(c, 0, vp(0x2000), vp(0x2000), 100, P(i32(50, 5)), None, None, 0, 4, None, 0,
                           None) == 3
    # import: bad kind; two dense pages of one head on one ring slot (P = 64,
    # one sink page, a ring of 256 / 64 + 2 = 6 slots: pages 1 and 7)
    assert lib.pkv_import_pages(c, 0, 1, P(i32(0)), P(i32(0)), P(i32(0)), P(u8(7)), P(u8(0)), P(u8(0)),
                                vp(0x2000), P(np.zeros(1, dtype=np.int64)), None, 0, None) == 1
    assert lib.pkv_import_pages(c, 0, 2, P(i32(1, 1)), P(i32(0, 0)), P(i32(1, 7)), P(u8(1, 1)), P(u8(0, 0)),
                                P(u8(0, 0)), vp(0x2000), P(np.zeros(2, dtype=np.int64)), None, 0, None) == 1
    assert "same dense slot" in lib.pkv_last_error().decode()


@pytest.mark.parametrize("kw,code", [(dict(adaptive_rank_error=1.0), 1), (dict(adaptive_rank_error=-0.1), 1),
                                     (dict(adaptive_rank_error=float("nan")), 1),
                                     (dict(adaptive_rank_error=0.2, dense_dtype=0), 6),
                                     (dict(adaptive_rank_error=0.2, page_size=16, max_rank=16), 6)])
def test_adaptive_rank_geometry_errors(pk, kw, code):
    """Adaptive ranks: eps must lie in [0, 1) and needs the bf16 32/64-token decomposition."""
    lib = pk.load_library()
    c = _cache(pk, **kw)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    assert lib.pkv_cache_check(c) == code
    assert lib.pkv_last_error()


def test_rank_zero_requests_need_adaptive_ranks(pk):
    """A rank of 0 is a request for a rank chosen per page: refused on the host
    (before any launch) unless the cache enables adaptive ranks; with them the
    remaining checks (duplicates, range) still apply."""
    lib = pk.load_library()
    vp = ctypes.c_void_p
    i32 = lambda *v: np.array(v, dtype=np.int32)
    u8 = lambda *v: np.array(v, dtype=np.uint8)
    P = lambda a: a.ctypes.data_as(vp)
    b, h, j = i32(0, 1), i32(0, 1), i32(2, 3)
    c = _cache(pk)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    assert lib.pkv_compress_pages(c, 0, 2, P(b), P(h), P(j), P(u8(0, 0)), P(u8(0, 0)), None, 0, None) == 3
    assert lib.pkv_prefill(c, 0, vp(0x2000), vp(0x2000), 128, P(i32(128, 128)), None, None, 0, 0, None, 0,
                           None) == 3
    ca = _cache(pk, adaptive_rank_error=0.2)
    ca.dense_pool = ca.factor_pool = ca.page_table = 0x1000
    assert lib.pkv_cache_check(ca) == 0
    assert lib.pkv_compress_pages(ca, 0, 2, P(i32(0, 0)), P(i32(1, 1)), P(i32(3, 3)), P(u8(0, 0)),
                                  P(u8(0, 0)), None, 0, None) == 1      # duplicate page
    assert lib.pkv_compress_pages(ca, 0, 2, P(b), P(h), P(j), P(u8(33, 0)), P(u8(0, 0)), None, 0, None) == 3


@pytest.mark.parametrize("kw,code", [(dict(key_rope_base=-1.0), 1), (dict(key_rope_base=float("inf")), 1),
                                     (dict(key_rope_base=float("nan")), 1),
                                     (dict(key_rope_base=1e6, dense_dtype=0, factor_dtype=0), 6),
                                     (dict(key_rope_base=1e6, factor_dtype=2), 6),
                                     (dict(key_rope_base=1e6, page_size=16, max_rank=16), 6),
                                     (dict(key_rope_base=1e6, head_dim=256), 6),
                                     (dict(key_rope_base=1e6, max_pages=(1 << 18) + 1), 6)])
def test_pre_rope_geometry_errors(pk, kw, code):
    """Pre-RoPE keys: the base must be 0 or positive and finite, and the
    geometry one the matrix-core kernels rotate (bf16, P = 32/64, d = 64/128,
    positions below 2^24)."""
    lib = pk.load_library()
    c = _cache(pk, **kw)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    assert lib.pkv_cache_check(c) == code
    assert lib.pkv_last_error()


def test_pre_rope_slot_holds_r_k_transposed(pk):
    """With keys cached before RoPE, R_K is stored as d x r4(rk): the page
    size grows by (r4(rk) - rk) d elements, and the slot is sized for it."""
    lib = pk.load_library()
    P, d = 64, 128
    r4 = lambda r: (r + 3) // 4 * 4
    c0 = _cache(pk, max_rank=30)
    c1 = _cache(pk, max_rank=30, key_rope_base=1e6)
    for rk, rv in [(16, 16), (13, 22), (30, 1)]:
        b0 = lib.pkv_factor_page_bytes(c0, rk, rv)
        b1 = lib.pkv_factor_page_bytes(c1, rk, rv)
        assert b0 == 2 * (P * r4(rk) + rk * d + rv * P + d * r4(rv))
        assert b1 == 2 * (P * r4(rk) + r4(rk) * d + rv * P + d * r4(rv))
    assert lib.pkv_factor_slot_bytes(c1) >= 2 * (P * 32 + 32 * d + 30 * P + d * 32)


def test_cache_bytes_argument_errors(pk):
    """pkv_cache_bytes checks its arguments before touching the page table."""
    from paper_2608_23843_amd import _lib
    lib = pk.load_library()
    c = _cache(pk)
    c.dense_pool = c.factor_pool = c.page_table = 0x1000
    f = _lib.PkvFootprint()
    seq = np.array([64, 64], dtype=np.int32)
    assert lib.pkv_cache_bytes(c, 0, None, ctypes.byref(f), None) == 1
    assert lib.pkv_cache_bytes(c, 0, seq.ctypes.data, None, None) == 1
    assert lib.pkv_cache_bytes(c, 2, seq.ctypes.data, ctypes.byref(f), None) == 1
    big = np.array([64, 8 * 64 + 1], dtype=np.int32)
    assert lib.pkv_cache_bytes(c, 0, big.ctypes.data, ctypes.byref(f), None) == 2
    assert lib.pkv_last_error()


@pytest.mark.parametrize("T,P,S,W,rho", [(16384, 32, 32, 32, 0.6), (16384, 32, 32, 32, 0.58755), (131072, 64, 64, 512, 0.5643),
                                         (32768, 64, 64, 256, 0.6), (1000, 32, 32, 32, 0.6), (100, 64, 64, 512, 0.6),
                                         (5000, 16, 40, 20, 0.3), (4096, 64, 0, 0, 0.05)])
def test_global_rank_matches_oracle_accounting(pk, T, P, S, W, rho):
    """pkv_global_rank (integer, host) against the oracle's accounting over the
    oracle's page plan, bit for bit."""
    kinds = oracle.plan_pages(T, P, S, W)
    n_fact = int(sum(min(P, T - j * P) for j, k in enumerate(kinds) if k == oracle.FACTOR))
    assert pk.global_rank(T, P, S, W, 128, rho) == accounting.global_rank(T - n_fact, n_fact, 128, rho)


def test_bandwidth_probe_argument_errors(pk):
    """pkv_bandwidth_probe checks its arguments before launching anything."""
    lib = pk.load_library()
    vp = ctypes.c_void_p
    g = ctypes.c_double(0.0)
    assert lib.pkv_bandwidth_probe(None, vp(0x1000), 1024, 0, 1, 64, 256, ctypes.byref(g), None) == 1
    assert lib.pkv_bandwidth_probe(vp(0x1000), vp(0x2000), 1000, 0, 1, 64, 256, ctypes.byref(g), None) == 1
    assert lib.pkv_bandwidth_probe(vp(0x1008), vp(0x2000), 1024, 0, 1, 64, 256, ctypes.byref(g), None) == 1
    assert lib.pkv_bandwidth_probe(vp(0x1000), vp(0x2000), 1024, 4, 1, 64, 256, ctypes.byref(g), None) == 1
    assert lib.pkv_bandwidth_probe(vp(0x1000), vp(0x2000), 1024, 0, 1, 64, 100, ctypes.byref(g), None) == 1
