"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with a retyped copy of itself: every check is
a printed number of the paper, a closed form, an invariant, a special case
that reduces to a textbook or LAPACK routine, or brute force on a tiny input.
Each is chosen so that a plausible slip in the oracle (a dropped term, a wrong
sign or index, a transposed operand, a missing 1/sqrt(d)) fails at least one.
"""
import math
import os

import numpy as np
import pytest

import oracle
from oracle import accounting, int4

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_storage.txt")


def _golden():
    out = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, val, tol, cite = line.split(None, 3)
            out[name] = (float(val), float(tol), cite)
    return out


# --------------------------------------------------------------------------
# Page plan
# --------------------------------------------------------------------------
def test_plan_paper_default_dense_region():
    """Section 4.1: with one sink page and W = P the dense region is the sink
    page, the most recently completed page and the current incomplete page.
    That prose is restated here independently of the oracle's rule."""
    P = 32
    for T in range(1, 40 * P + 1):
        kind = oracle.plan_pages(T, P, P, P)
        n_pages = -(-T // P)
        last_complete = T // P - 1
        incomplete = n_pages - 1 if T % P else None
        expect_dense = {0}
        if last_complete >= 0:
            expect_dense.add(last_complete)
        if incomplete is not None:
            expect_dense.add(incomplete)
        dense = {j for j in range(n_pages) if kind[j] == oracle.DENSE}
        fact = {j for j in range(n_pages) if kind[j] == oracle.FACTOR}
        assert dense == expect_dense, T
        assert fact == set(range(n_pages)) - expect_dense, T


def test_plan_tiny_workload_counts():
    """Tiny workload statement: T=256, P=16, 16 sink tokens and a 32-token
    window leave 13 middle pages factorized (pages 0, 14, 15 dense)."""
    kind = oracle.plan_pages(256, 16, 16, 32)
    assert list(np.nonzero(kind == oracle.DENSE)[0]) == [0, 14, 15]
    assert int((kind == oracle.FACTOR).sum()) == 13


def test_plan_incremental_invariants():
    """Section 3.3, Incremental Cache Update: a page is factorized once, never
    revisited, and a step converts at most one page (per layer and head)."""
    P, S, W = 16, 16, 48
    first_factor = {}
    prev = oracle.plan_pages(0, P, S, W, 64)
    for T in range(1, 64 * P + 1):
        cur = oracle.plan_pages(T, P, S, W, 64)
        became = np.nonzero((cur == oracle.FACTOR) & (prev != oracle.FACTOR))[0]
        assert len(became) <= 1
        assert not np.any((prev == oracle.FACTOR) & (cur != oracle.FACTOR)), "revisited"
        assert list(oracle.eligible_pages(T - 1, T, P, S, W)) == list(became)
        for j in became:
            assert j not in first_factor
            first_factor[j] = T
            # converted exactly when the page leaves the W-token window
            assert (j + 1) * P == T - W
        prev = cur
    n_complete_outside = 64 - (W // P) - 1  # all pages but the sink and the window
    assert len(first_factor) == n_complete_outside


def test_plan_empty_and_partial():
    assert len(oracle.plan_pages(0, 16, 16, 32)) == 0
    kind = oracle.plan_pages(17, 16, 0, 0)
    assert list(kind) == [oracle.FACTOR, oracle.DENSE]   # no sink, no window
    assert oracle.page_kind(5, 16, 0, 0, 3) == oracle.EMPTY


# --------------------------------------------------------------------------
# Storage accounting against the paper's printed numbers
# --------------------------------------------------------------------------
def test_accounting_matches_printed_numbers():
    g = _golden()
    gib = accounting.dense_kv_bytes(64, 8, 128 * 1024, 128, 2) / 2 ** 30
    v, tol, _ = g["dense_kv_gib_qwen3_32b_128k_bf16"]
    assert abs(gib - v) <= tol and gib == 32.0

    rho = accounting.page_storage_ratio(32, 16, 14, 128)
    v, tol, _ = g["rho_page_P32_rk16_rv14_d128"]
    assert abs(rho - v) <= tol

    # 16K tokens at P=32 are 512 pages, two of them dense (sink + last completed)
    whole = accounting.cache_ratio(512, 2, 32, 16, 14, 128)
    v, tol, _ = g["cache_ratio_P32_rk16_rv14_16k"]
    assert abs(whole - v) <= tol
    v, tol, _ = g["steady_state_fraction_of_raw"]
    assert abs(whole - v) <= tol
    v, tol, _ = g["steady_state_above_page_ratio_pp"]
    assert abs(100 * (whole - rho) - v) <= tol

    q = accounting.int4_cache_ratio(512, 2, 32, 16, 14, 128)
    v, tol, _ = g["int4_cache_ratio_P32_rk16_rv14_16k"]
    assert abs(q - v) <= tol
    # a flat 32-element grouping (not along the paper's directions) would not match
    flat = ((16 + 14) * (32 + 128) / 2 + 2 * ((16 + 14) * (32 + 128) / 32)) / (2 * 32 * 128 * 2)
    assert abs(((flat * 510 + 2) / 512) - v) > tol

    for (P, r), key in (((16, 9), "page_size_ratio_16_9_9"), ((32, 16), "page_size_ratio_32_16_16"),
                        ((64, 27), "page_size_ratio_64_27_27")):
        v, tol, _ = g[key]
        assert abs(accounting.page_storage_ratio(P, r, r, 128) - v) <= tol


def test_table5_footprint_consistent():
    """Table 5: the steady-state PuzzleKV footprint over Raw KV is 58.76%."""
    assert abs(1296.25 / 2205.90 - accounting.cache_ratio(512, 2, 32, 16, 14, 128)) < 2e-4


# --------------------------------------------------------------------------
# Truncated SVD
# --------------------------------------------------------------------------
def _householder_q(A):
    """Orthogonal Q of a QR factorization by Householder reflections (test-local)."""
    A = np.array(A, dtype=np.float64)
    m, n = A.shape
    Q = np.eye(m)
    for k in range(min(m - 1, n)):
        x = A[k:, k]
        alpha = -math.copysign(np.linalg.norm(x), x[0] if x[0] != 0 else 1.0)
        v = x.copy(); v[0] -= alpha
        nv = np.linalg.norm(v)
        if nv == 0:
            continue
        v /= nv
        A[k:, :] -= 2.0 * np.outer(v, v @ A[k:, :])
        Q[:, k:] -= 2.0 * np.outer(Q[:, k:] @ v, v)
    return Q


@pytest.mark.parametrize("shape", [(64, 128), (16, 64), (32, 128), (7, 5), (1, 8)])
def test_svd_full_reconstruction_and_orthogonality(shape):
    X = np.random.default_rng(1).standard_normal(shape)
    U, s, Rf, sw = oracle.svd_rows(X)
    assert sw > 0
    assert np.abs(U @ Rf - X).max() <= 1e-13 * np.abs(X).max() * max(shape)
    assert np.abs(U.T @ U - np.eye(shape[0])).max() < 1e-13
    G = Rf @ Rf.T
    assert np.abs(G - np.diag(np.diag(G))).max() < 1e-12 * s[0] ** 2
    assert np.all(np.diff(s) <= 0)
    assert np.allclose(np.linalg.norm(Rf, axis=1), s, rtol=1e-14, atol=0)


def test_svd_matches_lapack():
    """A special case reducing to a library routine: singular values and the
    rank-r projector agree with LAPACK (numpy.linalg.svd)."""
    rng = np.random.default_rng(2)
    X = rng.standard_normal((64, 24)) @ rng.standard_normal((24, 128)) + 0.05 * rng.standard_normal((64, 128))
    U, s, Rf, _ = oracle.svd_rows(X)
    Ul, sl, _ = np.linalg.svd(X)
    assert np.abs(s - sl).max() <= 1e-12 * sl[0]
    r = 24
    assert np.abs(U[:, :r] @ U[:, :r].T - Ul[:, :r] @ Ul[:, :r].T).max() < 1e-10


@pytest.mark.parametrize("r", [1, 4, 16, 24, 32, 63])
def test_eckart_young_tail(r):
    """Section 3.2: the rank-r truncation error is the tail of the spectrum,
    squared Frobenius error sum_{i>r} s_i^2 and spectral error s_{r+1}."""
    rng = np.random.default_rng(3)
    X = rng.standard_normal((64, 128)) * np.linspace(3, 0.1, 128)[None, :]
    L, R, s, _ = oracle.truncated_factors(X, r)
    E = X - L @ R
    assert abs(np.sum(E * E) - np.sum(s[r:] ** 2)) <= 1e-10 * np.sum(X * X)
    assert abs(np.linalg.norm(E, 2) - s[r]) <= 1e-10 * s[0]
    # truncation keeps the leading components: no other rank-r choice of the
    # computed components does better
    assert np.sum(E * E) <= np.sum((X - L[:, :max(r - 1, 0)] @ R[:max(r - 1, 0)]) ** 2)


def test_planted_svd_recovered():
    rng = np.random.default_rng(4)
    P, d = 32, 128
    Q1 = _householder_q(rng.standard_normal((P, P)))
    Q2 = _householder_q(rng.standard_normal((d, d)))[:, :P]
    sig = np.geomspace(50.0, 0.01, P)
    X = Q1 @ np.diag(sig) @ Q2.T
    U, s, Rf, _ = oracle.svd_rows(X)
    assert np.abs(s - sig).max() <= 1e-12 * sig[0]
    # each singular vector matches up to sign
    assert np.abs(np.abs(np.sum(U * Q1, axis=0)) - 1.0).max() < 1e-9
    W = Rf / s[:, None]
    assert np.abs(np.abs(np.sum(W.T * Q2, axis=0)) - 1.0).max() < 1e-9


def test_svd_brute_force_4x4():
    """Brute force on a 4x4 page: the squared singular values are the roots of
    the characteristic polynomial of X X^T (Faddeev-LeVerrier coefficients,
    roots by bisection between sign changes)."""
    rng = np.random.default_rng(5)
    X = rng.standard_normal((4, 4))
    A = X @ X.T
    n = 4
    c = [1.0]
    M = np.zeros_like(A)
    for k in range(1, n + 1):
        M = A @ M + c[-1] * np.eye(n)
        c.append(-np.trace(A @ M) / k)
    poly = lambda x: sum(ck * x ** (n - i) for i, ck in enumerate(c))
    hi = np.trace(A) + 1.0
    grid = np.linspace(-1e-9, hi, 200001)
    vals = poly(grid)
    roots = []
    for i in np.nonzero(np.sign(vals[:-1]) != np.sign(vals[1:]))[0]:
        a, b = grid[i], grid[i + 1]
        for _ in range(200):
            mid = 0.5 * (a + b)
            if np.sign(poly(mid)) == np.sign(poly(a)):
                a = mid
            else:
                b = mid
        roots.append(0.5 * (a + b))
    roots = np.sort(roots)[::-1]
    _, s, _, _ = oracle.svd_rows(X)
    assert len(roots) == 4
    assert np.abs(s ** 2 - roots).max() < 1e-9 * roots[0]


def test_svd_closed_forms():
    # diagonal: singular values are the sorted |x_ii|, ties keep the lower index
    X = np.zeros((4, 6)); X[0, 0], X[1, 1], X[2, 2], X[3, 3] = -2.0, 5.0, 2.0, 0.5
    U, s, Rf, _ = oracle.svd_rows(X)
    assert np.allclose(s, [5.0, 2.0, 2.0, 0.5], atol=0, rtol=0)
    assert np.argmax(np.abs(U[:, 1])) == 0 and np.argmax(np.abs(U[:, 2])) == 2
    # rank one: s1 = |u| |v|, the rest zero
    u = np.arange(1.0, 9.0); v = np.linspace(-1, 2, 16)
    _, s, _, _ = oracle.svd_rows(np.outer(u, v))
    assert abs(s[0] - np.linalg.norm(u) * np.linalg.norm(v)) < 1e-12 * s[0]
    assert np.abs(s[1:]).max() < 1e-12 * s[0]
    # 2x2: s^2 = (|X|_F^2 +- sqrt(|X|_F^4 - 4 det^2)) / 2
    X = np.array([[3.0, 1.0], [-2.0, 4.0]])
    f2 = np.sum(X * X); det = np.linalg.det(X)
    exp = np.sqrt([(f2 + math.sqrt(f2 ** 2 - 4 * det ** 2)) / 2, (f2 - math.sqrt(f2 ** 2 - 4 * det ** 2)) / 2])
    _, s, _, _ = oracle.svd_rows(X)
    assert np.abs(s - exp).max() < 1e-14 * exp[0]
    # orthogonal rows: all singular values 1
    Q = _householder_q(np.random.default_rng(6).standard_normal((8, 8)))
    _, s, _, _ = oracle.svd_rows(Q)
    assert np.abs(s - 1).max() < 1e-14


def test_svd_zero_page_and_rank_above_numerical_rank():
    X = np.zeros((16, 64))
    L, R, s, sw = oracle.truncated_factors(X, 8)
    assert np.all(s == 0) and np.all(R == 0)
    assert np.abs(L.T @ L - np.eye(8)).max() == 0
    rng = np.random.default_rng(7)
    X = rng.standard_normal((16, 3)) @ rng.standard_normal((3, 64))
    L, R, s, _ = oracle.truncated_factors(X, 6)
    assert np.abs(L @ R - X).max() < 1e-12 * np.abs(X).max()
    assert np.abs(L.T @ L - np.eye(6)).max() < 1e-13


def test_batch_matches_single():
    rng = np.random.default_rng(8)
    X = rng.standard_normal((5, 16, 64))
    ranks = [4, 1, 16, 8, 3]
    L, R, s, sw = oracle.truncated_factors_batch(X, ranks)
    for p in range(5):
        L1, R1, s1, _ = oracle.truncated_factors(X[p], ranks[p])
        assert np.array_equal(L[p, :, :ranks[p]], L1) and np.array_equal(R[p, :ranks[p]], R1)
        assert np.array_equal(s[p], s1)


# --------------------------------------------------------------------------
# Attention
# --------------------------------------------------------------------------
def _dense_head(rng, T, P, d, scale=1.0):
    n = -(-T // P)
    K = rng.standard_normal((n * P, d)) * scale
    V = rng.standard_normal((n * P, d))
    pages = [("dense", K[j * P:(j + 1) * P], V[j * P:(j + 1) * P]) for j in range(n)]
    return oracle.HeadCache(T, P, d, pages), K[:T], V[:T]


def test_attention_single_token():
    rng = np.random.default_rng(10)
    head, K, V = _dense_head(rng, 1, 16, 64)
    q = rng.standard_normal((3, 64))
    out, lse = oracle.attention(head, q)
    assert np.array_equal(out, np.repeat(V[:1], 3, axis=0))
    assert np.allclose(lse, q @ K[0] / 8.0, rtol=0, atol=1e-14)


def test_attention_two_token_closed_form():
    """T=2: o = sigmoid(s1 - s2) v1 + sigmoid(s2 - s1) v2, s_i = k_i . q / sqrt(d)."""
    rng = np.random.default_rng(11)
    d = 128
    head, K, V = _dense_head(rng, 2, 16, d)
    q = rng.standard_normal((1, d))
    s1, s2 = K[0] @ q[0] / math.sqrt(d), K[1] @ q[0] / math.sqrt(d)
    w1 = 1.0 / (1.0 + math.exp(s2 - s1))
    expect = w1 * V[0] + (1.0 - w1) * V[1]
    out, lse = oracle.attention(head, q)
    assert np.abs(out[0] - expect).max() < 1e-14
    assert abs(lse[0] - math.log(math.exp(s1) + math.exp(s2))) < 1e-13


def test_attention_uniform_scores_and_weights_sum_to_one():
    rng = np.random.default_rng(12)
    T, P, d = 77, 16, 64
    head, K, V = _dense_head(rng, T, P, d)
    out, lse = oracle.attention(head, np.zeros((1, d)))
    assert np.abs(out[0] - V.mean(axis=0)).max() < 1e-14
    assert abs(lse[0] - math.log(T)) < 1e-14
    # V = all ones: sum_t p_t = 1 exactly up to rounding
    ones = [(pg[0], pg[1], np.ones_like(pg[2])) for pg in head.pages]
    out, _ = oracle.attention(oracle.HeadCache(T, P, d, ones), rng.standard_normal((4, d)))
    assert np.abs(out - 1.0).max() < 1e-14


def test_attention_dominant_score():
    rng = np.random.default_rng(13)
    T, P, d = 40, 16, 64
    head, K, V = _dense_head(rng, T, P, d, scale=0.01)
    q = np.zeros((1, d)); q[0, 0] = 1.0
    K2 = K.copy(); K2[17] = 0.0; K2[17, 0] = 400.0          # score 50 for token 17
    n = -(-T // P)
    Kp = np.zeros((n * P, d)); Kp[:T] = K2
    Vp = np.zeros((n * P, d)); Vp[:T] = V
    pages = [("dense", Kp[j * P:(j + 1) * P], Vp[j * P:(j + 1) * P]) for j in range(n)]
    out, _ = oracle.attention(oracle.HeadCache(T, P, d, pages), q)
    assert np.abs(out[0] - V[17]).max() < 1e-18 + 1e-19 * T


def _factor_head(rng, T, P, d, ranks, full_rank=False):
    """Pages as exact factor pairs from the oracle SVD; returns the factor head
    and the dense head holding the same rebuilt K, V."""
    n = -(-T // P)
    fpages, dpages = [], []
    for j in range(n):
        K = rng.standard_normal((P, d)); V = rng.standard_normal((P, d))
        if j % 3 == 0 and not full_rank:
            fpages.append(("dense", K, V)); dpages.append(("dense", K, V))
            continue
        rk = min(P, d) if full_rank else ranks[j % len(ranks)]
        Lk, Rk, _, _ = oracle.truncated_factors(K, rk)
        Lv, Rv, _, _ = oracle.truncated_factors(V, rk)
        fpages.append(("factor", Lk, Rk, Lv, Rv))
        dpages.append(("dense", K if full_rank else Lk @ Rk, V if full_rank else Lv @ Rv))
    return oracle.HeadCache(T, P, d, fpages), oracle.HeadCache(T, P, d, dpages)


def test_attention_full_rank_factors_equal_dense():
    """Eq. (2) at r = min(P, d) is exact, so attention over full-rank factor
    pages equals dense attention over the original pages."""
    rng = np.random.default_rng(14)
    fh, dh = _factor_head(rng, 150, 16, 64, None, full_rank=True)
    q = rng.standard_normal((4, 64))
    o1, l1 = oracle.attention(fh, q)
    o2, l2 = oracle.attention(dh, q)
    assert np.abs(o1 - o2).max() < 1e-12
    assert np.abs(l1 - l2).max() < 1e-12


def test_pagewise_state_and_merge_equal_one_pass_softmax():
    """Eq. (4) per page then Eq. (5) over pages, in any order and grouping,
    equals one-pass softmax over the rebuilt cache (Eq. (1))."""
    rng = np.random.default_rng(15)
    T, P, d = 16 * 11 + 5, 16, 64
    fh, dh = _factor_head(rng, T, P, d, [4, 8, 3])
    q = rng.standard_normal((3, d)) * 2.0
    ref, lref = oracle.attention(fh, q)
    ref2, _ = oracle.attention(dh, q)
    assert np.abs(ref - ref2).max() < 1e-12
    n = len(fh.pages)
    for order, group in [(None, 0), (None, 1), (rng.permutation(n), 3), (rng.permutation(n), 5),
                         (np.arange(n)[::-1], 7)]:
        o, l = oracle.attention_pagewise(fh, q, order=order, group=group)
        assert np.abs(o - ref).max() < 1e-12
        assert np.abs(l - lref).max() < 1e-12


def test_attention_linear_in_values():
    rng = np.random.default_rng(16)
    T, P, d = 50, 16, 64
    head, K, V = _dense_head(rng, T, P, d)
    V2 = rng.standard_normal(V.shape)
    n = len(head.pages)
    def with_v(Vx):
        Vp = np.zeros((n * P, d)); Vp[:T] = Vx
        return oracle.HeadCache(T, P, d, [("dense", pg[1], Vp[j * P:(j + 1) * P])
                                          for j, pg in enumerate(head.pages)])
    q = rng.standard_normal((2, d))
    a, _ = oracle.attention(with_v(V), q)
    b, _ = oracle.attention(with_v(V2), q)
    c, _ = oracle.attention(with_v(2.0 * V - 3.0 * V2), q)
    assert np.abs(c - (2.0 * a - 3.0 * b)).max() < 1e-13


# --------------------------------------------------------------------------
# INT4 factor encoding (Section 4.3)
# --------------------------------------------------------------------------
def test_int4_balance_and_bounds():
    rng = np.random.default_rng(20)
    X = rng.standard_normal((64, 24)) @ rng.standard_normal((24, 128))
    L, R, s, _ = oracle.truncated_factors(X, 24)
    for which in ("K", "V"):
        e = int4.encode_page(which, L, R, s)
        # balancing leaves the product unchanged and splits sigma evenly
        assert np.abs(e["L_bal"] @ e["R_bal"] - L @ R).max() < 1e-11 * np.abs(X).max()
        assert np.allclose(np.linalg.norm(e["L_bal"], axis=0), np.sqrt(s[:24]), rtol=1e-12)
        assert np.allclose(np.linalg.norm(e["R_bal"], axis=1), np.sqrt(s[:24]), rtol=1e-12)
        for part, axis in (("L", int4.AXIS["L_" + which]), ("R", int4.AXIS["R_" + which])):
            codes, sc = e[part + "_codes"], e[part + "_scales"]
            x = e[part + "_bal"]
            assert codes.min() >= -7 and codes.max() <= 7
            assert np.all(sc.astype(np.float16).astype(np.float64) == sc)   # exact fp16
            err = np.abs(e[part + "_deq"] - x)
            lines = x if axis == 0 else x.T
            el = err if axis == 0 else err.T
            cl = codes if axis == 0 else codes.T
            for gi in range(sc.shape[0]):
                blk = slice(gi * 32, (gi + 1) * 32)
                assert np.all(el[blk] <= sc[gi][None, :] / 2 + 1e-15)
                # the largest magnitude of every run maps to code +-7
                idx = np.argmax(np.abs(lines[blk]), axis=0)
                assert np.all(np.abs(cl[blk][idx, np.arange(lines.shape[1])]) == 7)
    # directions: L_K column-wise -> scales (P/32, r); L_V row-wise -> (1, P) for r <= 32
    eK = int4.encode_page("K", L, R, s)
    eV = int4.encode_page("V", L, R, s)
    assert eK["L_scales"].shape == (2, 24) and eK["R_scales"].shape == (1, 128)
    assert eV["L_scales"].shape == (1, 64) and eV["R_scales"].shape == (1, 128)


def test_int4_zero_and_exact_grid():
    codes, sc = int4.quantize_lines(np.zeros((40, 3)), 0)
    assert np.all(codes == 0) and np.all(sc == 0)
    # values already on the grid code*s with s exactly representable survive exactly
    c = np.array([[-7, 3, 0, 7, -1]], dtype=np.float64).T
    x = c * 0.25
    codes, sc = int4.quantize_lines(x, 0)
    assert np.array_equal(codes[:, 0], c[:, 0].astype(np.int8)) and sc[0, 0] == 0.25
    # exact half steps round to the even code (reading: round half to even;
    # rounding half away from zero would give 1, 3, -1, -3, 7 at 0.5, 2.5,
    # -0.5, -2.5 and 6.5): the run's maximum 1.75 fixes s = 0.25 exactly
    h = np.array([[7, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5, -3.5, 6.5, -6.5]], dtype=np.float64).T
    codes, sc = int4.quantize_lines(h * 0.25, 0)
    assert sc[0, 0] == 0.25
    assert codes[:, 0].tolist() == [7, 0, 2, 2, 0, -2, -2, 4, -4, 6, -6]


# --------------------------------------------------------------------------
# Adaptive page rank (reconstruction-accuracy reading of Figure 2)
# --------------------------------------------------------------------------
def _orthonormal(n, rng):
    """An orthonormal basis from a Householder QR, independent of the oracle."""
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def test_adaptive_rank_hand_computed_spectrum():
    """sigma = (4, 3, 2, 1): |X|_F^2 = 30 and the tails after r = 1, 2, 3 are
    14, 5 and 1. With eps = 0.5 the budget is 7.5, first met at r = 2; with
    eps = 0.2 it is 1.2, met at r = 3; with eps = 0.1 (0.3) only r = 4 meets
    it. The page is built from that spectrum with independent orthonormal U
    and W, so the oracle's SVD is part of what is checked."""
    rng = np.random.default_rng(21)
    U = _orthonormal(4, rng)
    W = _orthonormal(12, rng)[:, :4]
    X = U @ np.diag([4.0, 3.0, 2.0, 1.0]) @ W.T
    _, s, _, _ = oracle.svd_rows(X)
    for eps, r in ((0.5, 2), (0.2, 3), (0.1, 4), (0.9, 1)):
        assert oracle.adaptive_rank(s, eps, 4) == r, (eps, r)
    assert oracle.adaptive_rank(s, 0.1, 2) == 2          # capped


def test_adaptive_rank_closed_forms():
    """An orthogonal page (all sigma = 1, n x n) needs r = ceil(n (1 - eps^2));
    a zero page needs rank 1; a rank-k page needs at most k at any eps > 0."""
    rng = np.random.default_rng(22)
    n = 16
    Q = _orthonormal(n, rng)
    _, s, _, _ = oracle.svd_rows(Q)
    for eps in (0.2, 0.5, 0.7):
        assert oracle.adaptive_rank(s, eps, n) == math.ceil(n * (1 - eps * eps) - 1e-9), eps
    _, s0, _, _ = oracle.svd_rows(np.zeros((8, 16)))
    assert oracle.adaptive_rank(s0, 0.2, 8) == 1
    Xk = rng.standard_normal((32, 5)) @ rng.standard_normal((5, 64))
    _, sk, _, _ = oracle.svd_rows(Xk)
    assert oracle.adaptive_rank(sk, 1e-6, 32) <= 5


@pytest.mark.parametrize("eps", [0.2, 0.05])
def test_adaptive_rank_meets_the_bound_by_brute_force(eps):
    """For random low-rank-plus-noise pages, the truncated factors at the
    chosen rank meet |X - L R|_F <= eps |X|_F (measured on the factors, not on
    the singular values), and one rank less does not."""
    rng = np.random.default_rng(23)
    for _ in range(6):
        X = rng.standard_normal((32, 6)) @ rng.standard_normal((6, 64)) + 0.3 * rng.standard_normal((32, 64))
        _, s, _, _ = oracle.svd_rows(X)
        r = oracle.adaptive_rank(s, eps, 32)
        L, R, _, _ = oracle.truncated_factors(X, r)
        assert np.linalg.norm(X - L @ R) <= eps * np.linalg.norm(X) * (1 + 1e-12)
        if r > 1:
            L1, R1, _, _ = oracle.truncated_factors(X, r - 1)
            assert np.linalg.norm(X - L1 @ R1) > eps * np.linalg.norm(X)


# --------------------------------------------------------------------------
# Pre-RoPE keys: rotary position embedding at cache access
# --------------------------------------------------------------------------
def test_rope_is_a_complex_multiplication():
    """RoPE read as in its original formulation: the pair (x_i, x_{i+d/2}) is
    the complex number x_i + j x_{i+d/2}, multiplied by exp(j pos theta_i)
    with theta_i = base^(-2i/d). Computed here with numpy's complex
    exponential, a different route from the oracle's real rotation, so a
    wrong sign, pairing or frequency fails."""
    rng = np.random.default_rng(31)
    d, base = 16, 1.0e4
    X = rng.standard_normal((7, d))
    pos = np.array([0, 1, 5, 100, 4097, 65536, 131071])
    Y = oracle.rope_rows(X, pos, base)
    h = d // 2
    theta = np.power(base, -np.arange(h) * 2.0 / d)
    z = (X[:, :h] + 1j * X[:, h:]) * np.exp(1j * pos[:, None] * theta[None, :])
    np.testing.assert_allclose(Y[:, :h], z.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Y[:, h:], z.imag, rtol=0, atol=1e-12)


def test_rope_closed_forms_and_invariants():
    """d = 2 has the single frequency 1: the unit key e_0 at position t
    becomes (cos t, sin t). Position 0 is the identity, every pair keeps its
    norm, and the score of two rotated vectors depends only on the distance
    of their positions (the relative-position property of RoPE)."""
    Y = oracle.rope_rows(np.array([[1.0, 0.0]] * 4), [0, 1, 2, 100], 1.0e6)
    t = np.array([0.0, 1.0, 2.0, 100.0])
    np.testing.assert_allclose(Y, np.stack([np.cos(t), np.sin(t)], 1), atol=1e-14)
    rng = np.random.default_rng(32)
    d = 128
    x = rng.standard_normal((3, d))
    np.testing.assert_array_equal(oracle.rope_rows(x, 0, 5e5), x)
    y = oracle.rope_rows(x, [3, 777, 120000], 5e5)
    np.testing.assert_allclose(np.hypot(y[:, :64], y[:, 64:]), np.hypot(x[:, :64], x[:, 64:]), rtol=1e-13)
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    s1 = oracle.rope_rows(q, 40, 1e6)[0] @ oracle.rope_rows(k, 1000, 1e6)[0]
    s2 = oracle.rope_rows(q, 40 + 90000, 1e6)[0] @ oracle.rope_rows(k, 1000 + 90000, 1e6)[0]
    s3 = q @ oracle.rope_rows(k, 960, 1e6)[0]
    assert abs(s1 - s2) < 1e-9 and abs(s1 - s3) < 1e-9


def test_attention_pre_rope_full_rank_equals_dense_over_rotated_keys():
    """A cache of pre-RoPE keys (dense pages and full-rank factor pages),
    attended with RoPE at access, equals plain attention over a dense cache
    whose keys were rotated beforehand by the complex form above: this pins
    that key t of page j sits at position j P + t."""
    rng = np.random.default_rng(33)
    P, d, g, base = 8, 16, 3, 1.0e4
    T = 5 * P + 3
    n = -(-T // P)
    h = d // 2
    theta = np.power(base, -np.arange(h) * 2.0 / d)
    K = rng.standard_normal((n * P, d))
    V = rng.standard_normal((n * P, d))
    pos = np.arange(n * P)
    z = (K[:, :h] + 1j * K[:, h:]) * np.exp(1j * pos[:, None] * theta[None, :])
    Krot = np.concatenate([z.real, z.imag], 1)
    pre, post = [], []
    for j in range(n):
        Kp, Vp = K[j * P:(j + 1) * P], V[j * P:(j + 1) * P]
        post.append(("dense", Krot[j * P:(j + 1) * P], Vp))
        if j in (1, 2, 3):
            Lk, Rk, _, _ = oracle.truncated_factors(Kp, P)
            Lv, Rv, _, _ = oracle.truncated_factors(Vp, P)
            pre.append(("factor", Lk, Rk, Lv, Rv))
        else:
            pre.append(("dense", Kp, Vp))
    q = rng.standard_normal((g, d))
    o1, l1 = oracle.attention(oracle.HeadCache(T, P, d, pre, key_rope_base=base), q)
    o2, l2 = oracle.attention(oracle.HeadCache(T, P, d, post), q)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-11)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-11)
    # and the rotation matters: without it the result differs
    o3, _ = oracle.attention(oracle.HeadCache(T, P, d, pre), q)
    assert np.abs(o3 - o2).max() > 1e-3


# --------------------------------------------------------------------------
# Global SVD baseline (Section 4.1 "Baselines"; Section 4.2 "Main Results";
# Appendix "Baseline Configurations")
# --------------------------------------------------------------------------
def test_global_svd_full_rank_lapack_and_projection():
    """At full rank the shared basis rebuilds the region exactly; the singular
    values are LAPACK's; B has orthonormal rows and A is the projection X B^T."""
    rng = np.random.default_rng(31)
    X = rng.standard_normal((300, 24)) * np.linspace(4.0, 0.2, 24)[None, :]
    A, B, s, sw = oracle.global_factors(X, 24)
    assert sw > 0 and A.shape == (300, 24) and B.shape == (24, 24)
    assert np.abs(A @ B - X).max() <= 1e-12 * np.abs(X).max()
    assert np.abs(B @ B.T - np.eye(24)).max() < 1e-13
    assert np.abs(A - X @ B.T).max() <= 1e-12 * np.abs(X).max()
    sl = np.linalg.svd(X, compute_uv=False)
    assert np.abs(s - sl).max() <= 1e-12 * sl[0]
    assert np.allclose(np.linalg.norm(A, axis=0), s, rtol=1e-13, atol=0)


@pytest.mark.parametrize("r", [1, 5, 12, 31])
def test_global_svd_eckart_young(r):
    """Truncating the shared basis at rank r leaves the spectral tail."""
    rng = np.random.default_rng(32)
    X = rng.standard_normal((500, 32)) * np.geomspace(5.0, 0.05, 32)[None, :]
    A, B, s, _ = oracle.global_factors(X, r)
    E = X - A @ B
    assert abs(np.sum(E * E) - np.sum(s[r:] ** 2)) <= 1e-10 * np.sum(X * X)
    assert abs(np.linalg.norm(E, 2) - s[r]) <= 1e-10 * s[0]


def test_global_svd_two_segments_closed_form():
    """A sequence whose first half lives in one 3-dimensional subspace and whose
    second half lives in an orthogonal one (the non-stationary case): its
    singular values are the union of the two halves' (9, 8, 7 and 3, 2, 1),
    so one shared basis of rank 3 keeps the first subspace exactly and loses
    the second entirely (squared error 3^2 + 2^2 + 1^2), while rank 6 is exact.
    Orthonormal factors come from an independent Householder QR."""
    rng = np.random.default_rng(33)
    d, n = 16, 40
    Wq = _householder_q(rng.standard_normal((d, d)))
    W1, W2 = Wq[:, :3].T, Wq[:, 3:6].T
    U1 = _householder_q(rng.standard_normal((n, n)))[:, :3]
    U2 = _householder_q(rng.standard_normal((n, n)))[:, :3]
    X = np.vstack([U1 @ np.diag([9.0, 8.0, 7.0]) @ W1, U2 @ np.diag([3.0, 2.0, 1.0]) @ W2])
    A, B, s, _ = oracle.global_factors(X, 3)
    assert np.abs(s[:6] - [9, 8, 7, 3, 2, 1]).max() < 1e-12 and np.abs(s[6:]).max() < 1e-12
    assert np.abs(B.T @ B - W1.T @ W1).max() < 1e-12
    E = X - A @ B
    assert abs(np.sum(E * E) - 14.0) < 1e-10
    assert np.abs(E[:n]).max() < 1e-12
    A6, B6, _, _ = oracle.global_factors(X, 6)
    assert np.abs(A6 @ B6 - X).max() < 1e-12


def test_global_rank_budget():
    """Rank matching. Without dense tokens the ratio is the paper's
    rho_global = r (S + d) / (S d) (Section 4.2): at S = 16K and 32K tokens,
    d = 128 and rho = 0.6 the largest rank within it is 76 (76.2 and 76.5
    before rounding down; the paper reports ranks of 76-78 for its inputs).
    With dense tokens (Appendix: the budget counts them), the stored elements
    of actual global factors plus the dense tokens stay within the budget at
    the chosen rank and exceed it one rank higher."""
    assert accounting.global_rank(0, 16384, 128, 0.6) == 76
    assert accounting.global_rank(0, 32768, 128, 0.6) == 76
    rng = np.random.default_rng(34)
    d, P = 32, 16
    n_dense, n_fact = 3 * P, 20 * P
    X = rng.standard_normal((n_fact, d))
    for rho in (0.3, 0.5, 0.6, 0.9):
        r = accounting.global_rank(n_dense, n_fact, d, rho)
        raw = 2 * (n_dense + n_fact) * d
        for rr, fits in ((r, True), (r + 1, False)):
            if rr > d:
                continue
            A, B, _, _ = oracle.global_factors(X, rr)
            stored = 2 * n_dense * d + 2 * (A.size + B.size)
            assert (stored <= rho * raw) == fits, (rho, rr)
    # matched to PuzzleKV's own whole-cache ratio at the paper's default
    # geometry (P = 32, (16, 14), d = 128, 16K tokens; the plan keeps the sink
    # page and the last completed page dense, the 58.76% of Section 4.5),
    # Global SVD gets rank 74
    kinds = oracle.plan_pages(16384, 32, 32, 32)
    n_dense_pages = int((kinds == oracle.DENSE).sum())
    assert n_dense_pages == 2
    rho_pkv = accounting.cache_ratio(512, n_dense_pages, 32, 16, 14, 128)
    assert abs(rho_pkv - 0.5876) < 5e-5
    assert accounting.global_rank(32 * n_dense_pages, 16384 - 32 * n_dense_pages, 128, rho_pkv) == 74


def test_global_head_attention_full_rank_equals_dense():
    """Attention over a head stored by Global SVD at full rank equals dense
    attention over the original keys and values: the coefficient rows are
    placed on the factorized pages in token order."""
    rng = np.random.default_rng(35)
    P, d, T, S, W = 16, 32, 16 * 9 + 5, 16, 16
    K = rng.standard_normal((T, d)); V = rng.standard_normal((T, d))
    kinds = oracle.plan_pages(T, P, S, W)
    rows = np.concatenate([np.arange(j * P, (j + 1) * P) for j, k in enumerate(kinds) if k == oracle.FACTOR])
    A_K, B_K, _, _ = oracle.global_factors(K[rows], d)
    A_V, B_V, _, _ = oracle.global_factors(V[rows], d)
    head = oracle.global_head(T, P, d, kinds, K, V, A_K, B_K, A_V, B_V)
    dense = oracle.HeadCache(T, P, d, [("dense", np.vstack([K[j * P:(j + 1) * P], np.zeros((max(0, (j + 1) * P - T), d))]),
                                        np.vstack([V[j * P:(j + 1) * P], np.zeros((max(0, (j + 1) * P - T), d))]))
                                       for j in range(len(kinds))])
    q = rng.standard_normal((3, d)) / np.sqrt(d)
    o1, l1 = oracle.attention(head, q)
    o2, l2 = oracle.attention(dense, q)
    assert np.abs(o1 - o2).max() < 1e-12 and np.abs(l1 - l2).max() < 1e-12
