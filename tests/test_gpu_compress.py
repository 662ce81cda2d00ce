"""GPU parity of the page decomposition (pkv_prefill / pkv_compress_pages)
against the oracle's one-sided Jacobi SVD, through the C ABI.

The truncated SVD is unique only up to signs, rotations inside repeated
singular values and ties at the cut, so the comparison uses sign-invariant
quantities on the exported factors: the singular values sigma_i = |R_i|
(Gram identity: R = L^T X has row norms sigma_i), the rank-r product L R
against the oracle's X_r where the spectrum has a gap at r, orthonormality of
L, and the Eckart-Young truncation error. Page-table entries are integers
and must match the plan bit for bit."""
import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, errors, storage_round

pytestmark = pytest.mark.gpu


def _prefill_case(B, Hkv, d, P, T, S, W, rank, dense_dtype, factor_dtype, r0, seed=0, rope=None,
                  outliers=0, rank_table=None):
    import torch
    import paper_2608_23843_amd as pk
    max_pages = -(-T // P)
    wl = synth.Workload("c", 91, B, Hkv, Hkv, d, P, T, S, W, r0, (rank,), dense_dtype, rope, outliers)
    K, V = synth.kv_layer(wl, seed, 0, T)
    max_rank = rank if rank_table is None else int(rank_table.max())
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, max_pages, max_rank, S, W, dense_dtype, factor_dtype)
    kt = torch.from_numpy(K).to(device="cuda", dtype=cache.qdtype).contiguous()
    vt = torch.from_numpy(V).to(device="cuda", dtype=cache.qdtype).contiguous()
    if rank_table is None:
        cache.prefill(0, kt, vt, [T] * B, default_rank=(rank, rank))
    else:
        rt = torch.from_numpy(rank_table.astype(np.uint8)).cuda().contiguous()
        cache.prefill(0, kt, vt, [T] * B, rank_k=rt, rank_v=rt)
    torch.cuda.synchronize()
    return cache, K, V, max_pages


def _export(cache, refs):
    b, h, j = zip(*refs)
    return cache.export_pages(0, list(b), list(h), list(j)).cpu().numpy().astype(np.float64)


def _unpack_factor(blk, P, d, R):
    Lk = blk[:P * R].reshape(P, R)
    Rk = blk[P * R:P * R + R * d].reshape(R, d)
    Lv = blk[P * R + R * d:2 * P * R + R * d].reshape(P, R)
    Rv = blk[2 * P * R + R * d:2 * P * R + 2 * R * d].reshape(R, d)
    return Lk, Rk, Lv, Rv


def _check_factor(L, R, X, r, gap_tol, orth_tol, sig_tol):
    """L (P x r), R (r x d) from the GPU, X the stored page (fp64).

    sig_tol is the relative storage rounding of a factor entry: a row norm of
    R moves by at most that fraction when R is stored (2^-8 for bf16, whose
    unit roundoff is 2^-8; ~0 for fp32). On top of it the fp32 Gram gives
    eigenvalues to about 1e-5 |G| = 1e-5 s_1^2."""
    _, s, _, _ = oracle.svd_rows(X)
    sig_gpu = np.linalg.norm(R, axis=1)
    bound = sig_tol * s[:r] + 1e-5 * s[0] ** 2 / np.maximum(s[:r], 1e-30) + 1e-6 * s[0]
    assert np.all(np.abs(sig_gpu - s[:r]) <= bound), (sig_gpu[:4], s[:4])
    assert np.abs(L.T @ L - np.eye(r)).max() <= orth_tol
    tail = np.sqrt(np.sum(s[r:] ** 2))
    err = np.linalg.norm(X - L @ R)
    assert err <= (1 + 1e-3) * tail + gap_tol * np.linalg.norm(X), (err, tail)
    if r < len(s) and s[r] < 0.5 * s[r - 1]:
        Lo, Ro, _, _ = oracle.truncated_factors(X, r)
        Xr = Lo @ Ro
        assert np.linalg.norm(L @ R - Xr) <= gap_tol * np.linalg.norm(Xr) + 1e-3 * tail


@pytest.mark.parametrize("factor_dtype,gap_tol,orth_tol,sig_tol",
                         [("f32", 1e-4, 1e-4, 1e-5), ("bf16", 6e-3, 1e-2, 4e-3)])
def test_prefill_llama_pages(factor_dtype, gap_tol, orth_tol, sig_tol):
    """Llama-3-8B page geometry (P=64, d=128, r=24 on rank-24 + noise pages)."""
    B, Hkv, d, P, S, W, r = 1, 2, 128, 64, 64, 256, 24
    T = 64 * 12 + 20
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, r, "bf16", factor_dtype, 24, rope=5e5,
                                     outliers=4)
    assert cache.device_status() == 0
    kind = oracle.plan_pages(T, P, S, W, npg)
    refs = [(0, h, j) for h in range(Hkv) for j in range(npg) if kind[j] == oracle.FACTOR]
    blocks = _export(cache, refs)
    R = cache.c.max_rank
    for (b, h, j), blk in zip(refs, blocks):
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
            _check_factor(L[:, :r], Rm[:r], X.astype(np.float64), r, gap_tol, orth_tol, sig_tol)
            assert np.all(L[:, r:] == 0) and np.all(Rm[r:] == 0)


def test_prefill_page_table_and_dense_pages_bit_exact():
    B, Hkv, d, P, S, W, r = 2, 2, 64, 16, 16, 48, 4
    T = 16 * 10 + 7
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, r, "bf16", "bf16", 4)
    slot, kind, rk, rv = cache.page_table_host(0)
    plan = oracle.plan_pages(T, P, S, W, npg)
    sink_pages = -(-S // P)
    ring = -(-W // P) + 2
    dslots = sink_pages + ring
    for b in range(B):
        for h in range(Hkv):
            assert np.array_equal(kind[b, h], plan)
            for j in range(npg):
                head = b * Hkv + h
                if plan[j] == oracle.FACTOR:
                    assert (slot[b, h, j], rk[b, h, j], rv[b, h, j]) == (head * npg + j, r, r)
                else:
                    ring_pos = j if j < sink_pages else sink_pages + (j - sink_pages) % ring
                    assert (slot[b, h, j], rk[b, h, j], rv[b, h, j]) == (head * dslots + ring_pos, 0, 0)
    refs = [(b, h, j) for b in range(B) for h in range(Hkv) for j in range(npg) if plan[j] == oracle.DENSE]
    blocks = _export(cache, refs)
    for (b, h, j), blk in zip(refs, blocks):
        rows = min(P, T - j * P)
        Kp = blk[:P * d].reshape(P, d)
        Vp = blk[P * d:2 * P * d].reshape(P, d)
        assert np.array_equal(Kp[:rows], K[b, h, j * P:j * P + rows])
        assert np.array_equal(Vp[:rows], V[b, h, j * P:j * P + rows])
        assert np.all(Kp[rows:] == 0) and np.all(Vp[rows:] == 0)


@pytest.mark.parametrize("P", [16, 32])
def test_prefill_small_pages_variable_ranks_fp32(P):
    """Several decompositions per wavefront (P < 64), fp32 pages and factors,
    per-page ranks including rank 1 and full rank P."""
    B, Hkv, d, S, W = 1, 2, 64, P, P
    T = P * 9
    npg = 9
    rng = np.random.default_rng(5)
    table = rng.choice([1, 3, P // 2, P], size=(B, Hkv, npg))
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, 0, "f32", "f32", P // 2, rank_table=table)
    assert cache.device_status() == 0
    kind = oracle.plan_pages(T, P, S, W, npg)
    refs = [(0, h, j) for h in range(Hkv) for j in range(npg) if kind[j] == oracle.FACTOR]
    blocks = _export(cache, refs)
    R = cache.c.max_rank
    for (b, h, j), blk in zip(refs, blocks):
        r = int(table[b, h, j])
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
            _check_factor(L[:, :r], Rm[:r], X.astype(np.float64), r, 1e-4, 1e-4, 1e-5)
            if r == P:
                assert np.abs(L[:, :r] @ Rm[:r] - X).max() <= 1e-5 * np.abs(X).max()


def test_incremental_compress_and_state_errors():
    """Append tokens one by one until a page leaves the window, compress it with
    pkv_compress_pages, and compare with the oracle; compressing it again
    raises the not-dense device bit and leaves the entry unchanged."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, d, P, S, W, r = 2, 2, 128, 64, 64, 128, 24
    T0, steps = 64 * 4 + 60, 40
    wl = synth.Workload("c", 92, B, Hkv, Hkv, d, P, T0, S, W, 24, (r,), "bf16", 5e5, 4,
                        decode_steps=steps)
    K, V = synth.kv_layer(wl, 0, 0)
    max_pages = -(-(T0 + steps) // P)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, max_pages, 32, S, W, "bf16", "bf16")
    kt = torch.from_numpy(K[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    vt = torch.from_numpy(V[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    cache.prefill(0, kt, vt, [T0] * B, default_rank=(r, r))
    converted = []
    for t in range(T0, T0 + steps):
        kn = torch.from_numpy(K[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        vn = torch.from_numpy(V[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        cache.append(0, kn, vn, [t] * B)
        new = oracle.eligible_pages(t, t + 1, P, S, W)
        for j in new:
            refs = [(b, h, int(j)) for b in range(B) for h in range(Hkv)]
            bb, hh, jj = zip(*refs)
            cache.compress_pages(0, bb, hh, jj, [r] * len(refs), [16] * len(refs))
            converted += refs
        slot, kind, rk, rv = cache.page_table_host(0)
        plan = oracle.plan_pages(t + 1, P, S, W, max_pages)
        assert np.array_equal(kind, np.broadcast_to(plan, kind.shape)), t
    assert cache.device_status() == 0
    assert converted, "the run must cross a window boundary"
    blocks = _export(cache, converted)
    R = cache.c.max_rank
    for (b, h, j), blk in zip(converted, blocks):
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        Xk = K[b, h, j * P:(j + 1) * P].astype(np.float64)
        Xv = V[b, h, j * P:(j + 1) * P].astype(np.float64)
        _check_factor(Lk[:, :r], Rk[:r], Xk, r, 6e-3, 1e-2, 4e-3)
        _check_factor(Lv[:, :16], Rv[:16], Xv, 16, 6e-3, 1e-2, 4e-3)
    # compressing a page that is already factorized: device bit, entry unchanged
    before = cache.page_table(0).clone()
    b, h, j = converted[0]
    cache.compress_pages(0, [b], [h], [j], [r], [r])
    assert cache.device_status() & pk._lib.PKV_DEV_NOT_DENSE
    assert torch.equal(before, cache.page_table(0))
    with pytest.raises(pk.PuzzleKVError, match="PKV_E_ARG"):
        cache.compress_pages(0, [0, 0], [0, 0], [5, 5], [r, r], [r, r])


def test_ring_overrun_is_reported():
    """Appending past the window without compressing the page that left it would
    overwrite a dense page: the append is refused with a device bit."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, d, P, S, W = 1, 1, 64, 16, 16, 16
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, 16, 4, S, W, "f32", "f32")
    row = torch.ones((1, 1, d), device="cuda")
    for t in range(16 * 5):
        cache.append(0, row, row, [t])
    assert cache.device_status() & pk._lib.PKV_DEV_RING_OVERRUN


def test_zero_page():
    import torch
    import paper_2608_23843_amd as pk
    P, d = 16, 64
    cache = pk.PuzzleKVCache(1, 1, 1, 1, d, P, 4, 4, 0, 0, "f32", "f32")
    z = torch.zeros((1, 1, 4 * P, d), device="cuda")
    cache.prefill(0, z, z, [4 * P], default_rank=(4, 4))
    blk = _export(cache, [(0, 0, 1)])[0]
    Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, 4)
    assert np.all(Rk == 0) and np.all(Rv == 0)
    assert np.abs(Lk.T @ Lk - np.eye(4)).max() < 1e-6


def test_prefill_bf16_pages_rank_above_signal():
    """Rank 32 on rank-24 + noise key and value pages (bf16 pages, fp32 factors,
    P = 64). The eight directions past the planted rank are noise directions
    whose Gram eigenvalues sit four to five decades below the largest one; the
    decomposition must still resolve them, so the Eckart-Young error is the
    optimal tail to 1e-4 and every singular value is right to fp32 Gram
    accuracy."""
    B, Hkv, d, P, S, W, r = 1, 2, 128, 64, 64, 256, 32
    T = 64 * 10
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, r, "bf16", "f32", 24, rope=1e6, outliers=4)
    assert cache.device_status() == 0
    kind = oracle.plan_pages(T, P, S, W, npg)
    refs = [(0, h, j) for h in range(Hkv) for j in range(npg) if kind[j] == oracle.FACTOR]
    blocks = _export(cache, refs)
    for (b, h, j), blk in zip(refs, blocks):
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, r)
        for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
            X = X.astype(np.float64)
            _check_factor(L, Rm, X, r, 1e-4, 1e-4, 1e-5)
            _, s, _, _ = oracle.svd_rows(X)
            tail = np.sqrt(np.sum(s[r:] ** 2))
            assert np.linalg.norm(X - L @ Rm) <= (1 + 1e-4) * tail, (j, np.linalg.norm(X - L @ Rm) / tail)


@pytest.mark.parametrize("P", [32, 64])
def test_prefill_bf16_pages_variable_ranks(P):
    """bf16 pages on the matrix-core decomposition (two pages per wavefront at
    P = 32), fp32 factors, per-page ranks including 1 and 32 (full rank at
    P = 32)."""
    B, Hkv, d, S, W = 2, 2, 128, P, P
    T = P * 9 + 5
    npg = 10
    rng = np.random.default_rng(7)
    table = rng.choice([1, 5, 16, 32], size=(B, Hkv, npg))
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, 0, "bf16", "f32", 24, rank_table=table,
                                     rope=5e5, outliers=4)
    assert cache.device_status() == 0
    kind = oracle.plan_pages(T, P, S, W, npg)
    refs = [(b, h, j) for b in range(B) for h in range(Hkv) for j in range(npg) if kind[j] == oracle.FACTOR]
    blocks = _export(cache, refs)
    R = cache.c.max_rank
    for (b, h, j), blk in zip(refs, blocks):
        r = int(table[b, h, j])
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
            _check_factor(L[:, :r], Rm[:r], X.astype(np.float64), r, 1e-4, 1e-4, 1e-5)
            assert np.all(L[:, r:] == 0) and np.all(Rm[r:] == 0)
            if r == P:
                assert np.abs(L[:, :r] @ Rm[:r] - X).max() <= 1e-5 * np.abs(X).max()


def test_rank_deficient_and_zero_pages_bf16():
    """A zero page and an exactly rank-5 page decomposed at rank 8 (bf16 pages,
    fp32 factors, P = 64). Directions past the page's rank have no eigenvalue
    of their own: L is completed to an orthonormal set, the matching rows of R
    vanish, and L R reproduces the page."""
    import torch
    import paper_2608_23843_amd as pk
    P, d, r = 64, 128, 8
    rng = np.random.default_rng(11)
    K = np.zeros((1, 1, 4 * P, d), dtype=np.float32)
    K[0, 0, P + 3:P + 8] = storage_round(rng.standard_normal((5, d)), "bf16")   # five nonzero rows
    K[0, 0, 2 * P:3 * P] = storage_round(rng.standard_normal((P, 5)) @ rng.standard_normal((5, d)), "bf16")
    V = np.zeros_like(K)
    cache = pk.PuzzleKVCache(1, 1, 1, 1, d, P, 4, r, 0, 0, "bf16", "f32")
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous()
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous()
    cache.prefill(0, kt, vt, [4 * P], default_rank=(r, r))
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    blocks = _export(cache, [(0, 0, 0), (0, 0, 1), (0, 0, 2)])
    for j, blk in enumerate(blocks):
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, r)
        X = K[0, 0, j * P:(j + 1) * P].astype(np.float64)
        for L, Rm, Xp in ((Lk, Rk, X), (Lv, Rv, np.zeros_like(X))):
            assert np.abs(L.T @ L - np.eye(r)).max() <= 1e-5, j
            if j == 2 and Xp is X:   # bf16 rounding makes this page full rank: a true rank-8 tail
                _check_factor(L, Rm, Xp, r, 1e-4, 1e-5, 1e-5)
            else:
                assert np.abs(L @ Rm - Xp).max() <= 1e-5 * max(np.abs(Xp).max(), 1.0), j
        if j == 0:
            assert np.all(Rk == 0) and np.all(Rv == 0)
        if j == 1:   # the five nonzero rows span the page: ranks 6..8 carry nothing
            assert np.abs(Rk[5:]).max() <= 1e-5 * np.abs(Rk).max()


def _adaptive_ok(s, r, eps, cap, band=1e-3):
    """r is an acceptable adaptive rank for singular values s: it meets the
    bound |X - X_r|_F <= eps |X|_F and r - 1 does not, both up to a relative
    band of the budget (the GPU decides the integer from fp32 eigenvalues of
    the Gram matrix, the oracle from fp64 singular values)."""
    E = float(np.sum(s ** 2))
    budget = eps * eps * E
    tail = lambda k: float(np.sum(s[k:] ** 2))
    if r < 1 or r > cap:
        return False
    meets = tail(r) <= budget * (1 + band) + 1e-30
    minimal = r == 1 or tail(r - 1) > budget * (1 - band) or r == cap and tail(cap) > budget
    return meets and minimal


@pytest.mark.parametrize("P,factor_dtype", [(64, "bf16"), (32, "bf16"), (64, "f32"), (64, "int4")])
def test_adaptive_ranks_prefill(P, factor_dtype):
    """Adaptive ranks (eps = 0.2, the paper's 80% reconstruction accuracy) on
    Qwen3-32B-like key and value pages: every factor page's chosen ranks meet
    the bound by the oracle's singular values of the stored page while one
    rank less does not, the page table holds them, fp32 factors reconstruct
    within the bound, and attention over the cache matches the oracle over the
    exported pages."""
    import torch
    import paper_2608_23843_amd as pk
    eps, d, S, W = 0.2, 128, P, 2 * P
    B, Hkv, G = 1, 2, 8
    T = P * 12 + 9
    cap = 32
    wl = synth.Workload("ad", 93, B, Hkv, Hkv * G, d, P, T, S, W, 24, (24,), "bf16", 1e6, 4)
    K, V = synth.kv_layer(wl, 0, 0, T)
    npg = -(-T // P)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * G, d, P, npg, cap, S, W, "bf16", factor_dtype,
                             adaptive_rank_error=eps)
    cache.prefill(0, torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous(), [T] * B, default_rank=(0, 0))
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    _, kind, rk, rv = cache.page_table_host(0)
    plan = oracle.plan_pages(T, P, S, W, npg)
    chosen = []
    for h in range(Hkv):
        assert np.array_equal(kind[0, h], plan)
        for j in np.flatnonzero(plan == oracle.FACTOR):
            for X, r in ((K[0, h, j * P:(j + 1) * P], int(rk[0, h, j])), (V[0, h, j * P:(j + 1) * P], int(rv[0, h, j]))):
                _, s, _, _ = oracle.svd_rows(X.astype(np.float64))
                assert _adaptive_ok(s, r, eps, cap), (h, j, r, oracle.adaptive_rank(s, eps, cap))
                chosen.append(r)
    assert len(set(chosen)) > 1, "the pages should need different ranks"
    # factors at the chosen ranks
    refs = [(0, h, int(j)) for h in range(Hkv) for j in np.flatnonzero(plan == oracle.FACTOR)]
    blocks = _export(cache, refs)
    R = cache.c.max_rank
    if factor_dtype == "f32":
        for (b, h, j), blk in zip(refs, blocks):
            Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
            for L, Rm, X, r in ((Lk, Rk, K[b, h, j * P:(j + 1) * P], int(rk[b, h, j])),
                                (Lv, Rv, V[b, h, j * P:(j + 1) * P], int(rv[b, h, j]))):
                X = X.astype(np.float64)
                assert np.linalg.norm(X - L[:, :r] @ Rm[:r]) <= eps * np.linalg.norm(X) * (1 + 1e-3)
                _check_factor(L[:, :r], Rm[:r], X, r, 1e-4, 1e-4, 1e-5)
    # attention over the whole cache against the oracle over the exported pages
    q = synth.queries(wl, 0, 0)
    out, _ = cache.attention(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous(), [T] * B)
    out = out.cpu().numpy().astype(np.float64)
    for h in range(Hkv):
        blk = cache.export_pages(0, [0] * npg, [h] * npg, list(range(npg))).cpu().numpy().astype(np.float64)
        pages = []
        for j in range(npg):
            o = blk[j]
            if plan[j] == oracle.FACTOR:
                a, c2 = int(rk[0, h, j]), int(rv[0, h, j])
                pages.append(("factor", o[:P * R].reshape(P, R)[:, :a], o[P * R:P * R + R * d].reshape(R, d)[:a],
                              o[P * R + R * d:2 * P * R + R * d].reshape(P, R)[:, :c2],
                              o[2 * P * R + R * d:2 * P * R + 2 * R * d].reshape(R, d)[:c2]))
            else:
                pages.append(("dense", o[:P * d].reshape(P, d), o[P * d:2 * P * d].reshape(P, d)))
        ro, _ = oracle.attention(oracle.HeadCache(T, P, d, pages), q[0, h * G:(h + 1) * G].astype(np.float64))
        ma, mr = errors(out[0, h * G:(h + 1) * G], ro)
        assert ma <= MAX_ABS and mr <= MEAN_REL, (h, ma, mr)


def test_adaptive_ranks_incremental_compress():
    """Pages compressed during decoding with a requested rank of 0 get ranks
    chosen per page, written to the table when the entry becomes FACTOR."""
    import torch
    import paper_2608_23843_amd as pk
    eps, B, Hkv, d, P, S, W = 0.2, 1, 2, 128, 64, 64, 128
    T0, steps = 64 * 4 + 60, 40
    wl = synth.Workload("c", 94, B, Hkv, Hkv, d, P, T0, S, W, 24, (24,), "bf16", 5e5, 4, decode_steps=steps)
    K, V = synth.kv_layer(wl, 0, 0)
    max_pages = -(-(T0 + steps) // P)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, max_pages, 32, S, W, "bf16", "f32", adaptive_rank_error=eps)
    cache.prefill(0, torch.from_numpy(K[:, :, :T0]).to("cuda", torch.bfloat16).contiguous(),
                  torch.from_numpy(V[:, :, :T0]).to("cuda", torch.bfloat16).contiguous(), [T0] * B,
                  default_rank=(24, 0))
    converted = []
    for t in range(T0, T0 + steps):
        cache.append(0, torch.from_numpy(K[:, :, t]).to("cuda", torch.bfloat16).contiguous(),
                     torch.from_numpy(V[:, :, t]).to("cuda", torch.bfloat16).contiguous(), [t] * B)
        for j in oracle.eligible_pages(t, t + 1, P, S, W):
            refs = [(0, h, int(j)) for h in range(Hkv)]
            bb, hh, jj = zip(*refs)
            cache.compress_pages(0, bb, hh, jj, [0] * len(refs), [0] * len(refs))
            converted += refs
    torch.cuda.synchronize()
    assert cache.device_status() == 0 and converted
    _, kind, rk, rv = cache.page_table_host(0)
    for (b, h, j) in converted:
        assert kind[b, h, j] == oracle.FACTOR
        for X, r in ((K[b, h, j * P:(j + 1) * P], int(rk[b, h, j])), (V[b, h, j * P:(j + 1) * P], int(rv[b, h, j]))):
            _, s, _, _ = oracle.svd_rows(X.astype(np.float64))
            assert _adaptive_ok(s, r, eps, 32), (h, j, r, oracle.adaptive_rank(s, eps, 32))
    # prefill kept the fixed key rank and chose the value ranks
    plan = oracle.plan_pages(T0, P, S, W, max_pages)
    for j in np.flatnonzero(plan == oracle.FACTOR):
        assert rk[0, 0, j] == 24


@pytest.mark.parametrize("case", range(8))
def test_random_geometries_matrix_core(case):
    """Seeded draws over the matrix-core decomposition: P in {32, 64}, d a
    multiple of 32 up to 256 (d < P gives Gram matrices of rank d), per-page
    ranks 1..min(P, d, 32), fp32 or bf16 factors, a planted page rank r0 and
    RoPE'd keys with outlier channels; every factor page of every head is
    checked against the oracle's SVD (sign-invariant)."""
    rng = np.random.default_rng(2000 + case)
    P = (32, 64)[case % 2]
    d = int(rng.choice([32, 64, 96, 128, 192, 256]))
    ft = ("f32", "bf16")[(case // 2) % 2]
    tols = (1e-4, 1e-4, 1e-5) if ft == "f32" else (6e-3, 1e-2, 4e-3)
    B, Hkv = int(rng.integers(1, 3)), int(rng.integers(1, 3))
    S, W = P * int(rng.integers(0, 2)), P * int(rng.integers(1, 3))
    T = P * int(rng.integers(4, 10)) + int(rng.integers(0, P))
    rmax = min(P, d, 32)
    npg = -(-T // P)
    table = rng.integers(1, rmax + 1, (B, Hkv, npg))
    r0 = int(rng.integers(2, rmax + 1))
    cache, K, V, npg = _prefill_case(B, Hkv, d, P, T, S, W, 0, "bf16", ft, r0, rank_table=table,
                                     rope=1e6, outliers=2, seed=case)
    assert cache.device_status() == 0
    kind = oracle.plan_pages(T, P, S, W, npg)
    refs = [(b, h, j) for b in range(B) for h in range(Hkv) for j in range(npg) if kind[j] == oracle.FACTOR]
    print("case %d: P=%d d=%d %s B=%d Hkv=%d T=%d S=%d W=%d r0=%d, %d factor pages"
          % (case, P, d, ft, B, Hkv, T, S, W, r0, len(refs)))
    blocks = _export(cache, refs)
    R = cache.c.max_rank
    for (b, h, j), blk in zip(refs, blocks):
        r = int(table[b, h, j])
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        for L, Rm, X in ((Lk, Rk, K[b, h, j * P:(j + 1) * P]), (Lv, Rv, V[b, h, j * P:(j + 1) * P])):
            _check_factor(L[:, :r], Rm[:r], X.astype(np.float64), r, *tols)
            assert np.all(L[:, r:] == 0) and np.all(Rm[r:] == 0)


def test_compress_refuses_pages_not_yet_eligible():
    """A page is factorized once, when it is complete and has left the window
    (Section 3.3, "Incremental Cache Update"). The page table records the rows
    each dense page holds (bit-exact against the plan at every step); a sink
    page is refused on the host (PKV_E_STATE), the current partial page and a
    complete page still inside the window raise PKV_DEV_NOT_ELIGIBLE and stay
    exactly as they were, and the same page is accepted once it has left."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, d, P, S, W, r = 1, 2, 128, 64, 64, 128, 16
    T0, steps = 64 * 4 + 10, 70
    wl = synth.Workload("c", 97, B, Hkv, Hkv, d, P, T0, S, W, 24, (r,), "bf16", 5e5, 4, decode_steps=steps)
    K, V = synth.kv_layer(wl, 0, 0)
    max_pages = -(-(T0 + steps) // P) + 1
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, max_pages, 32, S, W, "bf16", "bf16")
    kt = torch.from_numpy(K[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    vt = torch.from_numpy(V[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    cache.prefill(0, kt, vt, [T0] * B, default_rank=(r, r))

    def rows_ok(T):
        t = cache.page_table(0).cpu().numpy()
        plan = oracle.plan_pages(T, P, S, W, max_pages)
        want = np.array([min(P, T - j * P) if plan[j] == oracle.DENSE else 0 for j in range(max_pages)])
        return np.array_equal(t[..., 4], np.broadcast_to(plan, t[..., 4].shape)) and \
            np.array_equal(t[..., 7], np.broadcast_to(want, t[..., 7].shape))

    assert rows_ok(T0)
    with pytest.raises(pk.PuzzleKVError, match="PKV_E_STATE"):
        cache.compress_pages(0, [0], [0], [0], [r], [r])
    done = set()
    for t in range(T0, T0 + steps):
        kn = torch.from_numpy(K[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        vn = torch.from_numpy(V[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        cache.append(0, kn, vn, [t] * B)
        T = t + 1
        plan = oracle.plan_pages(T, P, S, W, max_pages)
        cur = (T - 1) // P                       # the page holding the newest token
        probes = [cur]                           # incomplete unless T is a multiple of P
        probes += [j for j in range(1, cur) if plan[j] == oracle.DENSE and j not in done]
        for j in sorted(set(probes)):
            if plan[j] == oracle.FACTOR:
                continue
            before = cache.page_table(0).clone()
            cache.compress_pages(0, [0], [1], [j], [r], [r])
            assert cache.device_status() == pk._lib.PKV_DEV_NOT_ELIGIBLE, (T, j)
            assert torch.equal(before, cache.page_table(0)), (T, j)
        for j in oracle.eligible_pages(t, T, P, S, W):
            cache.compress_pages(0, [0, 0], [0, 1], [int(j)] * 2, [r, r], [r, r])
            assert cache.device_status() == 0, (T, j)
            done.add(int(j))
        assert rows_ok(T), T
    assert done, "the run must cross a window boundary"


def test_import_refuses_two_dense_pages_on_one_slot():
    """Dense pages of one head live in a ring of ceil(W/P) + 2 slots: importing
    pages j and j + ring length together is refused on the host; importing the
    second while the first is still dense raises PKV_DEV_RING_OVERRUN and
    leaves the slot and the entry untouched."""
    import torch
    import paper_2608_23843_amd as pk
    P, d, S, W = 16, 64, 16, 32
    cache = pk.PuzzleKVCache(1, 1, 1, 1, d, P, 16, 4, S, W, "f32", "f32")
    ring = -(-W // P) + 2
    a = torch.full((2 * P * d,), 1.0, device="cuda")
    bsrc = torch.full((2 * P * d,), 2.0, device="cuda")
    with pytest.raises(pk.PuzzleKVError, match="PKV_E_ARG"):
        cache.import_pages(0, [0, 0], [0, 0], [1, 1 + ring], [oracle.DENSE] * 2, [0, 0], [0, 0],
                           torch.cat([a, bsrc]), [0, 2 * P * d])
    cache.import_pages(0, [0], [0], [1], [oracle.DENSE], [0], [0], a, [0])
    assert cache.device_status() == 0
    before = cache.page_table(0).clone()
    pool = cache.dense_pool.clone()
    cache.import_pages(0, [0], [0], [1 + ring], [oracle.DENSE], [0], [0], bsrc, [0])
    assert cache.device_status() == pk._lib.PKV_DEV_RING_OVERRUN
    assert torch.equal(before, cache.page_table(0))
    assert torch.equal(pool, cache.dense_pool)
    # the same page imported again replaces itself
    cache.import_pages(0, [0], [0], [1], [oracle.DENSE], [0], [0], bsrc, [0])
    assert cache.device_status() == 0


def test_compress_page_list_in_workspace_matches_batches():
    """pkv_compress_pages with a workspace (the page list copied to device
    memory, every page in one launch) and without one (launches of 96 pages):
    one window boundary of 128 (sequence, KV head) pairs, more than one
    launch's worth. Factor pool, page table and device status equal byte for
    byte between the two, and the factors agree with the oracle's SVD."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, d, P, S, W, r = 16, 8, 64, 32, 32, 64, 12
    T0 = 8 * P - 1
    wl = synth.Workload("cw", 93, B, Hkv, Hkv, d, P, T0, S, W, 12, (r,), "bf16", 5e5, 4, decode_steps=P)
    K, V = synth.kv_layer(wl, 0, 0)
    max_pages = -(-(T0 + P) // P) + 1
    caches = [pk.PuzzleKVCache(1, B, Hkv, Hkv, d, P, max_pages, 16, S, W, "bf16", "bf16") for _ in range(2)]
    kt = torch.from_numpy(K[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    vt = torch.from_numpy(V[:, :, :T0]).to("cuda", torch.bfloat16).contiguous()
    for c in caches:
        c.dense_pool.zero_()
        c.factor_pool.zero_()
        c.prefill(0, kt, vt, [T0] * B, default_rank=(r, r))
    refs = []
    for t in range(T0, T0 + P):
        kn = torch.from_numpy(K[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        vn = torch.from_numpy(V[:, :, t]).to("cuda", torch.bfloat16).contiguous()
        for c in caches:
            c.append(0, kn, vn, [t] * B)
        new = oracle.eligible_pages(t, t + 1, P, S, W)
        for j in new:
            refs = [(b, h, int(j)) for b in range(B) for h in range(Hkv)]
            bb, hh, jj = zip(*refs)
            assert len(refs) > 96
            caches[0].compress_pages(0, bb, hh, jj, [r] * len(refs), [8] * len(refs))
            caches[1].compress_pages(0, bb, hh, jj, [r] * len(refs), [8] * len(refs), workspace=None)
    torch.cuda.synchronize()
    assert refs, "the run must cross a window boundary"
    assert caches[0].device_status() == 0 and caches[1].device_status() == 0
    assert torch.equal(caches[0].factor_pool, caches[1].factor_pool)
    assert torch.equal(caches[0].table, caches[1].table)
    assert torch.equal(caches[0].dense_pool, caches[1].dense_pool)
    blocks = _export(caches[0], refs[::17])
    R = caches[0].c.max_rank
    for (b, h, j), blk in zip(refs[::17], blocks):
        Lk, Rk, Lv, Rv = _unpack_factor(blk, P, d, R)
        _check_factor(Lk[:, :r], Rk[:r], K[b, h, j * P:(j + 1) * P].astype(np.float64), r, 6e-3, 1e-2, 4e-3)
        _check_factor(Lv[:, :8], Rv[:8], V[b, h, j * P:(j + 1) * P].astype(np.float64), 8, 6e-3, 1e-2, 4e-3)
