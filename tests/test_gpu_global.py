"""GPU parity of the Global SVD baseline (Section 4.1 "Baselines"; Section 4.2;
Appendix "Baseline Configurations") through the C ABI.

* Decomposition: the truncated SVD with one basis per head is unique only up
  to signs and rotations inside repeated singular values, so the GPU factors
  are checked through sign-invariant quantities against the oracle's fp64
  Jacobi SVD of the same region: orthonormal basis rows, coefficients equal to
  the projection X B^T with the stored basis, coefficient column norms against
  the singular values, and the Eckart-Young reconstruction error against the
  oracle's spectral tail; where the spectrum has a gap at r the basis spans
  the oracle's subspace.
* Attention: the GPU result against the oracle's textbook attention over the
  GPU's own exported factors (coefficient rows placed on the factorized
  pages), max-abs <= 1e-2 and normwise mean-relative <= 1e-3.
* Page table: dense pages of the plan are DENSE with their rows, factorized
  pages are PKV_GLOBAL with the rank and their first coefficient row.
"""
import hashlib

import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, errors

pytestmark = pytest.mark.gpu

D = 128


def _wl(B, Hkv, g, P, T, S, W, seg, wid=120):
    return synth.Workload("global", wid, B, Hkv, Hkv * g, D, P, T, S, W, 24, (16,), "bf16", 1.0e6, 4,
                          segment_pages=seg)


def _region(T, P, S, W):
    kinds = oracle.plan_pages(T, P, S, W)
    rows = [np.arange(j * P, (j + 1) * P) for j, k in enumerate(kinds) if k == oracle.FACTOR]
    return kinds, (np.concatenate(rows) if rows else np.zeros(0, dtype=np.int64))


def _build(B, Hkv, g, P, S, W, seq, r, seg, max_tokens=None, wid=120):
    import torch
    import paper_2608_23843_amd as pk
    Tmax = max(seq)
    wl = _wl(B, Hkv, g, P, Tmax, S, W, seg, wid)
    K, V = synth.kv_layer(wl, 0, 0, Tmax)
    max_pages = max(1, -(-Tmax // P))
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "bf16")
    mt = max_tokens or max(32, -(-Tmax // 32) * 32)
    gs = pk.GlobalSVD(cache, r, mt)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous()
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous()
    gs.prefill(0, kt, vt, seq)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    return cache, gs, wl, K.astype(np.float64), V.astype(np.float64)


def _check_table(cache, seq, P, S, W, r):
    t = cache.page_table(0).cpu().numpy()
    slot = t[..., :4].copy().view(np.int32)[..., 0]
    for b, T in enumerate(seq):
        kinds = oracle.plan_pages(T, P, S, W, t.shape[2])
        for j, kd in enumerate(kinds):
            e = t[b, :, j]
            if kd == oracle.FACTOR:
                assert np.all(e[:, 4] == 3) and np.all(e[:, 5] == r) and np.all(e[:, 6] == r), (b, j)
                assert np.all(slot[b, :, j] == (j - (-(-S // P))) * P), (b, j)
            elif kd == oracle.DENSE:
                assert np.all(e[:, 4] == 1) and np.all(e[:, 7] == min(P, T - j * P)), (b, j)
            else:
                assert np.all(e[:, 4] == 0), (b, j)


_SVD = {}


def _oracle_svd(X, r):
    """The oracle's factors of a region at rank r (the full SVD is computed
    once per region and truncated)."""
    key = hashlib.sha1(np.ascontiguousarray(X).tobytes()).hexdigest()
    if key not in _SVD:
        _SVD[key] = oracle.global_factors(X, X.shape[1])
    A, B, sig, _ = _SVD[key]
    re = min(r, X.shape[0], X.shape[1])
    return A[:, :re], B[:re], sig


def _check_factors(X, Bk, Ak, r, gap):
    """X: the region (N x d, the stored bf16 values), Bk (r x d), Ak (N x r) from the GPU."""
    N = X.shape[0]
    A_o, B_o, sig = _oracle_svd(X, r)
    re = min(r, N, D)
    Bg = Bk[:re]
    # orthonormal basis rows (bf16 entries: 2^-9 relative each); a row is zero
    # only for a direction at rounding level of the fp32 Gram matrix
    nz = np.linalg.norm(Bg, axis=1) > 0.5
    assert np.all(nz[sig[:re] > 2.0 ** -11 * sig[0]])
    Gb = Bg[nz] @ Bg[nz].T
    assert np.abs(Gb - np.eye(int(nz.sum()))).max() < 1e-2
    # coefficients are the projection with the stored basis, rounded to bf16
    P_ = X @ Bg.T
    assert np.abs(Ak[:, :re] - P_).sum() <= 2.0 ** -8 * np.abs(P_).sum()
    # coefficient column norms against the singular values (fp32 Gram: its
    # eigenvalues are good to ~1e-6 of the largest, i.e. sigma to ~1e-3 sigma_1
    # near the bottom of a wide spectrum)
    cn = np.linalg.norm(Ak[:, :re], axis=0)
    assert np.all(np.abs(cn - sig[:re]) <= 1e-2 * sig[:re] + 2e-3 * sig[0]), np.abs(cn - sig[:re]).max()
    # Eckart-Young: the error is the spectral tail, plus the bf16 rounding of
    # the stored factors
    E = X - Ak[:, :re] @ Bg
    err = np.sqrt(np.sum(E * E))
    tail = np.sqrt(np.sum(sig[re:] ** 2))
    fro = np.sqrt(np.sum(X * X))
    assert tail - 1e-3 * fro <= err <= tail * (1 + 1e-3) + 4 * 2.0 ** -9 * fro, (err, tail, fro)
    if gap:
        Po = B_o.T @ B_o
        assert np.abs(Bg.T @ Bg - Po).max() < 2e-2
    return err / fro, tail / fro


def _attend_and_check(cache, gs, wl, K, V, seq, P, S, W, r, g):
    import torch
    q = synth.queries(wl, 0)
    qt = torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous()
    out, lse = gs.attention(0, qt, seq)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    lse = lse.cpu().numpy().astype(np.float64)
    ref = np.zeros_like(out)
    ref_lse = np.full_like(lse, -np.inf)
    for b, T in enumerate(seq):
        if T == 0:
            continue
        kinds, rows = _region(T, P, S, W)
        for h in range(cache.c.n_kv_heads):
            bk, bv, ak, av = (x.cpu().numpy().astype(np.float64) for x in gs.export(0, b, h, len(rows)))
            head = oracle.global_head(T, P, D, kinds, K[b, h], V[b, h], ak, bk, av, bv)
            o, l = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
            ref[b, h * g:(h + 1) * g] = o
            ref_lse[b, h * g:(h + 1) * g] = l
    ma, mr = errors(out, ref)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (ma, mr)
    fin = np.isfinite(ref_lse)
    assert np.all(np.abs(lse[fin] - ref_lse[fin]) <= 1e-3)
    assert np.all(out[~fin.repeat(D).reshape(out.shape)] == 0)
    return ma, mr


@pytest.mark.parametrize("r,seg,gap", [(40, 1, False), (77, 16, False), (24, 0, True)])
def test_global_svd_matches_oracle(r, seg, gap):
    """Two sequences of ragged lengths, two KV heads, P = 32, paper-default
    dense region; ranks covering one, two and three 32-rank steps; planted
    subspaces changing every page, every 16 pages, and never (one rank-24
    basis for the whole sequence: the values' spectrum then has a gap at
    r = 24 and the basis must span the oracle's subspace; the keys' RoPE
    leaves no such gap)."""
    B, Hkv, g, P, S, W = 2, 2, 4, 32, 32, 32
    seq = [32 * 70 + 11, 32 * 45]
    cache, gs, wl, K, V = _build(B, Hkv, g, P, S, W, seq, r, seg)
    _check_table(cache, seq, P, S, W, r)
    for b, T in enumerate(seq):
        _, rows = _region(T, P, S, W)
        for h in range(Hkv):
            bk, bv, ak, av = (x.cpu().numpy().astype(np.float64) for x in gs.export(0, b, h, len(rows)))
            _check_factors(K[b, h][rows], bk, ak, r, False)   # post-RoPE keys: no gap at r
            _check_factors(V[b, h][rows], bv, av, r, gap)
    _attend_and_check(cache, gs, wl, K, V, seq, P, S, W, r, g)


def test_global_svd_edges():
    """P = 64 with a 512-token window; a sequence with no factorized page, an
    empty one, one whose region spans several 4,096-token Gram chunks (a
    ragged last chunk), rank 1 and the full rank 128 (exact up to bf16)."""
    B, Hkv, g, P, S, W = 4, 1, 8, 64, 64, 512
    seq = [64 * 140 + 30, 300, 0, 64 * 20]
    for r in (1, 128):
        cache, gs, wl, K, V = _build(B, Hkv, g, P, S, W, seq, r, 4, wid=121)
        _check_table(cache, seq, P, S, W, r)
        for b, T in enumerate(seq):
            _, rows = _region(T, P, S, W)
            if len(rows) == 0:
                continue
            bk, bv, ak, av = (x.cpu().numpy().astype(np.float64) for x in gs.export(0, b, 0, len(rows)))
            for X, Bm, Am in ((K[b, 0][rows], bk, ak), (V[b, 0][rows], bv, av)):
                rel, tail = _check_factors(X, Bm, Am, r, False)
                if r == 128:
                    assert rel < 4 * 2.0 ** -9
        _attend_and_check(cache, gs, wl, K, V, seq, P, S, W, r, g)


def test_global_svd_errors():
    """Host-side refusals: region longer than max_tokens, rank outside 1..128,
    unsupported geometry, too small a workspace."""
    import torch
    import paper_2608_23843_amd as pk
    cache = pk.PuzzleKVCache(1, 1, 1, 4, D, 32, 64, 16, 32, 32, "bf16", "bf16")
    gs = pk.GlobalSVD(cache, 16, 64)
    k = torch.zeros((1, 1, 2048, D), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(pk.PuzzleKVError, match="PKV_E_SHAPE"):
        gs.prefill(0, k, k, [2048])
    with pytest.raises(pk.PuzzleKVError):
        pk.GlobalSVD(cache, 129, 64)
    c32 = pk.PuzzleKVCache(1, 1, 1, 4, 64, 32, 64, 16, 32, 32, "bf16", "bf16")
    with pytest.raises(pk.PuzzleKVError):
        pk.GlobalSVD(c32, 16, 64)
    import ctypes
    lib = pk.load_library()
    q = torch.zeros((1, 4, D), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((1, 4, D), dtype=torch.float32, device="cuda")
    ws = torch.zeros(16, dtype=torch.uint8, device="cuda")
    seq = np.array([64], dtype=np.int32)
    st = lib.pkv_global_attention(ctypes.byref(cache.c), ctypes.byref(gs.g), 0, q.data_ptr(),
                                  seq.ctypes.data_as(ctypes.c_void_p), out.data_ptr(), None, ws.data_ptr(), 16,
                                  None)
    assert st == pk._lib.PKV_E_WORKSPACE
