"""PuzzleKV CPU oracle (fp64) -- test infrastructure only.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product library
(``paper_2608_23843_amd``) never imports it, and it imports nothing from the
product: the two share no code.

The numeric work lives in ``oracle.c`` (plain C, no BLAS or LAPACK), compiled
with gcc into ``liboracle.so`` next to it; this module only marshals numpy
arrays. The INT4 factor encoding, an encoding rather than a numeric kernel,
is written in numpy in ``int4.py``. Storage accounting is in ``accounting.py``.

Parity status of each routine is listed with its pins in ``tests/``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

EMPTY, DENSE, FACTOR = 0, 1, 2
MAX_SWEEPS = 60

_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc (OpenMP, -O2). Returns the library path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    lib = ctypes.CDLL(_LIB)
    i32, i64, dbl = ctypes.c_int, ctypes.c_longlong, ctypes.c_double
    p = ctypes.c_void_p
    lib.orc_page_kind.argtypes = [i64, i32, i32, i32, i64]
    lib.orc_page_kind.restype = i32
    lib.orc_plan_pages.argtypes = [i64, i32, i32, i32, p, i64]
    lib.orc_plan_pages.restype = i64
    lib.orc_eligible_pages.argtypes = [i64, i64, i32, i32, i32, p, i64]
    lib.orc_eligible_pages.restype = i64
    lib.orc_svd_rows.argtypes = [i32, i32, p, p, p, p, i32]
    lib.orc_svd_rows.restype = i32
    lib.orc_truncated_factors.argtypes = [i32, i32, i32, p, p, p, p, i32]
    lib.orc_truncated_factors.restype = i32
    lib.orc_adaptive_rank.argtypes = [i32, p, dbl, i32]
    lib.orc_adaptive_rank.restype = i32
    lib.orc_truncated_factors_batch.argtypes = [i32, i32, i32, p, p, p, p, i32, p, p, i32]
    lib.orc_truncated_factors_batch.restype = None
    lib.orc_attention.argtypes = [i64, i32, i32, i32, i32, p, p, p, p, p, p, dbl, p, p]
    lib.orc_rope_rows.argtypes = [i32, i32, p, dbl, p]
    lib.orc_rope_rows.restype = i32
    lib.orc_attention.restype = i32
    lib.orc_attention_pagewise.argtypes = [i64, i32, i32, i32, i32, p, p, p, p, p, p, p, i32,
                                           p, p]
    lib.orc_attention_pagewise.restype = i32
    lib.orc_num_threads.argtypes = []
    lib.orc_num_threads.restype = i32
    lib.orc_set_num_threads.argtypes = [i32]
    lib.orc_set_num_threads.restype = None
    _ = dbl
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Sets the OpenMP threads of the oracle's parallel loops (timing only)."""
    _load().orc_set_num_threads(int(n))


# --------------------------------------------------------------------------
# Page plan (Section 3.3; Section 4.1 "Implementation")
# --------------------------------------------------------------------------
def page_kind(T: int, P: int, S: int, W: int, j: int) -> int:
    return int(_load().orc_page_kind(T, P, S, W, j))


def plan_pages(T: int, P: int, S: int, W: int, n: int | None = None) -> np.ndarray:
    """Kind of every logical page (0 empty, 1 dense, 2 factor), length n."""
    if n is None:
        n = -(-T // P) if T > 0 else 0
    kind = np.zeros(max(n, 1), dtype=np.uint8)
    _load().orc_plan_pages(T, P, S, W, _ptr(kind), n)
    return kind[:n]


def eligible_pages(T_prev: int, T_new: int, P: int, S: int, W: int) -> np.ndarray:
    """Pages that become factorized when the length grows from T_prev to T_new."""
    cap = max(1, -(-T_new // P))
    out = np.zeros(cap, dtype=np.int64)
    cnt = _load().orc_eligible_pages(T_prev, T_new, P, S, W, _ptr(out), cap)
    return out[:cnt].copy()


# --------------------------------------------------------------------------
# Truncated SVD (Section 3.2; Eq. (2))
# --------------------------------------------------------------------------
def svd_rows(X: np.ndarray, max_sweeps: int = MAX_SWEEPS):
    """One-sided Jacobi SVD of X (n x d): returns U (n x n), sig (n), Rf (n x d), sweeps.

    X = U @ Rf, columns of U orthonormal, rows of Rf = sig_k w_k^T."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    n, d = X.shape
    U = np.empty((n, n)); sig = np.empty(n); Rf = np.empty((n, d))
    sw = _load().orc_svd_rows(n, d, _ptr(X), _ptr(U), _ptr(sig), _ptr(Rf), max_sweeps)
    return U, sig, Rf, int(sw)


def truncated_factors(X: np.ndarray, r: int, max_sweeps: int = MAX_SWEEPS):
    """Eq. (2) factor pair of one page: L = U_r (P x r), R = Sigma_r W_r^T (r x d).

    Returns (L, R, sig, sweeps); sig holds all P singular values."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    P, d = X.shape
    L = np.empty((P, r)); R = np.empty((r, d)); sig = np.empty(P)
    sw = _load().orc_truncated_factors(P, d, r, _ptr(X), _ptr(L), _ptr(R), _ptr(sig),
                                       max_sweeps)
    return L, R, sig, int(sw)


def adaptive_rank(sig: np.ndarray, eps: float, cap: int) -> int:
    """Smallest r >= 1 with |X - X_r|_F <= eps |X|_F given the page's singular
    values in descending order (the reconstruction-accuracy reading of the
    paper's Figure 2), capped at cap."""
    sig = np.ascontiguousarray(sig, dtype=np.float64)
    return int(_load().orc_adaptive_rank(len(sig), _ptr(sig), float(eps), int(cap)))


def truncated_factors_batch(X: np.ndarray, ranks, max_sweeps: int = MAX_SWEEPS):
    """Eq. (2) for a batch X (n, P, d) with per-page ranks (OpenMP over pages).

    Returns L (n, P, rmax), R (n, rmax, d), sig (n, P), sweeps (n); entries past a
    page's own rank are unspecified."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    n, P, d = X.shape
    ranks = np.ascontiguousarray(np.broadcast_to(np.asarray(ranks, dtype=np.int32), (n,)))
    rmax = int(ranks.max()) if n else 1
    L = np.zeros((n, P, rmax)); R = np.zeros((n, rmax, d)); sig = np.empty((n, P))
    sweeps = np.empty(n, dtype=np.int32)
    if n:
        _load().orc_truncated_factors_batch(n, P, d, _ptr(ranks), _ptr(X), _ptr(L), _ptr(R),
                                            rmax, _ptr(sig), _ptr(sweeps), max_sweeps)
    # The C routine writes each page's L with leading dimension r_p inside the
    # rmax-wide slot; re-lay every page as a plain (P, r_p) block padded to rmax.
    Lout = np.zeros_like(L)
    Rout = np.zeros_like(R)
    for p in range(n):
        r = int(ranks[p])
        Lout[p, :, :r] = L[p].reshape(-1)[:P * r].reshape(P, r)
        Rout[p, :r, :] = R[p].reshape(-1)[:r * d].reshape(r, d)
    return Lout, Rout, sig, sweeps


def global_factors(X: np.ndarray, r: int, max_sweeps: int = MAX_SWEEPS):
    """Global SVD, the paper's controlled baseline (Section 4.1 "Baselines";
    Appendix "Baseline Configurations"): one basis shared by every token of the
    compressible region X (N x d) of one KV head, the rank-r truncated SVD
    X ~ U_r Sigma_r W_r^T stored as A = U_r Sigma_r (N x r), one coefficient
    row per token, and B = W_r^T (r x d), the shared basis.

    Computed with the same one-sided Jacobi as the page factors, applied to
    the d rows of X^T: X^T = J Y with J (d x d) = W and the rows of Y the
    sigma_k u_k^T, so B = J[:, :r]^T and A = Y[:r]^T. r is capped at
    min(N, d). Returns (A, B, sig, sweeps); sig holds all d singular values."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    N, d = X.shape
    r = int(min(r, N, d))
    J, sig, Y, sw = svd_rows(np.ascontiguousarray(X.T), max_sweeps)
    return np.ascontiguousarray(Y[:r].T), np.ascontiguousarray(J[:, :r].T), sig, sw


# --------------------------------------------------------------------------
# Attention (Eq. (1)) and page-wise state + merge (Eq. (4), Eq. (5))
# --------------------------------------------------------------------------
def rope_rows(X: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate-half RoPE of the rows of X (n, d) at positions pos (n,), fp64
    (Section 4.2; Appendix "RoPE Key Analysis")."""
    Y = np.array(np.atleast_2d(X), dtype=np.float64, order="C")
    pos = np.ascontiguousarray(np.broadcast_to(np.asarray(pos, dtype=np.int64), (Y.shape[0],)))
    if _load().orc_rope_rows(Y.shape[0], Y.shape[1], _ptr(pos), float(base), _ptr(Y)) != 0:
        raise ValueError("orc_rope_rows: d must be even and base > 0")
    return Y


class HeadCache:
    """Logical contents of one KV head: a list of pages.

    Each page is ("dense", K, V) with K, V of shape (P, d), or
    ("factor", L_K, R_K, L_V, R_V) with shapes (P, rk), (rk, d), (P, rv), (rv, d).
    Rows past the sequence length in the last page are ignored. key_rope_base
    > 0: the stored keys are pre-RoPE and the attention rotates key t to
    position t before the scores."""

    def __init__(self, T: int, P: int, d: int, pages, key_rope_base: float = 0.0):
        self.T, self.P, self.d = int(T), int(P), int(d)
        self.pages = list(pages)
        self.key_rope_base = float(key_rope_base)

    def pack(self):
        kind = np.zeros(len(self.pages), dtype=np.int32)
        rk = np.zeros(len(self.pages), dtype=np.int32)
        rv = np.zeros(len(self.pages), dtype=np.int32)
        off = np.zeros(len(self.pages), dtype=np.int64)
        chunks, pos = [], 0
        for j, pg in enumerate(self.pages):
            off[j] = pos
            if pg[0] == "dense":
                kind[j] = DENSE
                mats = [pg[1], pg[2]]
                assert pg[1].shape == (self.P, self.d) and pg[2].shape == (self.P, self.d)
            elif pg[0] == "factor":
                kind[j] = FACTOR
                Lk, Rk, Lv, Rv = pg[1:]
                rk[j], rv[j] = Lk.shape[1], Lv.shape[1]
                assert Lk.shape == (self.P, rk[j]) and Rk.shape == (rk[j], self.d)
                assert Lv.shape == (self.P, rv[j]) and Rv.shape == (rv[j], self.d)
                mats = [Lk, Rk, Lv, Rv]
            else:
                raise ValueError(pg[0])
            for m in mats:
                a = np.ascontiguousarray(m, dtype=np.float64).reshape(-1)
                chunks.append(a)
                pos += a.size
        data = np.concatenate(chunks) if chunks else np.zeros(1)
        return kind, rk, rv, off, data


def global_head(T: int, P: int, d: int, kinds, K: np.ndarray, V: np.ndarray, A_K: np.ndarray,
                B_K: np.ndarray, A_V: np.ndarray, B_V: np.ndarray) -> HeadCache:
    """The logical contents of one KV head stored by Global SVD: pages the plan
    `kinds` keeps dense hold K, V (rows of the whole sequence, T x d) as they
    are; the tokens of the factorized pages, in order, are the rows of A_K,
    A_V, rebuilt with the shared bases B_K, B_V. Each such page is written as a
    factor page (L = its rows of A, R = B), so attention over it is the same
    textbook softmax over the rebuilt keys and values."""
    pages, row = [], 0
    for j, kd in enumerate(kinds):
        if kd == FACTOR:
            pages.append(("factor", A_K[row:row + P], B_K, A_V[row:row + P], B_V))
            row += P
        else:
            Kp = np.zeros((P, d)); Vp = np.zeros((P, d))
            n = min(P, T - j * P)
            Kp[:n] = K[j * P:j * P + n]
            Vp[:n] = V[j * P:j * P + n]
            pages.append(("dense", Kp, Vp))
    if row != A_K.shape[0] or row != A_V.shape[0]:
        raise ValueError("coefficient rows (%d, %d) do not match the %d factorized tokens"
                         % (A_K.shape[0], A_V.shape[0], row))
    return HeadCache(T, P, d, pages)


def attention(head: HeadCache, q: np.ndarray):
    """Textbook softmax attention of the g queries q (g, d) over the rebuilt head.

    Returns (out (g, d), lse (g))."""
    q = np.ascontiguousarray(np.atleast_2d(q), dtype=np.float64)
    g = q.shape[0]
    kind, rk, rv, off, data = head.pack()
    out = np.empty((g, head.d)); lse = np.empty(g)
    rc = _load().orc_attention(head.T, head.P, head.d, g, len(head.pages), _ptr(kind), _ptr(rk),
                               _ptr(rv), _ptr(off), _ptr(data), _ptr(q), head.key_rope_base, _ptr(out),
                               _ptr(lse))
    if rc != 0:
        raise ValueError("orc_attention failed (%d)" % rc)
    return out, lse


def attention_pagewise(head: HeadCache, q: np.ndarray, order=None, group: int = 0):
    """Eq. (4) page states merged by Eq. (5), pages visited in `order`, merged in
    groups of `group` visited pages first. Returns (out, lse)."""
    if head.key_rope_base > 0:
        raise ValueError("the factor-form evaluation of Eq. (4) needs post-RoPE keys")
    q = np.ascontiguousarray(np.atleast_2d(q), dtype=np.float64)
    g = q.shape[0]
    kind, rk, rv, off, data = head.pack()
    out = np.empty((g, head.d)); lse = np.empty(g)
    ordp = None
    if order is not None:
        order = np.ascontiguousarray(order, dtype=np.int32)
        ordp = _ptr(order)
    rc = _load().orc_attention_pagewise(head.T, head.P, head.d, g, len(head.pages), _ptr(kind),
                                        _ptr(rk), _ptr(rv), _ptr(off), _ptr(data), _ptr(q), ordp,
                                        int(group), _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError("orc_attention_pagewise failed (%d)" % rc)
    return out, lse
