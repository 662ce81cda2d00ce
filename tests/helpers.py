"""Test-side helpers: build cache contents from the seeded generator, import
them into the GPU cache, and hand the same logical pages to the oracle.

Factor pages handed to both sides come from the oracle's own decomposition
(or are drawn directly by the generator), rounded to the storage type; no
input of the oracle ever comes from the GPU path."""
from __future__ import annotations

import numpy as np

import oracle
import synth

# Tolerance for floating-point parity of the attention output with bf16
# storage and fp32 accumulation: max-abs <= 1e-2 and normwise mean-relative
# error sum|gpu - ref| / sum|ref| <= 1e-3.
MAX_ABS = 1e-2
MEAN_REL = 1e-3


def errors(gpu: np.ndarray, ref: np.ndarray):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = np.abs(gpu - ref)
    max_abs = float(diff.max()) if diff.size else 0.0
    denom = float(np.abs(ref).sum())
    mean_rel = float(diff.sum() / denom) if denom > 0 else float(diff.sum())
    return max_abs, mean_rel


def storage_round(x, dtype: str):
    return synth.round_storage(np.asarray(x, dtype=np.float32), dtype).astype(np.float64)


def build_head_pages(K, V, T, P, S, W, ranks, factor_dtype, max_sweeps=60):
    """Logical pages of one KV head. K, V: (>= n_pages * P, d) storage-rounded
    arrays (rows past T may be anything). Factor pages are the oracle's Eq. (2)
    factors of the stored page, rounded to factor_dtype. ranks: per page
    (rank_k, rank_v) or one int for all. Returns a list of page tuples in the
    oracle.HeadCache format."""
    n = -(-T // P)
    kind = oracle.plan_pages(T, P, S, W, n)
    d = K.shape[1]
    pages = []
    for j in range(n):
        Kp = np.zeros((P, d)); Vp = np.zeros((P, d))
        rows = min(P, T - j * P)
        Kp[:rows] = K[j * P:j * P + rows]
        Vp[:rows] = V[j * P:j * P + rows]
        if kind[j] == oracle.FACTOR:
            r = ranks[j] if np.ndim(ranks) else ranks
            rk, rv = (r, r) if np.ndim(r) == 0 else r
            Lk, Rk, _, _ = oracle.truncated_factors(Kp, int(rk), max_sweeps)
            Lv, Rv, _, _ = oracle.truncated_factors(Vp, int(rv), max_sweeps)
            pages.append(("factor", storage_round(Lk, factor_dtype), storage_round(Rk, factor_dtype),
                          storage_round(Lv, factor_dtype), storage_round(Rv, factor_dtype)))
        else:
            pages.append(("dense", Kp, Vp))
    return pages


def import_head(cache, layer, b, h, pages, which=("dense", "factor")):
    """Writes logical pages of one head into the GPU cache via pkv_import_pages."""
    import torch
    for kind_name in which:
        idx = [j for j, pg in enumerate(pages) if pg[0] == kind_name]
        if not idx:
            continue
        dt = cache.qdtype if kind_name == "dense" else cache.fdtype
        chunks, offs, rk, rv, pos = [], [], [], [], 0
        for j in idx:
            pg = pages[j]
            mats = pg[1:]
            offs.append(pos)
            for m in mats:
                a = np.asarray(m, dtype=np.float32).reshape(-1)
                chunks.append(a)
                pos += a.size
            if kind_name == "factor":
                rk.append(pg[1].shape[1]); rv.append(pg[3].shape[1])
            else:
                rk.append(0); rv.append(0)
        src = torch.from_numpy(np.concatenate(chunks)).to(device=cache.device, dtype=dt)
        kinds = [oracle.DENSE if kind_name == "dense" else oracle.FACTOR] * len(idx)
        cache.import_pages(layer, [b] * len(idx), [h] * len(idx), idx, kinds, rk, rv, src, offs)


def oracle_head(T, P, d, pages):
    return oracle.HeadCache(T, P, d, pages)
