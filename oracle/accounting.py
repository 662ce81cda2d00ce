"""Storage accounting of the hybrid cache (test infrastructure, see oracle/__init__.py).

Plain restatements of the paper's storage formulas:
  * dense KV size 2 * L * H_kv * T * d elements (Section 1),
  * factor-page storage ratio rho_page = (r_K + r_V)(P + d) / (2 P d)
    (Section 3.3, Eq. (3); Appendix D.1, Eq. (6)),
  * whole-cache ratio when some pages stay dense (Section 4.5, "Memory
    Footprint": dense pages count at ratio 1),
  * INT4 factor storage, 4-bit codes plus one fp16 scale per run of at most 32
    elements along the direction Section 4.3 names for each factor,
  * Global SVD storage (Section 4.2, "Main Results": rho_global = r (S + d) /
    (S d) for an input of S tokens), with the rank matched to a budget
    counting the dense sink and window tokens as well (Appendix "Baseline
    Configurations").
"""
from __future__ import annotations


def dense_kv_bytes(layers: int, kv_heads: int, tokens: int, head_dim: int,
                   bytes_per_elem: int = 2) -> int:
    """Bytes of an uncompressed KV cache: 2 L H_kv T d elements."""
    return 2 * layers * kv_heads * tokens * head_dim * bytes_per_elem


def page_storage_ratio(P: int, r_k: int, r_v: int, d: int) -> float:
    """Eq. (3): storage of one factorized K/V page pair relative to dense."""
    return (r_k + r_v) * (P + d) / (2.0 * P * d)


def cache_ratio(n_pages: int, n_dense: int, P: int, r_k: int, r_v: int, d: int) -> float:
    """Whole-cache ratio: dense pages at 1, the others at rho_page."""
    rho = page_storage_ratio(P, r_k, r_v, d)
    return (rho * (n_pages - n_dense) + n_dense) / n_pages


def _runs(n: int, group: int = 32) -> int:
    return -(-n // group)


def int4_scale_count(P: int, r_k: int, r_v: int, d: int, group: int = 32) -> int:
    """fp16 scales of one INT4 factor page pair. Directions (Section 4.3):
    L_K column-wise, R_K column-wise, L_V row-wise, R_V column-wise; each line
    is cut into runs of at most `group` consecutive elements."""
    return (r_k * _runs(P, group)        # L_K: r_k columns of length P
            + d * _runs(r_k, group)       # R_K: d columns of length r_k
            + P * _runs(r_v, group)       # L_V: P rows of length r_v
            + d * _runs(r_v, group))      # R_V: d columns of length r_v


def int4_page_bytes(P: int, r_k: int, r_v: int, d: int, group: int = 32) -> float:
    """Bytes of one INT4 factor page pair: half a byte per code, 2 per scale."""
    codes = (r_k + r_v) * (P + d)
    return codes / 2.0 + 2.0 * int4_scale_count(P, r_k, r_v, d, group)


def int4_page_ratio(P: int, r_k: int, r_v: int, d: int, group: int = 32) -> float:
    """INT4 factor page pair relative to a dense bf16 page pair (2 P d * 2 bytes)."""
    return int4_page_bytes(P, r_k, r_v, d, group) / (2.0 * P * d * 2.0)


def int4_cache_ratio(n_pages: int, n_dense: int, P: int, r_k: int, r_v: int, d: int,
                     group: int = 32) -> float:
    rho = int4_page_ratio(P, r_k, r_v, d, group)
    return (rho * (n_pages - n_dense) + n_dense) / n_pages


def global_storage_elems(n_dense_tokens: int, n_factor_tokens: int, d: int, r: int) -> int:
    """Elements Global SVD stores for one KV head: K and V of the dense tokens,
    and for each of K and V the coefficients (one r-vector per factorized
    token) plus the shared r x d basis."""
    return 2 * n_dense_tokens * d + 2 * r * (n_factor_tokens + d)


def global_rank(n_dense_tokens: int, n_factor_tokens: int, d: int, rho: float) -> int:
    """Largest rank r (same for K and V, at most min(N, d)) whose whole-head
    storage, dense tokens included, stays within rho times the raw cache
    (2 T d elements, T = dense + factorized tokens); 0 if even rank 1 does not fit."""
    T = n_dense_tokens + n_factor_tokens
    budget = rho * 2.0 * T * d
    best = 0
    for r in range(1, min(n_factor_tokens, d) + 1):
        if global_storage_elems(n_dense_tokens, n_factor_tokens, d, r) <= budget:
            best = r
    return best
