"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds no part of the method's arithmetic: it only draws keys,
values, queries and per-page ranks, and rounds them to their storage type.
Both the oracle side and the GPU side of every test receive the same arrays
from here; neither imports the other.

Recipe (every draw comes from numpy's PCG64 seeded by
SeedSequence([seed, workload_id, tag, ...])):
  * per page j of one (layer, batch, kv head), independently for K and V:
    X_j = G_j W_j + 0.05 N_j with G_j (P x r0), W_j (r0 x d), N_j (P x d)
    all i.i.d. N(0, 1) -- pages with low-rank structure plus noise, the
    property the paper measures on real caches (Section 3.1);
  * keys (not the tiny workload): 4 channels per (layer, kv head), drawn
    without replacement, are scaled by 10 before RoPE; RoPE uses the
    rotate-half convention at absolute position t = j P + row with base
    5e5 (Llama-3-8B shape) or 1e6 (Qwen3-32B shape);
  * queries: per (batch, query head) i.i.d. N(0, 1/d);
  * ranks: fixed, or uniform over a set per (layer, batch, kv head, page);
  * storage rounding: bf16 round-to-nearest-even, or none for fp32;
  * non-stationary sequences (workloads with segment_pages != 1): the planted
    basis W is shared by runs of segment_pages consecutive pages and drawn
    afresh for the next run (0: one basis for the whole sequence), so the
    subspace the keys and values live in changes every segment.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import functools

import numpy as np

TAG_KEY, TAG_VALUE, TAG_OUTLIER, TAG_QUERY, TAG_RANK, TAG_FACTOR, TAG_TOKEN, TAG_GLOBAL = range(8)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int              # workload id used in the seed sequence
    batch: int
    kv_heads: int
    q_heads: int
    head_dim: int
    page: int             # P
    tokens: int           # T (prefill length)
    sink: int             # S, tokens
    window: int           # W, tokens
    r0: int               # rank of the planted page structure
    ranks: tuple          # rank choices for factorized pages
    dtype: str            # "f32" or "bf16"
    rope_base: float | None
    outliers: int
    layers: int = 1
    decode_steps: int = 0
    factor_dtype: str = ""  # storage of factor pages when it differs from dtype ("int4")
    ranks_v: tuple = ()     # rank choices of the value factors when they differ from the keys
    rank_error: float = 0.0  # > 0: each page's rank chosen for this relative reconstruction error
    key_rope: bool = False   # keys handed over before RoPE (the cache rotates them at access)
    segment_pages: int = 1   # pages sharing one planted basis (0: the whole sequence)
    global_rho: float = 0.0  # != 0: a Global SVD cache, its rank matched to this storage ratio
                             # (< 0: to the PuzzleKV ratio realized on the same inputs)

    @property
    def factors(self) -> str:
        return self.factor_dtype or self.dtype

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads


WORKLOADS = {
    # 1 layer, 1 KV head, 1 query head, d=64, P=16, T=256, sink 16, window 32, r=4, fp32.
    "tiny": Workload("tiny", 1, 1, 1, 1, 64, 16, 256, 16, 32, 4, (4,), "f32", None, 0),
    # Llama-3-8B-shaped layer: 32 q / 8 kv heads, d=128, P=64, T=32K, batch 1, r=24, bf16.
    # A decode step runs 32 such layers (Llama-3-8B's depth), each with its own
    # buffers: 32 x 76 MB is far beyond the 256 MB last-level cache, so every
    # layer's pages come from HBM.
    "llama8b_32k": Workload("llama8b_32k", 2, 1, 8, 32, 128, 64, 32768, 64, 256, 24, (24,),
                            "bf16", 5.0e5, 4, layers=32),
    # Qwen3-32B-shaped layer: 64 q / 8 kv heads, d=128, P=64, T=128K, batch 4,
    # r uniform over {16, 24, 32}; a decode step runs 64 such layers.
    "qwen32b_128k": Workload("qwen32b_128k", 3, 4, 8, 64, 128, 64, 131072, 64, 512, 24,
                             (16, 24, 32), "bf16", 1.0e6, 4, layers=64),
    # Incremental decode: Llama-3-8B heads, batch 32, prefill 16K then 512 steps, r=24.
    "llama8b_incremental": Workload("llama8b_incremental", 4, 32, 8, 32, 128, 64, 16384, 64,
                                    256, 24, (24,), "bf16", 5.0e5, 4, decode_steps=512),
    # The paper's default configuration on Qwen3-8B heads (32 q / 8 kv, d=128,
    # 36 layers): pages of 32 tokens, (r_K, r_V) = (16, 14), a 32-token sink
    # and a dense region of the last completed page plus the partial page
    # (W = P), 16K context, batch 1.
    "qwen8b_paper_default": Workload("qwen8b_paper_default", 6, 1, 8, 32, 128, 32, 16384, 32, 32, 24,
                                     (16,), "bf16", 1.0e6, 4, layers=36, ranks_v=(14,)),
    # The 128K Qwen3-32B-shaped layer with each page's ranks chosen for 80%
    # reconstruction accuracy (relative Frobenius error 0.2), at most 32.
    "qwen32b_128k_adaptive": Workload("qwen32b_128k_adaptive", 7, 4, 8, 64, 128, 64, 131072, 64, 512, 24,
                                      (32,), "bf16", 1.0e6, 4, layers=64, rank_error=0.2),
    # The 128K Qwen3-32B-shaped layer with keys cached before RoPE: the same
    # page model without the rotation; attention rotates keys at access.
    "qwen32b_128k_prerope": Workload("qwen32b_128k_prerope", 8, 4, 8, 64, 128, 64, 131072, 64, 512, 24,
                                     (16, 24, 32), "bf16", 1.0e6, 4, layers=64, key_rope=True),
    # One GPU's share of the 128K Qwen3-32B-shaped layers under 8-way tensor
    # parallelism by KV head: 1 kv head with its 8 q heads, batch 4, otherwise
    # as qwen32b_128k; 64 layers of ~152 MB each, far beyond the 256 MB
    # last-level cache.
    "qwen32b_128k_tp8": Workload("qwen32b_128k_tp8", 11, 4, 1, 8, 128, 64, 131072, 64, 512, 24,
                                 (16, 24, 32), "bf16", 1.0e6, 4, layers=64),
    # INT4 factors: Qwen3-32B heads, batch 8, T=128K.
    "qwen32b_int4": Workload("qwen32b_int4", 5, 8, 8, 64, 128, 64, 131072, 64, 512, 24,
                             (16, 24, 32), "bf16", 1.0e6, 4, factor_dtype="int4"),
    # Global SVD baseline at the 128K Qwen3-32B-shaped layer: one basis per
    # (sequence, KV head) over the compressible region, its rank matched to the
    # whole-cache storage PuzzleKV reaches on the same layer (ranks U{16,24,32}
    # pages, ratio 0.5643).
    "qwen32b_128k_global": Workload("qwen32b_128k_global", 9, 4, 8, 64, 128, 64, 131072, 64, 512, 24,
                                    (16, 24, 32), "bf16", 1.0e6, 4, layers=64, global_rho=0.5643),
    # Global SVD against PuzzleKV at the paper's default configuration
    # (Qwen3-8B heads, P = 32, (r_K, r_V) = (16, 14), S = W = 32, 16K,
    # batch 1), the Global SVD rank matched to PuzzleKV's realized whole-cache
    # ratio, on sequences whose planted subspace changes every
    # segment_pages pages (the comparison sweeps several values).
    "qwen8b_global": Workload("qwen8b_global", 10, 1, 8, 32, 128, 32, 16384, 32, 32, 24,
                              (16,), "bf16", 1.0e6, 4, layers=36, ranks_v=(14,), segment_pages=16,
                              global_rho=-1.0),
}


def rng(seed: int, wid: int, tag: int, *keys: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [int(seed), int(wid), int(tag)] + [int(k) for k in keys])))


# --------------------------------------------------------------------------
# Storage rounding
# --------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Values rounded to bf16 and returned as float32 (exactly representable)."""
    return bf16_to_f32(bf16_bits(np.asarray(x, dtype=np.float32)))


def round_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)


# --------------------------------------------------------------------------
# Keys, values, queries, ranks
# --------------------------------------------------------------------------
@functools.lru_cache(maxsize=8)
def _rope_table(n: int, d: int, base: float):
    """cos and sin (n x d/2, float32) of the rotate-half RoPE angles t * base^(-2i/d)."""
    half = d // 2
    inv = base ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.arange(n, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def _rope(x: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half RoPE of the rows of x (n x d) at positions 0 .. n-1."""
    n, d = x.shape
    half = d // 2
    c, s = _rope_table(n, d, base)
    a = x[:, :half]
    b = x[:, half:]
    out = np.empty_like(x)
    out[:, :half] = a * c - b * s
    out[:, half:] = b * c + a * s
    return out


def _low_rank_pages(g: np.random.Generator, n_pages: int, P: int, d: int, r0: int, seg: int = 1):
    G = g.standard_normal((n_pages, P, r0), dtype=np.float32)
    if seg == 1:
        W = g.standard_normal((n_pages, r0, d), dtype=np.float32)
    else:
        run = n_pages if seg <= 0 else seg
        Ws = g.standard_normal((-(-n_pages // run), r0, d), dtype=np.float32)
        W = np.repeat(Ws, run, axis=0)[:n_pages]
    N = g.standard_normal((n_pages, P, d), dtype=np.float32)
    N *= np.float32(0.05)
    N += np.matmul(G, W)
    return N.reshape(n_pages * P, d)


def outlier_channels(wl: Workload, seed: int, layer: int, h: int) -> np.ndarray:
    if wl.outliers <= 0:
        return np.zeros(0, dtype=np.int64)
    return rng(seed, wl.wid, TAG_OUTLIER, layer, h).choice(wl.head_dim, wl.outliers,
                                                           replace=False)


def kv_head(wl: Workload, seed: int, layer: int, b: int, h: int, tokens: int | None = None):
    """K and V (tokens x d, float32 holding storage-rounded values) of one KV head."""
    T = wl.tokens + wl.decode_steps if tokens is None else int(tokens)
    P, d = wl.page, wl.head_dim
    n_pages = -(-T // P)
    K = _low_rank_pages(rng(seed, wl.wid, TAG_KEY, layer, b, h), n_pages, P, d, wl.r0, wl.segment_pages)
    V = _low_rank_pages(rng(seed, wl.wid, TAG_VALUE, layer, b, h), n_pages, P, d, wl.r0, wl.segment_pages)
    ch = outlier_channels(wl, seed, layer, h)
    if ch.size:
        K[:, ch] *= np.float32(10.0)
    if wl.rope_base is not None and not wl.key_rope:
        K = _rope(K, wl.rope_base)
    return round_storage(K[:T], wl.dtype), round_storage(V[:T], wl.dtype)


def kv_layer(wl: Workload, seed: int, layer: int, tokens: int | None = None, workers: int = 0):
    """K, V of a whole layer: (batch, kv_heads, tokens, d) float32. Heads are
    independent streams, drawn in parallel threads when workers > 1 (the
    result does not depend on the thread count)."""
    T = wl.tokens + wl.decode_steps if tokens is None else int(tokens)
    K = np.empty((wl.batch, wl.kv_heads, T, wl.head_dim), dtype=np.float32)
    V = np.empty_like(K)

    def one(bh):
        b, h = bh
        K[b, h], V[b, h] = kv_head(wl, seed, layer, b, h, T)

    heads = [(b, h) for b in range(wl.batch) for h in range(wl.kv_heads)]
    if workers and workers > 1:
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            list(ex.map(one, heads))
    else:
        for bh in heads:
            one(bh)
    return K, V


def queries(wl: Workload, seed: int, step: int = 0) -> np.ndarray:
    """Decode queries (batch, q_heads, d), i.i.d. N(0, 1/d), storage-rounded."""
    out = np.empty((wl.batch, wl.q_heads, wl.head_dim), dtype=np.float32)
    for b in range(wl.batch):
        g = rng(seed, wl.wid, TAG_QUERY, step, b)
        out[b] = g.standard_normal((wl.q_heads, wl.head_dim)) / np.sqrt(wl.head_dim)
    return round_storage(out, wl.dtype)


def page_ranks(wl: Workload, seed: int, layer: int, n_pages: int, which: str = "k") -> np.ndarray:
    """Rank of every logical page, (batch, kv_heads, n_pages) uint8; uniform over
    wl.ranks when it holds several choices. which="v" gives the value ranks,
    which are the key ranks unless the workload sets ranks_v."""
    out = np.empty((wl.batch, wl.kv_heads, n_pages), dtype=np.uint8)
    if which == "v" and wl.ranks_v:
        assert len(wl.ranks_v) == 1, "value ranks: one fixed choice"
        out[:] = wl.ranks_v[0]
        return out
    choices = np.asarray(wl.ranks, dtype=np.uint8)
    for b in range(wl.batch):
        for h in range(wl.kv_heads):
            if len(choices) == 1:
                out[b, h] = choices[0]
            else:
                out[b, h] = rng(seed, wl.wid, TAG_RANK, layer, b, h).choice(choices, n_pages)
    return out


def factor_page(wl: Workload, seed: int, layer: int, b: int, h: int, j: int, r_k: int,
                r_v: int):
    """Factor pairs drawn directly (not from a decomposition), storage-rounded:
    L (P x r) ~ N(0, 1/P), R (r x d) ~ N(0, r0 P / r), so L R has the
    per-element scale of the planted pages. Used where a test needs a full-size
    cache whose factors must not come from the GPU decomposition."""
    g = rng(seed, wl.wid, TAG_FACTOR, layer, b, h, j)
    P, d = wl.page, wl.head_dim
    out = []
    for r in (r_k, r_v):
        L = g.standard_normal((P, r)) / np.sqrt(P)
        R = g.standard_normal((r, d)) * np.sqrt(wl.r0 * P / r)
        out += [round_storage(L, wl.dtype), round_storage(R, wl.dtype)]
    return tuple(out)


def decode_kv(wl: Workload, seed: int, layer: int, pos: int):
    """K and V rows (batch, kv_heads, d) for the token at position pos, drawn
    from the same page model as the prefill pages but from their own stream
    (one stream per decode position), with the key outliers and RoPE at pos
    (no RoPE for a workload that hands keys over before it)."""
    P, d = wl.page, wl.head_dim
    K = np.empty((wl.batch, wl.kv_heads, d), dtype=np.float32)
    V = np.empty_like(K)
    for b in range(wl.batch):
        g = rng(seed, wl.wid, TAG_TOKEN, layer, pos, b)
        for h in range(wl.kv_heads):
            for X in (K, V):
                x = g.standard_normal(wl.r0) @ g.standard_normal((wl.r0, d)) + 0.05 * g.standard_normal(d)
                X[b, h] = x
            ch = outlier_channels(wl, seed, layer, h)
            if ch.size:
                K[b, h, ch] *= 10.0
    if wl.rope_base is not None and not wl.key_rope:
        half = d // 2
        inv = wl.rope_base ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
        c, s = np.cos(pos * inv), np.sin(pos * inv)
        a, bb = K[..., :half].copy(), K[..., half:].copy()
        K[..., :half] = a * c - bb * s
        K[..., half:] = bb * c + a * s
    return round_storage(K, wl.dtype), round_storage(V, wl.dtype)


def global_factors(wl: Workload, seed: int, layer: int, b: int, h: int, n_rows: int, r: int):
    """Global SVD factors drawn directly (not from a decomposition),
    storage-rounded: coefficients A (n_rows x r) ~ N(0, r0 / r * d) per entry
    and a basis B (r x d) ~ N(0, 1/d), for K then V, so that A B has the
    per-element scale of the planted pages. Used where a cache of the right
    shape is needed without the GPU decomposition."""
    g = rng(seed, wl.wid, TAG_GLOBAL, layer, b, h)
    d = wl.head_dim
    out = []
    for _ in range(2):
        A = g.standard_normal((n_rows, r)) * np.sqrt(wl.r0 * d / r)
        B = g.standard_normal((r, d)) / np.sqrt(d)
        out += [round_storage(A, wl.dtype), round_storage(B, wl.dtype)]
    return tuple(out)
