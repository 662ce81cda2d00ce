"""PuzzleKV hot path on MI355X: Python binding of libpuzzlekv.so.

Argument marshalling only. Every step of the path (page planning on the host,
and on the device the decompositions, the append, the import / export copies
and the mixed-page attention) runs inside the C ABI declared in
include/puzzlekv.h. PyTorch supplies device memory and the current stream.
If the library is not built the import fails; there is no fallback.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import _lib
from ._lib import (PKV_BF16, PKV_DENSE, PKV_EMPTY, PKV_F32, PKV_FACTOR, PKV_GLOBAL, PKV_INT4, PKV_OP_ATTENTION,
                   PKV_OP_COMPRESS, PKV_OP_GLOBAL_ATTENTION, PKV_OP_GLOBAL_PREFILL, PKV_OP_IMPORT, PKV_OP_PREFILL,
                   PuzzleKVError, check)

__all__ = ["PuzzleKVCache", "GlobalSVD", "plan_pages", "eligible_pages", "global_rank", "load_library",
           "PuzzleKVError", "PKV_EMPTY", "PKV_DENSE", "PKV_FACTOR", "PKV_GLOBAL", "PKV_F32", "PKV_BF16", "PKV_INT4"]

_DTYPES = {"f32": PKV_F32, "fp32": PKV_F32, "float32": PKV_F32, "bf16": PKV_BF16, "bfloat16": PKV_BF16,
           "int4": PKV_INT4}


def load_library():
    return _lib.load()


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def plan_pages(T: int, P: int, S: int, W: int, n: int | None = None) -> np.ndarray:
    """pkv_plan_pages: kind of each logical page (0 empty, 1 dense, 2 factor)."""
    lib = _lib.load()
    if n is None:
        n = -(-T // P) if T > 0 else 0
    kind = np.zeros(max(n, 1), dtype=np.uint8)
    npg = ctypes.c_int64(0)
    check(lib.pkv_plan_pages(T, P, S, W, _np_ptr(kind), n, ctypes.byref(npg)), "pkv_plan_pages")
    return kind[:n]


def eligible_pages(T_prev: int, T_new: int, P: int, S: int, W: int) -> np.ndarray:
    """pkv_eligible_pages: pages that become factorized when T_prev grows to T_new."""
    lib = _lib.load()
    cap = max(1, -(-T_new // P))
    out = np.zeros(cap, dtype=np.int32)
    cnt = ctypes.c_int64(0)
    check(lib.pkv_eligible_pages(T_prev, T_new, P, S, W, _np_ptr(out), cap, ctypes.byref(cnt)),
          "pkv_eligible_pages")
    return out[:cnt.value].copy()


def global_rank(T: int, P: int, S: int, W: int, d: int, rho: float) -> int:
    """pkv_global_rank: Global SVD rank whose whole-head storage (dense tokens
    included) fits rho times the raw cache."""
    r = int(_lib.load().pkv_global_rank(T, P, S, W, d, float(rho)))
    if r < 0:
        raise ValueError("pkv_global_rank: invalid argument")
    return r


def bandwidth_probe(src, dst, mode: int, reps: int = 5, blocks: int = 2048, threads: int = 256, stream=None) -> float:
    """pkv_bandwidth_probe over device tensors src (and dst): GB/s of a plain
    streaming read (mode 0 grid-stride, 2 in 64 KB chunks per workgroup) or
    copy (modes 1 and 3)."""
    import torch
    lib = _lib.load()
    out = ctypes.c_double(0.0)
    check(lib.pkv_bandwidth_probe(src.data_ptr(), dst.data_ptr(), src.numel() * src.element_size(), mode, reps,
                                  blocks, threads, ctypes.byref(out), _stream_handle(torch, stream)),
          "pkv_bandwidth_probe")
    return float(out.value)


def _stream_handle(torch, stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _i32(x, n=None):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32).reshape(-1))
    if n is not None and a.size != n:
        raise ValueError("expected %d entries, got %d" % (n, a.size))
    return a


class PuzzleKVCache:
    """A hybrid paged KV cache in device memory (pools allocated with torch).

    Geometry follows pkv_cache: n_layers, batch, n_kv_heads, n_q_heads, head_dim
    (d), page_size (P), max_pages per (layer, sequence, KV head), max_rank,
    sink_tokens, window_tokens, dense and factor dtypes ("bf16" or "f32")."""

    def __init__(self, n_layers, batch, n_kv_heads, n_q_heads, head_dim, page_size, max_pages,
                 max_rank, sink_tokens, window_tokens, dense_dtype="bf16", factor_dtype="bf16",
                 device="cuda", adaptive_rank_error=0.0, key_rope_base=0.0):
        import torch
        self.torch = torch
        self.lib = _lib.load()
        c = _lib.PkvCache()
        c.n_layers, c.batch, c.n_kv_heads, c.n_q_heads = n_layers, batch, n_kv_heads, n_q_heads
        c.head_dim, c.page_size, c.max_pages, c.max_rank = head_dim, page_size, max_pages, max_rank
        c.sink_tokens, c.window_tokens = sink_tokens, window_tokens
        c.dense_dtype, c.factor_dtype = _DTYPES[dense_dtype], _DTYPES[factor_dtype]
        c.adaptive_rank_error = float(adaptive_rank_error)   # > 0: rank requests of 0 are chosen per page
        c.key_rope_base = float(key_rope_base)               # > 0: keys cached before RoPE
        self.c = c
        self.device = torch.device(device)
        lib = self.lib
        sizes = [lib.pkv_dense_pool_bytes(c), lib.pkv_factor_pool_bytes(c), lib.pkv_page_table_bytes(c)]
        if 0 in sizes:
            # report the geometry error the library found
            check(lib.pkv_cache_check(ctypes.byref(c)), "PuzzleKVCache")
        self.dense_pool = torch.empty(sizes[0], dtype=torch.uint8, device=self.device)
        self.factor_pool = torch.empty(sizes[1], dtype=torch.uint8, device=self.device)
        self.table = torch.empty(sizes[2], dtype=torch.uint8, device=self.device)
        c.dense_pool = self.dense_pool.data_ptr()
        c.factor_pool = self.factor_pool.data_ptr()
        c.page_table = self.table.data_ptr()
        check(lib.pkv_cache_check(ctypes.byref(c)), "PuzzleKVCache")
        self.qdtype = torch.bfloat16 if c.dense_dtype == PKV_BF16 else torch.float32
        self.fdtype = {PKV_BF16: torch.bfloat16, PKV_F32: torch.float32, PKV_INT4: torch.uint8}[c.factor_dtype]
        self.reset()

    # ---- geometry ----------------------------------------------------------
    @property
    def group(self) -> int:
        return self.c.n_q_heads // self.c.n_kv_heads

    def factor_page_bytes(self, rank_k: int, rank_v: int) -> int:
        return int(self.lib.pkv_factor_page_bytes(ctypes.byref(self.c), rank_k, rank_v))

    def workspace_bytes(self, op: int, n: int) -> int:
        return int(self.lib.pkv_workspace_bytes(ctypes.byref(self.c), op, n))

    def workspace(self, op: int, n: int):
        """A zero-filled workspace for `op` (see pkv_workspace_bytes)."""
        nb = self.workspace_bytes(op, n)
        return self.torch.zeros(max(nb, 1), dtype=self.torch.uint8, device=self.device)

    def page_table(self, layer: int):
        """Page-table entries of one layer as a (batch, n_kv_heads, max_pages, 8) uint8 tensor."""
        c = self.c
        per = c.batch * c.n_kv_heads * c.max_pages * 8
        return self.table[layer * per:(layer + 1) * per].view(c.batch, c.n_kv_heads, c.max_pages, 8)

    def page_table_host(self, layer: int):
        """(slot int32, kind, rank_k, rank_v) numpy arrays of one layer."""
        t = self.page_table(layer).cpu().numpy()
        slot = t[..., :4].copy().view(np.int32)[..., 0]
        return slot, t[..., 4].copy(), t[..., 5].copy(), t[..., 6].copy()

    # ---- operations --------------------------------------------------------
    def reset(self, layer: int = -1, stream=None):
        check(self.lib.pkv_cache_reset(ctypes.byref(self.c), layer, _stream_handle(self.torch, stream)),
              "pkv_cache_reset")

    def prefill(self, layer, k, v, seq_len, rank_k=None, rank_v=None, default_rank=None, stream=None):
        """k, v: device (batch, n_kv_heads, src_tokens, d). rank_k/rank_v: device uint8
        (batch, n_kv_heads, max_pages) or None with default_rank=(r_k, r_v)."""
        torch = self.torch
        assert k.is_contiguous() and v.is_contiguous() and k.dtype == self.qdtype
        seq = _i32(seq_len, self.c.batch)
        if rank_k is None:
            rk, rv = default_rank
            pk = pv = None
        else:
            rk = rv = 0
            for rt in (rank_k, rank_v):
                assert rt.dtype == torch.uint8 and rt.is_contiguous() and rt.is_cuda
                assert rt.numel() == self.c.batch * self.c.n_kv_heads * self.c.max_pages
            pk, pv = rank_k.data_ptr(), rank_v.data_ptr()
        check(self.lib.pkv_prefill(ctypes.byref(self.c), layer, k.data_ptr(), v.data_ptr(), k.shape[2],
                                   _np_ptr(seq), pk, pv, rk, rv, None, 0,
                                   _stream_handle(torch, stream)), "pkv_prefill")

    def append(self, layer, k_new, v_new, pos, stream=None):
        """k_new, v_new: device (batch, n_kv_heads, d); pos: host ints (token index per sequence)."""
        assert k_new.is_contiguous() and v_new.is_contiguous() and k_new.dtype == self.qdtype
        p = _i32(pos, self.c.batch)
        check(self.lib.pkv_append_kv(ctypes.byref(self.c), layer, k_new.data_ptr(), v_new.data_ptr(),
                                     _np_ptr(p), _stream_handle(self.torch, stream)), "pkv_append_kv")

    def compress_pages(self, layer, b, h, page, rank_k, rank_v, stream=None, workspace=True):
        """workspace: True (the cache's own, grown as needed: every page in one
        launch), a device uint8 tensor, or None (launches of 96 pages)."""
        b, h, page = _i32(b), _i32(h), _i32(page)
        n = b.size
        rk = np.ascontiguousarray(np.broadcast_to(np.asarray(rank_k, dtype=np.uint8), (n,)))
        rv = np.ascontiguousarray(np.broadcast_to(np.asarray(rank_v, dtype=np.uint8), (n,)))
        if workspace is True:
            need = self.workspace_bytes(PKV_OP_COMPRESS, n)
            ws = getattr(self, "_compress_ws", None)
            if ws is None or ws.numel() < need:
                ws = self._compress_ws = self.torch.empty(max(need, 256), dtype=self.torch.uint8,
                                                          device=self.device)
            workspace = ws
        ws_ptr, ws_n = (None, 0) if workspace is None else (workspace.data_ptr(), workspace.numel())
        check(self.lib.pkv_compress_pages(ctypes.byref(self.c), layer, n, _np_ptr(b), _np_ptr(h),
                                          _np_ptr(page), _np_ptr(rk), _np_ptr(rv), ws_ptr, ws_n,
                                          _stream_handle(self.torch, stream)), "pkv_compress_pages")

    def attention(self, layer, q, seq_len, out=None, lse=None, workspace=None, stream=None):
        """q: device (batch, n_q_heads, d) in the dense dtype. Returns (out, lse) fp32."""
        torch = self.torch
        c = self.c
        assert q.is_contiguous() and q.dtype == self.qdtype and tuple(q.shape) == (c.batch, c.n_q_heads, c.head_dim)
        seq = _i32(seq_len, c.batch)
        if out is None:
            out = torch.empty((c.batch, c.n_q_heads, c.head_dim), dtype=torch.float32, device=self.device)
        if lse is None:
            lse = torch.empty((c.batch, c.n_q_heads), dtype=torch.float32, device=self.device)
        need = self.workspace_bytes(PKV_OP_ATTENTION, int(seq.max()) if seq.size else 0)
        if workspace is None or workspace.numel() < need:
            # zero-filled on first use (the merge counters live in it)
            workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=self.device)
        check(self.lib.pkv_mixed_decode_attention(ctypes.byref(c), layer, q.data_ptr(), _np_ptr(seq),
                                                  out.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
                                                  workspace.numel(), _stream_handle(torch, stream)),
              "pkv_mixed_decode_attention")
        return out, lse

    def attention_noalloc(self, layer, q, seq_len, out, lse=None, stream=None):
        """pkv_mixed_decode_attention_noalloc: the same attention into caller
        buffers out (batch, n_q_heads, d) fp32 and lse (batch, n_q_heads) fp32
        or None, with the library's static scratch instead of a workspace."""
        c = self.c
        assert q.is_contiguous() and q.dtype == self.qdtype and tuple(q.shape) == (c.batch, c.n_q_heads, c.head_dim)
        assert out.is_contiguous() and out.dtype == self.torch.float32 and out.numel() == c.batch * c.n_q_heads * c.head_dim
        seq = _i32(seq_len, c.batch)
        check(self.lib.pkv_mixed_decode_attention_noalloc(ctypes.byref(c), layer, q.data_ptr(), _np_ptr(seq),
                                                          out.data_ptr(), None if lse is None else lse.data_ptr(),
                                                          _stream_handle(self.torch, stream)),
              "pkv_mixed_decode_attention_noalloc")
        return out, lse

    def import_pages(self, layer, b, h, page, kind, rank_k, rank_v, src, src_offset, stream=None):
        """src: device 1-D tensor (dense dtype for dense pages, factor dtype for factors)."""
        b, h, page = _i32(b), _i32(h), _i32(page)
        n = b.size
        kind = np.ascontiguousarray(np.asarray(kind, dtype=np.uint8).reshape(-1))
        rk = np.ascontiguousarray(np.asarray(rank_k, dtype=np.uint8).reshape(-1))
        rv = np.ascontiguousarray(np.asarray(rank_v, dtype=np.uint8).reshape(-1))
        off = np.ascontiguousarray(np.asarray(src_offset, dtype=np.int64).reshape(-1))
        assert src.is_contiguous() and kind.size == n and rk.size == n and rv.size == n and off.size == n
        check(self.lib.pkv_import_pages(ctypes.byref(self.c), layer, n, _np_ptr(b), _np_ptr(h),
                                        _np_ptr(page), _np_ptr(kind), _np_ptr(rk), _np_ptr(rv),
                                        src.data_ptr(), _np_ptr(off), None, 0,
                                        _stream_handle(self.torch, stream)), "pkv_import_pages")

    def int4_blob_bytes(self, rank_k: int, rank_v: int) -> int:
        """Size of the canonical INT4 page blob (pkv_int4_blob_bytes)."""
        return int(self.lib.pkv_int4_blob_bytes(ctypes.byref(self.c), rank_k, rank_v))

    def export_int4_pages(self, layer, b, h, page, stream=None):
        """Returns a device uint8 tensor (n, blob bytes at max_rank) of canonical INT4 blobs."""
        torch = self.torch
        b, h, page = _i32(b), _i32(h), _i32(page)
        n = b.size
        blk = self.int4_blob_bytes(self.c.max_rank, self.c.max_rank)
        dst = torch.zeros((max(n, 1), blk), dtype=torch.uint8, device=self.device)
        check(self.lib.pkv_export_int4_pages(ctypes.byref(self.c), layer, n, _np_ptr(b), _np_ptr(h),
                                             _np_ptr(page), dst.data_ptr(), _stream_handle(torch, stream)),
              "pkv_export_int4_pages")
        return dst[:n]

    def export_block_elems(self) -> int:
        return int(self.lib.pkv_export_block_elems(ctypes.byref(self.c)))

    def export_pages(self, layer, b, h, page, stream=None):
        """Returns a device fp32 tensor (n, export_block_elems) of logical page blocks."""
        torch = self.torch
        b, h, page = _i32(b), _i32(h), _i32(page)
        n = b.size
        blk = self.export_block_elems()
        dst = torch.empty((max(n, 1), blk), dtype=torch.float32, device=self.device)
        check(self.lib.pkv_export_pages(ctypes.byref(self.c), layer, n, _np_ptr(b), _np_ptr(h),
                                        _np_ptr(page), dst.data_ptr(), None, 0,
                                        _stream_handle(torch, stream)), "pkv_export_pages")
        return dst[:n]

    def compress_sweeps(self, stream=None) -> int:
        """Jacobi sweeps executed by decompositions on this device since the last call."""
        n = ctypes.c_uint64(0)
        check(self.lib.pkv_compress_sweeps(_stream_handle(self.torch, stream), ctypes.byref(n)),
              "pkv_compress_sweeps")
        return int(n.value)

    def footprint(self, seq_len, layer: int = -1, stream=None) -> dict:
        """Live KV footprint (pkv_cache_bytes) of `layer` (-1: every layer) for the
        sequences' lengths seq_len, as a dict of byte and page counts."""
        seq = _i32(seq_len, self.c.batch)
        f = _lib.PkvFootprint()
        check(self.lib.pkv_cache_bytes(ctypes.byref(self.c), layer, seq.ctypes.data, ctypes.byref(f),
                                       _stream_handle(self.torch, stream)), "pkv_cache_bytes")
        return {name: int(getattr(f, name)) for name, _ in f._fields_}

    def device_status(self, stream=None) -> int:
        bits = ctypes.c_uint32(0)
        check(self.lib.pkv_device_status(_stream_handle(self.torch, stream), ctypes.byref(bits)),
              "pkv_device_status")
        return int(bits.value)


class GlobalSVD:
    """Global SVD factors beside a PuzzleKVCache (pkv_global): one rank-r basis
    per (layer, sequence, KV head) and K/V, shared by the tokens of the
    compressible region; the cache's dense pool and page table hold the dense
    pages. Buffers are allocated with torch."""

    def __init__(self, cache: PuzzleKVCache, rank: int, max_tokens: int):
        torch = cache.torch
        self.cache, self.torch, self.lib = cache, torch, cache.lib
        g = _lib.PkvGlobal()
        g.rank, g.max_tokens = int(rank), int(max_tokens)
        nb = int(self.lib.pkv_global_basis_bytes(ctypes.byref(cache.c), ctypes.byref(g)))
        nc = int(self.lib.pkv_global_coef_bytes(ctypes.byref(cache.c), ctypes.byref(g)))
        if nb == 0 or nc == 0:
            raise PuzzleKVError(_lib.PKV_E_ARG, "GlobalSVD", "invalid geometry for Global SVD (rank %d, "
                                "max_tokens %d)" % (rank, max_tokens))
        self.basis = torch.zeros(nb, dtype=torch.uint8, device=cache.device)
        self.coef = torch.zeros(nc, dtype=torch.uint8, device=cache.device)
        g.basis, g.coef = self.basis.data_ptr(), self.coef.data_ptr()
        self.g = g

    def workspace(self, op: int, n: int):
        nb = self.cache.workspace_bytes(op, n)
        return self.torch.zeros(max(nb, 1), dtype=self.torch.uint8, device=self.cache.device)

    def prefill(self, layer, k, v, seq_len, workspace=None, stream=None):
        """k, v: device (batch, n_kv_heads, src_tokens, d) bf16."""
        c = self.cache
        assert k.is_contiguous() and v.is_contiguous() and k.dtype == c.qdtype
        seq = _i32(seq_len, c.c.batch)
        if workspace is None:
            workspace = self.workspace(PKV_OP_GLOBAL_PREFILL, int(seq.max()) if seq.size else 0)
        check(self.lib.pkv_global_prefill(ctypes.byref(c.c), ctypes.byref(self.g), layer, k.data_ptr(),
                                          v.data_ptr(), k.shape[2], _np_ptr(seq), workspace.data_ptr(),
                                          workspace.numel(), _stream_handle(self.torch, stream)),
              "pkv_global_prefill")

    def attention(self, layer, q, seq_len, out=None, lse=None, workspace=None, stream=None):
        torch, c = self.torch, self.cache.c
        assert q.is_contiguous() and q.dtype == self.cache.qdtype
        seq = _i32(seq_len, c.batch)
        if out is None:
            out = torch.empty((c.batch, c.n_q_heads, c.head_dim), dtype=torch.float32, device=self.cache.device)
        if lse is None:
            lse = torch.empty((c.batch, c.n_q_heads), dtype=torch.float32, device=self.cache.device)
        need = self.cache.workspace_bytes(PKV_OP_GLOBAL_ATTENTION, int(seq.max()) if seq.size else 0)
        if workspace is None or workspace.numel() < need:
            workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=self.cache.device)
        check(self.lib.pkv_global_attention(ctypes.byref(c), ctypes.byref(self.g), layer, q.data_ptr(), _np_ptr(seq),
                                            out.data_ptr(), lse.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                            _stream_handle(torch, stream)), "pkv_global_attention")
        return out, lse

    def export(self, layer, b, h, n_rows, stream=None):
        """(B_K, B_V, A_K, A_V) of one head as device fp32: (r, d), (r, d), (n_rows, r), (n_rows, r)."""
        torch, c, r = self.torch, self.cache.c, self.g.rank
        bk = torch.empty((r, c.head_dim), dtype=torch.float32, device=self.cache.device)
        bv = torch.empty_like(bk)
        ak = torch.empty((max(n_rows, 1), r), dtype=torch.float32, device=self.cache.device)
        av = torch.empty_like(ak)
        check(self.lib.pkv_global_export(ctypes.byref(c), ctypes.byref(self.g), layer, b, h, n_rows, bk.data_ptr(),
                                         bv.data_ptr(), ak.data_ptr(), av.data_ptr(), _stream_handle(torch, stream)),
              "pkv_global_export")
        return bk, bv, ak[:n_rows], av[:n_rows]
