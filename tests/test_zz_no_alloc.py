"""pkv_mixed_decode_attention_noalloc (no workspace, static scratch) against
pkv_mixed_decode_attention with a caller workspace, through the C ABI: two
calls in a row on different caches, the second with a smaller input (fewer
sequences, fewer KV heads, shorter sequences), each within the attention
parity bar of the workspace call's output and of the oracle. The calls run
alone on the GPU (the scratch is shared by every call on a device)."""
import ctypes

import numpy as np
import pytest

import oracle
import synth
from helpers import MAX_ABS, MEAN_REL, build_head_pages, errors, import_head, oracle_head

pytestmark = pytest.mark.gpu


def _case(B, Hkv, g, d, P, seq_lens, S, W, r, wid):
    import paper_2608_23843_amd as pk
    Tmax = max(seq_lens)
    max_pages = -(-Tmax // P)
    wl = synth.Workload("noalloc", wid, B, Hkv, Hkv * g, d, P, Tmax, S, W, 8, (r,), "bf16", None, 0)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, d, P, max_pages, r, S, W, "bf16", "bf16")
    heads = {}
    for b, T in enumerate(seq_lens):
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, b, h, max_pages * P)
            pages = build_head_pages(K.astype(np.float64), V.astype(np.float64), T, P, S, W, r, "bf16")
            import_head(cache, 0, b, h, pages)
            heads[(b, h)] = oracle_head(T, P, d, pages)
    return cache, wl, heads


def test_noalloc_matches_workspace_call_twice():
    import torch
    import paper_2608_23843_amd as pk
    cases = [(4, 8, 8, 128, 64, [64 * 90 + 5, 64 * 70, 64 * 88, 3000], 64, 256, 24, 98),
             (2, 4, 4, 128, 32, [1500, 900], 32, 32, 16, 99)]
    for (B, Hkv, g, d, P, seq, S, W, r, wid) in cases:
        cache, wl, heads = _case(B, Hkv, g, d, P, seq, S, W, r, wid)
        q = synth.queries(wl, 0)
        qt = torch.from_numpy(q).to(device="cuda", dtype=torch.bfloat16).contiguous()
        ref_out, ref_lse = cache.attention(0, qt, seq)
        out = torch.full((B, Hkv * g, d), float("nan"), dtype=torch.float32, device="cuda")
        lse = torch.full((B, Hkv * g), float("nan"), dtype=torch.float32, device="cuda")
        lib = pk.load_library()
        seq_np = np.ascontiguousarray(seq, dtype=np.int32)
        st = lib.pkv_mixed_decode_attention_noalloc(ctypes.byref(cache.c), 0, ctypes.c_void_p(qt.data_ptr()),
                                                    seq_np.ctypes.data_as(ctypes.c_void_p),
                                                    ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(lse.data_ptr()),
                                                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0, lib.pkv_last_error()
        torch.cuda.synchronize()
        assert cache.device_status() == 0
        o, ro = out.cpu().numpy().astype(np.float64), ref_out.cpu().numpy().astype(np.float64)
        ma, mr = errors(o, ro)
        assert ma <= MAX_ABS and mr <= MEAN_REL, (B, ma, mr)
        assert float((lse - ref_lse).abs().max()) <= 1e-4
        ref = np.zeros_like(o)
        for (b, h), head in heads.items():
            ref[b, h * g:(h + 1) * g], _ = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ma, mr = errors(o, ref)
        assert ma <= MAX_ABS and mr <= MEAN_REL, (B, ma, mr)


def test_noalloc_refuses_too_many_heads():
    """batch * n_kv_heads above PKV_NOALLOC_MAX_HEADS: PKV_E_WORKSPACE before any launch."""
    import torch
    import paper_2608_23843_amd as pk
    cache = pk.PuzzleKVCache(1, 129, 16, 16, 64, 16, 2, 4, 0, 0, "bf16", "bf16")
    q = torch.zeros((129, 16, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((129, 16, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(pk.PuzzleKVError, match="PKV_E_WORKSPACE"):
        cache.attention_noalloc(0, q, [16] * 129, out)
