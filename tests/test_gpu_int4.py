"""GPU parity of the INT4 factor pages (Section 4.3 "Quantization
Compatibility"), through the C ABI.

* Attention: factor pages are the oracle's Eq. (2) factors, balanced and
  quantized by the oracle (oracle/int4.py), packed into the canonical INT4
  blob and imported; the oracle attends over the same dequantized factors.
  Bar: max-abs <= 1e-2, normwise mean-relative <= 1e-3.
* Layout: exporting the imported pages returns the blobs bit for bit, and the
  dequantized export equals code x scale exactly.
* Compression: the GPU's INT4 pages are compared with the oracle quantizer
  applied to the GPU's own fp32 factors of the same pages (a cache with fp32
  factors, same kernel): scales agree to within one fp16 step (the two sides
  balance with slightly different sigma), codes agree except where the
  quotient x / scale lies within 1e-3 of a rounding boundary.
* End to end: GPU compression then GPU attention against the oracle on the
  GPU's own dequantized factors."""
import numpy as np
import pytest

import oracle
import synth
from oracle import int4 as q4
from helpers import MAX_ABS, MEAN_REL, errors

pytestmark = pytest.mark.gpu

P, D = 64, 128


def _wl(B, Hkv, g, T, S, W, seed_wid=95):
    return synth.Workload("int4case", seed_wid, B, Hkv, Hkv * g, D, P, T, S, W, 24, (16, 24, 32), "bf16",
                          1e6, 4)


def _bf16(x):
    return synth.round_storage(np.asarray(x, dtype=np.float32), "bf16").astype(np.float64)


def _blob(enc_k, enc_v):
    """Canonical blob of one page from the oracle encodings of K and V."""
    parts = [enc_k["L_codes"], enc_k["R_codes"], enc_v["L_codes"], enc_v["R_codes"]]
    codes = np.concatenate([np.asarray(c, dtype=np.int8).reshape(-1) for c in parts]).view(np.uint8)
    sc = [enc_k["L_scales"], enc_k["R_scales"], enc_v["L_scales"], enc_v["R_scales"]]
    scales = np.concatenate([np.asarray(s, dtype=np.float16).reshape(-1) for s in sc]).view(np.uint8)
    return np.concatenate([codes, scales])


def _encode_head(K, V, T, S, W, rank_of):
    """Logical pages of one head: dense pages as stored (bf16), factor pages as
    the oracle's INT4 encoding of its own Eq. (2) factors."""
    n = -(-T // P)
    kind = oracle.plan_pages(T, P, S, W, n)
    pages, blobs = [], {}
    for j in range(n):
        rows = min(P, T - j * P)
        Kp = np.zeros((P, D)); Vp = np.zeros((P, D))
        Kp[:rows] = K[j * P:j * P + rows]
        Vp[:rows] = V[j * P:j * P + rows]
        if kind[j] == oracle.FACTOR:
            rk, rv = rank_of(j)
            Lk, Rk, sk, _ = oracle.truncated_factors(Kp, rk)
            Lv, Rv, sv, _ = oracle.truncated_factors(Vp, rv)
            ek, ev = q4.encode_page("K", Lk, Rk, sk), q4.encode_page("V", Lv, Rv, sv)
            pages.append(("factor", ek["L_deq"], ek["R_deq"], ev["L_deq"], ev["R_deq"]))
            blobs[j] = _blob(ek, ev)
        else:
            pages.append(("dense", Kp, Vp))
    return pages, blobs


def _import(cache, b, h, pages, blobs):
    import torch
    dense = [j for j, pg in enumerate(pages) if pg[0] == "dense"]
    if dense:
        src = torch.from_numpy(np.concatenate([np.concatenate([pages[j][1].reshape(-1), pages[j][2].reshape(-1)])
                                               for j in dense]).astype(np.float32)).to("cuda", torch.bfloat16)
        offs = [i * 2 * P * D for i in range(len(dense))]
        cache.import_pages(0, [b] * len(dense), [h] * len(dense), dense, [oracle.DENSE] * len(dense),
                           [0] * len(dense), [0] * len(dense), src, offs)
    fac = sorted(blobs)
    if fac:
        offs, pos = [], 0
        for j in fac:
            offs.append(pos)
            pos += blobs[j].size
        src = torch.from_numpy(np.concatenate([blobs[j] for j in fac])).to("cuda")
        rk = [pages[j][1].shape[1] for j in fac]
        rv = [pages[j][3].shape[1] for j in fac]
        cache.import_pages(0, [b] * len(fac), [h] * len(fac), fac, [oracle.FACTOR] * len(fac), rk, rv, src, offs)


def _attend(cache, wl, seq_lens, heads, g, seed=0):
    import torch
    q = synth.queries(wl, seed)
    qt = torch.from_numpy(q).to(device="cuda", dtype=torch.bfloat16).contiguous()
    out, lse = cache.attention(0, qt, seq_lens)
    torch.cuda.synchronize()
    assert cache.device_status() == 0
    out = out.cpu().numpy().astype(np.float64)
    ref = np.zeros_like(out)
    for (b, h), head in heads.items():
        o, _ = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
        ref[b, h * g:(h + 1) * g] = o
    return out, ref


def test_int4_storage_size():
    """5,344 bytes per page pair at ranks 24/24 (16.3% of the 32 KB dense pair)."""
    import paper_2608_23843_amd as pk
    cache = pk.PuzzleKVCache(1, 1, 1, 8, D, P, 4, 32, 64, 64, "bf16", "int4")
    assert cache.factor_page_bytes(24, 24) == 5344
    # keys: A_K codes + scales, B_K scales + codes; values: B_V codes + scales, A_V scales + codes
    assert cache.factor_page_bytes(16, 32) == (16 * 32 + 16 * 4 + 256 + 16 * 64) + (32 * 64 + 256 + 128 + 32 * 32)
    # the canonical blob: int8 codes of the four factors, then the oracle's scale counts in fp16
    assert cache.int4_blob_bytes(24, 24) == 2 * (64 * 24 + 24 * 128) + 2 * (2 * 24 + 128 + 64 + 128)


@pytest.mark.parametrize("seq_lens,ranks", [([64 * 40 + 17, 64 * 33], None), ([64 * 12, 0, 100], (16, 24))])
def test_int4_attention_matches_oracle(seq_lens, ranks):
    import paper_2608_23843_amd as pk
    B, Hkv, g, S, W = len(seq_lens), 2, 8, 64, 128
    Tmax = max(seq_lens)
    wl = _wl(B, Hkv, g, Tmax, S, W)
    max_pages = -(-Tmax // P)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "int4")
    rng = np.random.default_rng(7)
    heads = {}
    for b, T in enumerate(seq_lens):
        if T == 0:
            continue
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, b, h, max_pages * P)
            K, V = _bf16(K), _bf16(V)
            rks = {j: (ranks or tuple(int(x) for x in rng.choice([16, 17, 24, 32], 2))) for j in range(max_pages)}
            pages, blobs = _encode_head(K, V, T, S, W, lambda j: rks[j])
            _import(cache, b, h, pages, blobs)
            heads[(b, h)] = oracle.HeadCache(T, P, D, pages)
            # the layout round trip: export returns the imported blobs, and the
            # dequantized export is code x scale
            fac = sorted(blobs)
            if fac:
                got = cache.export_int4_pages(0, [b] * len(fac), [h] * len(fac), fac).cpu().numpy()
                for i, j in enumerate(fac):
                    assert np.array_equal(got[i, :blobs[j].size], blobs[j]), (b, h, j)
                blk = cache.export_pages(0, [b] * len(fac), [h] * len(fac), fac).cpu().numpy()
                R = 32
                for i, j in enumerate(fac):
                    pg = pages[j]
                    rk, rv = pg[1].shape[1], pg[3].shape[1]
                    o = blk[i]
                    Lk = o[:P * R].reshape(P, R); Rk = o[P * R:P * R + R * D].reshape(R, D)
                    off = P * R + R * D
                    Lv = o[off:off + P * R].reshape(P, R); Rv = o[off + P * R:off + P * R + R * D].reshape(R, D)
                    assert np.array_equal(Lk[:, :rk], pg[1].astype(np.float32))
                    assert np.array_equal(Rk[:rk], pg[2].astype(np.float32))
                    assert np.array_equal(Lv[:, :rv], pg[3].astype(np.float32))
                    assert np.array_equal(Rv[:rv], pg[4].astype(np.float32))
    out, ref = _attend(cache, wl, seq_lens, heads, g)
    ma, mr = errors(out, ref)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (ma, mr)


def test_int4_attention_one_chunk_per_head():
    """256 heads of six pages each (B=32, 8 KV heads): every head is one
    workgroup's chunk, which normalizes its own output (no partial or merge);
    pages 1 and 2 of every head are INT4 factor pages."""
    import paper_2608_23843_amd as pk
    B, Hkv, g, S, W = 32, 8, 8, 64, 128
    T = 6 * 64 - 7
    wl = _wl(B, Hkv, g, T, S, W, seed_wid=97)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, 6, 32, S, W, "bf16", "int4")
    rng = np.random.default_rng(13)
    heads = {}
    for b in range(B):
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, b, h, 6 * P)
            K, V = _bf16(K), _bf16(V)
            rks = {j: tuple(int(x) for x in rng.choice([16, 24, 32], 2)) for j in range(6)}
            pages, blobs = _encode_head(K, V, T, S, W, lambda j: rks[j])
            assert sorted(blobs) == [1, 2]
            _import(cache, b, h, pages, blobs)
            heads[(b, h)] = oracle.HeadCache(T, P, D, pages)
    out, ref = _attend(cache, wl, [T] * B, heads, g)
    ma, mr = errors(out, ref)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (ma, mr)


@pytest.mark.parametrize("g", [1, 5, 16])
def test_int4_attention_query_groups(g):
    """Query groups below, between and above 8: at most 8 queries the kernel
    carries the lo half of the O^T update in the padding columns 8-15 and
    folds those rows back at the merge; 16 queries use both halves of every
    product for queries."""
    import paper_2608_23843_amd as pk
    seq_lens = [64 * 21 + 5, 64 * 9]
    B, Hkv, S, W = len(seq_lens), 2, 64, 128
    Tmax = max(seq_lens)
    wl = _wl(B, Hkv, g, Tmax, S, W, seed_wid=96)
    max_pages = -(-Tmax // P)
    cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "int4")
    rng = np.random.default_rng(11)
    heads = {}
    for b, T in enumerate(seq_lens):
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, b, h, max_pages * P)
            K, V = _bf16(K), _bf16(V)
            rks = {j: tuple(int(x) for x in rng.choice([8, 17, 24, 32], 2)) for j in range(max_pages)}
            pages, blobs = _encode_head(K, V, T, S, W, lambda j: rks[j])
            _import(cache, b, h, pages, blobs)
            heads[(b, h)] = oracle.HeadCache(T, P, D, pages)
    out, ref = _attend(cache, wl, seq_lens, heads, g)
    ma, mr = errors(out, ref)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (g, ma, mr)


def _near_tie(x, s):
    qv = np.abs(x / np.where(s > 0, s, 1.0))
    return np.abs(qv - np.floor(qv) - 0.5) < 1e-3


def test_int4_compress_codes_and_scales():
    """GPU quantizer vs the oracle quantizer on the GPU's own factors."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, g, S, W = 1, 2, 8, 64, 128
    T = 64 * 12
    wl = _wl(B, Hkv, g, T, S, W)
    max_pages = T // P + 1
    K, V = synth.kv_layer(wl, 0, 0, T)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    ranks = np.full((B, Hkv, max_pages), 24, dtype=np.uint8)
    ranks[0, 0, 3] = 16
    ranks[0, 1, 4] = 32
    ranks[0, 1, 5] = 20
    rt = torch.from_numpy(ranks).cuda()
    c4 = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "int4")
    cf = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "f32")
    c4.prefill(0, kt, vt, [T], rank_k=rt, rank_v=rt)
    cf.prefill(0, kt, vt, [T], rank_k=rt, rank_v=rt)
    torch.cuda.synchronize()
    assert c4.device_status() == 0 and cf.device_status() == 0
    kinds = oracle.plan_pages(T, P, S, W)
    fac = [j for j, k in enumerate(kinds) if k == oracle.FACTOR]
    n_bad = n_codes = 0
    for h in range(Hkv):
        blobs = c4.export_int4_pages(0, [0] * len(fac), [h] * len(fac), fac).cpu().numpy()
        blk = cf.export_pages(0, [0] * len(fac), [h] * len(fac), fac).cpu().numpy().astype(np.float64)
        R = 32
        for i, j in enumerate(fac):
            r = int(ranks[0, h, j])
            o = blk[i]
            L = {"K": o[:P * R].reshape(P, R)[:, :r], "V": o[P * R + R * D:2 * P * R + R * D].reshape(P, R)[:, :r]}
            Rm = {"K": o[P * R:P * R + R * D].reshape(R, D)[:r],
                  "V": o[2 * P * R + R * D:2 * P * R + 2 * R * D].reshape(R, D)[:r]}
            # the blob of this page
            nc = 2 * (P * r + r * D)
            codes = blobs[i][:nc].view(np.int8).astype(np.int64)
            scales = blobs[i][nc:nc + 2 * (2 * r + D + P + D)].view(np.float16).astype(np.float64)
            cs = {"K": (codes[:P * r].reshape(P, r), codes[P * r:P * r + r * D].reshape(r, D)),
                  "V": (codes[P * r + r * D:2 * P * r + r * D].reshape(P, r), codes[2 * P * r + r * D:].reshape(r, D))}
            ss = {"K": (scales[:2 * r].reshape(2, r), scales[2 * r:2 * r + D].reshape(1, D)),
                  "V": (scales[2 * r + D:2 * r + D + P].reshape(1, P), scales[2 * r + D + P:].reshape(1, D))}
            for which in ("K", "V"):
                sig = np.linalg.norm(Rm[which], axis=1)    # rows of R = Sigma W^T
                Lt, Rt = q4.balance(L[which], Rm[which], sig)
                for (mat, axis, got_c, got_s) in ((Lt, q4.AXIS["L_" + which], cs[which][0], ss[which][0]),
                                                  (Rt, q4.AXIS["R_" + which], cs[which][1], ss[which][1])):
                    ref_c, ref_s = q4.quantize_lines(mat, axis)
                    assert got_s.shape == ref_s.shape
                    rel = np.abs(got_s - ref_s) / np.maximum(ref_s, 1e-30)
                    assert np.all((got_s == ref_s) | (rel <= 2.0 ** -10)), (h, j, which, rel.max())
                    # codes where both sides used the same scale and the quotient is not near a tie
                    lines = mat if axis == 0 else mat.T
                    gl = got_c if axis == 0 else got_c.T
                    rl = ref_c if axis == 0 else ref_c.T
                    s_el = np.repeat(ref_s, q4.GROUP, axis=0)[:lines.shape[0]]
                    g_el = np.repeat(got_s, q4.GROUP, axis=0)[:lines.shape[0]]
                    same = (s_el == g_el) & ~_near_tie(lines, s_el)
                    n_codes += int(same.sum())
                    n_bad += int((gl[same] != rl[same]).sum())
                    assert np.all(np.abs(got_c) <= 7)
    assert n_codes > 50000
    assert n_bad == 0, n_bad


def test_int4_compress_then_attention():
    """GPU prefill (decompose + balance + quantize) then GPU attention against
    the oracle attending over the GPU's own dequantized factors."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, g, S, W = 2, 2, 8, 64, 256
    seq = [64 * 20 + 5, 64 * 17]
    T = max(seq)
    wl = _wl(B, Hkv, g, T, S, W)
    max_pages = -(-T // P)
    K, V = synth.kv_layer(wl, 0, 0, T)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    c4 = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "int4")
    c4.prefill(0, kt, vt, seq, default_rank=(24, 24))
    torch.cuda.synchronize()
    heads = {}
    R = 32
    for b in range(B):
        n = -(-seq[b] // P)
        for h in range(Hkv):
            blk = c4.export_pages(0, [b] * n, [h] * n, list(range(n))).cpu().numpy().astype(np.float64)
            kinds = oracle.plan_pages(seq[b], P, S, W, n)
            pages = []
            for j in range(n):
                o = blk[j]
                if kinds[j] == oracle.FACTOR:
                    pages.append(("factor", o[:P * R].reshape(P, R)[:, :24], o[P * R:P * R + R * D].reshape(R, D)[:24],
                                  o[P * R + R * D:2 * P * R + R * D].reshape(P, R)[:, :24],
                                  o[2 * P * R + R * D:2 * P * R + 2 * R * D].reshape(R, D)[:24]))
                else:
                    pages.append(("dense", o[:P * D].reshape(P, D), o[P * D:2 * P * D].reshape(P, D)))
            heads[(b, h)] = oracle.HeadCache(seq[b], P, D, pages)
    out, ref = _attend(c4, wl, seq, heads, g)
    ma, mr = errors(out, ref)
    assert ma <= MAX_ABS and mr <= MEAN_REL, (ma, mr)


def test_int4_workspace_reuse_across_chunk_counts():
    """INT4 kernel: one workspace serves calls whose lengths give different
    chunk counts (B = 1, 8 KV heads: 2,000 tokens split into 32 chunks, 2,100
    into 17); every call agrees with a call on a fresh workspace to the
    kernel's precision and with the oracle to the parity bar, and the claim
    and merge counters read zero afterwards."""
    import torch
    import paper_2608_23843_amd as pk
    B, Hkv, g, S, W = 1, 8, 8, 64, 128
    lens = (2000, 2100)
    wl = _wl(B, Hkv, g, max(lens), S, W, seed_wid=96)
    max_pages = -(-max(lens) // P)
    caches, heads_of = [], []
    for T in lens:
        cache = pk.PuzzleKVCache(1, B, Hkv, Hkv * g, D, P, max_pages, 32, S, W, "bf16", "int4")
        heads = {}
        for h in range(Hkv):
            K, V = synth.kv_head(wl, 0, 0, 0, h, max_pages * P)
            pages, blobs = _encode_head(_bf16(K), _bf16(V), T, S, W, lambda j: (24, 16))
            _import(cache, 0, h, pages, blobs)
            heads[(0, h)] = oracle.HeadCache(T, P, D, pages)
        caches.append(cache)
        heads_of.append(heads)
    sizes = [caches[0].workspace_bytes(pk.PKV_OP_ATTENTION, T) for T in lens]
    assert sizes[0] != sizes[1], "the two lengths must give different partial layouts"
    q = synth.queries(wl, 0)
    qt = torch.from_numpy(q).to(device="cuda", dtype=torch.bfloat16).contiguous()
    ws = caches[0].workspace(pk.PKV_OP_ATTENTION, 4096)
    for rep in range(2):
        for cache, T, heads in zip(caches, lens, heads_of):
            out, lse = cache.attention(0, qt, [T], workspace=ws)
            fresh, lse_f = cache.attention(0, qt, [T], workspace=cache.workspace(pk.PKV_OP_ATTENTION, T))
            torch.cuda.synchronize()
            assert cache.device_status() == 0
            # pages reach the waves in a dynamic order, which moves the lazy
            # max's rescale points and with them the fp16 roundings of the
            # weights, so two calls agree only to the kernel's own precision
            # (stale counters would give garbage or nothing at all)
            o = out.cpu().numpy().astype(np.float64)
            ma, mr = errors(o, fresh.cpu().numpy().astype(np.float64))
            assert ma <= 1e-3 and mr <= 1e-4, (T, rep, ma, mr)
            assert float((lse - lse_f).abs().max()) <= 1e-4
            ref = np.zeros_like(o)
            for (b, h), head in heads.items():
                ref[b, h * g:(h + 1) * g], _ = oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
            ma, mr = errors(o, ref)
            assert ma <= MAX_ABS and mr <= MEAN_REL, (T, rep, ma, mr)
    heads = B * Hkv
    counters = (4 * heads + 255) // 256 * 256 + 256 * heads
    assert int(ws[:counters].count_nonzero()) == 0
