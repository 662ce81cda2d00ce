#!/usr/bin/env python3
"""Benchmark of the PuzzleKV hot path on one MI355X.

Workload (default qwen32b_128k): Qwen3-32B-shaped layer -- 64 query heads over
8 KV heads, d=128, pages of 64 tokens, batch 4, 131072 cached tokens per
sequence, 64-token sink and 512-token window dense, every other page stored as
bf16 factors with a per-page rank drawn from {16, 24, 32}. A decode step runs
64 layers, each with its own cache buffers: append the new token, factorize
pages that leave the window (the host planner decides; none at this length
inside a short run), and mixed-page decode attention.

--workload qwen32b_int4: the same heads and length at batch 8 with factor
pages stored as INT4 codes plus fp16 scales (Section 4.3), one layer per step.

Setup (untimed): the seeded generator draws layer 0's prompt K/V, the GPU
decomposition builds its hybrid cache (timed separately for pages/s), and the
layer's buffers are copied into the 63 other layers. Inputs are resident in
HBM when the timed region starts.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
EVENT_STRIDE = 8   # decode steps: the attention call of every EVENT_STRIDE-th layer is timed with events
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_23843_amd", "csrc", f)
                  for f in ("attention.inl", "attention_mfma.inl", "attention_q4.inl", "attention_launch.inl",
                            "global_svd.inl")]


def log(msg: str) -> None:
    print("[bench %7.1fs] %s" % (time.time() - T0, msg), file=sys.stderr, flush=True)


T0 = time.time()


def kernel_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", "attention_%s_traffic.txt" % workload)


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source; else None."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_hash") != kernel_hash() or vals.get("workload") != workload:
        return None
    try:
        return float(vals["bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen32b_128k")
    ap.add_argument("--layers", type=int, default=0, help="layers per step (default: the workload's)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--tokens", type=int, default=0, help="override the cached length T")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU-baseline budget for the oracle (0 disables)")
    ap.add_argument("--workers", type=int, default=16, help="host threads for input generation")
    ap.add_argument("--no-calibration", action="store_true",
                    help="skip the HBM read/copy bandwidth sweep (for short profiling runs)")
    ap.add_argument("--compare", action="store_true",
                    help="Global SVD workloads: also compare its accuracy with PuzzleKV's at the same budget")
    return ap.parse_args()


def factor_logical_bytes(factors, P, d, rk, rv):
    """Bytes of one factor page pair at its logical ranks (Eq. (3) storage):
    (r_K + r_V)(P + d) elements; INT4 adds one fp16 scale per run of up to 32
    elements along the paper's directions to its half-byte codes."""
    if factors == "int4":
        runs = lambda n: -(-n // 32)
        scales = rk * runs(P) + d * runs(rk) + P * runs(rv) + d * runs(rv)
        return (rk + rv) * (P + d) // 2 + 2 * scales
    return (rk + rv) * (P + d) * (4 if factors == "f32" else 2)


def attention_bytes(factors, ranks_np, ranks_v_np, seq_len, P, d, B, Hkv, Hq, S, W):
    """Algorithmic bytes one attention launch must move: every factor page pair
    at its logical ranks (padding the slot layout adds is not counted), the
    dense pages up to the sequence length, the page-table entries, the
    queries, out and lse."""
    total = 0
    fpb = {}
    for b in range(B):
        T = int(seq_len[b])
        n = -(-T // P)
        sink_pages = -(-S // P)
        jmax = (T - W) // P - 1 if T - W >= 0 else -1
        for h in range(Hkv):
            for j in range(n):
                if sink_pages <= j <= jmax:
                    r = (int(ranks_np[b, h, j]), int(ranks_v_np[b, h, j]))
                    if r not in fpb:
                        fpb[r] = factor_logical_bytes(factors, P, d, *r)
                    total += fpb[r]
                else:
                    rows = min(P, T - j * P)
                    total += 2 * rows * d * 2
            total += n * 8
    total += B * Hq * d * 2 + B * Hq * d * 4 + B * Hq * 4
    return total


def compress_work(kinds, ranks_np, ranks_v_np, B, Hkv, P, d, sweeps_total):
    """FLOPs of one prefill's decompositions (a page pair is a K and a V
    decomposition). Useful: the Gram matrix X X^T (2 P^2 d) and the projection
    R = L^T X at the page's rank (2 r P d). Executed, as the matrix-core kernel
    runs it: Gram; the QR of G (P steps, each lane forming the pivot norm, its
    dot and its update: 6 P^3); each Jacobi sweep (P - 1 steps of P lanes, a
    P-long dot and update each: 4 P^2 (P - 1)); the projection for all 32 rank
    slots (2 * 32 P d)."""
    import numpy as np
    fact = np.nonzero(np.asarray(kinds) == 2)[0]
    r = ranks_np[:, :, fact].astype(np.float64)          # [B][Hkv][pages]
    rv = ranks_v_np[:, :, fact].astype(np.float64)
    n_dec = 2 * r.size
    useful = 2 * r.size * 2.0 * P * P * d + (2.0 * r * P * d).sum() + (2.0 * rv * P * d).sum()
    executed = n_dec * (2.0 * P * P * d + 6.0 * P ** 3 + 2.0 * 32 * P * d) + sweeps_total * 4.0 * P * P * (P - 1)
    return {"sweeps": sweeps_total / max(n_dec, 1), "useful": useful, "executed": executed}


def chosen_ranks(cache, kinds, max_pages, eps):
    """The (rank_k, rank_v) the decomposition chose for layer 0, read from its page table."""
    import numpy as np
    import paper_2608_23843_amd as pk
    _, _, rk, rv = cache.page_table_host(0)
    rk = np.ascontiguousarray(rk[:, :, :max_pages]).astype(np.uint8)
    rv = np.ascontiguousarray(rv[:, :, :max_pages]).astype(np.uint8)
    fac = np.flatnonzero(np.asarray(kinds) == pk.PKV_FACTOR)
    log("ranks chosen for relative error %.2f: mean r_K %.2f, mean r_V %.2f over %d factor pages per head"
        % (eps, rk[:, :, fac].mean(), rv[:, :, fac].mean(), len(fac)))
    return rk, rv


def cpu_baseline(wl, seed, seq_T, K_dense, V_dense, q, budget_s, layers, ranks, ranks_v):
    """The oracle on a bounded sample: whole (sequence, KV head) heads of one
    layer at the full length, factor pages drawn by the generator, timed until
    the budget is spent; extrapolated to the step (all heads, all layers)."""
    import numpy as np
    import oracle
    import synth
    from oracle import int4 as q4
    P, d, g = wl.page, wl.head_dim, wl.group
    int4 = wl.factors == "int4"
    kinds = oracle.plan_pages(seq_T, P, wl.sink, wl.window)
    times, heads = [], []
    for b in range(wl.batch):
        for h in range(wl.kv_heads):
            pages = []
            encoded = {}
            for j, kd in enumerate(kinds):
                if kd == oracle.FACTOR:
                    Lk, Rk, Lv, Rv = synth.factor_page(wl, seed, 0, b, h, j, int(ranks[b, h, j]),
                                                       int(ranks_v[b, h, j]))
                    if int4:
                        encoded[j] = [q4.encode_page(w, L, R, np.linalg.norm(R, axis=1))
                                      for w, L, R in (("K", Lk, Rk), ("V", Lv, Rv))]
                        pages.append(None)
                    else:
                        pages.append(("factor", Lk, Rk, Lv, Rv))
                else:
                    Kp, Vp = K_dense[(b, h, j)], V_dense[(b, h, j)]
                    pages.append(("dense", Kp, Vp))
            t = time.time()
            for j, (ek, ev) in encoded.items():   # INT4: dequantization is part of the timed work
                pages[j] = ("factor",) + tuple(
                    q4.dequantize_lines(e[c + "_codes"], e[c + "_scales"], q4.AXIS[c + "_" + w])
                    for e, w in ((ek, "K"), (ev, "V")) for c in ("L", "R"))
            head = oracle.HeadCache(seq_T, P, d, pages, key_rope_base=wl.rope_base if wl.key_rope else 0.0)
            oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
            times.append(time.time() - t)
            heads.append((b, h))
            if sum(times) >= budget_s:
                break
        if sum(times) >= budget_s:
            break
    per_head = sum(times) / len(times)
    n_heads = wl.batch * wl.kv_heads
    us_step = per_head * n_heads * layers * 1e6
    return {
        "value": us_step, "unit": "us/step", "cores": oracle.num_threads(), "kind": "oracle",
        "sample": "%d of %d (sequence, KV head) heads of one layer at T=%d (fp64 %srebuild + %ssoftmax), "
                  "%.2f s per head, extrapolated x%d heads x%d layers"
                  % (len(times), n_heads, seq_T, "INT4 dequantization + " if int4 else "",
                     "key RoPE + " if wl.key_rope else "", per_head, n_heads, layers),
    }


def hbm_calibration(achieved_gbps):
    """Streaming read and copy rates of this chip (pkv_bandwidth_probe over
    2 GiB, beyond the 256 MB last-level cache; the best of a sweep of access
    patterns and launch shapes), and the attention's rate against them."""
    import torch
    import paper_2608_23843_amd as pk
    n = 2 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    best = {"read": (0.0, ""), "copy": (0.0, "")}
    for mode in (0, 2, 1, 3):
        name = "copy" if mode & 1 else "read"
        for threads in (256, 512):
            for blocks in (256, 512, 1024, 2048, 4096):
                gbps = pk.bandwidth_probe(src, dst, mode, reps=5, blocks=blocks, threads=threads)
                if gbps > best[name][0]:
                    best[name] = (gbps, "%s, %d x %d threads" % ("64 KB chunks per workgroup" if mode & 2 else
                                                                 "grid-stride", blocks, threads))
    del src, dst
    torch.cuda.empty_cache()
    out = {"read_gbps": round(best["read"][0], 1), "read_shape": best["read"][1],
           "copy_gbps": round(best["copy"][0], 1), "copy_shape": best["copy"][1],
           "attention_frac_of_read": round(achieved_gbps / best["read"][0], 4),
           "attention_frac_of_copy": round(achieved_gbps / best["copy"][0], 4),
           "probe": "pkv_bandwidth_probe over 2 GiB, 16-byte loads, best of 5 launches per shape"}
    log("HBM calibration: read %.0f GB/s (%s), copy %.0f GB/s (%s); attention at %.3f of read"
        % (best["read"][0], best["read"][1], best["copy"][0], best["copy"][1], achieved_gbps / best["read"][0]))
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_extras(wl, seed, T, K_dense, V_dense, q, comp_X, ranks_np, ranks_v_np, comp_refs):
    """The rest of the oracle baseline: one head's attention on a single
    thread, and the oracle's decomposition (fp64 one-sided Jacobi) on a sample
    of up to 4,096 of the prompt's factorizable page pairs on all threads and
    on a single thread (a 64-pair slice)."""
    import numpy as np
    import oracle
    threads = oracle.num_threads()
    extras = {"cpu_model": cpu_model()}
    oracle.set_num_threads(1)
    try:
        one = cpu_baseline(wl, seed, T, K_dense, V_dense, q, 0.0, 1, ranks_np, ranks_v_np)
        n_heads = wl.batch * wl.kv_heads
        extras["value_1thread"] = one["value"] * n_heads   # one layer, all heads, 1 thread
        extras["unit_1thread"] = "us per layer (all heads), 1 thread, extrapolated from one head"
        if comp_X is not None and wl.rank_error == 0:
            n1 = min(64, len(comp_refs))
            X1 = np.concatenate([comp_X[:n1], comp_X[len(comp_refs):len(comp_refs) + n1]])
            r1 = np.array([ranks_np[b, h, j] for b, h, j in comp_refs[:n1]] +
                          [ranks_v_np[b, h, j] for b, h, j in comp_refs[:n1]], dtype=np.int32)
            t = time.time()
            oracle.truncated_factors_batch(X1, r1)
            extras["compress_page_pairs_per_s_1thread"] = round(n1 / (time.time() - t), 2)
    finally:
        oracle.set_num_threads(threads)
    if comp_X is not None and wl.rank_error == 0:
        n = len(comp_refs)
        rk = np.array([ranks_np[b, h, j] for b, h, j in comp_refs] + [ranks_v_np[b, h, j] for b, h, j in comp_refs],
                      dtype=np.int32)
        t = time.time()
        oracle.truncated_factors_batch(comp_X, rk)
        dt = time.time() - t
        extras["compress_page_pairs_per_s"] = round(n / dt, 2)
        extras["compress_sample"] = ("%d page pairs (K and V, P=%d, d=%d) of the prompt's factorizable pages, "
                                     "fp64 one-sided Jacobi, %d threads, %.1f s" % (n, wl.page, wl.head_dim,
                                                                                     threads, dt))
    log("CPU extras: %s" % json.dumps(extras))
    return extras


def global_attention_bytes(P, d, g, r, seq_len, S, W):
    """Algorithmic bytes of one Global SVD attention launch, per (sequence, KV
    head): the coefficient rows of the region (r bf16 values for K and for V
    per token), the two bases (r x d each), the dense pages up to the length
    and their page-table entries. The caller adds the queries, out and lse."""
    total = 0
    for T in seq_len:
        n_pages = -(-T // P)
        sink_pages = -(-S // P)
        t1 = (T - W) // P * P if T >= W else 0
        n_reg = max(0, t1 - sink_pages * P)
        total += 2 * n_reg * r * 2 + 2 * r * d * 2 + 2 * (T - n_reg) * d * 2 + (n_pages - n_reg // P) * 8
    return total


def _rel(a, b):
    import numpy as np
    return float(np.abs(a - b).sum() / max(np.abs(b).sum(), 1e-300))


def global_comparison(wl, seed, settings, log_fn):
    """Global SVD against PuzzleKV at one budget (Section 4.2 "Main Results",
    a matched rho), on sequences whose planted subspace changes every
    `segment_pages` pages: reconstruction error of the compressible region
    and attention error against exact dense attention (the oracle, fp64) for
    random queries and for retrieval queries (each query head points at one
    random key of the region, so its softmax is peaked), both methods' factors
    computed on the GPU."""
    import dataclasses
    import numpy as np
    import torch
    import oracle
    import paper_2608_23843_amd as pk
    import synth
    P, d, S, W, T, B, Hkv, g = wl.page, wl.head_dim, wl.sink, wl.window, wl.tokens, wl.batch, wl.kv_heads, wl.group
    rk, rv = wl.ranks[0], (wl.ranks_v or wl.ranks)[0]
    kinds = oracle.plan_pages(T, P, S, W)
    fac = [j for j, k in enumerate(kinds) if k == oracle.FACTOR]
    rows = np.concatenate([np.arange(j * P, (j + 1) * P) for j in fac])
    out = []
    for seg in settings:
        w = dataclasses.replace(wl, segment_pages=seg)
        K, V = synth.kv_layer(w, seed, 0, T)
        kt = torch.from_numpy(K).to("cuda", torch.bfloat16).contiguous()
        vt = torch.from_numpy(V).to("cuda", torch.bfloat16).contiguous()
        cache = pk.PuzzleKVCache(1, B, Hkv, w.q_heads, d, P, len(kinds), max(rk, rv), S, W, "bf16", "bf16")
        cache.prefill(0, kt, vt, [T] * B, default_rank=(rk, rv))
        fp = cache.footprint([T] * B, layer=0)
        rho = (fp["dense_bytes"] + fp["factor_bytes"]) / fp["raw_bytes"]
        r = pk.global_rank(T, P, S, W, d, rho)
        gc = pk.PuzzleKVCache(1, B, Hkv, w.q_heads, d, P, len(kinds), 1, S, W, "bf16", "bf16")
        gs = pk.GlobalSVD(gc, r, -(-len(rows) // 32) * 32)
        gs.prefill(0, kt, vt, [T] * B)
        torch.cuda.synchronize()
        status = cache.device_status()
        # reconstruction of the region
        num = {"pkv": [0.0, 0.0], "global": [0.0, 0.0]}
        den = [0.0, 0.0]
        R = cache.c.max_rank
        for b in range(B):
            for h in range(Hkv):
                blk = cache.export_pages(0, [b] * len(fac), [h] * len(fac), fac).cpu().numpy().astype(np.float64)
                bk, bv, ak, av = (x.cpu().numpy().astype(np.float64) for x in gs.export(0, b, h, len(rows)))
                for i, (X, Ag, Bg) in enumerate(((K[b, h][rows].astype(np.float64), ak, bk),
                                                 (V[b, h][rows].astype(np.float64), av, bv))):
                    den[i] += float(np.sum(X * X))
                    Eg = X - Ag @ Bg
                    num["global"][i] += float(np.sum(Eg * Eg))
                    rr = rk if i == 0 else rv
                    off = 0 if i == 0 else P * R + R * d
                    Lp = blk[:, off:off + P * R].reshape(-1, P, R)[:, :, :rr]
                    Rp = blk[:, off + P * R:off + P * R + R * d].reshape(-1, R, d)[:, :rr]
                    Ep = X.reshape(-1, P, d) - np.matmul(Lp, Rp)
                    num["pkv"][i] += float(np.sum(Ep * Ep))
        rec = {m: [float(np.sqrt(num[m][i] / den[i])) for i in range(2)] for m in num}
        # attention against dense attention
        rng = np.random.default_rng(seed + 77)
        q_rand = synth.queries(w, seed, 0)
        q_ret = np.empty_like(q_rand)
        for b in range(B):
            for h in range(Hkv):
                for i in range(g):
                    kk = K[b, h][rows[rng.integers(len(rows))]].astype(np.float64)
                    q_ret[b, h * g + i] = 12.0 * np.sqrt(d) * kk / np.sum(kk * kk)   # score of that key: 12
        q_ret = synth.round_storage(q_ret, "bf16")
        att = {}
        for name, qv in (("random", q_rand), ("retrieval", q_ret)):
            qt = torch.from_numpy(qv).to("cuda", torch.bfloat16).contiguous()
            o_p, _ = cache.attention(0, qt, [T] * B)
            o_g, _ = gs.attention(0, qt, [T] * B)
            torch.cuda.synchronize()
            o_p, o_g = o_p.cpu().numpy().astype(np.float64), o_g.cpu().numpy().astype(np.float64)
            ref = np.zeros_like(o_p)
            for b in range(B):
                for h in range(Hkv):
                    pages = []
                    for j in range(len(kinds)):
                        Kp = np.zeros((P, d)); Vp = np.zeros((P, d))
                        n = min(P, T - j * P)
                        Kp[:n] = K[b, h, j * P:j * P + n]; Vp[:n] = V[b, h, j * P:j * P + n]
                        pages.append(("dense", Kp, Vp))
                    ref[b, h * g:(h + 1) * g], _ = oracle.attention(oracle.HeadCache(T, P, d, pages),
                                                                    qv[b, h * g:(h + 1) * g].astype(np.float64))
            att[name] = {"pkv": _rel(o_p, ref), "global": _rel(o_g, ref)}
        status |= cache.device_status() | gc.device_status()
        rho_g = (2 * (T * B * Hkv - len(rows) * B * Hkv) * d + 2 * r * (len(rows) + d) * B * Hkv) / (2.0 * T * d * B * Hkv)
        row = {"segment_pages": seg, "rho_pkv": round(rho, 5), "global_rank": r, "rho_global": round(rho_g, 5),
               "recon_rel_err": {"pkv": [round(x, 5) for x in rec["pkv"]], "global": [round(x, 5) for x in rec["global"]]},
               "attn_rel_err": {k: {m: round(v, 6) for m, v in d_.items()} for k, d_ in att.items()},
               "device_status": status}
        log_fn("comparison, segments of %s pages: %s" % (seg, json.dumps(row)))
        out.append(row)
        del cache, gc, gs, kt, vt
        torch.cuda.empty_cache()
    return out


def global_cpu_baseline(wl, seed, T, r, budget_s, layers):
    """The oracle's Global SVD attention (every factorized token rebuilt from
    its coefficients and the basis, then textbook softmax) on whole heads of
    one layer, coefficients and bases drawn by the generator, timed until the
    budget is spent; extrapolated to the step."""
    import numpy as np
    import oracle
    import synth
    P, d, g = wl.page, wl.head_dim, wl.group
    kinds = oracle.plan_pages(T, P, wl.sink, wl.window)
    n_reg = int((kinds == oracle.FACTOR).sum()) * P
    q = synth.queries(wl, seed, 0)
    times = []
    for b in range(wl.batch):
        for h in range(wl.kv_heads):
            K, V = synth.kv_head(wl, seed, 0, b, h, T)
            A_K, B_K, A_V, B_V = synth.global_factors(wl, seed, 0, b, h, n_reg, r)
            t = time.time()
            head = oracle.global_head(T, P, d, kinds, K, V, A_K, B_K, A_V, B_V)
            oracle.attention(head, q[b, h * g:(h + 1) * g].astype(np.float64))
            times.append(time.time() - t)
            if sum(times) >= budget_s:
                break
        if sum(times) >= budget_s:
            break
    per_head = sum(times) / len(times)
    n_heads = wl.batch * wl.kv_heads
    return {"value": per_head * n_heads * layers * 1e6, "unit": "us/step", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "%d of %d (sequence, KV head) heads of one layer at T=%d (fp64 rebuild of %d factorized "
                      "tokens at rank %d + softmax), %.2f s per head, extrapolated x%d heads x%d layers"
                      % (len(times), n_heads, T, n_reg, r, per_head, n_heads, layers)}


def run_global(args, wl):
    """Global SVD baseline: prefill (Gram, eigenvectors, projection) timed on
    layer 0, the layer copied into the others, then attention over every layer
    per decode step. The baseline is built from the prompt and attended at
    its length; decode steps re-attend the same cache with new queries."""
    import numpy as np
    import torch
    import paper_2608_23843_amd as pk
    import synth
    layers = args.layers or wl.layers
    B, Hkv, Hq, d, P, T = wl.batch, wl.kv_heads, wl.q_heads, wl.head_dim, wl.page, wl.tokens
    S, W, g = wl.sink, wl.window, wl.group
    n_steps = args.warmup + args.steps
    kinds = pk.plan_pages(T, P, S, W)
    n_reg = int((kinds == pk.PKV_FACTOR).sum()) * P
    K, V = synth.kv_layer(wl, args.seed, 0, T, workers=args.workers)
    kt = torch.from_numpy(K).to("cuda", torch.bfloat16)
    vt = torch.from_numpy(V).to("cuda", torch.bfloat16)
    del K, V
    rho = wl.global_rho
    if rho < 0:   # matched to PuzzleKV's realized ratio on the same inputs
        pc = pk.PuzzleKVCache(1, B, Hkv, Hq, d, P, len(kinds), max(wl.ranks + wl.ranks_v), S, W, "bf16", "bf16")
        pc.prefill(0, kt, vt, [T] * B, default_rank=(wl.ranks[0], (wl.ranks_v or wl.ranks)[0]))
        fp = pc.footprint([T] * B, layer=0)
        rho = (fp["dense_bytes"] + fp["factor_bytes"]) / fp["raw_bytes"]
        del pc
    r = pk.global_rank(T, P, S, W, d, rho)
    log("workload %s: B=%d Hq=%d Hkv=%d d=%d P=%d T=%d layers=%d, Global SVD rank %d for ratio %.5f"
        % (wl.name, B, Hq, Hkv, d, P, T, layers, r, rho))
    cache = pk.PuzzleKVCache(layers, B, Hkv, Hq, d, P, len(kinds), 1, S, W, "bf16", "bf16")
    gs = pk.GlobalSVD(cache, r, -(-n_reg // 32) * 32)
    ws_p = gs.workspace(pk.PKV_OP_GLOBAL_PREFILL, T)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pre_ms = []
    for rep in range(3):
        torch.cuda.synchronize()
        ev0.record()
        gs.prefill(0, kt, vt, [T] * B, workspace=ws_p)
        ev1.record()
        torch.cuda.synchronize()
        pre_ms.append(ev0.elapsed_time(ev1))
    status = cache.device_status()
    log("Global SVD prefill (Gram + eigenvectors + projection) of one layer: %.3f ms (best of 3), status %d"
        % (min(pre_ms), status))
    del kt, vt, ws_p
    torch.cuda.empty_cache()
    for buf in (cache.dense_pool, cache.table, gs.basis, gs.coef):
        per = buf.numel() // layers
        for layer in range(1, layers):
            buf[layer * per:(layer + 1) * per].copy_(buf[:per])
    torch.cuda.synchronize()
    ws = gs.workspace(pk.PKV_OP_GLOBAL_ATTENTION, T)
    out = torch.empty((B, Hq, d), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    qs = [torch.from_numpy(synth.queries(wl, args.seed, s)).to("cuda", torch.bfloat16).contiguous()
          for s in range(n_steps)]
    stream = torch.cuda.current_stream()
    pool = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps * layers)]
    marks = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize()
    import gc as _gc
    _gc.collect()
    _gc.disable()
    calls = []
    for s in range(n_steps):
        timed = s >= args.warmup
        if s == args.warmup:
            torch.cuda.synchronize()
            marks[0].record(stream)
        for layer in range(layers):
            ev = timed and layer % EVENT_STRIDE == 0   # as in the PuzzleKV decode steps
            if ev:
                e0, e1 = pool[len(calls)]
                e0.record(stream)
            gs.attention(layer, qs[s], [T] * B, out=out, lse=lse, workspace=ws)
            if ev:
                e1.record(stream)
                calls.append((e0, e1))
    marks[1].record(stream)
    torch.cuda.synchronize()
    _gc.enable()
    status |= cache.device_status()
    ms_per_step = marks[0].elapsed_time(marks[1]) / args.steps
    call_ms = np.array([a.elapsed_time(b) for a, b in calls])
    attn_us = float(call_ms.mean() * 1e3)
    if not np.isfinite(out.cpu().numpy()).all():
        raise RuntimeError("non-finite attention output")
    abytes = global_attention_bytes(P, d, g, r, [T] * B, S, W) * Hkv + B * Hq * (d * 2 + d * 4 + 4)
    achieved = abytes / (attn_us * 1e-6) / 1e9
    log("decode: %.3f ms/step, Global SVD attention %.1f us/layer (median %.1f), %.1f GB/s, status %d"
        % (ms_per_step, attn_us, float(np.median(call_ms) * 1e3), achieved, status))
    result = {
        "metric": "Global SVD decode attention time per decode step (%d layers, %d/%d heads, %dK context, one "
                  "rank-%d basis per KV head)" % (layers, Hq, Hkv, T // 1024, r),
        "value": round(ms_per_step * 1e3, 2), "unit": "us/step", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d, "page": P,
                   "tokens": T, "sink": S, "window": W, "global_rank": r, "storage_ratio": round(rho, 5),
                   "segment_pages": wl.segment_pages, "layers": layers,
                   "step": "Global SVD attention per layer (the baseline is not updated while decoding)"},
        "attention_us_per_layer": round(attn_us, 2),
        "attention_us_median": round(float(np.median(call_ms) * 1e3), 2),
        "attention_us_p90": round(float(np.percentile(call_ms * 1e3, 90)), 2),
        "attention_samples": int(call_ms.size),
        "attention_algorithmic_bytes": int(abytes),
        "attention_gbps": round(achieved, 1),
        "global_prefill_ms_per_layer": round(min(pre_ms), 3),
        "device_status": status,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(wl.name)},
    }
    del cache, gs, ws
    torch.cuda.empty_cache()
    if not args.no_calibration:
        result["hbm_calibration"] = hbm_calibration(achieved)
    if args.cpu_seconds > 0:
        log("CPU baseline (oracle), budget %.0f s" % args.cpu_seconds)
        result["cpu_baseline"] = global_cpu_baseline(wl, args.seed, T, r, args.cpu_seconds, layers)
        result["cpu_baseline"]["cpu_model"] = cpu_model()
    if args.compare:
        result["comparison"] = global_comparison(wl, args.seed, (1, 4, 16, 64, 0), log)
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(asked for --gpus %d, WORLD_SIZE=%d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_23843_amd as pk
    import synth

    pk.load_library()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.workload]
    if args.tokens:
        import dataclasses
        wl = dataclasses.replace(wl, tokens=args.tokens, name=wl.name + "_T%d" % args.tokens)
    if wl.global_rho != 0:
        return run_global(args, wl)
    layers = args.layers or wl.layers
    B, Hkv, Hq, d, P, T = wl.batch, wl.kv_heads, wl.q_heads, wl.head_dim, wl.page, wl.tokens
    S, W = wl.sink, wl.window
    n_steps = args.warmup + args.steps
    max_pages = -(-(T + n_steps + 1) // P) + 1
    max_rank = max(wl.ranks + wl.ranks_v)
    log("workload %s: B=%d Hq=%d Hkv=%d d=%d P=%d T=%d layers=%d" % (wl.name, B, Hq, Hkv, d, P, T, layers))

    # ---- inputs ----------------------------------------------------------------
    K, V = synth.kv_layer(wl, args.seed, 0, T, workers=args.workers)
    log("generated layer-0 K/V (%.1f GB fp32 on host)" % (2 * K.nbytes / 1e9))
    kinds = pk.plan_pages(T, P, S, W)
    dense_idx = [j for j, kd in enumerate(kinds) if kd == pk.PKV_DENSE]
    K_dense = {(b, h, j): K[b, h, j * P:(j + 1) * P].astype(np.float64)
               for b in range(B) for h in range(Hkv) for j in dense_idx}
    V_dense = {(b, h, j): V[b, h, j * P:(j + 1) * P].astype(np.float64)
               for b in range(B) for h in range(Hkv) for j in dense_idx}
    # a sample of the prompt's factorizable pages for the oracle's decomposition
    # baseline (up to 4,096 page pairs, taken in order over heads and pages)
    fac_idx = [j for j, kd in enumerate(kinds) if kd == pk.PKV_FACTOR]
    comp_refs = [(b, h, j) for b in range(B) for h in range(Hkv) for j in fac_idx][:4096]
    comp_X = np.stack([K[b, h, j * P:(j + 1) * P] for b, h, j in comp_refs] +
                      [V[b, h, j * P:(j + 1) * P] for b, h, j in comp_refs]).astype(np.float64) if comp_refs else None
    bf = torch.bfloat16
    kt = torch.from_numpy(K).to("cuda", bf)
    del K
    vt = torch.from_numpy(V).to("cuda", bf)
    del V
    ranks_np = synth.page_ranks(wl, args.seed, 0, max_pages)
    ranks_v_np = synth.page_ranks(wl, args.seed, 0, max_pages, "v")
    if wl.rank_error > 0:   # rank 0: the decomposition chooses each page's ranks
        ranks_np[:] = 0
        ranks_v_np[:] = 0
    req_np, req_v_np = ranks_np.copy(), ranks_v_np.copy()   # what prefill and compress_pages ask for
    ranks = torch.from_numpy(ranks_np).cuda().contiguous()
    ranks_v = torch.from_numpy(ranks_v_np).cuda().contiguous()

    rope_base = wl.rope_base if wl.key_rope else 0.0   # > 0: keys cached before RoPE
    cache = pk.PuzzleKVCache(layers, B, Hkv, Hq, d, P, max_pages, max_rank, S, W, wl.dtype, wl.factors,
                             adaptive_rank_error=wl.rank_error, key_rope_base=rope_base)
    log("cache: factor pool %.1f GB, dense pool %.2f GB" % (cache.factor_pool.numel() / 1e9,
                                                            cache.dense_pool.numel() / 1e9))

    # ---- batched page decomposition (prefill of layer 0) ----------------------
    n_fact = int((kinds == pk.PKV_FACTOR).sum()) * B * Hkv
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    comp_ms = []
    cache.compress_sweeps()   # clear the device's sweep counter
    for rep in range(3):
        torch.cuda.synchronize()
        ev0.record()
        cache.prefill(0, kt, vt, [T] * B, rank_k=ranks, rank_v=ranks_v)
        ev1.record()
        torch.cuda.synchronize()
        comp_ms.append(ev0.elapsed_time(ev1))
    sweeps = cache.compress_sweeps() / 3.0
    status = cache.device_status()
    fp = cache.footprint([T] * B, layer=0)   # live KV footprint of the prefilled layer
    fp_ratio = (fp["dense_bytes"] + fp["factor_bytes"]) / fp["raw_bytes"]
    fp_slots = (fp["dense_bytes"] + fp["factor_slot_bytes"]) / fp["raw_bytes"]
    log("live KV footprint at T=%d: %.5f of raw (slots with padding: %.5f)" % (T, fp_ratio, fp_slots))
    if wl.rank_error > 0:
        ranks_np, ranks_v_np = chosen_ranks(cache, kinds, max_pages, wl.rank_error)
    comp_ms_best = min(comp_ms)
    pages_per_s = n_fact / (comp_ms_best / 1e3)
    comp = compress_work(kinds, ranks_np, ranks_v_np, B, Hkv, P, d, sweeps)
    log("prefill/decomposition: %d page pairs in %.2f ms (%.3g pairs/s, %.2f sweeps per decomposition, "
        "useful %.2f TFLOP/s, executed %.2f TFLOP/s), status %d"
        % (n_fact, comp_ms_best, pages_per_s, comp["sweeps"], comp["useful"] / comp_ms_best / 1e9,
           comp["executed"] / comp_ms_best / 1e9, status))
    del kt, vt
    torch.cuda.empty_cache()

    # ---- replicate layer 0 into the other layers --------------------------------
    per_d = cache.dense_pool.numel() // layers
    per_f = cache.factor_pool.numel() // layers
    per_t = cache.table.numel() // layers
    for layer in range(1, layers):
        cache.dense_pool[layer * per_d:(layer + 1) * per_d].copy_(cache.dense_pool[:per_d])
        cache.factor_pool[layer * per_f:(layer + 1) * per_f].copy_(cache.factor_pool[:per_f])
        cache.table[layer * per_t:(layer + 1) * per_t].copy_(cache.table[:per_t])
    torch.cuda.synchronize()
    log("replicated layer 0 into %d layers" % layers)

    # ---- decode steps ------------------------------------------------------------
    ws = cache.workspace(pk.PKV_OP_ATTENTION, T + n_steps + 1)
    out = torch.empty((B, Hq, d), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    qs = [torch.from_numpy(synth.queries(wl, args.seed, s)).to("cuda", bf).contiguous() for s in range(n_steps)]
    toks = [tuple(torch.from_numpy(x).to("cuda", bf).contiguous() for x in synth.decode_kv(wl, args.seed, 0, T + s))
            for s in range(n_steps)]
    stream = torch.cuda.current_stream()
    # every event is created (and one pair exercised) before the timed region
    pool = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps * layers)]
    pool[0][0].record(stream)
    pool[0][1].record(stream)
    step_marks = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize()
    call_events = []
    comp_events = []   # (start, end, page pairs) of the compress calls in the timed steps
    step_start = step_end = None
    compress_calls = 0
    # the host only enqueues in the timed loop; a garbage-collector pass there
    # could leave the GPU idle between a call's start event and its launch
    import gc
    gc.collect()
    gc.disable()
    for s in range(n_steps):
        timed = s >= args.warmup
        if s == args.warmup:
            torch.cuda.synchronize()
            step_start = step_marks[0]
            step_start.record(stream)
        pos = T + s
        new_pages = pk.eligible_pages(pos, pos + 1, P, S, W)
        for layer in range(layers):
            cache.append(layer, toks[s][0], toks[s][1], [pos] * B)
            if len(new_pages):
                bb, hh, jj = zip(*[(b, h, int(j)) for b in range(B) for h in range(Hkv) for j in new_pages])
                rr = [int(req_np[b, h, j]) for b, h, j in zip(bb, hh, jj)]
                rv = [int(req_v_np[b, h, j]) for b, h, j in zip(bb, hh, jj)]
                if timed:
                    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    c0.record(stream)
                cache.compress_pages(layer, bb, hh, jj, rr, rv)
                if timed:
                    c1.record(stream)
                    comp_events.append((c0, c1, len(bb)))
                compress_calls += 1
            # the attention's duration: events around every eighth layer's call
            # (events around every call added ~0.2-0.4 ms per 64-layer step of
            # their own to the step time)
            ev = timed and layer % EVENT_STRIDE == 0
            if ev:
                e0, e1 = pool[len(call_events)]
                e0.record(stream)
            cache.attention(layer, qs[s], [pos + 1] * B, out=out, lse=lse, workspace=ws)
            if ev:
                e1.record(stream)
                call_events.append((e0, e1))
        if s == 0:
            torch.cuda.synchronize()
            log("first step done")
    step_end = step_marks[1]
    step_end.record(stream)
    torch.cuda.synchronize()
    gc.enable()
    status |= cache.device_status()
    ms_total = step_start.elapsed_time(step_end)
    ms_per_step = ms_total / args.steps
    call_ms = np.array([a.elapsed_time(b) for a, b in call_events])
    attn_us = float(call_ms.mean() * 1e3)
    pct = np.percentile(call_ms * 1e3, [10, 50, 90, 99])
    log("decode: %.3f ms/step, attention %.1f us/layer (p10 %.1f, median %.1f, p90 %.1f, p99 %.1f, max %.1f), "
        "status %d" % (ms_per_step, attn_us, pct[0], pct[1], pct[2], pct[3], float(call_ms.max() * 1e3), status))
    per_step = call_ms.reshape(args.steps, -1).mean(axis=1) * 1e3
    log("attention us/layer by timed step: " + " ".join("%.1f" % x for x in per_step))
    if not np.isfinite(out.float().cpu().numpy()).all():
        raise RuntimeError("non-finite attention output")

    comp_decode = None
    if comp_events:
        cms = sum(a.elapsed_time(b) for a, b, _ in comp_events)
        npairs = sum(n for _, _, n in comp_events)
        comp_decode = {"calls": len(comp_events), "page_pairs": npairs, "ms_total": round(cms, 3),
                       "page_pairs_per_s": round(npairs / (cms * 1e-3), 1)}
        log("compress during the timed steps: %d calls, %d page pairs, %.3f ms, %.3g page pairs/s"
            % (len(comp_events), npairs, cms, npairs / (cms * 1e-3)))

    if wl.rank_error > 0:   # ranks of the pages compressed during the decode steps too
        ranks_np, ranks_v_np = chosen_ranks(cache, pk.plan_pages(T + n_steps, P, S, W), max_pages, wl.rank_error)
    mid_T = T + args.warmup + args.steps // 2 + 1
    abytes = attention_bytes(wl.factors, ranks_np, ranks_v_np, [mid_T] * B, P, d, B, Hkv, Hq, S, W)
    achieved = abytes / (attn_us * 1e-6) / 1e9
    traffic = measured_traffic(wl.name)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": traffic}

    metrics = {
        "qwen32b_128k": "mixed-page decode attention time per decode step (64 layers, Qwen3-32B heads, 128K context)",
        "qwen8b_paper_default": "mixed-page decode attention time per decode step (36 layers, Qwen3-8B heads, "
                                "16K context, pages of 32 tokens, (r_K, r_V) = (16, 14))",
        "qwen32b_128k_adaptive": "mixed-page decode attention time per decode step (64 layers, Qwen3-32B "
                                 "heads, 128K context, page ranks chosen for relative error 0.2)",
        "qwen32b_128k_prerope": "mixed-page decode attention time per decode step (64 layers, Qwen3-32B "
                                "heads, 128K context, keys cached before RoPE and rotated at access)",
        "qwen32b_int4": "mixed-page decode attention time per decode step (INT4 factor pages, Qwen3-32B heads, "
                        "128K context, batch 8)",
        "qwen32b_128k_tp8": "mixed-page decode attention time per decode step (64 layers, one GPU's share of "
                            "Qwen3-32B heads under 8-way tensor parallelism: 1 KV head, 8 query heads, 128K "
                            "context)",
    }
    result = {
        "metric": metrics.get(wl.name, "mixed-page decode attention time per decode step"),
        "value": round(ms_per_step * 1e3, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.factors == "bf16" else "int4 factors, fp16/bf16 MFMA, fp32 accumulate",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
                   "page": P, "tokens": T, "sink": S, "window": W, "ranks": list(wl.ranks), "ranks_v": list(wl.ranks_v or wl.ranks),
                   "rank_error": wl.rank_error, "keys_before_rope": wl.key_rope,
                   "factor_storage": wl.factors,
                   "layers": layers, "step": "append + planner + compress-when-eligible + attention per layer"},
        "attention_us_per_layer": round(attn_us, 2),
        "attention_us_median": round(float(pct[1]), 2),
        "attention_us_p90": round(float(pct[2]), 2),
        "attention_samples": int(call_ms.size),
        "attention_algorithmic_bytes": int(abytes),
        "attention_gbps": round(achieved, 1),
        "compress_page_pairs_per_s": round(pages_per_s, 1),
        "compress_decompositions_per_s": round(2 * pages_per_s, 1),
        "compress_ms_per_layer_prefill": round(comp_ms_best, 3),
        "compress_sweeps_per_decomposition": round(comp["sweeps"], 3),
        "compress_useful_tflops": round(comp["useful"] / comp_ms_best / 1e9, 3),
        "compress_executed_tflops": round(comp["executed"] / comp_ms_best / 1e9, 3),
        "compress_calls_in_run": compress_calls,
        "footprint_ratio": round(fp_ratio, 5),
        "footprint_ratio_slots": round(fp_slots, 5),
        "device_status": status,
        "roofline": roofline,
    }
    if comp_decode:
        result["compress_during_decode"] = comp_decode
    if not args.no_calibration:
        result["hbm_calibration"] = hbm_calibration(achieved)
    if args.cpu_seconds > 0:
        log("CPU baseline (oracle), budget %.0f s" % args.cpu_seconds)
        q0 = synth.queries(wl, args.seed, 0)
        result["cpu_baseline"] = cpu_baseline(wl, args.seed, T, K_dense, V_dense, q0, args.cpu_seconds,
                                              layers, ranks_np, ranks_v_np)
        # the ranks the cache holds (requested, or chosen by the decomposition)
        result["cpu_baseline"].update(cpu_extras(wl, args.seed, T, K_dense, V_dense, q0, comp_X, ranks_np,
                                                 ranks_v_np, comp_refs))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
