// Batched per-page truncated decomposition (Section 3.3: the Gram matrix
// G = X X^T of a P x d page, its top-r eigenvectors L, and R = L^T X, which
// equal the rank-r truncated-SVD factors of Eq. (2) because P < d).
//
// One wavefront handles 64 / P decompositions; inside a group of P lanes,
// lane c owns column c of G and column c of the accumulated rotation J, both
// in registers. The eigenvectors come from one-sided Jacobi on G: pairs of
// columns are rotated until they are orthogonal, using the xor ordering
// (step m pairs column c with column c ^ m, m = 1 .. P-1), so the partner is
// always one lane-xor away and every pair meets once per sweep. At
// convergence G J = J diag(lambda) and lambda_c = j_c . (G j_c).
// Included by pkv_kernels.hip.

namespace pkv {

constexpr int kMaxSweeps = 32;

enum { SRC_CACHE = 0, SRC_PREFILL = 1 };

struct CompressSrc {
    int mode;
    const void *k, *v;        // prefill source [B][Hkv][src_tokens][d]
    int64_t src_tokens;
    SeqArgs off;              // prefill: item offset of sequence b (off.len[B] = total)
    const uint8_t *rank_k, *rank_v;
    int def_rk, def_rv;
    const CompressItem *list;   // compress: the items in device memory, when set (else the launch's items);
                                // the matrix-core kernel takes it through its kList instantiation
};

__device__ inline float wave_shfl_xor(float v, int m) { return __shfl_xor(v, m, 64); }

// Factor storage marker for INT4 pages (balanced, quantized factors).
struct q4_t {};
template <typename TF> struct is_q4 { static constexpr bool value = false; };
template <> struct is_q4<q4_t> { static constexpr bool value = true; };

// One decomposition of a compress or prefill launch: which page, which half
// (K or V), its ranks and where its P x d values are. A page that may not be
// factorized now (compress mode: not dense, incomplete, in the sink or still
// inside the window) raises its status bit when `report` is set and leaves
// the decomposition inactive.
struct DecompRef {
    bool active;
    int b, h, j, rk, rv, which;
    const void *X;
    bool transposed;   // X is V^T (d x P), the dense slot's value layout
};

// kList: compress items come from src.list (device memory), else from the
// launch's items (a template parameter: the runtime choice cost the
// register-bound decomposition kernel a spill).
template <typename TX, bool kList = false>
__device__ inline DecompRef decode_decomp(const Geo &g, const pkv_page *table, const char *dense,
                                          const CompressItems &items, const CompressSrc &src, int64_t q,
                                          int64_t n_decomp, bool report) {
    DecompRef r{};
    r.active = q < n_decomp;
    r.rk = r.rv = 1;
    r.which = (int)(q & 1);
    if (!r.active) return r;
    const int64_t item = q >> 1;
    if (src.mode == SRC_CACHE) {
        const CompressItem it = kList ? src.list[item] : items.it[item];
        r.b = it.b; r.h = it.h; r.j = it.j; r.rk = it.rk; r.rv = it.rv;
        const int64_t head = g.head_index(r.b, r.h);
        const pkv_page e = table[head * g.max_pages + r.j];
        const unsigned int refusal = compress_refusal(g, table, head, r.j);
        if (refusal) {
            if (report) raise_status(refusal);
            r.active = false;
        } else {
            const TX *slot = (const TX *)(dense + e.slot * g.dense_slot_bytes);
            r.X = r.which == 0 ? slot : slot + (int64_t)g.P * g.d;
            r.transposed = r.which == 1;
        }
    } else {
        int bb = 0;
        while (bb + 1 < src.off.n - 1 && src.off.len[bb + 1] <= item) ++bb;
        const int64_t local = item - src.off.len[bb];
        const int64_t nf = (src.off.len[bb + 1] - src.off.len[bb]) / g.Hkv;
        r.b = bb;
        r.h = (int)(local / nf);
        r.j = g.sink_pages + (int)(local % nf);
        const int64_t head = g.head_index(r.b, r.h);
        if (src.rank_k) {
            const int rmax = min(g.max_rank, min(g.P, g.d));
            const int rmin = g.rank_err > 0.f ? 0 : 1;   // 0: chosen per page
            r.rk = max(rmin, min((int)src.rank_k[head * g.max_pages + r.j], rmax));
            r.rv = max(rmin, min((int)src.rank_v[head * g.max_pages + r.j], rmax));
        } else {
            r.rk = src.def_rk;
            r.rv = src.def_rv;
        }
        const TX *base = (const TX *)(r.which == 0 ? src.k : src.v);
        r.X = base + (head * src.src_tokens + (int64_t)r.j * g.P) * g.d;
    }
    return r;
}

template <typename TX, typename TF, int P>
__global__ __launch_bounds__(64) void k_compress(Geo g, pkv_page *table, const char *dense, char *factor,
                                                 CompressItems items, CompressSrc src, int64_t n_decomp) {
    constexpr int D = 64 / P;                           // decompositions per wave
    constexpr int PAD = sizeof(TX) == 2 ? 2 : 1;        // one dword of row padding
    extern __shared__ unsigned char smem_raw[];
    const int d = g.d, ld_x = d + PAD;
    TX *sX_all = (TX *)smem_raw;

    const int lane = threadIdx.x;
    const int grp = lane / P, c = lane % P;
    const int64_t q = (int64_t)blockIdx.x * D + grp;    // decomposition index
    TX *sX = sX_all + (int64_t)grp * P * ld_x;

    // ---- which page, which half (K or V), ranks, source --------------------
    const DecompRef ref = src.list ? decode_decomp<TX, true>(g, table, dense, items, src, q, n_decomp, c == 0)
                                   : decode_decomp<TX, false>(g, table, dense, items, src, q, n_decomp, c == 0);
    bool active = ref.active;
    const int b = ref.b, h = ref.h, j = ref.j, rk = ref.rk, rv = ref.rv, which = ref.which;
    const TX *X = (const TX *)ref.X;
    const bool transposed = ref.transposed;

    // ---- stage X (P x d) in LDS -------------------------------------------
    if (active) {
        if (!transposed) {
            for (int i = c; i < P * d; i += P) sX[(i / d) * ld_x + (i % d)] = X[i];
        } else {
            for (int i = c; i < P * d; i += P) {      // X[t][k] = Vt[k][t]
                const int k = i / P, t = i % P;
                sX[t * ld_x + k] = X[i];
            }
        }
    }
    __syncthreads();

    // ---- Gram column c: G[k][c] = x_k . x_c ---------------------------------
    float gcol[P], jcol[P];
#pragma unroll
    for (int k = 0; k < P; ++k) { gcol[k] = 0.f; jcol[k] = (k == c) ? 1.f : 0.f; }
    if (active) {
        for (int kk = 0; kk < d; ++kk) {
            const float xc = to_f32(sX[c * ld_x + kk]);
#pragma unroll
            for (int k = 0; k < P; ++k) gcol[k] = fmaf(to_f32(sX[k * ld_x + kk]), xc, gcol[k]);
        }
    }

    // ---- one-sided Jacobi on G ---------------------------------------------
    // Columns are carried as d_c * g~_c (and d_c * j~_c: J takes the same
    // rotations, so the same scale). Rotating the pair (c, p) by (cs, sn) is
    // then g~_c += mu g~_p, d_c *= cs with mu = +-tan * d_p / d_c: one fma per
    // element of G and of J instead of two. |g_c|^2 is carried along (from
    // the pair's alpha, beta, gamma) and recomputed, with the scales folded
    // back in, at the start of every sweep. G is first divided by its
    // Frobenius norm, so no scaled entry can overflow within a sweep
    // (d_c >= 2^-32 after 63 rotations).
    float nrm2 = 0.f;
#pragma unroll
    for (int k = 0; k < P; ++k) nrm2 = fmaf(gcol[k], gcol[k], nrm2);
    float fro2 = nrm2;
    for (int m = 1; m < P; m <<= 1) fro2 += wave_shfl_xor(fro2, m);
    const float gnorm = sqrtf(fro2);
    const float ginv = fro2 > 0.f ? 1.f / gnorm : 0.f;
#pragma unroll
    for (int k = 0; k < P; ++k) gcol[k] *= ginv;
    // Rotation threshold P 2^-23 on the cosine of two columns; for factors
    // stored in bf16 ten times that (two sweeps fewer of ~12, the rank-r
    // reconstruction moving by ~1e-4 |X|, far below bf16 rounding). fp32
    // factors keep the tight threshold.
    constexpr float kTolFactor = std::is_same<TF, uint16_t>::value ? 10.f : 1.f;
    const float tol = kTolFactor * (float)P * 1.1920929e-7f;
    const float tiny2 = fro2 > 0.f ? tol * tol : 0.f;  // relative to |G|_F^2 = 1

    // Only the top r eigenvectors are stored, and a column whose G-image is
    // orthogonal to every other column's is an exact eigenvector whatever
    // the remaining pairs do (G j_c _|_ G j_p for all p gives G^2 j_c || j_c).
    // So a sweep counts as converged when no pair involving one of the r
    // columns of largest |G j| (ranked during the previous sweep; all
    // columns in the first) still needed a rotation.
    const int r_need = which == 0 ? rk : rv;
    float dsc = 1.f, alpha = 0.f;
    bool top = true;
    int sweeps = 0;
    bool more = true;
    while (more && sweeps < kMaxSweeps) {
        ++sweeps;
        int larger = 0;   // columns ranked above this one during this sweep
        alpha = 0.f;
#pragma unroll
        for (int k = 0; k < P; ++k) {
            gcol[k] *= dsc;
            jcol[k] *= dsc;
            alpha = fmaf(gcol[k], gcol[k], alpha);
        }
        dsc = 1.f;
        int rotated = 0;
        for (int m = 1; m < P; ++m) {
            float pg[P];
            float gt = 0.f;
#pragma unroll
            for (int k = 0; k < P; ++k) {
                pg[k] = wave_shfl_xor(gcol[k], m);
                gt = fmaf(gcol[k], pg[k], gt);
            }
            const float beta = wave_shfl_xor(alpha, m);
            const float dp = wave_shfl_xor(dsc, m);
            const int top_p = __shfl_xor(top ? 1 : 0, m, 64);
            larger += (beta > alpha || (beta == alpha && (c ^ m) < c)) ? 1 : 0;
            const float gamma = gt * dsc * dp;
            const bool lo = c < (c ^ m);
            const float a_lo = lo ? alpha : beta, a_hi = lo ? beta : alpha;
            // rotation parameters without branches; the hardware reciprocal
            // and reciprocal square root (about 1 ulp) suffice here, the
            // eigenvectors are renormalized at the end
            const bool rot = a_lo > tiny2 && a_hi > tiny2 && fabsf(gamma) > tol * sqrtf(a_lo * a_hi);
            const float zeta = (a_hi - a_lo) * __builtin_amdgcn_rcpf(2.f * gamma);
            const float tz = __builtin_copysignf(
                __builtin_amdgcn_rcpf(fabsf(zeta) + __builtin_amdgcn_sqrtf(fmaf(zeta, zeta, 1.f))), zeta);
            const float t = rot ? tz : 0.f;
            const float cs = rot ? __builtin_amdgcn_rsqf(fmaf(t, t, 1.f)) : 1.f;
            rotated |= (rot && (top || top_p)) ? 1 : 0;
            const float t_eff = lo ? -t : t;       // the lower column takes -sn
            const float mu = t_eff * (dp * __builtin_amdgcn_rcpf(dsc));
#pragma unroll
            for (int k = 0; k < P; ++k) gcol[k] = fmaf(mu, pg[k], gcol[k]);
#pragma unroll
            for (int k = 0; k < P; ++k) {
                const float pj = wave_shfl_xor(jcol[k], m);
                jcol[k] = fmaf(mu, pj, jcol[k]);
            }
            const float s_eff = cs * t_eff;
            alpha = fmaf(cs * cs, alpha, fmaf(2.f * cs * s_eff, gamma, s_eff * s_eff * beta));
            dsc *= cs;
        }
        const bool top_new = larger < r_need;
        more = __any(rotated || top_new != top);   // converged only on a settled ranking
        top = top_new;
    }
    if (active && c == 0) {
        count_sweeps(sweeps);
        if (more) raise_status(PKV_DEV_NO_CONVERGE);
    }
#pragma unroll
    for (int k = 0; k < P; ++k) {
        gcol[k] *= dsc * gnorm;   // back to G J
        jcol[k] *= dsc;
    }

    // ---- eigenvalues, order (descending; ties keep the lower index) --------
    // Rotations by tiny angles round cos to 1 and grow |j_c| slightly, so each
    // eigenvector is renormalized; lambda_c is the Rayleigh quotient.
    float jn2 = 0.f, lam = 0.f;
#pragma unroll
    for (int k = 0; k < P; ++k) {
        jn2 = fmaf(jcol[k], jcol[k], jn2);
        lam = fmaf(jcol[k], gcol[k], lam);
    }
    lam /= jn2;
    const float jinv = 1.f / sqrtf(jn2);
#pragma unroll
    for (int k = 0; k < P; ++k) jcol[k] *= jinv;
    int rho = 0;
    const int base = grp * P;
    for (int k = 0; k < P; ++k) {
        const float lk = __shfl(lam, base + k, 64);
        rho += (lk > lam) || (lk == lam && k < c);
    }

    if (!active) return;

    // ---- outputs ------------------------------------------------------------
    const int rk4 = r4(rk), rv4 = r4(rv);
    const FactorLayout fl = factor_layout(P, d, rk, rv);
    TF *Ak = (TF *)(factor + (g.head_index(b, h) * g.max_pages + j) * g.factor_slot_bytes);
    TF *Bk = Ak + fl.bk, *Bvt = Ak + fl.bvt, *Avt = Ak + fl.avt;
    const int r = which == 0 ? rk : rv;
    const int rr4 = which == 0 ? rk4 : rv4;
    if (which == 0) {
        if (rho < rk4)
            for (int t = 0; t < P; ++t) st(Ak, (int64_t)t * rk4 + rho, rho < rk ? jcol[t] : 0.f);
    } else {
        if (rho < rv)
            for (int t = 0; t < P; ++t) st(Avt, (int64_t)rho * P + t, jcol[t]);
    }
    // R row rho = sum_t L[t][rho] X[t][:], in chunks of 16 columns
    for (int k0 = 0; k0 < d; k0 += 16) {
        float acc[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) acc[u] = 0.f;
        for (int t = 0; t < P; ++t) {
            const float lt = jcol[t];
#pragma unroll
            for (int u = 0; u < 16; ++u) acc[u] = fmaf(lt, to_f32(sX[t * ld_x + k0 + u]), acc[u]);
        }
        if (which == 0) {
            if (rho < rk)
#pragma unroll
                for (int u = 0; u < 16; ++u) st(Bk, (int64_t)rho * d + k0 + u, acc[u]);
        } else {
            if (rho < rv4)
#pragma unroll
                for (int u = 0; u < 16; ++u) st(Bvt, (int64_t)(k0 + u) * rv4 + rho, rho < rv ? acc[u] : 0.f);
        }
    }
    (void)r; (void)rr4;
}

template <typename TX, typename TF, int P>
hipError_t launch_compress_t(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                             int64_t n_decomp) {
    constexpr int D = 64 / P;
    const int pad = sizeof(TX) == 2 ? 2 : 1;
    size_t smem = (size_t)D * P * (L.geo.d + pad) * sizeof(TX);
    const int64_t blocks = ceil_div(n_decomp, D);
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL((k_compress<TX, TF, P>), dim3((unsigned)blocks), dim3(64), smem, L.stream, L.geo,
                       p.table, p.dense, p.factor, items, src, n_decomp);
    return hipGetLastError();
}

template <typename TX, typename TF>
hipError_t launch_compress_p(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                             int64_t n_decomp) {
    switch (L.geo.P) {
    case 16: return launch_compress_t<TX, TF, 16>(L, items, src, n_decomp);
    case 32: return launch_compress_t<TX, TF, 32>(L, items, src, n_decomp);
    case 64: return launch_compress_t<TX, TF, 64>(L, items, src, n_decomp);
    default: return hipErrorInvalidValue;
    }
}

inline bool compress_qr_supported(const Geo &g);
hipError_t launch_compress_qr(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                              int64_t n_decomp);

// bf16 pages of 32 or 64 tokens take the matrix-core path (k_compress_qr);
// fp32 pages and 16-token pages the one-wave Gram + Jacobi kernel above.
hipError_t launch_compress_any(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                               int64_t n_decomp) {
    if (n_decomp <= 0) return hipSuccess;
    if (compress_qr_supported(L.geo)) return launch_compress_qr(L, items, src, n_decomp);
    if (L.geo.key_t) return hipErrorInvalidValue;   // R_K^T slots: stored by the matrix-core kernel only
    // INT4 caches are validated to bf16 pages of 64 tokens with d = 128: the
    // matrix-core kernel above always takes them
    if (L.geo.factor_dtype == PKV_INT4) return hipErrorInvalidValue;
    const bool db = L.geo.dense_dtype == PKV_BF16, fb = L.geo.factor_dtype == PKV_BF16;
    if (db && fb) return launch_compress_p<uint16_t, uint16_t>(L, items, src, n_decomp);
    if (db) return launch_compress_p<uint16_t, float>(L, items, src, n_decomp);
    if (fb) return launch_compress_p<float, uint16_t>(L, items, src, n_decomp);
    return launch_compress_p<float, float>(L, items, src, n_decomp);
}

hipError_t launch_compress(const LaunchCtx &L, const CompressItems &items) {
    CompressSrc src{};
    src.mode = SRC_CACHE;
    return launch_compress_any(L, items, src, 2LL * items.n);
}

hipError_t launch_compress_list(const LaunchCtx &L, const CompressItem *list, int64_t n) {
    CompressItems items{};
    CompressSrc src{};
    src.mode = SRC_CACHE;
    src.list = list;
    return launch_compress_any(L, items, src, 2 * n);
}

hipError_t launch_prefill_compress(const LaunchCtx &L, const void *k, const void *v, int64_t src_tokens,
                                   const int32_t *item_offsets, int64_t n_items, const uint8_t *rank_k,
                                   const uint8_t *rank_v, int def_rk, int def_rv) {
    CompressItems items{};
    CompressSrc src{};
    src.mode = SRC_PREFILL;
    src.k = k;
    src.v = v;
    src.src_tokens = src_tokens;
    src.off.n = L.geo.B + 1;
    for (int i = 0; i <= L.geo.B; ++i) src.off.len[i] = item_offsets[i];
    src.rank_k = rank_k;
    src.rank_v = rank_v;
    src.def_rk = def_rk;
    src.def_rv = def_rv;
    return launch_compress_any(L, items, src, 2 * n_items);
}

}  // namespace pkv
