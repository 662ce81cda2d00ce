// Mixed-page decode attention on the matrix cores (bf16 pages and factors,
// d = 64 or 128, P = 16, 32 or 64, ranks <= 32, query group <= 16).
//
// One wavefront owns one (sequence, KV head) and a chunk of pages. All four
// contractions of a factor page (Eq. (4)) are 16x16x32 bf16 MFMAs with the
// query group in the N dimension:
//   Z^T = R_K Q^T        (M = rank,  K = d)       R_K   stored r x d
//   S^T = L_K Z^T        (M = token, K = rank)    L_K   stored P x r4
//   Y^T = L_V^T E^T      (M = rank,  K = token)   L_V^T stored r x P
//   O^T += R_V^T Y^T     (M = dim,   K = rank)    R_V^T stored d x r4
// Each stored operand has its contraction index contiguous, so every lane
// loads its A-operand slice straight from HBM. The accumulator layout of one
// product (lane l holds rows 4(l/16)..4(l/16)+3 of column l%16 of each 16-row
// tile) is reused as the B operand of the next: two 16-row tiles give a lane
// exactly the 8 K-entries {4(l/16)+e} and {16+4(l/16)+e}, so the A operand is
// read in that same permuted K order (two 8-byte loads) and no data moves
// between lanes. fp32 intermediates (Z, exp weights, Y) enter the MFMA as a
// bf16 hi/lo pair (two MFMAs), keeping about 16 mantissa bits; Q and the
// stored pages are exact in bf16. Dense pages use S^T = K Q^T and
// O^T += V^T E^T with V stored transposed.
// Included by pkv_kernels.hip.

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kRescaleLog2 = 8.0f;   // keep the running max until a page exceeds it by 2^8

__device__ inline f32x4 mfma_bf16(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8 ld_b8(const uint16_t *p) { return *(const bf16x8 *)p; }
__device__ inline bf16x4 ld_b4(const uint16_t *p) { return *(const bf16x4 *)p; }
__device__ inline bf16x8 cat4(const bf16x4 &a, const bf16x4 &b) {
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ inline bf16x4 zero4() { return bf16x4{0, 0, 0, 0}; }
__device__ inline bf16x8 zero8() { return bf16x8{0, 0, 0, 0, 0, 0, 0, 0}; }

// 8 fp32 values (two accumulator tiles) -> bf16 hi + lo operands.
__device__ inline void split_hi_lo(const f32x4 &x0, const f32x4 &x1, bf16x8 &hi, bf16x8 &lo) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const __bf16 h0 = (__bf16)x0[e];
        const __bf16 h1 = (__bf16)x1[e];
        hi[e] = h0;
        hi[4 + e] = h1;
        lo[e] = (__bf16)(x0[e] - (float)h0);
        lo[4 + e] = (__bf16)(x1[e] - (float)h1);
    }
}

template <int D, int P>
__global__ __launch_bounds__(64) void k_attn_mfma(Geo g, const pkv_page *table, const char *dense,
                                                  const char *factor, const uint16_t *q, SeqArgs seq,
                                                  int ppc, int n_chunks, float *part,
                                                  unsigned int *counters, float *out, float *lse) {
    constexpr int KD = D / 32;         // K-steps over the head dimension
    constexpr int DT = D / 16;         // 16-row tiles over the head dimension
    constexpr int TT = P / 16;         // 16-row tiles over the page tokens
    constexpr int KS = (P + 31) / 32;  // K-steps over the page tokens

    const int chunk = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    const int G = g.g;
    const int lane = threadIdx.x;
    const int n = lane & 15, j4 = lane >> 4;
    const int64_t T = seq.len[b];
    const int64_t n_pages = ceil_div(T, P);
    const int64_t j0 = (int64_t)chunk * ppc;
    const int64_t j1 = min<int64_t>(j0 + ppc, n_pages);
    const float c2 = kLog2e / sqrtf((float)D);

    // query group as the B operand (K = d, N = query head)
    bf16x8 qb[KD];
    {
        const uint16_t *qp = q + ((int64_t)b * g.Hq + (int64_t)h * G + n) * D + 8 * j4;
#pragma unroll
        for (int s = 0; s < KD; ++s) qb[s] = n < G ? ld_b8(qp + 32 * s) : zero8();
    }

    f32x4 o[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_part = 0.f;

    for (int64_t j = j0; j < j1; ++j) {
        const pkv_page e = table[head * g.max_pages + j];
        const int rows = (int)min<int64_t>(P, T - j * P);
        f32x4 st[TT];
        bf16x8 eh[KS], el[KS];

        // online softmax over this page's scores st (scaled to log2 units here)
        auto softmax = [&](void) {
            float pm = -INFINITY;
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int tok = 16 * tt + 4 * j4 + v;
                    const float s = tok < rows ? st[tt][v] * c2 : -INFINITY;
                    st[tt][v] = s;
                    pm = fmaxf(pm, s);
                }
            pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
            pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
            if (pm > m_run + kRescaleLog2 || m_run == -INFINITY) {
                const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - pm);
#pragma unroll
                for (int t = 0; t < DT; ++t) o[t] *= alpha;
                l_part *= alpha;
                m_run = pm;
            }
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float ex = exp2f(st[tt][v] - m_run);
                    st[tt][v] = ex;
                    l_part += ex;
                }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const f32x4 z4 = f32x4{0.f, 0.f, 0.f, 0.f};
                split_hi_lo(st[2 * ks], 2 * ks + 1 < TT ? st[2 * ks + 1] : z4, eh[ks], el[ks]);
            }
        };

        if (e.kind == PKV_FACTOR) {
            const int rk = e.rank_k, rv = e.rank_v, rk4 = r4(rk), rv4 = r4(rv);
            const uint16_t *Ak = (const uint16_t *)(factor + e.slot * g.factor_slot_bytes);
            const uint16_t *Bk = Ak + (int64_t)P * rk4;
            const uint16_t *Avt = Bk + (int64_t)rk * D;
            const uint16_t *Bvt = Avt + (int64_t)rv * P;

            // ---- issue every load of the page ------------------------------
            bf16x8 bk[2][KD];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const int row = 16 * rt + n;
#pragma unroll
                for (int s = 0; s < KD; ++s)
                    bk[rt][s] = row < rk ? ld_b8(Bk + (int64_t)row * D + 32 * s + 8 * j4) : zero8();
            }
            bf16x8 ak[TT];
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                const uint16_t *ap = Ak + (int64_t)(16 * tt + n) * rk4;
                ak[tt] = cat4(4 * j4 < rk4 ? ld_b4(ap + 4 * j4) : zero4(),
                              16 + 4 * j4 < rk4 ? ld_b4(ap + 16 + 4 * j4) : zero4());
            }
            bf16x8 av[2][KS];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const int row = 16 * rt + n;
                const uint16_t *ap = Avt + (int64_t)row * P;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    av[rt][ks] = cat4(row < rv ? ld_b4(ap + 32 * ks + 4 * j4) : zero4(),
                                      (row < rv && 32 * ks + 16 < P) ? ld_b4(ap + 32 * ks + 16 + 4 * j4)
                                                                      : zero4());
            }
            bf16x8 bv[DT];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const uint16_t *bp = Bvt + (int64_t)(16 * dt + n) * rv4;
                bv[dt] = cat4(4 * j4 < rv4 ? ld_b4(bp + 4 * j4) : zero4(),
                              16 + 4 * j4 < rv4 ? ld_b4(bp + 16 + 4 * j4) : zero4());
            }

            // ---- Z^T = R_K Q^T --------------------------------------------
            f32x4 z[2];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                z[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (rk > 16 * rt)
#pragma unroll
                    for (int s = 0; s < KD; ++s) z[rt] = mfma_bf16(bk[rt][s], qb[s], z[rt]);
            }
            bf16x8 zh, zl;
            split_hi_lo(z[0], z[1], zh, zl);
            // ---- S^T = L_K Z^T ----------------------------------------------
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                st[tt] = mfma_bf16(ak[tt], zh, f32x4{0.f, 0.f, 0.f, 0.f});
                st[tt] = mfma_bf16(ak[tt], zl, st[tt]);
            }
            softmax();
            // ---- Y^T = L_V^T E^T ----------------------------------------------
            f32x4 y[2];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                y[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (rv > 16 * rt)
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) {
                        y[rt] = mfma_bf16(av[rt][ks], eh[ks], y[rt]);
                        y[rt] = mfma_bf16(av[rt][ks], el[ks], y[rt]);
                    }
            }
            bf16x8 yh, yl;
            split_hi_lo(y[0], y[1], yh, yl);
            // ---- O^T += R_V^T Y^T ---------------------------------------------
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                o[dt] = mfma_bf16(bv[dt], yh, o[dt]);
                o[dt] = mfma_bf16(bv[dt], yl, o[dt]);
            }
        } else if (e.kind == PKV_DENSE) {
            const uint16_t *K = (const uint16_t *)(dense + e.slot * g.dense_slot_bytes);
            const uint16_t *Vt = K + (int64_t)P * D;
            bf16x8 kk[TT][KD];
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int s = 0; s < KD; ++s) kk[tt][s] = ld_b8(K + (int64_t)(16 * tt + n) * D + 32 * s + 8 * j4);
            bf16x8 vv[DT][KS];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const uint16_t *vp = Vt + (int64_t)(16 * dt + n) * P;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const int t0 = 32 * ks + 4 * j4, t1 = 32 * ks + 16 + 4 * j4;
                    bf16x4 lo = ld_b4(vp + t0);
                    bf16x4 hi = 32 * ks + 16 < P ? ld_b4(vp + t1) : zero4();
#pragma unroll
                    for (int u = 0; u < 4; ++u) {   // rows past the sequence may hold anything
                        if (t0 + u >= rows) lo[u] = (__bf16)0.f;
                        if (t1 + u >= rows) hi[u] = (__bf16)0.f;
                    }
                    vv[dt][ks] = cat4(lo, hi);
                }
            }
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                st[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < KD; ++s) st[tt] = mfma_bf16(kk[tt][s], qb[s], st[tt]);
            }
            softmax();
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    o[dt] = mfma_bf16(vv[dt][ks], eh[ks], o[dt]);
                    o[dt] = mfma_bf16(vv[dt][ks], el[ks], o[dt]);
                }
        } else {
            if (lane == 0) raise_status(PKV_DEV_BAD_PAGE);
        }
    }

    // ---- partial state of the chunk ---------------------------------------
    l_part += __shfl_xor(l_part, 16, 64);
    l_part += __shfl_xor(l_part, 32, 64);
    if (n < G) {
        const int64_t p = partial_index(head, chunk, n_chunks, n, G, D);
        if (j4 == 0) {
            part[p] = m_run;
            part[p + 1] = l_part;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int v = 0; v < 4; ++v) part[p + 2 + 16 * dt + 4 * j4 + v] = o[dt][v];
    }
    publish_and_merge(g, head, n_chunks, part, counters, out, lse, T, lane);
}

inline bool mfma_supported(const Geo &g) {
    return g.dense_dtype == PKV_BF16 && g.factor_dtype == PKV_BF16 && (g.d == 64 || g.d == 128) &&
           (g.P == 16 || g.P == 32 || g.P == 64) && g.max_rank <= 32 && g.g <= 16;
}

hipError_t launch_attn_mfma(const LaunchCtx &L, const AttnPlan &plan, const uint16_t *q, const SeqArgs &seq,
                            float *part, unsigned int *counters, float *out, float *lse) {
    LayerPtrs p = layer_ptrs(L);
    const Geo &g = L.geo;
    dim3 grid(plan.n_chunks, g.B * g.Hkv);
#define PKV_LAUNCH_MFMA(DD, PP)                                                                          \
    hipLaunchKernelGGL((k_attn_mfma<DD, PP>), grid, dim3(64), 0, L.stream, g, p.table, p.dense, p.factor, q, \
                       seq, plan.pages_per_chunk, plan.n_chunks, part, counters, out, lse)
    if (g.d == 128) {
        if (g.P == 64) PKV_LAUNCH_MFMA(128, 64);
        else if (g.P == 32) PKV_LAUNCH_MFMA(128, 32);
        else PKV_LAUNCH_MFMA(128, 16);
    } else {
        if (g.P == 64) PKV_LAUNCH_MFMA(64, 64);
        else if (g.P == 32) PKV_LAUNCH_MFMA(64, 32);
        else PKV_LAUNCH_MFMA(64, 16);
    }
#undef PKV_LAUNCH_MFMA
    return hipGetLastError();
}

}  // namespace pkv
