// Global SVD, the paper's controlled baseline for compression granularity
// (Section 4.1 "Baselines"; Section 4.2 "Main Results"; Appendix "Baseline
// Configurations"): for each (layer, sequence, KV head) and each of K and V,
// one rank-r basis shared by every token of the compressible region (the
// pages the plan factorizes; sink and window pages stay dense as in
// PuzzleKV). With X the region (N x d):
//   G = X^T X (d x d)                          k_global_gram, matrix cores
//   B = W_r^T, the top-r eigenvectors of G     k_global_eigen, one-sided Jacobi
//   A = X B^T (N x r), one row per token       k_global_project, matrix cores
// so X ~ A B (A = U_r Sigma_r, B = W_r^T: the rank-r truncated SVD). Decode
// attention reads the factors directly (k_attn_global): Z = B_K q once per
// workgroup, scores A_K Z per token, Y = sum_t p_t A_V[t] accumulated in the
// rank space, and O = Y B_V once per wave at the end; factorized tokens are
// never rebuilt into K or V.
// Included by pkv_kernels.hip.

namespace pkv {

constexpr int kGGramTok = 4096;    // tokens per Gram workgroup
constexpr int kGProjTok = 1024;    // tokens per projection workgroup
constexpr int kGEigThreads = 512;  // eigen workgroup: 8 threads per column pair
constexpr int kGMaxSweeps = 40;
constexpr int kGAttnWaves = 8;

// Compressible region of a sequence of T tokens: tokens [t0, t1) (the
// factor pages of the plan, contiguous).
__host__ __device__ inline void global_range(const Geo &g, int64_t T, int64_t &t0, int64_t &t1) {
    t0 = (int64_t)g.sink_pages * g.P;
    t1 = T - g.W >= 0 ? (T - g.W) / g.P * g.P : 0;
    if (t1 < t0) t1 = t0;
}

// Byte offsets of one (layer, sequence, KV head)'s factors.
__host__ __device__ inline int64_t gbasis_head_bytes(const GlobalGeo &gg, int d) { return 3LL * gg.r8 * d * 2; }
__host__ __device__ inline int64_t gcoef_head_bytes(const GlobalGeo &gg) { return 2LL * gg.r8 * gg.max_tokens * 2; }

typedef float g_f32x16 __attribute__((ext_vector_type(16)));

// ---- Gram matrix ------------------------------------------------------------
//
// One 256-thread workgroup per (chunk of kGGramTok tokens, K/V, head). Tiles of
// 64 tokens are staged in LDS transposed (dim-major), so that the operand of
// the 32x32x16 bf16 MFMA -- eight consecutive tokens of one dim -- is one
// 16-byte LDS read; wave w accumulates the 64 x 64 quadrant (w / 2, w % 2) of
// G in fp32 over the chunk (products of bf16 values are exact). The partial
// sums of the chunks are added in order by the eigen kernel.
__global__ __launch_bounds__(256) void k_global_gram(Geo g, const uint16_t *k, const uint16_t *v, int64_t src_tokens,
                                                     SeqArgs seq, float *part, int n_chunks) {
    constexpr int D = 128, TT = 64, PITCH = TT + 8;
    __shared__ __align__(16) uint16_t xs[D * PITCH];
    const int chunk = blockIdx.x, which = blockIdx.y;
    const int64_t head = blockIdx.z;
    const int b = (int)(head / g.Hkv);
    int64_t t0, t1;
    global_range(g, seq.len[b], t0, t1);
    const int64_t c0 = t0 + (int64_t)chunk * kGGramTok;
    const int64_t c1 = min<int64_t>(t1, c0 + kGGramTok);
    const uint16_t *X = (which ? v : k) + head * src_tokens * D;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int I = wave >> 1, J = wave & 1;
    const int row = lane & 31, kg = lane >> 5;
    g_f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[a][c] = g_f32x16{};
    // thread (wave, lane) moves dims 8 (wave + 4 i) .. +7 of token `lane`
    uint4 stage[4];
    auto load = [&](int64_t tb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t t = tb + lane;
            stage[i] = t < c1 ? *(const uint4 *)(X + t * D + 8 * (wave + 4 * i)) : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    if (c0 < c1) load(c0);
    for (int64_t tb = c0; tb < c1; tb += TT) {
        __syncthreads();   // the previous tile's operands have been read
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint16_t *e = (const uint16_t *)&stage[i];
            const int dim0 = 8 * (wave + 4 * i);
#pragma unroll
            for (int u = 0; u < 8; ++u) xs[(dim0 + u) * PITCH + lane] = e[u];
        }
        __syncthreads();
        if (tb + TT < c1) load(tb + TT);   // next tile in flight during the products
#pragma unroll
        for (int ks = 0; ks < TT / 16; ++ks) {
            bf16x8 a[2], bb[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                a[t] = *(const bf16x8 *)(xs + (64 * I + 32 * t + row) * PITCH + 16 * ks + 8 * kg);
                bb[t] = *(const bf16x8 *)(xs + (64 * J + 32 * t + row) * PITCH + 16 * ks + 8 * kg);
            }
#pragma unroll
            for (int ti = 0; ti < 2; ++ti)
#pragma unroll
                for (int tj = 0; tj < 2; ++tj)
                    acc[ti][tj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ti], bb[tj], acc[ti][tj], 0, 0, 0);
        }
    }
    // C[m][n] of a 32x32 tile sits in lane n + 32 ((m / 4) % 2), register
    // (m % 4) + 4 (m / 8)
    float *out = part + ((head * 2 + which) * (int64_t)n_chunks + chunk) * D * D;
#pragma unroll
    for (int ti = 0; ti < 2; ++ti)
#pragma unroll
        for (int tj = 0; tj < 2; ++tj)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = 64 * I + 32 * ti + 4 * kg + (i & 3) + 8 * (i >> 2);
                const int n = 64 * J + 32 * tj + row;
                out[m * D + n] = acc[ti][tj][i];
            }
}

// ---- eigenvectors of G --------------------------------------------------------
//
// One 512-thread workgroup per (K/V, head). G (the chunk partials added in
// order, then scaled to unit Frobenius norm) sits in LDS column by column.
// One-sided Jacobi rotates pairs of columns until every pair is orthogonal to
// a cosine of d 2^-23; the pairs of a round are disjoint (round-robin
// ordering: 64 pairs per round, 127 rounds per sweep, every pair once), eight
// threads per pair, each holding 16 rows. At convergence the columns are
// lambda_c w_c (G W = W Lambda): their norms are the eigenvalues and their
// directions the eigenvectors, i.e. the right singular vectors of X. The r
// largest become the basis rows, in decreasing order (ties: lower column);
// a column whose norm is at most 2^-24 of |G|_F was never rotated (it is zero
// to working precision) and gives a zero row, which loses nothing of the
// region but a component at rounding level.
__global__ __launch_bounds__(kGEigThreads) void k_global_eigen(Geo g, GlobalGeo gg, const float *part, int n_chunks,
                                                               char *basis_layer) {
    constexpr int D = 128, PITCH = D + 4;
    __shared__ float Gs[D * PITCH];   // column c at Gs[c * PITCH + row]
    __shared__ float s_norm[D];
    __shared__ int s_rank[D];
    __shared__ float s_red[kGEigThreads / 64];
    __shared__ int s_rot;
    const int which = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int tid = threadIdx.x;
    const float *src = part + (head * 2 + which) * (int64_t)n_chunks * D * D;
    // sum the partials (fixed order) and the squared Frobenius norm
    float f2 = 0.f;
    for (int e = tid; e < D * D; e += kGEigThreads) {
        float x = 0.f;
        for (int c = 0; c < n_chunks; ++c) x += src[(int64_t)c * D * D + e];
        const int m = e / D, n = e % D;   // G[m][n], stored as column n
        Gs[n * PITCH + m] = x;
        f2 = fmaf(x, x, f2);
    }
    for (int o = 32; o >= 1; o >>= 1) f2 += __shfl_xor(f2, o, 64);
    if ((tid & 63) == 0) s_red[tid >> 6] = f2;
    __syncthreads();
    float fro2 = 0.f;
#pragma unroll
    for (int w = 0; w < kGEigThreads / 64; ++w) fro2 += s_red[w];
    const float inv = fro2 > 0.f ? 1.f / sqrtf(fro2) : 0.f;
    for (int e = tid; e < D * D; e += kGEigThreads) {
        const int m = e / D, n = e % D;
        Gs[n * PITCH + m] *= inv;
    }
    __syncthreads();
    const float tol = (float)D * 0x1p-23f;
    const float tiny2 = 0x1p-48f;   // |column|^2 below this (G scaled to |G|_F = 1): no direction
    const int p = tid >> 3, sub = tid & 7;
    int sweeps = 0;
    bool converged = fro2 == 0.f;
    while (!converged && sweeps < kGMaxSweeps) {
        if (tid == 0) s_rot = 0;
        __syncthreads();
        int rotated = 0;
        for (int round = 0; round < D - 1; ++round) {
            const int ci = p == 0 ? D - 1 : (round + p) % (D - 1);
            const int cj = p == 0 ? round : (round - p + D - 1) % (D - 1);
            float *gi = Gs + ci * PITCH + 16 * sub;
            float *gj = Gs + cj * PITCH + 16 * sub;
            float xi[16], xj[16];
#pragma unroll
            for (int u = 0; u < 16; u += 4) {
                *(f32x4 *)(xi + u) = *(const f32x4 *)(gi + u);
                *(f32x4 *)(xj + u) = *(const f32x4 *)(gj + u);
            }
            float al = 0.f, be = 0.f, ga = 0.f;
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                al = fmaf(xi[u], xi[u], al);
                be = fmaf(xj[u], xj[u], be);
                ga = fmaf(xi[u], xj[u], ga);
            }
#pragma unroll
            for (int o = 1; o < 8; o <<= 1) {
                al += __shfl_xor(al, o, 64);
                be += __shfl_xor(be, o, 64);
                ga += __shfl_xor(ga, o, 64);
            }
            if (al > tiny2 && be > tiny2 && fabsf(ga) > tol * sqrtf(al * be)) {
                const float zeta = (be - al) / (2.f * ga);
                const float t = (zeta >= 0.f ? 1.f : -1.f) / (fabsf(zeta) + sqrtf(1.f + zeta * zeta));
                const float c = 1.f / sqrtf(1.f + t * t), s = c * t;
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const float a = xi[u], bv = xj[u];
                    xi[u] = c * a - s * bv;
                    xj[u] = fmaf(s, a, c * bv);
                }
#pragma unroll
                for (int u = 0; u < 16; u += 4) {
                    *(f32x4 *)(gi + u) = *(const f32x4 *)(xi + u);
                    *(f32x4 *)(gj + u) = *(const f32x4 *)(xj + u);
                }
                rotated = 1;
            }
            __syncthreads();
        }
        if (rotated) s_rot = 1;
        __syncthreads();
        converged = s_rot == 0;
        ++sweeps;
        __syncthreads();
    }
    if (!converged && tid == 0) raise_status(PKV_DEV_NO_CONVERGE);
    // eigenvalues (column norms) and their order
    if (tid < D) {
        float n2 = 0.f;
        for (int m = 0; m < D; ++m) n2 = fmaf(Gs[tid * PITCH + m], Gs[tid * PITCH + m], n2);
        s_norm[tid] = sqrtf(n2);
    }
    __syncthreads();
    if (tid < D) {
        const float me = s_norm[tid];
        int rk = 0;
        for (int c = 0; c < D; ++c) rk += (s_norm[c] > me || (s_norm[c] == me && c < tid)) ? 1 : 0;
        s_rank[tid] = rk;
    }
    __syncthreads();
    // basis rows: B (r8 x d) row-major for K and V, B_V^T (d x r8) for V
    uint16_t *bk = (uint16_t *)(basis_layer + head * gbasis_head_bytes(gg, D));
    uint16_t *bv = bk + (int64_t)gg.r8 * D, *bvt = bv + (int64_t)gg.r8 * D;
    uint16_t *brow = which ? bv : bk;
    for (int e = tid; e < gg.r8 * D; e += kGEigThreads) brow[e] = 0;
    if (which)
        for (int e = tid; e < gg.r8 * D; e += kGEigThreads) bvt[e] = 0;
    __syncthreads();
    for (int e = tid; e < D * D; e += kGEigThreads) {
        const int c = e / D, m = e % D;   // column c, row (dim) m
        const int rk = s_rank[c];
        if (rk >= gg.r) continue;
        const float nc = s_norm[c];
        const float val = nc * nc > tiny2 ? Gs[c * PITCH + m] / nc : 0.f;
        const uint16_t hv = f32_to_bf16(val);
        brow[(int64_t)rk * D + m] = hv;
        if (which) bvt[(int64_t)m * gg.r8 + rk] = hv;
    }
}

// ---- coefficients A = X B^T ------------------------------------------------------
//
// One 256-thread workgroup per (block of kGProjTok tokens, K/V, head); each
// wave takes 16-token tiles. Lane (i, q) = (lane % 16, lane / 16) holds, for
// each 32-dim step, dims 32 s + 8 q .. +7 of basis row 16 rt + i and of token
// row i of the tile, which are both the A and the B operand layout of the
// 16x16x32 MFMA. Keys: C = B X^T (rank x token), lane (token, q) ends with
// ranks 4q .. 4q+3 of each rank tile, stored to the token-major A_K. Values:
// C = X B^T (token x rank), lane (rank, q) ends with tokens 4q .. 4q+3,
// stored to A_V^T, which is rank-major inside each 32-token unit: unit u's
// block of r8 x 32 values is contiguous, so the attention reads a unit's
// A_V^T as whole 128-byte lines, as it reads the unit's A_K rows.
template <int RT>
__global__ __launch_bounds__(256) void k_global_project(Geo g, GlobalGeo gg, const uint16_t *k, const uint16_t *v,
                                                        int64_t src_tokens, SeqArgs seq, const char *basis_layer,
                                                        char *coef_layer) {
    constexpr int D = 128;
    const int blk = blockIdx.x, which = blockIdx.y;
    const int64_t head = blockIdx.z;
    const int b = (int)(head / g.Hkv);
    int64_t t0, t1;
    global_range(g, seq.len[b], t0, t1);
    const int64_t n_rows = t1 - t0;
    const int64_t r0 = (int64_t)blk * kGProjTok;
    if (r0 >= n_rows) return;
    const int64_t r1 = min<int64_t>(n_rows, r0 + kGProjTok);
    const uint16_t *X = (which ? v : k) + (head * src_tokens + t0) * D;
    const uint16_t *Bm = (const uint16_t *)(basis_layer + head * gbasis_head_bytes(gg, D)) + (which ? (int64_t)gg.r8 * D : 0);
    uint16_t *Ak = (uint16_t *)(coef_layer + head * gcoef_head_bytes(gg));
    uint16_t *Avt = Ak + (int64_t)gg.max_tokens * gg.r8;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = lane & 15, q = lane >> 4;
    bf16x8 bop[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int s = 0; s < 4; ++s)
            bop[rt][s] = 16 * rt + i < gg.r8 ? ld_b8(Bm + (int64_t)(16 * rt + i) * D + 32 * s + 8 * q) : zero8();
    for (int64_t tb = r0 + 16 * wave; tb < r1; tb += 64) {
        bf16x8 xo[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) xo[s] = ld_b8(X + (tb + i) * D + 32 * s + 8 * q);   // tb + 16 <= r1 (N is a multiple of 32)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            f32x4 c = zero_f4();
            if (which == 0) {
#pragma unroll
                for (int s = 0; s < 4; ++s) c = mfma_bf16(bop[rt][s], xo[s], c);
                if (16 * rt + 4 * q < gg.r8) {
                    uint32_t lo = (uint32_t)f32_to_bf16(c[0]) | ((uint32_t)f32_to_bf16(c[1]) << 16);
                    uint32_t hi = (uint32_t)f32_to_bf16(c[2]) | ((uint32_t)f32_to_bf16(c[3]) << 16);
                    *(uint2 *)(Ak + (tb + i) * gg.r8 + 16 * rt + 4 * q) = make_uint2(lo, hi);
                }
            } else {
#pragma unroll
                for (int s = 0; s < 4; ++s) c = mfma_bf16(xo[s], bop[rt][s], c);
                if (16 * rt + i < gg.r8) {
                    uint32_t lo = (uint32_t)f32_to_bf16(c[0]) | ((uint32_t)f32_to_bf16(c[1]) << 16);
                    uint32_t hi = (uint32_t)f32_to_bf16(c[2]) | ((uint32_t)f32_to_bf16(c[3]) << 16);
                    *(uint2 *)(Avt + (tb & ~(int64_t)31) * gg.r8 + (16 * rt + i) * 32 + (tb & 31) + 4 * q) =
                        make_uint2(lo, hi);
                }
            }
        }
    }
}

// ---- decode attention over the global factors ------------------------------------
//
// Grid (chunk, head), eight waves per workgroup. The compressible region is
// cut into 32-token units; chunk c takes a contiguous run of units and its
// waves take every eighth one. Per wave:
//   Z^T = B_K Q^T once (M = rank, K = d), as hi/lo bf16 B operands over KS
//       32-rank steps (rank tile (ks, rt) row m -> rank 32 ks + rank_row(rt, m),
//       so a lane's two tiles of a step hold ranks 32 ks + 8q .. +7);
//   per unit: S^T = A_K Z^T (M = token, K = rank; the A_K rows of the two
//       token tiles follow the token map, so the exp weights land as the B
//       operand of the token contraction), online softmax with a lazy max,
//       Y^T += A_V^T E^T (M = rank, K = token), l from a ones x E^T product;
//   dense pages (sink, window) of the chunk: S^T = K Q^T, O^T += V^T E^T;
//   at the end O^T += B_V^T Y^T (M = dim, K = rank).
// Ranks at or past r8 read as zero through buffer range checks, which zeroes
// the matching rows of Z and Y; the A_K rank blocks and the A_V^T rank rows
// at or past r8 are not read (they would hold the next token's or the next
// unit's values). Waves merge in LDS; workgroups
// publish partials merged by Eq. (5) as in the page kernels.
template <int KS>
struct GWave {
    f32x4 o[8];         // O^T tiles (d = 128), dense pages and the final product
    f32x4 y[KS][2];     // Y^T tiles
    f32x4 l;            // normalizer (every row holds its column's value)
    float m_run;        // running max, log2 units
};

template <int KS>
__device__ inline void g_softmax(GWave<KS> &w, f32x4 (&st)[2], int rows, int q, float c2) {
    float pm = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            if (token_row<32>(tt, 4 * q + v) >= rows) st[tt][v] = -INFINITY;
            pm = fmaxf(pm, st[tt][v]);
        }
    if (__builtin_amdgcn_ballot_w64(pm * c2 > w.m_run + kLazyLog2) != 0) {
        pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
        const float m_new = fmaxf(w.m_run, pm * c2);
        const float alpha = w.m_run == -INFINITY ? 0.f : exp2f(w.m_run - m_new);
#pragma unroll
        for (int t = 0; t < 8; ++t) w.o[t] *= alpha;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) w.y[ks][rt] *= alpha;
        w.l *= alpha;
        w.m_run = m_new;
    }
    const float nm = -w.m_run;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) st[tt][v] = __builtin_amdgcn_exp2f(fmaf(st[tt][v], c2, nm));
}

template <int KS>
struct GUnitOps {
    bf16x8 ak[2][KS];   // A_K row token_row(tt, n), ranks 32 ks + 8q .. +7
    bf16x8 av[KS][2];   // A_V^T row 32 ks + rank_row(rt, n), tokens 8q .. +7 of the unit
};

template <int KS>
__device__ inline void g_issue_unit(GUnitOps<KS> &f, __amdgpu_buffer_rsrc_t rak, __amdgpu_buffer_rsrc_t ravt,
                                    int64_t u0, int r8, int n, int q) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        const uint32_t off = 2u * ((uint32_t)(u0 + token_row<32>(tt, n)) * (uint32_t)r8 + 8u * q);
        // rank blocks at or past r8 read nothing: an offset past the
        // resource returns zeros without a memory access
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) f.ak[tt][ks] = bld8(rak, 32 * ks + 8 * q < r8 ? off + 64u * ks : kOOB, 0u);
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            const uint32_t rank = 32u * ks + (uint32_t)rank_row(rt, n);
            f.av[ks][rt] = bld8(ravt, rank < (uint32_t)r8 ? 2u * ((uint32_t)u0 * (uint32_t)r8 + 32u * rank + 8u * q) : kOOB, 0u);
        }
}

template <int KS>
__device__ inline void g_unit(GWave<KS> &w, const GUnitOps<KS> &f, const bf16x8 (&zh)[KS], const bf16x8 (&zl)[KS],
                              int q, float c2) {
    f32x4 st[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        st[tt] = zero_f4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            st[tt] = mfma_bf16(f.ak[tt][ks], zh[ks], st[tt]);
            st[tt] = mfma_bf16(f.ak[tt][ks], zl[ks], st[tt]);
        }
    }
    g_softmax<KS>(w, st, 32, q, c2);
    bf16x8 eh, el;
    split_tiles(st[0], st[1], eh, el);
    const bf16x8 ones = bf16x8{1, 1, 1, 1, 1, 1, 1, 1};
    w.l = mfma_bf16(ones, eh, w.l);
    w.l = mfma_bf16(ones, el, w.l);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            w.y[ks][rt] = mfma_bf16(f.av[ks][rt], eh, w.y[ks][rt]);
            w.y[ks][rt] = mfma_bf16(f.av[ks][rt], el, w.y[ks][rt]);
        }
}

// One dense page (rows valid tokens), in units of 32 tokens.
template <int KS>
__device__ inline void g_dense_page(GWave<KS> &w, const bf16x8 (&qb)[4], const uint16_t *K, int P, int rows_page,
                                    int n, int q, float c2) {
    const uint16_t *Vt = K + (int64_t)P * 128;
    for (int half = 0; half * 32 < rows_page; ++half) {
        const int rows = min(32, rows_page - 32 * half);
        f32x4 st[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
            st[tt] = zero_f4();
            const uint16_t *kp = K + (int64_t)(32 * half + token_row<32>(tt, n)) * 128 + 8 * q;
#pragma unroll
            for (int s = 0; s < 4; ++s) st[tt] = mfma_bf16(ld_b8(kp + 32 * s), qb[s], st[tt]);
        }
        g_softmax<KS>(w, st, rows, q, c2);
        bf16x8 eh, el;
        split_tiles(st[0], st[1], eh, el);
        const bf16x8 ones = bf16x8{1, 1, 1, 1, 1, 1, 1, 1};
        w.l = mfma_bf16(ones, eh, w.l);
        w.l = mfma_bf16(ones, el, w.l);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            bf16x8 vv = ld_b8(Vt + (int64_t)(16 * dt + n) * P + 32 * half + 8 * q);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (8 * q + u >= rows) vv[u] = (__bf16)0.f;   // columns past the page's rows may hold anything
            w.o[dt] = mfma_bf16(vv, eh, w.o[dt]);
            w.o[dt] = mfma_bf16(vv, el, w.o[dt]);
        }
    }
}

template <int KS>
__global__ __launch_bounds__(64 * kGAttnWaves, 1) void k_attn_global(Geo g, GlobalGeo gg, const pkv_page *__restrict__ table,
                                                                      const char *__restrict__ dense,
                                                                      const char *__restrict__ basis_layer,
                                                                      const char *__restrict__ coef_layer,
                                                                      const uint16_t *__restrict__ q, SeqArgs seq,
                                                                      int n_chunks, Partials pp, float *out, float *lse) {
    constexpr int D = 128, NW = kGAttnWaves;
    const int chunk = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    const int G = g.g;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int lane = threadIdx.x % 64;
    const int n = lane & 15, q4 = lane >> 4;
    const int64_t T = seq.len[b];
    const float c2 = kLog2e / sqrtf((float)D);
    int64_t t0, t1;
    global_range(g, T, t0, t1);
    const int64_t n_units = (t1 - t0) / 32;
    const int64_t upc = ceil_div(n_units, n_chunks);
    const int64_t ub = (int64_t)chunk * upc, ue = min<int64_t>(n_units, ub + upc);

    bf16x8 qb[4];
    {
        const uint16_t *qp = q + ((int64_t)b * g.Hq + (int64_t)h * G + n) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < 4; ++s) qb[s] = n < G ? ld_b8(qp + 32 * s) : zero8();
    }
    GWave<KS> w;
#pragma unroll
    for (int t = 0; t < 8; ++t) w.o[t] = zero_f4();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) w.y[ks][rt] = zero_f4();
    w.l = zero_f4();
    w.m_run = -INFINITY;

    const char *bh = basis_layer + head * gbasis_head_bytes(gg, D);
    const char *ch = coef_layer + head * gcoef_head_bytes(gg);
    const __amdgpu_buffer_rsrc_t rbk = section_rsrc(bh, (uint32_t)(2 * gg.r8 * D));
    const __amdgpu_buffer_rsrc_t rbvt = section_rsrc(bh + 4 * gg.r8 * D, (uint32_t)(2 * gg.r8 * D));
    // A_K up to the region's last row: reads past r8 in that row return zero
    // rather than rows the projection never wrote
    const __amdgpu_buffer_rsrc_t rak = section_rsrc(ch, (uint32_t)(2 * (t1 - t0) * gg.r8));
    const __amdgpu_buffer_rsrc_t ravt =
        section_rsrc(ch + 2 * (int64_t)gg.max_tokens * gg.r8, (uint32_t)(2 * (int64_t)gg.max_tokens * gg.r8));

    if (ub < ue) {
        // Z^T = B_K Q^T as hi/lo B operands of the score product
        bf16x8 zh[KS], zl[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            f32x4 z[2];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                z[rt] = zero_f4();
                const uint32_t rank = 32u * ks + (uint32_t)rank_row(rt, n);
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    z[rt] = mfma_bf16(bld8(rbk, 2u * (rank * D + 32u * s + 8u * q4), 0u), qb[s], z[rt]);
            }
            split_tiles(z[0], z[1], zh[ks], zl[ks]);
        }
        // the wave's units, each unit's operands loaded one step ahead (at
        // ranks above 96 the second operand set would not fit the registers)
        constexpr bool kAhead = KS <= 3;
        GUnitOps<KS> cur, nxt;
        int64_t u = ub + wave;
        if (kAhead && u < ue) g_issue_unit<KS>(cur, rak, ravt, u * 32, gg.r8, n, q4);
        for (; u < ue; u += NW) {
            if (kAhead) {
                if (u + NW < ue) g_issue_unit<KS>(nxt, rak, ravt, (u + NW) * 32, gg.r8, n, q4);
                g_unit<KS>(w, cur, zh, zl, q4, c2);
                cur = nxt;
            } else {
                g_issue_unit<KS>(cur, rak, ravt, u * 32, gg.r8, n, q4);
                g_unit<KS>(w, cur, zh, zl, q4, c2);
            }
        }
    }
    // dense pages: sink pages, then the pages after the region, dealt out over
    // (chunk, wave)
    {
        const int64_t n_pages = ceil_div(T, g.P);
        const int64_t n_sink = min<int64_t>(g.sink_pages, n_pages);
        const int64_t jw = max<int64_t>(g.sink_pages, t1 / g.P);
        const int64_t n_dense = n_sink + max<int64_t>(0, n_pages - jw);
        const pkv_page *tab = table + head * g.max_pages;
        for (int64_t i = chunk + (int64_t)n_chunks * wave; i < n_dense; i += (int64_t)n_chunks * NW) {
            const int64_t j = i < n_sink ? i : jw + (i - n_sink);
            const pkv_page e = tab[j];
            if (e.kind != PKV_DENSE) {
                if (lane == 0) raise_status(PKV_DEV_BAD_PAGE);
                continue;
            }
            g_dense_page<KS>(w, qb, (const uint16_t *)(dense + e.slot * g.dense_slot_bytes), g.P,
                             (int)min<int64_t>(g.P, T - j * g.P), n, q4, c2);
        }
        // the region's last page must be held by the global factors
        if (chunk == 0 && wave == 0 && t1 > t0 && tab[t1 / g.P - 1].kind != PKV_GLOBAL && lane == 0)
            raise_status(PKV_DEV_BAD_PAGE);
    }
    // O^T += B_V^T Y^T
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        bf16x8 yh, yl;
        split_tiles(w.y[ks][0], w.y[ks][1], yh, yl);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const bf16x8 a = bld8(rbvt, 2u * ((16u * dt + n) * (uint32_t)gg.r8 + 32u * ks + 8u * q4), 0u);
            w.o[dt] = mfma_bf16(a, yh, w.o[dt]);
            w.o[dt] = mfma_bf16(a, yl, w.o[dt]);
        }
    }

    // ---- merge the wave states (Eq. (5)) into the chunk's partial --------------
    __shared__ float s_m[NW][16], s_l[NW][16];
    __shared__ __align__(16) float s_o[NW][16][D + 4];
    if (q4 == 0) {
        s_m[wave][n] = w.m_run;
        s_l[wave][n] = w.l[0];
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int v = 0; v < 4; ++v) s_o[wave][n][16 * dt + 4 * q4 + v] = w.o[dt][v];
    __syncthreads();
    // four dims per thread, one 16-byte store with the coherent cache policy of st_dev
    const __amdgpu_buffer_rsrc_t rpo =
        __builtin_amdgcn_make_buffer_rsrc(pp.o + pp.oi(head, 0, 0, chunk), (short)0, G * D * 4, kBufferDword3);
    for (int f = threadIdx.x; f < G * D / 4; f += 64 * NW) {
        const int qi = (4 * f) / D, k = (4 * f) % D;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, s_m[ww][qi]);
        f32x4 acc = zero_f4();
        float l = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
            const float sc = s_m[ww][qi] == -INFINITY ? 0.f : exp2f(s_m[ww][qi] - M);
            acc += sc * lds_ld4(&s_o[ww][qi][k]);
            l = fmaf(sc, s_l[ww][qi], l);
        }
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), rpo, 16u * (uint32_t)f, 0, 16);
        if (k == 0) {
            st_dev(&pp.m[pp.mi(head, qi, chunk)], M);
            st_dev(&pp.l[pp.mi(head, qi, chunk)], l);
        }
    }
    // the wave-state block is free once every thread has passed the publish barrier
    publish_and_merge<64 * NW>(g, head, pp, out, lse, T, &s_o[0][0][0]);
}

// ---- launches -----------------------------------------------------------------------

inline GlobalLayer global_layer(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl) {
    GlobalLayer p;
    const int64_t heads = (int64_t)L.geo.B * L.geo.Hkv;
    p.basis = (char *)gl->basis + (int64_t)L.layer * heads * gbasis_head_bytes(gg, L.geo.d);
    p.coef = (char *)gl->coef + (int64_t)L.layer * heads * gcoef_head_bytes(gg);
    return p;
}

int global_gram_chunks(const Geo &g, int64_t max_T) {
    int64_t t0, t1;
    global_range(g, max_T, t0, t1);
    return (int)std::max<int64_t>(1, ceil_div(t1 - t0, kGGramTok));
}

int64_t global_prefill_workspace_bytes(const Geo &g, int64_t max_T) {
    return (int64_t)g.B * g.Hkv * 2 * global_gram_chunks(g, max_T) * 128 * 128 * 4;
}

int global_attention_chunks(const Geo &g, int64_t max_T) {
    int64_t t0, t1;
    global_range(g, max_T, t0, t1);
    const int64_t heads = (int64_t)g.B * g.Hkv;
    const int64_t units = (t1 - t0) / 32;
    const int64_t want = ceil_div(256, heads);
    return (int)std::max<int64_t>(1, std::min<int64_t>(want, ceil_div(units, kGAttnWaves)));
}

int64_t global_attention_workspace_bytes(const Geo &g, int64_t max_T) {
    return partials_bytes((int64_t)g.B * g.Hkv, global_attention_chunks(g, max_T), g.g, g.d);
}

hipError_t launch_global_prefill(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, const void *k,
                                 const void *v, int64_t src_tokens, const SeqArgs &seq, int64_t max_T, void *ws) {
    const Geo &g = L.geo;
    const GlobalLayer gp = global_layer(L, gg, gl);
    const int heads = g.B * g.Hkv;
    const int n_chunks = global_gram_chunks(g, max_T);
    int64_t t0, t1;
    global_range(g, max_T, t0, t1);
    hipLaunchKernelGGL(k_global_gram, dim3(n_chunks, 2, heads), dim3(256), 0, L.stream, g, (const uint16_t *)k,
                       (const uint16_t *)v, src_tokens, seq, (float *)ws, n_chunks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_global_eigen, dim3(2, heads), dim3(kGEigThreads), 0, L.stream, g, gg, (const float *)ws,
                       n_chunks, gp.basis);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int blocks = (int)std::max<int64_t>(1, ceil_div(t1 - t0, kGProjTok));
    const dim3 grid(blocks, 2, heads);
    switch ((gg.r8 + 15) / 16) {
#define PKV_GPROJ(RT)                                                                                        \
    case RT:                                                                                                 \
        hipLaunchKernelGGL(k_global_project<RT>, grid, dim3(256), 0, L.stream, g, gg, (const uint16_t *)k,  \
                           (const uint16_t *)v, src_tokens, seq, (const char *)gp.basis, gp.coef);           \
        break;
        PKV_GPROJ(1) PKV_GPROJ(2) PKV_GPROJ(3) PKV_GPROJ(4) PKV_GPROJ(5) PKV_GPROJ(6) PKV_GPROJ(7) PKV_GPROJ(8)
#undef PKV_GPROJ
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_global_attention(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, const void *q,
                                   const SeqArgs &seq, int64_t max_T, float *out, float *lse, void *ws) {
    const Geo &g = L.geo;
    const GlobalLayer gp = global_layer(L, gg, gl);
    LayerPtrs p = layer_ptrs(L);
    const int n_chunks = global_attention_chunks(g, max_T);
    const Partials pp = make_partials(ws, (int64_t)g.B * g.Hkv, n_chunks, g.g, g.d);
    const dim3 grid(n_chunks, g.B * g.Hkv);
    switch ((gg.r8 + 31) / 32) {
#define PKV_GATT(KS)                                                                                          \
    case KS:                                                                                                  \
        hipLaunchKernelGGL(k_attn_global<KS>, grid, dim3(64 * kGAttnWaves), 0, L.stream, g, gg, p.table,      \
                           p.dense, (const char *)gp.basis, (const char *)gp.coef, (const uint16_t *)q, seq,  \
                           n_chunks, pp, out, lse);                                                           \
        break;
        PKV_GATT(1) PKV_GATT(2) PKV_GATT(3) PKV_GATT(4)
#undef PKV_GATT
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Export of one head's factors as fp32: B_K, B_V (r x d), A_K, A_V (n_rows x r).
__global__ void k_global_export(GlobalGeo gg, const char *basis_head, const char *coef_head, int64_t n_rows,
                                float *bk, float *bv, float *ak, float *av) {
    constexpr int D = 128;
    const uint16_t *Bk = (const uint16_t *)basis_head, *Bv = Bk + (int64_t)gg.r8 * D;
    const uint16_t *Ak = (const uint16_t *)coef_head, *Avt = Ak + (int64_t)gg.max_tokens * gg.r8;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t e = i0; e < (int64_t)gg.r * D; e += stride) {
        const int64_t a = e / D, m = e % D;
        bk[e] = bf16_to_f32(Bk[a * D + m]);
        bv[e] = bf16_to_f32(Bv[a * D + m]);
    }
    for (int64_t e = i0; e < n_rows * gg.r; e += stride) {
        const int64_t t = e / gg.r, a = e % gg.r;
        ak[e] = bf16_to_f32(Ak[t * gg.r8 + a]);
        av[e] = bf16_to_f32(Avt[(t & ~(int64_t)31) * gg.r8 + a * 32 + (t & 31)]);
    }
}

hipError_t launch_global_export(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, int b, int h,
                                int64_t n_rows, float *bk, float *bv, float *ak, float *av) {
    const GlobalLayer gp = global_layer(L, gg, gl);
    const int64_t head = L.geo.head_index(b, h);
    hipLaunchKernelGGL(k_global_export, dim3(256), dim3(256), 0, L.stream, gg,
                       (const char *)gp.basis + head * gbasis_head_bytes(gg, L.geo.d),
                       (const char *)gp.coef + head * gcoef_head_bytes(gg), n_rows, bk, bv, ak, av);
    return hipGetLastError();
}

}  // namespace pkv
