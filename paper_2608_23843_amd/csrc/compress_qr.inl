// Batched per-page truncated decomposition for bf16 pages of P = 32 or 64
// tokens: the path pkv_compress_pages and pkv_prefill take for bf16 dense
// pages (Section 3.3, Eq. (2)). The result is the one k_compress computes --
// the top-r eigenvectors L of the page's Gram matrix G = X X^T and R = L^T X,
// the rank-r truncated-SVD factors -- reached in four phases per wavefront
// (one page half for P = 64, two for P = 32, one per 32-lane half):
//
//  1. G by matrix-core products (32x32x16 bf16: exact products, fp32
//     accumulation) with operands loaded straight from the page, then one
//     permlane32 swap per pair of accumulator registers so that lane c holds
//     all of column c of G (rows in the accumulator's row order, which no
//     later step depends on).
//  2. A backward-stable QR of G: modified Gram-Schmidt with the columns taken
//     in order of decreasing norm, keeping only R. The computed R is the exact
//     R of G + dG with |dG| ~ eps |G| (Bjorck), and with G Pi = Q R the matrix
//     G Q = Pi R^T has the eigenvectors of G as its left singular vectors and
//     the eigenvalues as its singular values. Its rows are graded, so the
//     Jacobi iteration converges in about half the sweeps it needs on G
//     itself. Row k of R is written to LDS and read by the lane pivoted at
//     step k, which no longer needs its column of G: no register indexing,
//     no transposition buffer.
//  3. One-sided Jacobi on the columns of Pi R^T (xor pairing inside 32-lane
//     halves, partner columns fetched with ds_swizzle, which costs a third of
//     a ds_bpermute; pairs across halves are met by swapping 16-lane rows
//     between groups of steps), without accumulating the rotations: at
//     convergence the columns are lambda_c u_c with u_c the eigenvectors, so
//     L is the normalized columns, orthonormal to the rotation threshold.
//  4. Ranking and eigenvectors; then R = L^T X with L staged in LDS: on
//     32x32x16 bf16 matrix-core products at P = 64 (L as a bf16 hi + lo
//     pair against the exact page) for bf16 and INT4 factors, otherwise
//     fp32 fmas with each lane owning two output dims; stores.
//     The page is read again here: holding it from phase 1 would take 64
//     more registers per lane (two waves per SIMD instead of three) or 16 KB
//     of LDS per wave, and the kernel is bound by its vector-ALU issue, not
//     by the second read (about 0.2 TB/s).
// Included by pkv_kernels.hip after compress.inl.

namespace pkv {

typedef __bf16 cq_bf16x8 __attribute__((ext_vector_type(8)));
typedef float cq_f32x16 __attribute__((ext_vector_type(16)));

constexpr float kCqTiny2 = 3.5527137e-15f;   // (2^-24)^2: a column below this (|G|_F = 1) is zero

// Eight consecutive dims of page row `row`, dims k0..k0+7, as an MFMA operand.
__device__ inline cq_bf16x8 cq_load8(const uint16_t *X, bool transposed, int P, int d, int row, int k0) {
    if (!transposed) return __builtin_bit_cast(cq_bf16x8, *(const uint4 *)(X + (int64_t)row * d + k0));
    uint32_t w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
        w[u] = (uint32_t)X[(int64_t)(k0 + 2 * u) * P + row] | ((uint32_t)X[(int64_t)(k0 + 2 * u + 1) * P + row] << 16);
    return __builtin_bit_cast(cq_bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
}

// Page element (t, k) as fp32.
__device__ inline float cq_elem(const uint16_t *X, bool transposed, int P, int d, int t, int k) {
    return bf16_to_f32(transposed ? X[(int64_t)k * P + t] : X[(int64_t)t * d + k]);
}

typedef float cq_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 cq_bf16x2 __attribute__((ext_vector_type(2)));

// Two fp32 values as a packed bf16 pair, rounded to nearest even.
__device__ inline uint32_t cq_pack_bf16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(cq_f32x2{a, b}, cq_bf16x2));
}
// Two fp32 values -> bf16 pair hi and bf16 pair lo of the remainders
// (hi + lo carries 16 significant bits).
__device__ inline void cq_split2(float a, float b, uint32_t &hi, uint32_t &lo) {
    hi = cq_pack_bf16(a, b);
    lo = cq_pack_bf16(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}
// Page dims k and k + 1 (k even) over tokens t0..t0+7 as two MFMA operands:
// one 4-byte read per token row, split into its even and odd dim.
__device__ inline void cq_load_dim_pair(const uint16_t *X, bool transposed, int P, int d, int k, int t0,
                                        cq_bf16x8 &be, cq_bf16x8 &bo) {
    if (transposed) {   // d x P: eight tokens of one dim are contiguous
        be = __builtin_bit_cast(cq_bf16x8, *(const uint4 *)(X + (int64_t)k * P + t0));
        bo = __builtin_bit_cast(cq_bf16x8, *(const uint4 *)(X + (int64_t)(k + 1) * P + t0));
        return;
    }
    uint32_t w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = *(const uint32_t *)(X + (int64_t)(t0 + i) * d + k);
    uint32_t e[4], o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        e[i] = __builtin_amdgcn_perm(w[2 * i + 1], w[2 * i], 0x05040100u);   // low halves: dim k
        o[i] = __builtin_amdgcn_perm(w[2 * i + 1], w[2 * i], 0x07060302u);   // high halves: dim k + 1
    }
    be = __builtin_bit_cast(cq_bf16x8, make_uint4(e[0], e[1], e[2], e[3]));
    bo = __builtin_bit_cast(cq_bf16x8, make_uint4(o[0], o[1], o[2], o[3]));
}

__device__ inline float cq_f(int v) { return __int_as_float(v); }
__device__ inline int cq_i(float v) { return __float_as_int(v); }

// Partner values for xor pairing step M < 32 (inside each 32-lane half).
template <int P, int M>
__device__ __forceinline__ void cq_swz(const float (&a)[P], float (&pa)[P], float s0, float &p0, float s1, float &p1,
                                       int s2, int &p2) {
    constexpr int pat = (M << 10) | 0x1f;   // bitmask mode: and 0x1f, or 0, xor M
#pragma unroll
    for (int k = 0; k < P; ++k) pa[k] = cq_f(__builtin_amdgcn_ds_swizzle(cq_i(a[k]), pat));
    p0 = cq_f(__builtin_amdgcn_ds_swizzle(cq_i(s0), pat));
    p1 = cq_f(__builtin_amdgcn_ds_swizzle(cq_i(s1), pat));
    p2 = __builtin_amdgcn_ds_swizzle(s2, pat);
}

// Value of lane `src` (within this lane's P-lane group) of every group.
template <int P>
__device__ __forceinline__ float cq_group_bcast(float v, int src0, int src1, int grp) {
    if constexpr (P == 64) {
        return cq_f(__builtin_amdgcn_readlane(cq_i(v), src0));
    } else {
        const float a = cq_f(__builtin_amdgcn_readlane(cq_i(v), src0));
        const float b = cq_f(__builtin_amdgcn_readlane(cq_i(v), src1));
        return grp ? b : a;
    }
}

// Sum over the lanes of a P-lane group.
template <int P>
__device__ __forceinline__ float cq_group_sum(float v) {
    v += cq_f(__builtin_amdgcn_ds_swizzle(cq_i(v), (1 << 10) | 0x1f));
    v += cq_f(__builtin_amdgcn_ds_swizzle(cq_i(v), (2 << 10) | 0x1f));
    v += cq_f(__builtin_amdgcn_ds_swizzle(cq_i(v), (4 << 10) | 0x1f));
    v += cq_f(__builtin_amdgcn_ds_swizzle(cq_i(v), (8 << 10) | 0x1f));
    v += cq_f(__builtin_amdgcn_ds_swizzle(cq_i(v), (16 << 10) | 0x1f));
    if constexpr (P == 64) v += cq_f(__builtin_amdgcn_ds_bpermute((int)(((threadIdx.x & 63) ^ 32) << 2), cq_i(v)));
    return v;
}

// Minimum over the lanes of a P-lane group.
template <int P>
__device__ __forceinline__ int cq_group_min(int v) {
    v = min(v, __builtin_amdgcn_ds_swizzle(v, (1 << 10) | 0x1f));
    v = min(v, __builtin_amdgcn_ds_swizzle(v, (2 << 10) | 0x1f));
    v = min(v, __builtin_amdgcn_ds_swizzle(v, (4 << 10) | 0x1f));
    v = min(v, __builtin_amdgcn_ds_swizzle(v, (8 << 10) | 0x1f));
    v = min(v, __builtin_amdgcn_ds_swizzle(v, (16 << 10) | 0x1f));
    if constexpr (P == 64) v = min(v, __builtin_amdgcn_ds_bpermute((int)(((threadIdx.x & 63) ^ 32) << 2), v));
    return v;
}

// Adaptive rank from the group's column norms: with key the squared norm of
// this lane's column and lam its eigenvalue of G, the smallest r whose r
// largest eigenvalues leave |X|_F^2 - (their sum) <= eps2 |X|_F^2; P + 1 when
// none does. Ties rank the lower lane first.
template <int P>
__device__ __forceinline__ int cq_adaptive_rank(float key, float lam, float xnorm2, float eps2, int c, int grp) {
    float head = lam;   // energy of the columns ranked at or above this one
    int above = 0;
    for (int k = 0; k < P; ++k) {
        const float kk = cq_group_bcast<P>(key, k, 32 + k, grp);
        const float lk = cq_group_bcast<P>(lam, k, 32 + k, grp);
        const bool up = kk > key || (kk == key && k < c);
        head += up ? lk : 0.f;
        above += up ? 1 : 0;
    }
    const bool ok = xnorm2 - head <= eps2 * xnorm2;
    return cq_group_min<P>(ok ? above + 1 : P + 1);
}

// LDS floats per wavefront: R's row buffer (64), L staged as 64 x 32, inverse
// singular values (64), the position -> token table (64); INT4 adds R~'s
// codes (32 x d bytes) and L~'s scales ((P/32) r8 or P <= 64).
__host__ __device__ inline int cq_wave_lds(int d, bool q4) { return 64 + 64 * 32 + 64 + 64 + (q4 ? 8 * d + 64 : 0); }

// Rank of `key` among the P lanes of the group: descending, ties to the lower lane.
template <int P>
__device__ __forceinline__ int cq_rank(float key, int c, int grp) {
    int rho = 0;
    for (int k = 0; k < P; ++k) {
        const float kk = cq_group_bcast<P>(key, k, 32 + k, grp);
        rho += (kk > key) || (kk == key && k < c);
    }
    return rho;
}

// One wavefront per workgroup. kAdapt (a cache with adaptive ranks): a rank
// of 0 asks for the rank chosen from the spectrum. The packed factor slot
// places V's sections after K's rank, so the V decomposition of a page must
// know K's rank before it stores: the two halves of the wavefront hold K and
// V at P = 32, and at P = 64 the wavefront decomposes K, then V. With fixed
// ranks every P = 64 decomposition is a wavefront of its own.
template <typename TF, int P, bool kAdapt, bool kList = false>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3)))
void k_compress_qr(Geo g, pkv_page *table, const char *dense, char *factor, CompressItems items, CompressSrc src,
                   int64_t n_decomp) {
    static_assert(P == 32 || P == 64, "P = 32 or 64");
    constexpr int D = 64 / P;                          // decompositions per pass
    constexpr int kPasses = P == 64 && kAdapt ? 2 : 1;
    constexpr bool kQ4 = is_q4<TF>::value;
    extern __shared__ float cq_smem[];
    const int d = g.d;
    const int lane = threadIdx.x;
    int *cq_tok = (int *)(cq_smem + 64 + 64 * 32 + 64);   // position -> token, per group
    const int grp = P == 64 ? 0 : lane >> 5;
    const int c = P == 64 ? lane : lane & 31;
    int rk_first = 0;   // two passes: the K rank chosen by the first
    for (int kv = 0; kv < kPasses; ++kv) {
    // K and V of a page are decompositions 2i and 2i + 1 of the launch, so
    // a pass is active exactly when the other one is
    const int64_t q = ((int64_t)blockIdx.x * kPasses + kv) * D + grp;

    const DecompRef ref = decode_decomp<uint16_t, kList>(g, table, dense, items, src, q, n_decomp, c == 0);
    const bool active = ref.active;
    const uint16_t *X = (const uint16_t *)ref.X;

    // ---- 1. Gram matrix by MFMA, lane c <- column c ------------------------
    float gc[P];
    float xnorm2 = 0.f;   // |X|_F^2 of this lane's page half
    {
        const int row = lane & 31, kh = lane >> 5;
        if constexpr (P == 64) {
            cq_f32x16 c00 = {}, c01 = {}, c10 = {}, c11 = {};
            float e2 = 0.f;
            if (active) {
                for (int s = 0; s < d / 16; ++s) {
                    const int k0 = 16 * s + 8 * kh;
                    const cq_bf16x8 a0 = cq_load8(X, ref.transposed, P, d, row, k0);
                    const cq_bf16x8 a1 = cq_load8(X, ref.transposed, P, d, 32 + row, k0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) e2 = fmaf((float)a1[u], (float)a1[u], fmaf((float)a0[u], (float)a0[u], e2));
                    c00 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, a0, c00, 0, 0, 0);
                    c01 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, a1, c01, 0, 0, 0);
                    c10 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, a0, c10, 0, 0, 0);
                    c11 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, a1, c11, 0, 0, 0);
                }
            }
            // C[m][n] sits in lane 32 (m/4 % 2) + n; swapping the upper half of
            // the column-tile-0 accumulator with the lower half of column tile 1
            // gives lane c all of column c (rows 0..31), likewise for rows 32..63.
            xnorm2 = cq_group_sum<64>(e2);   // |X|_F^2: every element was loaded by one lane
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const auto r0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(c00[i]), __float_as_uint(c01[i]), false, false);
                const auto r1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(c10[i]), __float_as_uint(c11[i]), false, false);
                gc[i] = __uint_as_float(r0[0]);
                gc[16 + i] = __uint_as_float(r0[1]);
                gc[32 + i] = __uint_as_float(r1[0]);
                gc[48 + i] = __uint_as_float(r1[1]);
            }
        } else {
            // two pages per wave: each lane feeds both pages' operands
            const uint64_t xbits = (uint64_t)(uintptr_t)X;
            const uint64_t x0 = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(xbits >> 32), 0) << 32) |
                                (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)xbits, 0);
            const uint64_t x1 = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(xbits >> 32), 32) << 32) |
                                (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)xbits, 32);
            const int act0 = __builtin_amdgcn_readlane(active ? 1 : 0, 0);
            const int act1 = __builtin_amdgcn_readlane(active ? 1 : 0, 32);
            const int tr0 = __builtin_amdgcn_readlane(ref.transposed ? 1 : 0, 0);
            const int tr1 = __builtin_amdgcn_readlane(ref.transposed ? 1 : 0, 32);
            cq_f32x16 cg0 = {}, cg1 = {};
            float e0 = 0.f, e1 = 0.f;
            for (int s = 0; s < d / 16; ++s) {
                const int k0 = 16 * s + 8 * kh;
                if (act0) {
                    const cq_bf16x8 a = cq_load8((const uint16_t *)(uintptr_t)x0, tr0, P, d, row, k0);
                    cg0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, cg0, 0, 0, 0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) e0 = fmaf((float)a[u], (float)a[u], e0);
                }
                if (act1) {
                    const cq_bf16x8 a = cq_load8((const uint16_t *)(uintptr_t)x1, tr1, P, d, row, k0);
                    cg1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, cg1, 0, 0, 0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) e1 = fmaf((float)a[u], (float)a[u], e1);
                }
            }
            const float n0 = cq_group_sum<64>(e0), n1 = cq_group_sum<64>(e1);
            xnorm2 = grp ? n1 : n0;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(cg0[i]), __float_as_uint(cg1[i]), false, false);
                gc[i] = __uint_as_float(r[0]);
                gc[16 + i] = __uint_as_float(r[1]);
            }
        }
    }

    // ---- 2. QR of G by modified Gram-Schmidt, R only -----------------------
    float nrm2 = 0.f;
#pragma unroll
    for (int e = 0; e < P; ++e) nrm2 = fmaf(gc[e], gc[e], nrm2);
    const float fro2 = cq_group_sum<P>(nrm2);
    const float gnorm = sqrtf(fro2);
    const float ginv = fro2 > 0.f ? 1.f / gnorm : 0.f;
#pragma unroll
    for (int e = 0; e < P; ++e) gc[e] *= ginv;
    nrm2 *= ginv * ginv;
    // Pivot order: decreasing column norm. The columns are first moved so that
    // the k-th pivot sits in lane k: row k of R then becomes the column of
    // lane k, and the xor pairing of the Jacobi steps meets rows of similar
    // size early (about 1.4 sweeps fewer than leaving row k in the pivot's
    // lane). tok_of[k] records which token's column that is; the
    // eigenvectors' entries come out in this order.
    {
        const int prank = cq_rank<P>(nrm2, c, grp);
        const int daddr = ((P == 64 ? 0 : grp * 32) + prank) << 2;
#pragma unroll
        for (int e = 0; e < P; ++e) gc[e] = cq_f(__builtin_amdgcn_ds_permute(daddr, cq_i(gc[e])));
        cq_tok[grp * P + c] = __builtin_amdgcn_ds_permute(daddr, c);   // token of this lane's column
    }
    float *rowbuf = cq_smem + grp * P;
    bool done = false;
    for (int k = 0; k < P; ++k) {
        const int piv0 = k;
        const int piv1 = P == 64 ? k : 32 + k;
        float x[P];
#pragma unroll
        for (int e = 0; e < P; ++e) x[e] = cq_group_bcast<P>(gc[e], piv0, piv1, grp);
        float da = 0.f, db = 0.f;
#pragma unroll
        for (int e = 0; e < P; e += 2) {
            da = fmaf(x[e], gc[e], da);
            db = fmaf(x[e + 1], gc[e + 1], db);
        }
        const float dot = da + db;
        // the pivot's column is x, so its dot is |x|^2: no lane sums squares
        const float nx2 = cq_group_bcast<P>(dot, piv0, piv1, grp);
        const float inv = nx2 > kCqTiny2 ? __builtin_amdgcn_rsqf(nx2) : 0.f;
        const float rk = done ? 0.f : dot * inv;          // R[k][c]
        const float f = done ? 0.f : rk * inv;            // projection coefficient
#pragma unroll
        for (int e = 0; e < P; ++e) gc[e] = fmaf(-f, x[e], gc[e]);
        rowbuf[c] = rk;
        __builtin_amdgcn_wave_barrier();
        if (c == k) {   // the pivot's column is finished: it takes row k of R
#pragma unroll
            for (int e = 0; e < P; ++e) gc[e] = rowbuf[e];
            done = true;
        }
        __builtin_amdgcn_wave_barrier();
    }

    // ---- 3. one-sided Jacobi on the columns of Pi R^T -----------------------
    // Columns are carried as d_c * a~_c: rotating the pair (c, p) is then
    // a~_c += mu a~_p, d_c *= cos, one fma per element. |a_c|^2 is carried
    // along and recomputed with the scales folded back in every sweep.
    //
    // Sweep order at P = 64: the xor steps m = 1..31 pair lanes inside each
    // 32-lane half (ds_swizzle). The pairs across the halves are met by
    // moving columns instead of fetching across halves: with the 16-lane rows
    // holding quarters [A B | C D], swapping rows 1 and 2 gives [A C | B D]
    // and steps m = 16..31 pair A-C and B-D; swapping rows 0 and 2 then gives
    // [B C | A D] for A-D and B-C. Every pair meets once per sweep, all 63
    // steps are swizzles, and a row swap costs about one permlane per value.
    //
    // Convergence: the iteration stops after a sweep in which the ranking of
    // the r largest columns did not change and no pair touching them needed a
    // rotation by more than sqrt(tol) in cosine: Jacobi converges
    // quadratically, so what such a sweep leaves is below tol.
    // Threshold on the cosine of two columns: P 2^-23, a hundred times that
    // for bf16 factors (7.6e-4 at P = 64), below the 2^-9 rounding of every
    // stored entry of L. fp32 factors, and INT4 factors (quantized from
    // exactly what an fp32 cache stores), keep the tight one.
    constexpr float kTolFactor = std::is_same<TF, uint16_t>::value ? 100.f : 1.f;
    const float tol = kTolFactor * (float)P * 1.1920929e-7f;
    const float tol2 = tol * tol;   // the tests compare squares: |gamma| > tol sqrt(a_lo a_hi)
    // requested rank, 0 for a rank chosen from the spectrum (adaptive ranks).
    // Then each sweep estimates that rank from the current column norms, and
    // the two columns after it are converged too (at most r_cap): a sweep
    // that changes the estimate is never the last.
    const int r_req = ref.which == 0 ? ref.rk : ref.rv;
    const int r_cap = min(g.max_rank, min(P, d));
    const bool adaptive = kAdapt ? __any(r_req == 0) : false;
    const float eps2 = g.rank_err * g.rank_err;
    int r_need = r_req > 0 ? r_req : r_cap;
    // tag = top flag << 8 | column id: the id travels with the column, so
    // equal norms (zero columns) are ranked the same way wherever they sit
    float dsc = 1.f, alpha = 0.f;
    int tag = (1 << 8) | c, larger = 0;
    int sweeps = 0;
    bool more = true;
    int rotated = 0;
    auto step = [&](int m) {
        float pg[P], beta, dp;
        int tag_p;
        switch (m) {
#define PKV_CQ_CASE(M) \
    case M: cq_swz<P, M>(gc, pg, alpha, beta, dsc, dp, tag, tag_p); break;
            PKV_CQ_CASE(1) PKV_CQ_CASE(2) PKV_CQ_CASE(3) PKV_CQ_CASE(4) PKV_CQ_CASE(5) PKV_CQ_CASE(6)
            PKV_CQ_CASE(7) PKV_CQ_CASE(8) PKV_CQ_CASE(9) PKV_CQ_CASE(10) PKV_CQ_CASE(11) PKV_CQ_CASE(12)
            PKV_CQ_CASE(13) PKV_CQ_CASE(14) PKV_CQ_CASE(15) PKV_CQ_CASE(16) PKV_CQ_CASE(17) PKV_CQ_CASE(18)
            PKV_CQ_CASE(19) PKV_CQ_CASE(20) PKV_CQ_CASE(21) PKV_CQ_CASE(22) PKV_CQ_CASE(23) PKV_CQ_CASE(24)
            PKV_CQ_CASE(25) PKV_CQ_CASE(26) PKV_CQ_CASE(27) PKV_CQ_CASE(28) PKV_CQ_CASE(29) PKV_CQ_CASE(30)
            default: cq_swz<P, 31>(gc, pg, alpha, beta, dsc, dp, tag, tag_p); break;
#undef PKV_CQ_CASE
        }
        // one accumulation chain (three fewer adds per step than four
        // partial sums, and measured faster); the partner lane sums the same
        // products in the same order, so both see the same gt
        float gt = 0.f;
#pragma unroll
        for (int e = 0; e < P; ++e) gt = fmaf(gc[e], pg[e], gt);
        const int partner = c ^ m;
        larger += (int)(beta > alpha) | ((int)(beta == alpha) & (int)((tag_p & 255) < (tag & 255)));
        const float gamma = gt * dsc * dp;
        const bool lo = c < partner;
        const float a_lo = lo ? alpha : beta, a_hi = lo ? beta : alpha;
        const float prod = a_lo * a_hi, g2 = gamma * gamma;
        const bool rot = a_lo > kCqTiny2 && a_hi > kCqTiny2 && g2 > tol2 * prod;
        const float zeta = (a_hi - a_lo) * __builtin_amdgcn_rcpf(2.f * gamma);
        const float tz = __builtin_copysignf(
            __builtin_amdgcn_rcpf(fabsf(zeta) + __builtin_amdgcn_sqrtf(fmaf(zeta, zeta, 1.f))), zeta);
        const float t = rot ? tz : 0.f;
        const float cs = rot ? __builtin_amdgcn_rsqf(fmaf(t, t, 1.f)) : 1.f;
        // a rotation touching the top columns above sqrt(tol) in cosine
        rotated |= (rot && ((tag | tag_p) >> 8) && g2 > tol * prod) ? 1 : 0;
        const float t_eff = lo ? -t : t;   // the lower column takes -sin
        const float mu = t_eff * (dp * __builtin_amdgcn_rcpf(dsc));
#pragma unroll
        for (int e = 0; e < P; ++e) gc[e] = fmaf(mu, pg[e], gc[e]);
        const float s_eff = cs * t_eff;
        alpha = fmaf(cs * cs, alpha, fmaf(2.f * cs * s_eff, gamma, s_eff * s_eff * beta));
        dsc *= cs;
    };
    while (more && sweeps < kMaxSweeps) {
        ++sweeps;
        larger = 0;
        float aa = 0.f, ab = 0.f;
#pragma unroll
        for (int e = 0; e < P; e += 2) {
            gc[e] *= dsc;
            gc[e + 1] *= dsc;
            aa = fmaf(gc[e], gc[e], aa);
            ab = fmaf(gc[e + 1], gc[e + 1], ab);
        }
        alpha = aa + ab;
        dsc = 1.f;
        rotated = 0;
        for (int m = 1; m < 32; ++m) step(m);
        if constexpr (P == 64) {
            // rows 1 <-> 2: three permlanes move two values
            auto swap12 = [](float &x, float &y) {
                const auto t1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
                const auto t2 = __builtin_amdgcn_permlane16_swap(t1[0], t1[1], false, false);
                const auto t3 = __builtin_amdgcn_permlane32_swap(t2[0], t2[1], false, false);
                x = __uint_as_float(t3[0]);
                y = __uint_as_float(t3[1]);
            };
            // rows 0 <-> 2: one permlane and one select per value
            const bool keep = ((lane >> 4) & 1) == ((lane >> 5) & 1);   // rows 0 and 3 take the second half-copy
            auto swap02 = [keep](float &x) {
                const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
                x = __uint_as_float(keep ? t[1] : t[0]);
            };
            float ti = __int_as_float(tag), li = __int_as_float(larger);
#pragma unroll
            for (int e = 0; e < P; e += 2) swap12(gc[e], gc[e + 1]);
            swap12(alpha, dsc);
            swap12(ti, li);
            tag = __float_as_int(ti);
            larger = __float_as_int(li);
            for (int m = 16; m < 32; ++m) step(m);
            ti = __int_as_float(tag);
            li = __int_as_float(larger);
#pragma unroll
            for (int e = 0; e < P; ++e) swap02(gc[e]);
            swap02(alpha);
            swap02(dsc);
            swap02(ti);
            swap02(li);
            tag = __float_as_int(ti);
            larger = __float_as_int(li);
            for (int m = 16; m < 32; ++m) step(m);
        }
        bool moved = false;
        if (adaptive) {
            const float a2 = fmaxf(alpha, 0.f);
            const int est = cq_adaptive_rank<P>(a2, sqrtf(a2) * gnorm, xnorm2, eps2, c, grp);
            const int rn = r_req > 0 ? r_req : min(r_cap, est + 2);
            moved = rn != r_need;
            r_need = rn;
        }
        const int top_new = larger < r_need ? 1 : 0;
        more = __any(rotated || moved || top_new != (tag >> 8));   // converged only on a settled ranking
        tag = (top_new << 8) | (tag & 255);
    }
    if (active && c == 0) {
        count_sweeps(sweeps);
        if (more) raise_status(PKV_DEV_NO_CONVERGE);
    }

    // ---- 4. eigenvalues, ranking, eigenvectors -----------------------------
    float an2a = 0.f, an2b = 0.f;
#pragma unroll
    for (int e = 0; e < P; e += 2) {
        gc[e] *= dsc;
        gc[e + 1] *= dsc;
        an2a = fmaf(gc[e], gc[e], an2a);
        an2b = fmaf(gc[e + 1], gc[e + 1], an2b);
    }
    const float an2 = an2a + an2b;
    const float lam = sqrtf(an2) * gnorm;   // eigenvalue of G (column norm of G Q J)
    const int rho = cq_rank<P>(an2, c, grp);
    const bool tinycol = !(an2 > kCqTiny2);
    // Adaptive rank: the smallest r with |X - X_r|_F^2 = |X|_F^2 - (sum of the
    // r largest eigenvalues of G) <= eps^2 |X|_F^2, capped at r_cap (only the
    // r_cap largest columns are converged, and only they enter the sums used).
    int r_own = r_req;
    if (adaptive) {
        const int cand = cq_adaptive_rank<P>(an2, lam, xnorm2, eps2, c, grp);
        if (r_req == 0) r_own = max(1, min(cand, r_cap));
    }
    {
        // A column at rounding level starts from the unit vector of its own
        // id k (the row of R it began as; ids travel with the columns): the
        // columns above it are combinations of rows of R before k, which are
        // upper triangular with nonzero diagonals, so e_k is never in their span.
        const int cid = tag & 255;
        const float inv = tinycol ? 0.f : __builtin_amdgcn_rsqf(an2);
#pragma unroll
        for (int e = 0; e < P; ++e) gc[e] = tinycol ? (e == cid ? 1.f : 0.f) : gc[e] * inv;
    }
    // The normalized columns are orthonormal to the rotation threshold. For
    // fp32 factor storage one Gram-Schmidt pass in rank order makes them
    // orthonormal to rounding (bf16 storage rounds far above the threshold).
    // A column at rounding level (rank-deficient page) has no direction of
    // its own: its unit vector is made orthogonal to the columns ranked above
    // it by Gram-Schmidt in rank order (twice).
    {
        constexpr bool kAll = std::is_same<TF, float>::value;
        const bool any_tiny = __any(tinycol && rho < r_need);
        if (kAll || any_tiny) {
            const int rmax = max(__builtin_amdgcn_readlane(r_need, 0), __builtin_amdgcn_readlane(r_need, 63));
            const int passes = any_tiny ? 2 : 1;
            const bool mine = kAll || tinycol;   // columns this pass orthogonalizes
            for (int pass = 0; pass < passes; ++pass) {
                for (int i = 0; i < rmax; ++i) {
                    const uint64_t bal = __ballot(rho == i);
                    const int piv0 = __builtin_ctzll(bal);
                    const int piv1 = P == 64 ? piv0 : 32 + __builtin_ctzll(bal >> 32);
                    float x[P];
#pragma unroll
                    for (int e = 0; e < P; ++e) x[e] = cq_group_bcast<P>(gc[e], piv0, piv1, grp);
                    float dot = 0.f;
#pragma unroll
                    for (int e = 0; e < P; ++e) dot = fmaf(x[e], gc[e], dot);
                    if (rho > i && mine)
#pragma unroll
                        for (int e = 0; e < P; ++e) gc[e] = fmaf(-dot, x[e], gc[e]);
                    __builtin_amdgcn_wave_barrier();
                    if (rho == i + 1 && mine) {
                        float n2 = 0.f;
#pragma unroll
                        for (int e = 0; e < P; ++e) n2 = fmaf(gc[e], gc[e], n2);
                        const float inv = n2 > 0.f ? __builtin_amdgcn_rsqf(n2) : 0.f;
#pragma unroll
                        for (int e = 0; e < P; ++e) gc[e] *= inv;
                    }
                }
            }
        }
    }

    // ---- 5. R = L^T X and the stores -----------------------------------------
    // L goes to LDS (sL[t][rank], 32 ranks, zero past r). Each lane then owns
    // two output dims for every rank: one 4-byte load per page row (a row is
    // one coalesced 256-byte read across the lanes) and 64 fmas against the
    // row's L entries, read as broadcasts.
    // the page's K and V ranks (each chosen by its own half when adaptive)
    int rk, rv;
    if constexpr (P == 64) {
        if (kAdapt) {   // kv = 0 decomposes K (its sections do not depend on rv), kv = 1 V
            if (kv == 0) rk_first = r_own;
            rk = rk_first;
            rv = r_own;
        } else {
            rk = ref.rk;
            rv = ref.rv;
        }
    } else {
        rk = __builtin_amdgcn_readlane(r_own, 0);    // lanes 0..31 decompose K, 32..63 V
        rv = __builtin_amdgcn_readlane(r_own, 32);
    }
    const int which = ref.which;
    const int r = which == 0 ? rk : rv;
    if (active && c == 0 && r_req == 0) {   // the chosen rank goes into the page's entry
        uint8_t *ent = (uint8_t *)(table + g.head_index(ref.b, ref.h) * g.max_pages + ref.j);
        ent[which == 0 ? offsetof(pkv_page, rank_k) : offsetof(pkv_page, rank_v)] = (uint8_t)r;
    }
    float *sL = cq_smem + 64 + grp * (P * 32);   // this group's P x 32 block
    float *sInvSig = cq_smem + 64 + 64 * 32 + grp * 32;
    {
        const float sig = sqrtf(fmaxf(lam, 0.f));
        const float scale = kQ4 ? sqrtf(sig) : 1.f;   // INT4: L~ = U Sigma^(1/2)
        if (rho < 32) {
            const int *tok = cq_tok + grp * P;
#pragma unroll
            for (int e = 0; e < P; ++e) sL[tok[e] * 32 + rho] = (rho < r && active) ? gc[e] * scale : 0.f;
            sInvSig[rho] = sig > 0.f ? 1.f / sig : 0.f;
        }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
    if (!active) return;

    const int64_t slot_off = (g.head_index(ref.b, ref.h) * g.max_pages + ref.j) * g.factor_slot_bytes;
    constexpr int kCols = 2;                      // dims per lane per pass
    int8_t *sRc = (int8_t *)(cq_smem + 64 + 64 * 32 + 64 + 64);   // INT4 only: R~ codes (P = 64: one group per wave)
    Int4Layout f4{};
    if constexpr (kQ4) f4 = int4_layout(P, d, rk, rv);
    // bf16 and INT4 factors at P = 64: the projection on the matrix cores.
    // 32x32x16 bf16 products with A = L^T (rank lane % 32; tokens
    // 16 s + 8 (lane / 32) + 0..7 of k-step s) split into bf16 hi + lo, so L
    // enters with 16 significant bits, and B = X, exact. Lane (n, h) owns
    // dims k = 64 J + 2 n and k + 1 in two accumulator tiles, so one
    // 4-byte page read feeds both; accumulator register v holds rank
    // 8 (v / 4) + 4 h + v % 4 of its dim. fp32 factors take the exact VALU
    // loop below.
    constexpr bool kMfmaProj = P == 64 && !std::is_same<TF, float>::value;
    if constexpr (kMfmaProj) {
        const int n = lane & 31, h = lane >> 5;
        float isg[16];   // INT4: 1 / sigma of this lane's ranks
        if constexpr (kQ4) {
#pragma unroll
            for (int v = 0; v < 16; ++v) isg[v] = sInvSig[8 * (v >> 2) + 4 * h + (v & 3)];
        }
        // one block of 64 dims at a time: two accumulator tiles
#pragma unroll 1
        for (int k = 2 * n; k - 2 * n < d; k += 64) {
            cq_f32x16 ae = {}, ao = {};
            const bool kin = k < d;
            // an offset the compiler cannot see is zero: the L operands are
            // rebuilt from LDS in every block rather than hoisted out of the
            // loop and held (32 more registers, spilled to scratch memory)
            int z;
            asm volatile("v_mov_b32 %0, 0" : "=v"(z));
            const float *sLz = sL + z;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                uint32_t hw[4], lw[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    cq_split2(sLz[(16 * s + 8 * h + 2 * i) * 32 + n], sLz[(16 * s + 8 * h + 2 * i + 1) * 32 + n], hw[i], lw[i]);
                const cq_bf16x8 ahi = __builtin_bit_cast(cq_bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
                const cq_bf16x8 alo = __builtin_bit_cast(cq_bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
                cq_bf16x8 be = {}, bo = {};
                if (kin) cq_load_dim_pair(X, ref.transposed, P, d, k, 16 * s + 8 * h, be, bo);
                ae = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, be, ae, 0, 0, 0);
                ao = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, bo, ao, 0, 0, 0);
                ae = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, be, ae, 0, 0, 0);
                ao = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, bo, ao, 0, 0, 0);
            }
            if (!kin) continue;
            if constexpr (kQ4) {
                // R~ = Sigma^(-1/2) R (the products used L~ = L Sigma^(1/2));
                // a dim's scale spans all ranks: this lane's 16 and lane ^ 32's
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    cq_f32x16 &a = u == 0 ? ae : ao;
                    float amax = 0.f;
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        a[v] *= isg[v];
                        if (8 * (v >> 2) + 4 * h + (v & 3) < r) amax = fmaxf(amax, fabsf(a[v]));
                    }
                    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(amax), __float_as_uint(amax),
                                                                     false, false);
                    amax = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));   // the same in both lanes
                    const uint16_t hs = f16_rne((double)amax / (double)kQ4Max);
                    if (h == 0)
                        *(uint16_t *)(factor + slot_off + (which == 0 ? q4_rk_scale(f4, k + u) : q4_rv_scale(f4, k + u))) = hs;
                    const float sc = half_bits_to_f32(hs);
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int rr = 8 * (v >> 2) + 4 * h + (v & 3);
                        const int8_t code = (int8_t)(rr < r ? q4_code(a[v], sc) : 0);
                        if (which == 0) sRc[rr * d + k + u] = code;
                        else sRc[(k + u) * 32 + rr] = code;
                    }
                }
            } else {
                const int rk4 = r4(rk), rv4 = r4(rv);
                const FactorLayout fl = factor_layout(P, d, rk, rv, g.key_t != 0);
                uint16_t *Ak = (uint16_t *)(factor + slot_off);
                if (which == 0 && !g.key_t) {
                    uint16_t *Bk = Ak + fl.bk;             // R_K, rk x d: dims k, k + 1 side by side
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int a = 8 * (v >> 2) + 4 * h + (v & 3);
                        if (a < rk) *(uint32_t *)(Bk + (int64_t)a * d + k) = cq_pack_bf16(ae[v], ao[v]);
                    }
                } else {
                    // R_K^T (d x r4(rk)) or R_V^T (d x r4(rv)), zero past the rank:
                    // four consecutive ranks per 8-byte store
                    const int rw = which == 0 ? rk4 : rv4;
                    uint16_t *Bt = Ak + (which == 0 ? fl.bk : fl.bvt);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int a0 = 8 * j + 4 * h;
                        if (a0 >= rw) continue;
                        *(uint2 *)(Bt + (int64_t)k * rw + a0) =
                            make_uint2(cq_pack_bf16(ae[4 * j], ae[4 * j + 1]), cq_pack_bf16(ae[4 * j + 2], ae[4 * j + 3]));
                        *(uint2 *)(Bt + (int64_t)(k + 1) * rw + a0) =
                            make_uint2(cq_pack_bf16(ao[4 * j], ao[4 * j + 1]), cq_pack_bf16(ao[4 * j + 2], ao[4 * j + 3]));
                    }
                }
            }
        }
    }
    for (int k0 = 0; k0 < (kMfmaProj ? 0 : d); k0 += kCols * P) {
        const int k = k0 + kCols * c;
        const bool kin = k < d;
        float acc[kCols][32];
#pragma unroll
        for (int u = 0; u < kCols; ++u)
#pragma unroll
            for (int a = 0; a < 32; ++a) acc[u][a] = 0.f;
        for (int t = 0; t < P; ++t) {
            float x0 = 0.f, x1 = 0.f;
            if (kin) {
                if (!ref.transposed) {
                    const uint32_t w = *(const uint32_t *)(X + (int64_t)t * d + k);
                    x0 = __uint_as_float(w << 16);
                    x1 = __uint_as_float(w & 0xffff0000u);
                } else {
                    x0 = bf16_to_f32(X[(int64_t)k * P + t]);
                    x1 = bf16_to_f32(X[(int64_t)(k + 1) * P + t]);
                }
            }
            const float4 *lrow = (const float4 *)(sL + t * 32);
#pragma unroll
            for (int a4 = 0; a4 < 8; ++a4) {
                const float4 l = lrow[a4];
                acc[0][4 * a4 + 0] = fmaf(l.x, x0, acc[0][4 * a4 + 0]);
                acc[0][4 * a4 + 1] = fmaf(l.y, x0, acc[0][4 * a4 + 1]);
                acc[0][4 * a4 + 2] = fmaf(l.z, x0, acc[0][4 * a4 + 2]);
                acc[0][4 * a4 + 3] = fmaf(l.w, x0, acc[0][4 * a4 + 3]);
                acc[1][4 * a4 + 0] = fmaf(l.x, x1, acc[1][4 * a4 + 0]);
                acc[1][4 * a4 + 1] = fmaf(l.y, x1, acc[1][4 * a4 + 1]);
                acc[1][4 * a4 + 2] = fmaf(l.z, x1, acc[1][4 * a4 + 2]);
                acc[1][4 * a4 + 3] = fmaf(l.w, x1, acc[1][4 * a4 + 3]);
            }
        }
        if (!kin) continue;
        if constexpr (kQ4) {
            // R~ = Sigma^(-1/2) R: the accumulation used L~ = L Sigma^(1/2), so
            // divide by sigma. R~'s scales run down a column (one dim, all
            // ranks), which this lane holds: its scale goes to the slot and
            // its codes to LDS (K: [rank][dim], V: [dim][rank]) for packing.
#pragma unroll
            for (int u = 0; u < kCols; ++u) {
                float amax = 0.f;
#pragma unroll
                for (int a = 0; a < 32; ++a) {
                    acc[u][a] *= sInvSig[a];
                    if (a < r) amax = fmaxf(amax, fabsf(acc[u][a]));
                }
                const uint16_t hs = f16_rne((double)amax / (double)kQ4Max);
                *(uint16_t *)(factor + slot_off + (which == 0 ? q4_rk_scale(f4, k + u) : q4_rv_scale(f4, k + u))) = hs;
                const float sc = half_bits_to_f32(hs);
#pragma unroll
                for (int a = 0; a < 32; ++a) {
                    const int8_t code = (int8_t)(a < r ? q4_code(acc[u][a], sc) : 0);
                    if (which == 0) sRc[a * d + k + u] = code;
                    else sRc[(k + u) * 32 + a] = code;
                }
            }
        } else {
            const int rk4 = r4(rk), rv4 = r4(rv);
            const FactorLayout fl = factor_layout(P, d, rk, rv, g.key_t != 0);
            TF *Ak = (TF *)(factor + slot_off);
            if (which == 0 && g.key_t) {
                TF *Bkt = Ak + fl.bk;                      // R_K^T, d x r4(rk), zero past rk
#pragma unroll
                for (int a = 0; a < 32; ++a)
                    if (a < rk4) {
                        st(Bkt, (int64_t)k * rk4 + a, acc[0][a]);
                        st(Bkt, (int64_t)(k + 1) * rk4 + a, acc[1][a]);
                    }
            } else if (which == 0) {
                TF *Bk = Ak + fl.bk;                       // R_K, rk x d
#pragma unroll
                for (int a = 0; a < 32; ++a)
                    if (a < rk) {
                        st(Bk, (int64_t)a * d + k, acc[0][a]);
                        st(Bk, (int64_t)a * d + k + 1, acc[1][a]);
                    }
            } else {
                TF *Bvt = Ak + fl.bvt;                     // R_V^T, d x r4(rv), zero past rv
#pragma unroll
                for (int a = 0; a < 32; ++a)
                    if (a < rv4) {
                        st(Bvt, (int64_t)k * rv4 + a, acc[0][a]);
                        st(Bvt, (int64_t)(k + 1) * rv4 + a, acc[1][a]);
                    }
            }
        }
    }
    if constexpr (kQ4) {
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
        float *sScale = (float *)(sRc + 32 * d);
        q4_store_codes(factor + slot_off, f4, P, d, r, which, sL, sRc, sScale, lane);
    } else {
        // L: A_K = L_K (P x r4(rk), zero past rk) row by row, A_V^T = L_V^T (rv x P)
        const FactorLayout fl = factor_layout(P, d, rk, rv, g.key_t != 0);
        TF *Ak = (TF *)(factor + slot_off);
        const int t = c;
        if (which == 0) {
            const int rk4 = r4(rk);
            for (int a = 0; a < rk4; ++a) st(Ak, (int64_t)t * rk4 + a, sL[t * 32 + a]);
        } else {
            TF *Avt = Ak + fl.avt;
            for (int a = 0; a < rv; ++a) st(Avt, (int64_t)a * P + t, sL[t * 32 + a]);
        }
    }
    }   // passes
}

// Whether the matrix-core decomposition covers this geometry.
inline bool compress_qr_supported(const Geo &g) {
    return g.dense_dtype == PKV_BF16 && (g.P == 32 || g.P == 64) && g.d % 16 == 0 && g.d <= 256;
}

template <typename TF, int P, bool kAdapt>
hipError_t launch_compress_qr_a(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                                int64_t n_decomp) {
    constexpr int per_wave = (64 / P) * (P == 64 && kAdapt ? 2 : 1);   // decompositions per wavefront
    const size_t smem = (size_t)cq_wave_lds(L.geo.d, is_q4<TF>::value) * sizeof(float);
    const int64_t blocks = ceil_div(n_decomp, (int64_t)per_wave);
    LayerPtrs p = layer_ptrs(L);
    if (src.list)
        hipLaunchKernelGGL((k_compress_qr<TF, P, kAdapt, true>), dim3((unsigned)blocks), dim3(64), smem, L.stream,
                           L.geo, p.table, p.dense, p.factor, items, src, n_decomp);
    else
        hipLaunchKernelGGL((k_compress_qr<TF, P, kAdapt>), dim3((unsigned)blocks), dim3(64), smem, L.stream,
                           L.geo, p.table, p.dense, p.factor, items, src, n_decomp);
    return hipGetLastError();
}

template <typename TF, int P>
hipError_t launch_compress_qr_t(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                                int64_t n_decomp) {
    return L.geo.rank_err > 0.f ? launch_compress_qr_a<TF, P, true>(L, items, src, n_decomp)
                                : launch_compress_qr_a<TF, P, false>(L, items, src, n_decomp);
}

hipError_t launch_compress_qr(const LaunchCtx &L, const CompressItems &items, const CompressSrc &src,
                              int64_t n_decomp) {
    const int ft = L.geo.factor_dtype;
    if (ft == PKV_INT4) {
        if (L.geo.P != 64) return hipErrorInvalidValue;
        return launch_compress_qr_t<q4_t, 64>(L, items, src, n_decomp);
    }
    if (L.geo.P == 64)
        return ft == PKV_BF16 ? launch_compress_qr_t<uint16_t, 64>(L, items, src, n_decomp)
                              : launch_compress_qr_t<float, 64>(L, items, src, n_decomp);
    return ft == PKV_BF16 ? launch_compress_qr_t<uint16_t, 32>(L, items, src, n_decomp)
                          : launch_compress_qr_t<float, 32>(L, items, src, n_decomp);
}

}  // namespace pkv
