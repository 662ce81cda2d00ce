// Mixed-page decode attention on the matrix cores (bf16 pages and factors,
// d = 64 or 128, P = 16, 32 or 64, ranks <= 32, query group <= 16).
//
// One wavefront streams a set of pages of one (sequence, KV head). All four
// contractions of a factor page (Eq. (4)) are 16x16x32 bf16 MFMAs with the
// query group in the N dimension:
//   Z^T = R_K Q^T        (M = rank,  K = d)       R_K   stored r x d
//   S^T = L_K Z^T        (M = token, K = rank)    L_K   stored P x r4
//   Y^T = L_V^T E^T      (M = rank,  K = token)   L_V^T stored r x P
//   O^T += R_V^T Y^T     (M = dim,   K = rank)    R_V^T stored d x r4
// The accumulator of one product becomes the B operand of the next without
// moving data between lanes: lane (n, q) = (lane % 16, lane / 16) holds rows
// 4q..4q+3 of column n of each 16-row tile, and the M rows of the tiles are
// assigned to ranks (tokens) so that two tiles give the lane exactly the K
// entries 8q..8q+7 a B operand needs, in natural order:
//   rank tile rt,  row m  ->  rank  8 (m / 4) + 4 rt + m % 4
//   token tile tt, row m  ->  token 32 (tt / 2) + 8 (m / 4) + 4 (tt % 2) + m % 4   (P >= 32)
// Every A operand is then one contiguous 16-byte slice of a stored row.
// fp32 intermediates (Z, exp weights, Y) enter the MFMA as a bf16 hi/lo pair
// (two MFMAs), keeping about 16 mantissa bits; Q and the stored pages are
// exact in bf16. Dense pages use S^T = K Q^T and O^T += V^T E^T with V stored
// transposed. The normalizer is a fifth product, ones x E^T, so it needs no
// per-token additions.
//
// Caches of pre-RoPE keys (ROPE): a factor page's keys are rebuilt on the
// matrix cores and rotated before the scores, since RoPE does not commute
// with the factorization. K^T = R_K^T L_K^T (M = dim, K = rank, N = token,
// R_K^T stored d x r4) comes out with lane (n, q) holding token n and dims
// 8q..8q+7 of each 32-dim chunk over a pair of dim tiles (the rank-tile map
// read as a dim map), which is the A operand layout of S^T = K Q^T. The
// rotate-half pairs (i, i + d/2) sit in the same lane, so the rotation needs
// no data movement. Keys are rotated by their offset within the unit (a
// table shared by every unit) and the query group by the unit's first
// position, once per unit; both enter S^T as fp16 hi/lo pairs. Dense keys
// are rotated the same way from their bf16 operands.
//
// Factor operands are read with buffer loads, one resource per section of the
// slot sized to that section: rank rows past the page's rank fall outside it
// and read as zero, which also zeroes the matching entries of Z and Y, so the
// K columns a lane reads past a row's end (always finite data of the same
// page) multiply zeros. A page that is not a factor page gets empty
// resources. Each wave keeps its loads half a page ahead of its math (see
// k_attn_mfma).
// Included by pkv_kernels.hip.

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMfmaWaves = 8;     // wavefronts per workgroup, bf16 kernel (two per SIMD)
constexpr int kMfmaWavesQ4 = 12;  // INT4 kernel: three per SIMD to cover its dependency stalls
template <bool Q4>
constexpr int attn_waves() { return Q4 ? kMfmaWavesQ4 : kMfmaWaves; }
constexpr int kQ4DenseStage = 256;   // dense pages of one head a workgroup can queue (INT4 kernel)
// The running max (log2 units) is raised only when a score exceeds it by more
// than this; below that the exp weights stay under 2^32 and the fp32 sums
// cannot overflow, so most pages skip the cross-lane max and the rescale.
constexpr float kLazyLog2 = 32.0f;
constexpr float kLazyLog2Q4 = 4.0f;   // INT4 kernel: weights stay at most 2^4 (fp16 operands)
constexpr int kBufferDword3 = 0x00020000; // raw buffer, 32-bit data format

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
__device__ inline f32x4 zero_f4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Row maps of the 16-row tiles (see the header comment).
__device__ inline int rank_row(int rt, int m) { return 8 * (m >> 2) + 4 * rt + (m & 3); }
template <int P>
__device__ inline int token_row(int tt, int m) {
    return P >= 32 ? 32 * (tt >> 1) + 8 * (m >> 2) + 4 * (tt & 1) + (m & 3) : m;
}

__device__ inline __amdgpu_buffer_rsrc_t section_rsrc(const char *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(base), (short)0, (int)bytes, kBufferDword3);
}
// Buffer loads: per-lane byte offset `voff` (range checked), wave-uniform
// byte offset `soff`.
__device__ inline bf16x8 bld8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ inline bf16x4 bld4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

// Two fp32 values -> bf16 hi pair (round to nearest) and bf16 lo pair of the
// remainders, as packed dwords.
__device__ inline void split2(float a, float b, uint32_t &hi, uint32_t &lo) {
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
    const float ha = __builtin_bit_cast(float, h << 16), hb = __builtin_bit_cast(float, h & 0xffff0000u);
    hi = h;
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a - ha, b - hb}, bf16x2));
}
// Two accumulator tiles -> hi and lo B operands (K entries 8q..8q+7).
__device__ inline void split_tiles(const f32x4 &x0, const f32x4 &x1, bf16x8 &hi, bf16x8 &lo) {
    uint32_t h0, h1, h2, h3, l0, l1, l2, l3;
    split2(x0[0], x0[1], h0, l0);
    split2(x0[2], x0[3], h1, l1);
    split2(x1[0], x1[1], h2, l2);
    split2(x1[2], x1[3], h3, l3);
    hi = __builtin_bit_cast(bf16x8, u32x4{h0, h1, h2, h3});
    lo = __builtin_bit_cast(bf16x8, u32x4{l0, l1, l2, l3});
}
// One tile (the other half of K zero).
__device__ inline void split_tile(const f32x4 &x0, bf16x8 &hi, bf16x8 &lo) {
    uint32_t h0, h1, l0, l1;
    split2(x0[0], x0[1], h0, l0);
    split2(x0[2], x0[3], h1, l1);
    hi = __builtin_bit_cast(bf16x8, u32x4{h0, h1, 0u, 0u});
    lo = __builtin_bit_cast(bf16x8, u32x4{l0, l1, 0u, 0u});
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ inline f32x4 mfma_f16(const f16x8 &a, const f16x8 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// fp32 pair -> fp16 hi (toward zero) and lo (the remainder), as packed words.
// The remainder a - hi is one mixed-precision fma with hi as its fp16
// operand (the -1 is kept opaque so the compiler keeps the fma form); hi and
// lo together keep about 22 bits.
__device__ inline void split2_f16(float a, float b, uint32_t &hi, uint32_t &lo) {
    const f16x2 h = __builtin_bit_cast(f16x2, __builtin_amdgcn_cvt_pkrtz(a, b));
    float m1 = -1.f;
    asm("" : "+v"(m1));
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(fmaf((float)h[0], m1, a), fmaf((float)h[1], m1, b)));
}

// Operand slices of one factor page held by one lane, in two halves: the key
// factors feed phase 1 (scores and softmax), the value factors phase 2.
template <int D, int P>
struct KeyOps {
    bf16x8 bk[2][D / 32];  // R_K row rank_row(rt, n), d-chunk s
    bf16x8 ak[P / 16];     // L_K row token_row(tt, n), ranks 8q..8q+7
};
template <int D, int P>
struct ValueOps {
    bf16x8 av[2][(P + 31) / 32];  // L_V^T row rank_row(rt, n), tokens of K-step ks
    bf16x8 bv[D / 16];            // R_V^T row 16 dt + n, ranks 8q..8q+7
};

// Per page: one buffer resource per section and the page-dependent parts of
// the lane offsets. Lane-constant offsets live in LaneOffs.
struct PageRes {
    __amdgpu_buffer_rsrc_t ak, bk, bvt, avt;
    int rk, rv, rk4, rv4;
    int kst;   // ROPE: elements per row of the bk section (d for dense K, r4(rk) for R_K^T)
    int kcs;   // ROPE: byte step of one 32-dim chunk (64 along a dense K row, 32 rows of R_K^T)
};
struct LaneOffs {
    uint32_t bk[2], av[2];   // R_K / L_V^T row rank_row(rt, n), chunk q
    uint32_t tok0;           // token_row(0, n)
};

// One step of a wave's stream: a factor page, or a unit of min(P, 32)
// tokens of a dense page (`half` = which unit), so that dense pages flow
// through the same pipelined loop and operand registers as factor pages.
struct Unit {
    pkv_page e;   // e.kind == PKV_EMPTY: no unit
    int64_t j;    // logical page
    int half;     // dense pages: unit index within the page
};
template <int P>
__device__ constexpr int dense_unit_tokens() { return P < 32 ? P : 32; }

template <int D, int P, bool ROPE = false>
__device__ inline PageRes unit_res(const char *factor, int64_t fslot_bytes, const char *dense, int64_t dslot_bytes,
                                   const Unit &u) {
    PageRes r;
    r.kst = D;
    r.kcs = 64;
    if (u.e.kind == PKV_DENSE) {
        // K rows of the unit feed the R_K registers (the same rank_row lane
        // map serves as the token map of two 16-row tiles), V^T columns of
        // the unit the R_V^T registers with row length P.
        constexpr int UT = dense_unit_tokens<P>();
        const char *base = dense + u.e.slot * dslot_bytes;
        r.rk = r.rv = 0;
        r.rk4 = 0;
        r.rv4 = P;
        r.ak = section_rsrc(base, 0u);
        r.avt = section_rsrc(base, 0u);
        r.bk = section_rsrc(base + 2 * UT * u.half * D, (uint32_t)(2 * UT * D));
        r.bvt = section_rsrc(base + 2 * P * D + 2 * UT * u.half, (uint32_t)(2 * (D * P - UT * u.half)));
        return r;
    }
    const bool is_f = u.e.kind == PKV_FACTOR;
    r.rk = is_f ? u.e.rank_k : 0;
    r.rv = is_f ? u.e.rank_v : 0;
    r.rk4 = r4(r.rk);
    r.rv4 = r4(r.rv);
    if (ROPE) {
        r.kst = r.rk4;
        r.kcs = 64 * r.rk4;
    }
    const FactorLayout fl = factor_layout(P, D, r.rk, r.rv, ROPE);
    const char *base = factor + (is_f ? u.e.slot : 0) * fslot_bytes;
    r.ak = section_rsrc(base, (uint32_t)(2 * fl.bk));
    r.bk = section_rsrc(base + 2 * fl.bk, (uint32_t)(2 * (fl.bvt - fl.bk)));
    r.bvt = section_rsrc(base + 2 * fl.bvt, (uint32_t)(2 * (fl.avt - fl.bvt)));
    r.avt = section_rsrc(base + 2 * fl.avt, (uint32_t)(2 * (fl.end - fl.avt)));
    return r;
}

// Pre-RoPE caches: the key chunks of one rotate-half pair (s0, s0 + d/64).
// Dense K: row rank_row(rt, n), columns 32 s + 8q..8q+7 (row length d);
// R_K^T: row 32 s + rank_row(rt, n), columns 8q..8q+7 (row length r4(rk)).
template <int D, int P>
__device__ inline void issue_key_pair_rope(KeyOps<D, P> &f, const PageRes &r, int n, int q, int s0) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        const uint32_t vb = 2u * ((uint32_t)rank_row(rt, n) * (uint32_t)r.kst + 8u * q);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int s = s0 + k * (D / 64);
            f.bk[rt][s] = bld8(r.bk, vb, (uint32_t)s * (uint32_t)r.kcs);
        }
    }
}

// first_pair: pre-RoPE caches, the first rotate-half pair whose key chunks
// are still to be loaded (the earlier ones were issued during phase 1)
template <int D, int P, bool ROPE = false>
__device__ inline void issue_key_loads(KeyOps<D, P> &f, const PageRes &r, const LaneOffs &lo, int n, int q,
                                       int first_pair = 0) {
    if constexpr (ROPE) {
#pragma unroll
        for (int s0 = 0; s0 < D / 64; ++s0)
            if (s0 >= first_pair) issue_key_pair_rope<D, P>(f, r, n, q, s0);
    } else {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int s = 0; s < D / 32; ++s) f.bk[rt][s] = bld8(r.bk, lo.bk[rt] + 64u * s, 0u);
    }
    const uint32_t v_ak = 2u * (lo.tok0 * r.rk4 + 8 * q);
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) {
        const uint32_t toff = P >= 32 ? 32u * (tt >> 1) + 4u * (tt & 1) : 0u;
        f.ak[tt] = bld8(r.ak, v_ak, 2u * toff * r.rk4);
    }
}

template <int D, int P>
__device__ inline void issue_value_loads(ValueOps<D, P> &f, const PageRes &r, const LaneOffs &lo, int n, int q) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ks = 0; ks < (P + 31) / 32; ++ks)
            f.av[rt][ks] = P >= 32 ? bld8(r.avt, lo.av[rt] + 64u * ks, 0u) : cat4(bld4(r.avt, lo.av[rt], 0u), zero4());
    const uint32_t v_bv = 2u * (n * r.rv4 + 8 * q);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) f.bv[dt] = bld8(r.bvt, v_bv, 32u * dt * r.rv4);
}

// Running softmax state of one wave: O^T tiles, the normalizer (every row of
// `l` holds its column's value) and the running max (log2 units).
template <int D>
struct WaveState {
    f32x4 o[D / 16];
    f32x4 l;
    float m_run;
};

// Online softmax over one page's raw scores st (Eq. (5) state update): the
// running max is raised (and the state rescaled) only when needed, then st
// holds the exp weights. Rows at or past `rows` are masked (dense pages only;
// factor pages are complete).
template <int D, int P, bool MASK, int LAZY = (int)kLazyLog2>
__device__ inline void page_exp(WaveState<D> &w, f32x4 (&st)[P / 16], int rows, int q, float c2) {
    constexpr int TT = P / 16, DT = D / 16;
    float pm = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            if (MASK && token_row<P>(tt, 4 * q + v) >= rows) st[tt][v] = -INFINITY;
            pm = fmaxf(pm, st[tt][v]);
        }
    if (__builtin_amdgcn_ballot_w64(pm * c2 > w.m_run + (float)LAZY) != 0) {
        pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
        const float m_new = fmaxf(w.m_run, pm * c2);
        const float alpha = w.m_run == -INFINITY ? 0.f : exp2f(w.m_run - m_new);
#pragma unroll
        for (int t = 0; t < DT; ++t) w.o[t] *= alpha;
        w.l *= alpha;
        w.m_run = m_new;
    }
    const float nm = -w.m_run;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) st[tt][v] = __builtin_amdgcn_exp2f(fmaf(st[tt][v], c2, nm));
}

// bf16 pages: the exp weights become hi/lo B operands of the token
// contraction, and the normalizer (every row of w.l) is a ones x E^T product.
template <int D, int P, bool MASK>
__device__ inline void page_softmax(WaveState<D> &w, f32x4 (&st)[P / 16], bf16x8 (&eh)[(P + 31) / 32],
                                    bf16x8 (&el)[(P + 31) / 32], int rows, int q, float c2) {
    constexpr int TT = P / 16, KS = (P + 31) / 32;
    page_exp<D, P, MASK>(w, st, rows, q, c2);
    const bf16x8 ones = bf16x8{1, 1, 1, 1, 1, 1, 1, 1};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (2 * ks + 1 < TT) split_tiles(st[2 * ks], st[2 * ks + 1], eh[ks], el[ks]);
        else split_tile(st[2 * ks], eh[ks], el[ks]);
        w.l = mfma_bf16(ones, eh[ks], w.l);
        w.l = mfma_bf16(ones, el[ks], w.l);
    }
}

// Phase 1 of a unit. Factor page: Z^T = R_K Q^T, S^T = L_K Z^T, softmax.
// Dense unit: the same first product with the unit's K rows in the R_K
// registers is already S^T (two 16-token tiles); softmax with tokens at or
// past `rows` masked. Either way the exp weights come out as hi/lo B operands
// of the token contraction (a dense unit uses K-step 0 only).
template <int D, int P>
__device__ inline void unit_phase1(WaveState<D> &w, const KeyOps<D, P> &f, const bf16x8 (&qb)[D / 32], bool dense,
                                   int rows, bf16x8 (&eh)[(P + 31) / 32], bf16x8 (&el)[(P + 31) / 32], int q,
                                   float c2) {
    // both rank tiles hold ranks below 16 (rank_row), so neither is skipped
    // for small ranks; rows past the rank read as zero
    f32x4 z[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        z[rt] = zero_f4();
#pragma unroll
        for (int s = 0; s < D / 32; ++s) z[rt] = mfma_bf16(f.bk[rt][s], qb[s], z[rt]);
    }
    if (dense) {
        bf16x8 eh1[1], el1[1];
        page_softmax<D, 32, true>(w, z, eh1, el1, rows, q, c2);
        eh[0] = eh1[0];
        el[0] = el1[0];
        return;
    }
    bf16x8 zh, zl;
    split_tiles(z[0], z[1], zh, zl);
    f32x4 st[P / 16];
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) {
        st[tt] = mfma_bf16(f.ak[tt], zh, zero_f4());
        st[tt] = mfma_bf16(f.ak[tt], zl, st[tt]);
    }
    page_softmax<D, P, false>(w, st, eh, el, P, q, c2);
}

// RoPE angles in revolutions: w_i = theta_i / 2 pi is held in LDS as
// wh + wl (fp64 on the way). The rotation of position t0 + tau is split as
// R(t0 + tau) = R(t0) R(tau), and q . R(t0) R(tau) k = (R(-t0) q) . (R(tau) k):
// the keys of a unit are rotated by their offset tau from the unit's start
// with cos / sin (tau theta_i) from a table shared by every unit, and the
// query group is rotated once per unit by -t0 theta_i. Both angles come from
// the fraction of their product with w_i (split exactly with an fma, right
// to ~2^-24 revolutions at any position below 2^24), and the hardware sine
// and cosine take revolutions.
__device__ inline float rope_frac(float t0, float wh, float wl) {
    const float p = t0 * wh;
    const float e = fmaf(t0, wh, -p);
    return __builtin_amdgcn_fractf(__builtin_amdgcn_fractf(p) + fmaf(t0, wl, e));
}

// Rotates the pairs (x0[u], x1[u]) of one lane's key row: x0[u] is dim
// 32 s + 8 q + u, x1[u] its partner d/2 above; ct / st: cos and sin of
// tau theta_i for the row's offset tau.
__device__ inline void rope_pair(float (&x0)[8], float (&x1)[8], int s, int q, const float *ct, const float *st) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i0 = 32 * s + 8 * q + 4 * h;
        const f32x4 c = *(const f32x4 *)(ct + i0);
        const f32x4 sn = *(const f32x4 *)(st + i0);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float a = x0[4 * h + v], b = x1[4 * h + v];
            x0[4 * h + v] = fmaf(a, c[v], -b * sn[v]);
            x1[4 * h + v] = fmaf(b, c[v], a * sn[v]);
        }
    }
}

// fp32 entries -> fp16 hi/lo operands (8 dims of one chunk).
__device__ inline void split8_f16(const float (&x)[8], f16x8 &hi, f16x8 &lo) {
    uint32_t hd[4], ld[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) split2_f16(x[2 * u], x[2 * u + 1], hd[u], ld[u]);
    hi = __builtin_bit_cast(f16x8, u32x4{hd[0], hd[1], hd[2], hd[3]});
    lo = __builtin_bit_cast(f16x8, u32x4{ld[0], ld[1], ld[2], ld[3]});
}

// LDS tables of a pre-RoPE cache: w_i as wh + wl (D floats); cos and sin of
// tau theta_i for tau < P (rows of D/2 + 4 floats, padded against bank
// conflicts); the query group in fp32 in the lanes' B operand layout
// ([chunk][lane][8]); per wave, cos | sin of t0 theta_i of its current unit.
template <int D, int P>
struct RopeLds {
    static constexpr int kRow = D / 2 + 4;
    const float *rw, *ct, *st, *qf;
    float *r0;
};

// One rotate-half pair of 32-dim chunks (s0, s0 + d/64) of the query group
// rotated by -t0 theta_i, as fp16 hi/lo B operands of the score product
// (about 22 bits): [0] chunk s0, [1] chunk s0 + d/64.
template <int D, int P>
__device__ inline void rope_query(const RopeLds<D, P> &L, int s0, int lane, int q, f16x8 (&qh)[2], f16x8 (&ql)[2]) {
    float a[8], b[8];
    const float *pa = L.qf + (s0 * 64 + lane) * 8, *pb = L.qf + ((s0 + D / 64) * 64 + lane) * 8;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i0 = 32 * s0 + 8 * q + 4 * h;
        const f32x4 xa = *(const f32x4 *)(pa + 4 * h), xb = *(const f32x4 *)(pb + 4 * h);
        const f32x4 c = *(const f32x4 *)(L.r0 + i0), sn = *(const f32x4 *)(L.r0 + D / 2 + i0);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            a[4 * h + v] = fmaf(xa[v], c[v], xb[v] * sn[v]);
            b[4 * h + v] = fmaf(xb[v], c[v], -xa[v] * sn[v]);
        }
    }
    split8_f16(a, qh[0], ql[0]);
    split8_f16(b, qh[1], ql[1]);
}

// Phase 1 of a unit of a pre-RoPE cache. Factor page: per token tile,
// K^T = R_K^T L_K^T, rotation by the token's offset tau, S^T = K Q^T against
// the query group rotated by -t0 theta_i; rank entries at or past r4(rk) of
// the L_K operand are zeroed (the R_K^T operand holds the next row's values
// there). Dense unit: the K rows are rotated, then the same product. Keys and
// queries enter it as fp16 hi/lo pairs (three products: hi hi, lo hi, hi lo).
// The loops take one rotate-half pair of 32-dim chunks at a time, outermost,
// so only that pair of the rotated query is held, and a pair's key chunks are
// free once it is done: pair_done(s0) is called then (but not after the last
// pair), for the next unit's loads of those chunks. t0: position of the
// unit's first token.
template <int D, int P, typename PairDone>
__device__ inline void unit_phase1_rope(WaveState<D> &w, const KeyOps<D, P> &f, const RopeLds<D, P> &L,
                                        bool dense, int rows, bf16x8 (&eh)[(P + 31) / 32],
                                        bf16x8 (&el)[(P + 31) / 32], int n, int q, float c2, int64_t t0, int rk4,
                                        PairDone pair_done) {
    constexpr int R = RopeLds<D, P>::kRow;
    const int lane = q * 16 + n;
    if (lane < D / 2) {
        const float fr = rope_frac((float)t0, L.rw[lane], L.rw[D / 2 + lane]);
        L.r0[lane] = __builtin_amdgcn_cosf(fr);
        L.r0[D / 2 + lane] = __builtin_amdgcn_sinf(fr);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the wave's row is written before it is read
    if (dense) {
        f32x4 z[2] = {zero_f4(), zero_f4()};
#pragma unroll
        for (int s0 = 0; s0 < D / 64; ++s0) {
            f16x8 qh[2], ql[2];
            rope_query<D, P>(L, s0, lane, q, qh, ql);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const int tau = rank_row(rt, n);
                float x[2][8];
#pragma unroll
                for (int k = 0; k < 2; ++k)
#pragma unroll
                    for (int u = 0; u < 8; ++u) x[k][u] = (float)f.bk[rt][s0 + k * (D / 64)][u];
                rope_pair(x[0], x[1], s0, q, L.ct + tau * R, L.st + tau * R);
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    f16x8 hi, lo;
                    split8_f16(x[k], hi, lo);
                    z[rt] = mfma_f16(hi, qh[k], z[rt]);
                    z[rt] = mfma_f16(lo, qh[k], z[rt]);
                    z[rt] = mfma_f16(hi, ql[k], z[rt]);
                }
            }
            if (s0 + 1 < D / 64) pair_done(s0);
        }
        bf16x8 eh1[1], el1[1];
        page_softmax<D, 32, true>(w, z, eh1, el1, rows, q, c2);
        eh[0] = eh1[0];
        el[0] = el1[0];
        return;
    }
    const bool m_lo = 8 * q < rk4, m_hi = 8 * q + 4 < rk4;
    bf16x8 a[P / 16];
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) {
        u32x4 am = __builtin_bit_cast(u32x4, f.ak[tt]);
        if (!m_lo) am[0] = am[1] = 0u;
        if (!m_hi) am[2] = am[3] = 0u;
        a[tt] = __builtin_bit_cast(bf16x8, am);
    }
    f32x4 st[P / 16];
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) st[tt] = zero_f4();
#pragma unroll
    for (int s0 = 0; s0 < D / 64; ++s0) {
        f16x8 qh[2], ql[2];
        rope_query<D, P>(L, s0, lane, q, qh, ql);
#pragma unroll
        for (int tt = 0; tt < P / 16; ++tt) {
            const int tau = token_row<P>(tt, n);
            float x[2][8];
#pragma unroll
            for (int k = 0; k < 2; ++k)
#pragma unroll
                for (int hp = 0; hp < 2; ++hp) {
                    const f32x4 kt = mfma_bf16(f.bk[hp][s0 + k * (D / 64)], a[tt], zero_f4());
#pragma unroll
                    for (int v = 0; v < 4; ++v) x[k][4 * hp + v] = kt[v];
                }
            rope_pair(x[0], x[1], s0, q, L.ct + tau * R, L.st + tau * R);
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                f16x8 hi, lo;
                split8_f16(x[k], hi, lo);
                st[tt] = mfma_f16(hi, qh[k], st[tt]);
                st[tt] = mfma_f16(lo, qh[k], st[tt]);
                st[tt] = mfma_f16(hi, ql[k], st[tt]);
            }
        }
        if (s0 + 1 < D / 64) pair_done(s0);
    }
    page_softmax<D, P, false>(w, st, eh, el, P, q, c2);
}

// Phase 2 of a unit. Factor page: Y^T = L_V^T E^T, O^T += R_V^T Y^T. Dense
// unit: O^T += V^T E^T with the unit's V^T columns in the R_V^T registers;
// columns at or past `rows` may hold anything, so they are zeroed.
template <int D, int P>
__device__ inline void unit_phase2(WaveState<D> &w, const ValueOps<D, P> &f, bool dense, int rows,
                                   const bf16x8 (&eh)[(P + 31) / 32], const bf16x8 (&el)[(P + 31) / 32], int q) {
    bf16x8 bh, bl;
    if (dense) {
        bh = eh[0];
        bl = el[0];
    } else {
        f32x4 y[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            y[rt] = zero_f4();
#pragma unroll
            for (int ks = 0; ks < (P + 31) / 32; ++ks) {
                y[rt] = mfma_bf16(f.av[rt][ks], eh[ks], y[rt]);
                y[rt] = mfma_bf16(f.av[rt][ks], el[ks], y[rt]);
            }
        }
        split_tiles(y[0], y[1], bh, bl);
    }
    const bool mask = dense && rows < 32;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
        bf16x8 vv = f.bv[dt];
        if (mask) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (8 * q + u >= rows) vv[u] = (__bf16)0.f;
        }
        w.o[dt] = mfma_bf16(vv, bh, w.o[dt]);
        w.o[dt] = mfma_bf16(vv, bl, w.o[dt]);
    }
}

}  // namespace pkv

#include "attention_q4.inl"

namespace pkv {

// A page-table entry read at a wave-uniform address, as scalars: the page's
// buffer resources then live in scalar registers.
__device__ inline pkv_page unpack_entry(uint2 ent) {
    pkv_page e;
    e.slot = (int32_t)__builtin_amdgcn_readfirstlane((int)ent.x);
    const unsigned int meta = (unsigned int)__builtin_amdgcn_readfirstlane((int)ent.y);
    e.kind = (uint8_t)(meta & 0xffu);
    e.rank_k = (uint8_t)((meta >> 8) & 0xffu);
    e.rank_v = (uint8_t)((meta >> 16) & 0xffu);
    e.rows = 0;
    return e;
}

// One workgroup of eight wavefronts per CU (two per SIMD) streams a chunk of
// one head's pages; each wave keeps its own running state, and the states
// are merged in LDS at the end. Per wave the loads run half a page ahead of
// the math: phase 1 of page i reads the key operands, which are then refilled
// with page i+1's while phase 2 of page i reads the value operands, refilled
// in turn with page i+1's. One operand set per wave keeps the register budget
// at two waves per SIMD.
template <int D, int P, bool Q4, bool ROPE = false, bool FOLD = false>
__global__ __launch_bounds__(64 * attn_waves<Q4>(), 1) void k_attn_mfma(Geo g, const pkv_page *__restrict__ table,
                                                                  const char *__restrict__ dense,
                                                                  const char *__restrict__ factor,
                                                                  const uint16_t *__restrict__ q, SeqArgs seq,
                                                                  int sched, int n_chunks, Partials pp, float *out,
                                                                  float *lse) {
    constexpr int KD = D / 32, DT = D / 16, KS = (P + 31) / 32;
    constexpr int NW = attn_waves<Q4>();
    const int chunk = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    const int G = g.g;
    // wave index as a scalar: everything derived from it (page indices, the
    // page resources) stays wave-uniform
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int lane = threadIdx.x % 64;
    const int n = lane & 15, q4 = lane >> 4;
    const int64_t T = seq.len[b];
    const int64_t n_pages = ceil_div(T, P);
    const float c2 = kLog2e / sqrtf((float)D);

    // query group as the B operand (K = d, N = query head)
    bf16x8 qb[KD];
    {
        const uint16_t *qp = q + ((int64_t)b * g.Hq + (int64_t)h * G + n) * D + 8 * q4;
#pragma unroll
        for (int s = 0; s < KD; ++s) qb[s] = n < G ? ld_b8(qp + 32 * s) : zero8();
        // completed before the page loop (a load still pending on entry
        // would make the first wait inside the loop body a full drain on
        // every page); the bf16 path first issues its first table reads
    }

    // merge buffers; the INT4 kernel also keeps its O^T accumulators in s_o
    // (rows padded to D + 4 floats against bank conflicts)
    __shared__ float s_m[NW][16], s_l[NW][16];
    __shared__ __align__(16) float s_o[NW][16][D + 4];

    WaveState<D> w;
#pragma unroll
    for (int t = 0; t < DT; ++t) w.o[t] = zero_f4();
    w.m_run = -INFINITY;
    w.l = zero_f4();

    // Pages are handed out dynamically: every wave of every workgroup of a
    // head takes the head's next page from one device-wide counter, so the
    // waves and CUs that the memory system serves faster simply take more
    // pages and all finish together. A dense page becomes P / 32 units of up
    // to 32 tokens that flow through the same pipelined loop (and operand
    // registers) as factor pages.
    const uint2 *tab = (const uint2 *)(table + head * g.max_pages);
    constexpr int UT = dense_unit_tokens<P>();
    // claim: take the head's next page index and start reading its entry
    struct Claim {
        int64_t j;
        uint2 raw;
    };
    // A claim is issued (the atomic) at the top of a loop iteration and taken
    // (its result read) at the bottom: the vector memory counter is in
    // order, so waiting for an atomic issued after the next page's loads
    // would also wait for those loads and serialize every page.
    auto issue_claim = [&]() -> unsigned int {
        unsigned int k = 0u;
        if (lane == 0) k = __hip_atomic_fetch_add(pp.claim(head), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return k;
    };
    auto take_claim = [&](unsigned int k) -> Claim {
        // pinned here: hoisted up to the atomic, the read of its result would
        // wait for every load issued before it
        asm volatile("" : "+v"(k));
        Claim c;
        // the claim word is unsigned: widened as such, a stale or wrapped
        // value can only fail the range check, never index below the table
        c.j = (int64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)k);
        c.raw = c.j < n_pages ? tab[c.j] : make_uint2(0u, 0u);
        return c;
    };
    if constexpr (Q4) {
        // INT4 factor pages stream through the pipelined loop; dense pages met
        // on the way are queued (a head has at most as many dense pages as
        // dense slots, which the host keeps within the queue) and done after.
        __shared__ int s_dense[kQ4DenseStage];
        __shared__ unsigned int s_nd;
        // the query group times c2 (scores come out in log2 units) as fp16 B
        // operands, elements of pairs 1 and 3 (e = 2, 3, 6, 7) also divided
        // by 16 for the raw key words; one copy per workgroup (every wave
        // serves this head), read per page instead of held in registers
        __shared__ f16x8 s_qh[4][64];
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): the query
        if (threadIdx.x == 0) s_nd = 0u;
        if (wave == 0) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                f16x8 h;
#pragma unroll
                for (int e = 0; e < 8; ++e) h[e] = (_Float16)((float)qb[s][e] * ((e & 2) ? 0.0625f * c2 : c2));
                s_qh[s][lane] = h;
            }
        }
        Q4State w4;
        w4.ol = &s_o[wave][n][4 * q4];
        w4.l = 0.f;
        w4.m_run = -INFINITY;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) lds_st4(w4.ol + 16 * dt, zero_f4());
        __syncthreads();
        const Q4Consts kq4 = q4_consts(n);
        Claim ahead = take_claim(issue_claim());
        // pre: a claim issued while ahead.j < n_pages, taken by the first step
        auto next_factor = [&](unsigned int pre) -> pkv_page {
            bool have_pre = true;
            while (ahead.j < n_pages) {
                const pkv_page e = unpack_entry(ahead.raw);
                const int64_t j = ahead.j;
                ahead = take_claim(have_pre ? pre : issue_claim());
                have_pre = false;
                if (e.kind == PKV_FACTOR) return e;
                if (lane == 0) {
                    if (e.kind == PKV_DENSE) {
                        const unsigned int di = atomicAdd(&s_nd, 1u);
                        if (di < (unsigned int)kQ4DenseStage) s_dense[di] = (int)j;
                        else raise_status(PKV_DEV_BAD_PAGE);   // more dense pages than a head can hold
                    } else {
                        raise_status(PKV_DEV_BAD_PAGE);
                    }
                }
            }
            pkv_page none;
            none.kind = PKV_EMPTY;
            return none;
        };
        Q4Key ko;
        Q4ValY vy;
        Q4ValO vo;
        pkv_page cur;
        cur.kind = PKV_EMPTY;
        pkv_page nxt = next_factor(ahead.j < n_pages ? issue_claim() : 0u);
        while (cur.kind == PKV_FACTOR || nxt.kind == PKV_FACTOR) {
            const unsigned int pre = ahead.j < n_pages ? issue_claim() : 0u;
            const Q4Res nres = q4_res(factor, g.factor_slot_bytes, nxt);
            const bool live = cur.kind == PKV_FACTOR;
            if (live) {
                f32x4 st[4];
                // scores start from -(m_run + 2^4 units), or 0 on the first page
                q4_scores(ko, s_qh, lane, st, kq4, w4.m_run == -INFINITY ? 0.f : -(w4.m_run + kQ4UnitLog2));
                q4_issue_key_loads(ko, nres, n, q4);
                q4_exp_shifted<D, FOLD>(w4, st);
                f16x8 yh, yl;
                q4_values_y<FOLD>(vy, st, yh, yl, kq4);
                q4_issue_y_loads(vy, nres, n, q4);
                q4_values_o<D, FOLD>(w4, vo, yh, yl, kq4);
                q4_issue_o_loads(vo, nres, n, q4);
            } else {
                q4_issue_key_loads(ko, nres, n, q4);
                q4_issue_y_loads(vy, nres, n, q4);
                q4_issue_o_loads(vo, nres, n, q4);
            }
            cur = nxt;
            nxt = next_factor(pre);
        }
        __syncthreads();
        const int nd = (int)min(s_nd, (unsigned int)kQ4DenseStage);
        // the bf16 query group is read again here rather than kept in
        // registers through the stream
        const uint16_t *qp = q + ((int64_t)b * g.Hq + (int64_t)h * G + n) * D + 8 * q4;
        for (int i = wave; i < nd; i += NW) {
            const int64_t j = s_dense[i];
            const pkv_page e = unpack_entry(tab[j]);
            bf16x8 qd[KD];
#pragma unroll
            for (int s = 0; s < KD; ++s) qd[s] = n < G ? ld_b8(qp + 32 * s) : zero8();
            q4_dense_page<D, FOLD>(w4, qd, dense, g.dense_slot_bytes, e.slot, (int)min<int64_t>(P, T - j * P), n, q4, c2);
        }
        w.m_run = w4.m_run;
        w.l[0] = w4.l;
    } else {
    // bf16 pages are handed to the workgroup in blocks of NW consecutive
    // pages, one per wave: round k, wave w streams page block_k + w. The
    // eight waves of a CU then read eight neighbouring slots together, which
    // a read-only probe of this access pattern measured 4% faster than
    // claiming page by page per wave (6.26 against 6.0 TB/s). Wave 0 takes a
    // block one round ahead with one device-scope atomic on the head's
    // counter; the block goes through LDS at the round's barrier.
    //
    // The barrier is inside take_page and nowhere else in the loop, and every
    // wave calls take_page once per round until the round whose block starts
    // past the sequence (the same round for all waves: its base is read from
    // LDS): a wave whose page of a round is past the end takes the next round
    // at once. So all waves arrive at the same number of barriers, whatever
    // mix of factor pages and multi-unit dense pages each one streams.
    __shared__ unsigned int s_blk[4];
    int round = 0;
    bool blocks_done = false;
    // Wave 0's block claim is issued at the top of a loop iteration and read
    // at the bottom of the same iteration (the vector memory counter is in
    // order: read later, its wait would also cover the loads issued after
    // it); the value is held until take_page publishes it. A claim is taken
    // synchronously only where none is held: the last rounds, when a wave's
    // page is past the end.
    //
    // With wave_claims (kSchedWaveClaims, set by the host for pre-RoPE caches, and for streams
    // of few pages per wave) each wave instead claims one page at a time after
    // the same static round 0, with the same issue-ahead scheme and no
    // barrier (a claim k is page n_chunks NW + k). The round barrier keeps the
    // waves in step: the two waves of a SIMD then run the same phase of their
    // pages at once, which costs compute-bound pages (pre-RoPE), and a round
    // holding a two-unit dense page lasts twice as long for all eight waves,
    // which costs a stream of few rounds.
    const bool wave_claims = ROPE || (sched & kSchedWaveClaims) != 0;
    // With kSchedReverse the k-th page handed out is page n_pages - 1 - k:
    // the window's dense pages (two units each) are taken first, and the last
    // claims of every head are factor pages (set by the host for long streams).
    const bool reverse = (sched & kSchedReverse) != 0;
    auto page_of = [&](int64_t k) -> int64_t { return k >= n_pages ? n_pages : reverse ? n_pages - 1 - k : k; };
    const unsigned int claim_step = wave_claims ? 1u : (unsigned int)NW;
    unsigned int blk_next = 0u;
    bool blk_ready = false, need_blk = false;   // wave 0 only, unless wave_claims
    auto sync_claim = [&]() -> unsigned int {
        unsigned int k = 0u;
        if (lane == 0) k = __hip_atomic_fetch_add(pp.claim(head), claim_step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return (unsigned int)__builtin_amdgcn_readfirstlane((int)k);
    };
    auto needs_blk = [&]() -> bool { return (wave_claims || wave == 0) && need_blk; };
    auto issue_blk = [&]() -> unsigned int {
        unsigned int k = 0u;
        if (lane == 0) k = __hip_atomic_fetch_add(pp.claim(head), claim_step, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return k;
    };
    auto take_blk = [&](unsigned int k) {
        asm volatile("" : "+v"(k));
        blk_next = (unsigned int)__builtin_amdgcn_readfirstlane((int)k);
        blk_ready = true;
        need_blk = false;
    };
    // Round 0 is static: workgroup c streams block c (pages c NW .. c NW +
    // NW - 1) with no claim, and the head's counter hands out the blocks
    // after the first n_chunks (a claim k is block n_chunks NW + k). The
    // first table entries, wave 0's claim of the next block and the query
    // are then in flight together: one memory round trip before the first
    // page's loads instead of four in a row.
    auto take_page = [&]() -> Claim {
        unsigned int base;
        if (round == 0) {
            base = (unsigned int)chunk * (unsigned int)NW;
            if (wave_claims || wave == 0) need_blk = true;
        } else if (wave_claims) {
            const unsigned int v = blk_ready ? blk_next : sync_claim();
            blk_ready = false;
            need_blk = true;
            ++round;
            Claim c;
            c.j = page_of((int64_t)v + (int64_t)n_chunks * NW);
            if (c.j >= n_pages) blocks_done = true;
            c.raw = c.j < n_pages ? tab[c.j] : make_uint2(0u, 0u);
            return c;
        } else {
            if (wave == 0) {
                const unsigned int v = blk_ready ? blk_next : sync_claim();
                if (lane == 0) s_blk[round & 3] = v + (unsigned int)n_chunks * (unsigned int)NW;
                blk_ready = false;
                need_blk = true;
            }
            // LDS write complete, then the round barrier; no vector-memory wait
            // (loads of the units in flight stay in flight across it)
            __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
            asm volatile("s_barrier" ::: "memory");
            base = (unsigned int)__builtin_amdgcn_readfirstlane((int)s_blk[round & 3]);
        }
        ++round;
        if ((int64_t)base >= n_pages) blocks_done = true;
        Claim c;
        c.j = page_of((int64_t)base + wave);
        c.raw = c.j < n_pages ? tab[c.j] : make_uint2(0u, 0u);
        return c;
    };
    Claim ahead = take_page();                              // round 0
    const unsigned int pre0 = needs_blk() ? issue_blk() : 0u;   // round 1's block
    __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): query, first table entries, claim
    // pre-RoPE keys: w_i = theta_i / 2 pi = base^(-2i/d) / 2 pi as wh + wl
    // (fp64 on the way), i < d/2; the table of cos / sin (tau theta_i) for
    // tau < P; the query group in fp32. Shared by the workgroup.
    RopeLds<D, P> rl{};
    if constexpr (ROPE) {
        constexpr int R = RopeLds<D, P>::kRow;
        __shared__ float s_rw[D];
        __shared__ float s_rt[2][P * R];
        __shared__ float s_qf[KD * 64 * 8];
        __shared__ float s_r0[NW][D];
        if (threadIdx.x < D / 2) {
            const int i = (int)threadIdx.x;
            const double th = exp2(-(2.0 * i / D) * log2((double)g.rope_base));
            const double wv = th * 0.15915494309189533577;   // 1 / (2 pi)
            const float wh = (float)wv;
            s_rw[i] = wh;
            s_rw[D / 2 + i] = (float)(wv - (double)wh);
        }
        if (wave == 0) {
#pragma unroll
            for (int s = 0; s < KD; ++s)
#pragma unroll
                for (int u = 0; u < 8; ++u) s_qf[(s * 64 + lane) * 8 + u] = (float)qb[s][u];
        }
        __syncthreads();
        for (int idx = (int)threadIdx.x; idx < P * (D / 2); idx += 64 * NW) {
            const int tau = idx / (D / 2), i = idx % (D / 2);
            const float fr = rope_frac((float)tau, s_rw[i], s_rw[D / 2 + i]);
            s_rt[0][tau * R + i] = __builtin_amdgcn_cosf(fr);
            s_rt[1][tau * R + i] = __builtin_amdgcn_sinf(fr);
        }
        __syncthreads();
        rl.rw = s_rw;
        rl.ct = s_rt[0];
        rl.st = s_rt[1];
        rl.qf = s_qf;
        rl.r0 = s_r0[wave];
    }
    Unit pending;                 // second and later units of a dense page
    pending.e.kind = PKV_EMPTY;
    pending.j = 0;
    pending.half = 0;
    // pre: wave 0's block claim issued at the top of this iteration (needs_blk held)
    auto next_unit = [&](unsigned int pre) -> Unit {
        if (needs_blk()) take_blk(pre);
        if (pending.e.kind == PKV_DENSE) {
            Unit u = pending;
            const int next_half = u.half + 1;
            if ((int64_t)next_half * UT >= min<int64_t>(P, T - u.j * P)) pending.e.kind = PKV_EMPTY;
            else pending.half = next_half;
            return u;
        }
        while (!blocks_done) {
            const Claim c = ahead;
            ahead = take_page();
            if (c.j >= n_pages) continue;   // this wave's page of the round is past the end
            Unit u;
            u.e = unpack_entry(c.raw);
            u.j = c.j;
            u.half = 0;
            if (u.e.kind == PKV_FACTOR) return u;
            if (u.e.kind == PKV_DENSE) {
                if (UT < min<int64_t>(P, T - u.j * P)) {
                    pending = u;
                    pending.half = 1;
                }
                return u;
            }
            if (lane == 0) raise_status(PKV_DEV_BAD_PAGE);
        }
        Unit none;
        none.e.kind = PKV_EMPTY;
        none.j = 0;
        none.half = 0;
        return none;
    };

    auto unit_rows = [&](const Unit &u) -> int {
        return (int)min<int64_t>(UT, T - u.j * P - (int64_t)UT * u.half);
    };

    LaneOffs lo;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        lo.bk[rt] = 2u * (rank_row(rt, n) * D + 8 * q4);
        lo.av[rt] = 2u * (rank_row(rt, n) * P + (P >= 32 ? 8 : 4) * q4);
    }
    lo.tok0 = token_row<P>(0, n);
    // The loop starts one step early with an empty unit, so the loads of the
    // first unit are issued by the loop body itself, in the order every later
    // unit's are: the waits the compiler places at the top of the body then
    // count only the loads that unit really needs. The page after the next
    // is claimed one iteration ahead, hiding its table read.
    KeyOps<D, P> ko;
    ValueOps<D, P> vo;
    Unit cur;
    cur.e.kind = PKV_EMPTY;
    cur.j = 0;
    cur.half = 0;
    Unit nxt = next_unit(pre0);
    while (cur.e.kind != PKV_EMPTY || nxt.e.kind != PKV_EMPTY) {
        const unsigned int pre = needs_blk() ? issue_blk() : 0u;
        const PageRes nres = unit_res<D, P, ROPE>(factor, g.factor_slot_bytes, dense, g.dense_slot_bytes, nxt);
        bf16x8 eh[KS], el[KS];
        const int rows = unit_rows(cur);
        const bool live = cur.e.kind != PKV_EMPTY, dns = cur.e.kind == PKV_DENSE;
        if (live) {
            if constexpr (ROPE)
                unit_phase1_rope<D, P>(w, ko, rl, dns, rows, eh, el, n, q4, c2,
                                       cur.j * P + (int64_t)UT * cur.half, r4(cur.e.rank_k),
                                       [&](int s0) { issue_key_pair_rope<D, P>(ko, nres, n, q4, s0); });
            else
                unit_phase1<D, P>(w, ko, qb, dns, rows, eh, el, q4, c2);
        }
        // pre-RoPE: the pairs but the last were issued during phase 1
        issue_key_loads<D, P, ROPE>(ko, nres, lo, n, q4, ROPE && live ? D / 64 - 1 : 0);
        if (live) unit_phase2<D, P>(w, vo, dns, rows, eh, el, q4);
        issue_value_loads<D, P>(vo, nres, lo, n, q4);
        cur = nxt;
        nxt = next_unit(pre);
    }
    }

    // ---- merge the wave states (Eq. (5)) into the chunk's partial ---------
    float l_col = w.l[0];
    if constexpr (Q4) {   // lane shares of the normalizer
        l_col += __shfl_xor(l_col, 16, 64);
        l_col += __shfl_xor(l_col, 32, 64);
    }
    if (q4 == 0) {
        s_m[wave][n] = w.m_run;
        s_l[wave][n] = l_col;
    }
    if constexpr (!Q4) {   // the INT4 kernel accumulated in s_o already
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int v = 0; v < 4; ++v) s_o[wave][n][16 * dt + 4 * q4 + v] = w.o[dt][v];
    }
    __syncthreads();
    // a head's only workgroup writes out and lse itself (no partial, counter
    // or merge); otherwise the chunk's partial is published
    const bool single = pp.nc == 1;
    // four dims per thread: the wave weights once per query and dims, and one
    // 16-byte store with the coherent cache policy of st_dev
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
            // INT4 at <= 8 queries: rows 8-15 hold the lo parts of rows 0-7
            const f32x4 o = FOLD ? lds_ld4(&s_o[ww][qi][k]) + lds_ld4(&s_o[ww][qi + 8][k]) : lds_ld4(&s_o[ww][qi][k]);
            acc += sc * o;
            l = fmaf(sc, s_l[ww][qi], l);
        }
        if constexpr (Q4) {   // back from the INT4 kernel's units of 2^-4
            acc *= kQ4Unit;
            l *= kQ4Unit;
        }
        if (single) {   // Eq. (5) with one partial: normalize
            const bool empty = T <= 0 || !(l > 0.f);
            float *o = out + ((int64_t)b * g.Hq + h * G + qi) * D + k;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = empty ? 0.f : acc[i] / l;
            if (lse && k == 0) lse[(int64_t)b * g.Hq + h * G + qi] = empty ? -INFINITY : (M + log2f(l)) * kLn2;
            continue;
        }
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), rpo, 16u * (uint32_t)f, 0, 16);
        if (k == 0) {
            st_dev(&pp.m[pp.mi(head, qi, chunk)], M);
            st_dev(&pp.l[pp.mi(head, qi, chunk)], l);
        }
    }
    if (single) {   // every claim of this workgroup has returned: clear the head's claim word
        if (threadIdx.x == 0) __hip_atomic_store(pp.claim(head), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    // the wave-state block is free once every thread has passed the publish barrier
    publish_and_merge<64 * NW>(g, head, pp, out, lse, T, &s_o[0][0][0]);
}

inline bool mfma_supported(const Geo &g) {
    if (g.factor_dtype == PKV_INT4) return true;   // validated on the host (bf16 dense, P = 64, d = 128)
    return g.dense_dtype == PKV_BF16 && g.factor_dtype == PKV_BF16 && (g.d == 64 || g.d == 128) &&
           (g.P == 16 || g.P == 32 || g.P == 64) && g.max_rank <= 32 && g.g <= 16;
}

hipError_t launch_attn_mfma(const LaunchCtx &L, const AttnPlan &plan, const uint16_t *q, const SeqArgs &seq,
                            const Partials &pp, float *out, float *lse) {
    LayerPtrs p = layer_ptrs(L);
    const Geo &g = L.geo;
    dim3 grid(plan.n_chunks, g.B * g.Hkv);
#define PKV_LAUNCH_MFMA(DD, PP)                                                                         \
    hipLaunchKernelGGL((k_attn_mfma<DD, PP, false>), grid, dim3(64 * kMfmaWaves), 0, L.stream, g, p.table,   \
                       p.dense, p.factor, q, seq, plan.sched, plan.n_chunks, pp, out, lse)
#define PKV_LAUNCH_MFMA_ROPE(DD, PP)                                                                    \
    hipLaunchKernelGGL((k_attn_mfma<DD, PP, false, true>), grid, dim3(64 * kMfmaWaves), 0, L.stream, g,      \
                       p.table, p.dense, p.factor, q, seq, plan.sched, plan.n_chunks, pp, out, lse)
    if (g.key_t) {   // pre-RoPE keys (validated on the host: d = 64/128, P = 32/64)
        if (g.d == 128) {
            if (g.P == 64) PKV_LAUNCH_MFMA_ROPE(128, 64);
            else PKV_LAUNCH_MFMA_ROPE(128, 32);
        } else {
            if (g.P == 64) PKV_LAUNCH_MFMA_ROPE(64, 64);
            else PKV_LAUNCH_MFMA_ROPE(64, 32);
        }
    } else if (g.factor_dtype == PKV_INT4) {
        if (g.g <= 8)   // padding columns 8-15 carry the lo half of the O^T update
            hipLaunchKernelGGL((k_attn_mfma<128, 64, true, false, true>), grid, dim3(64 * kMfmaWavesQ4), 0, L.stream,
                               g, p.table, p.dense, p.factor, q, seq, plan.sched, plan.n_chunks, pp, out, lse);
        else
            hipLaunchKernelGGL((k_attn_mfma<128, 64, true>), grid, dim3(64 * kMfmaWavesQ4), 0, L.stream, g, p.table,
                               p.dense, p.factor, q, seq, plan.sched, plan.n_chunks, pp, out, lse);
    } else if (g.d == 128) {
        if (g.P == 64) PKV_LAUNCH_MFMA(128, 64);
        else if (g.P == 32) PKV_LAUNCH_MFMA(128, 32);
        else PKV_LAUNCH_MFMA(128, 16);
    } else {
        if (g.P == 64) PKV_LAUNCH_MFMA(64, 64);
        else if (g.P == 32) PKV_LAUNCH_MFMA(64, 32);
        else PKV_LAUNCH_MFMA(64, 16);
    }
#undef PKV_LAUNCH_MFMA
#undef PKV_LAUNCH_MFMA_ROPE
    return hipGetLastError();
}

}  // namespace pkv
