// Mixed-page decode attention over INT4 factor pages (Section 4.3): the
// balanced factors L~ = U Sigma^(1/2), R~ = Sigma^(1/2) W^T are stored as
// 4-bit codes (offset-binary, nibble c + 8) with fp16 scales (layout:
// int4_layout). Per factor page the four products of Eq. (4) run on the
// matrix cores with the codes turned into exact small numbers in registers,
// and every scale applied where it is a diagonal of the product:
//   Z^T = R~_K Q^T       fp16 MFMA, A = raw code word (exact), B = q o s_K
//                        (the R~_K column scale folded into the query); the
//                        raw words' offset is one more product, -beta x B,
//                        used as the accumulator's start
//   S^T = L~_K Z^T       fp16 MFMA, A = raw code word, B = s o Z (the L~_K
//                        scale folded into Z in fp32, one B per 32-token run)
//                        as fp16 hi/lo; started from -beta x B
//   Y^T = L~_V^T E'^T    fp16 MFMA, A = raw code word, B = E' = E x (row
//                        scale of L~_V) in fp16; started from -beta x E'
//   O^T += s .* (R~_V^T Y^T)  fp16 MFMA, A = raw code word, B = Y hi/lo,
//                        started from -beta x Y; output row c scaled by the
//                        column scale of R~_V
// The exp weights, l and O^T are kept in units of 2^-4 so every fp16 operand
// stays in range and out of the subnormals.
// With at most 8 queries per group, columns 8-15 of every 16x16 product are
// padding; the O^T update then takes Y hi in columns 0-7 and Y lo in columns
// 8-15 of one B operand (one product per dim tile instead of two), the lo
// parts accumulate in the wave's rows 8-15 of O^T, and those rows are added
// to rows 0-7 when the wave states are merged (lanes n and n + 8 keep the
// same running max so both rows share every rescale).
// Unpacking a word of eight nibbles n = c + 8 takes one and-or per pair of
// codes: masked into the low mantissa of 1024.0 (fp16, quantum 1) a nibble
// at bits 0-3 gives 1024 + n and one at bits 4-7 gives 1024 + 16 n, both
// exact. Elements whose nibble sits at bits 4-7 carry the factor 16, which
// the other operand (or the scale) divides out exactly. Dense pages (bf16) are queued and done after the stream.
// Included by attention_mfma.inl.

namespace pkv {


// Loop-invariant unpack constants, held in registers (kept opaque so the
// compiler forms one v_and_or_b32 per pair of codes).
struct Q4Consts {
    uint32_t m0, m1;     // masks of the nibbles at bits 0-3 and 4-7 of each half
    uint32_t h16;        // fp16 1024.0 in both halves
    uint32_t h16y;       // Y^T rows: 1024.0, or 64.0 in lanes whose row (rank) is 2 or 3 mod 4
    f16x8 nbeta_y;       // -beta, divided by 16 in the same lanes
};
__device__ inline Q4Consts q4_consts(int n) {
    Q4Consts k;
    k.m0 = 0x000f000fu;
    k.m1 = 0x00f000f0u;
    k.h16 = 0x64006400u;
    k.h16y = (n & 2) ? 0x54005400u : 0x64006400u;
    k.nbeta_y = f16x8{-1032, -1032, -1152, -1152, -1032, -1032, -1152, -1152} *
                ((n & 2) ? (_Float16)0.0625f : (_Float16)1.f);
    asm("" : "+s"(k.m0));
    asm("" : "+s"(k.m1));
    asm("" : "+v"(k.h16));
    asm("" : "+v"(k.h16y));
    return k;
}

// Element e of a word sits at bit int4_nib(e); the pairs (0,1), (2,3), (4,5),
// (6,7) sit at bits (0, 16), (4, 20), (8, 24), (12, 28).
// Eight codes -> fp16 1024 + n (pairs 0 and 2) and 1024 + 16 n (pairs 1 and 3), exact.
// With the magic 64.0 instead (quantum 1/16) the same word gives those
// values divided by 16, also exact.
__device__ inline f16x8 q4_frag_raw(uint32_t x, const Q4Consts &k, uint32_t magic) {
    const uint32_t y = x >> 8;
    u32x4 p;
    p[0] = (x & k.m0) | magic;
    p[1] = (x & k.m1) | magic;
    p[2] = (y & k.m0) | magic;
    p[3] = (y & k.m1) | magic;
    return __builtin_bit_cast(f16x8, p);
}
__device__ inline f16x8 q4_frag_raw(uint32_t x, const Q4Consts &k) { return q4_frag_raw(x, k, k.h16); }
// Scale words of one lane with pairs 1 and 3 divided by 16 (exact unless subnormal).
__device__ inline u32x4 q4_scale_div16(const u32x4 &sc) {
    const f16x2 r16 = f16x2{(_Float16)0.0625f, (_Float16)0.0625f};
    const uint32_t s1 = sc[1], s3 = sc[3];
    u32x4 o = sc;
    o[1] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, s1) * r16);
    o[3] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, s3) * r16);
    return o;
}
__device__ inline void split_tiles_f16(const f32x4 &x0, const f32x4 &x1, f16x8 &hi, f16x8 &lo) {
    uint32_t h0, h1, h2, h3, l0, l1, l2, l3;
    split2_f16(x0[0], x0[1], h0, l0);
    split2_f16(x0[2], x0[3], h1, l1);
    split2_f16(x1[0], x1[1], h2, l2);
    split2_f16(x1[2], x1[3], h3, l3);
    hi = __builtin_bit_cast(f16x8, u32x4{h0, h1, h2, h3});
    lo = __builtin_bit_cast(f16x8, u32x4{l0, l1, l2, l3});
}

// Within each 16-lane row, lanes 8-15 take `src` of lane n - 8 and lanes 0-7
// keep `keep` (DPP row rotate by 8, written to banks 2 and 3 only).
__device__ inline uint32_t row_hi_from_lo(uint32_t keep, uint32_t src) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)keep, (int)src, 0x128, 0xf, 0xc, false);
}
__device__ inline float row_hi_from_lo(float keep, float src) {
    return __uint_as_float(row_hi_from_lo(__float_as_uint(keep), __float_as_uint(src)));
}
// B operand of the folded O^T update: Y hi in lanes 0-7 of each row, Y lo of
// lane n - 8 in lanes 8-15.
__device__ inline f16x8 fold_hi_lo(const f16x8 &hi, const f16x8 &lo) {
    const u32x4 h = __builtin_bit_cast(u32x4, hi), l = __builtin_bit_cast(u32x4, lo);
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = row_hi_from_lo(h[i], l[i]);
    return __builtin_bit_cast(f16x8, o);
}

// Operand words of one INT4 factor page held by one lane.
struct Q4Key {
    u32x4 bkc[2];   // R~_K codes, rank row rank_row(rt, n): word s = dims 32s + 8q .. +7
    u32x4 bks[4];   // R~_K scales of those dims: [s] -> 4 fp16 pairs
    u32x4 akc;      // L~_K codes, word tt = token row token_row(tt, n), ranks 8q .. +7
    u32x4 aks[2];   // L~_K scales of those ranks, run 0 (tiles 0, 1) and run 1 (tiles 2, 3)
};
// Value operands in two parts: those of Y^T (used right after the page's
// softmax) and those of O^T (used one pipeline step later).
struct Q4ValY {
    u32x4 avc;      // L~_V^T codes, word 2 rt + ks = rank row rank_row(rt, n), tokens 32 ks + 8q .. +7
    u32x4 avs[2];   // L~_V scales of the lane's score rows token_row(tt, 4q + v): word (2 tt + v/2)
};
struct Q4ValO {
    u32x4 bvc[2];   // R~_V^T codes, word dt = dim 16 dt + n, ranks 8q .. +7
    u32x4 bvs[4];   // R~_V scales of the lane's output rows 16 dt + 4q + v: word (2 dt + v/2)
};

// Per page: one resource for the key half and one for the value half (each
// ends with the section whose rows can pass the rank), and section offsets.
struct Q4Res {
    __amdgpu_buffer_rsrc_t k, v;
    uint32_t bkc, bks, aks;        // key half (akc starts at 0)
    uint32_t bvs, avs, avc, pad;   // value half (bvc starts at 0)
    int kqk, kqv;                  // groups of 8 ranks present
};
__device__ inline Q4Res q4_res(const char *factor, int64_t slot_bytes, const pkv_page &e) {
    Q4Res r;
    const bool is_f = e.kind == PKV_FACTOR;
    const int rk = is_f ? e.rank_k : 0, rv = is_f ? e.rank_v : 0;
    const Int4Layout f = int4_layout(64, 128, rk, rv);
    const char *base = factor + (is_f ? e.slot : 0) * slot_bytes;
    r.k = section_rsrc(base, is_f ? (uint32_t)f.keys_end : 0u);
    r.v = section_rsrc(base + f.bvc, is_f ? (uint32_t)(f.end - f.bvc) : 0u);
    r.bkc = (uint32_t)f.bkc;
    r.bks = (uint32_t)f.bks;
    r.aks = (uint32_t)f.aks;
    r.bvs = (uint32_t)(f.bvs - f.bvc);
    r.avs = (uint32_t)(f.avs - f.bvc);
    r.avc = (uint32_t)(f.avc - f.bvc);
    r.pad = (uint32_t)(f.pad - f.bvc);
    r.kqk = r8(rk) / 8;
    r.kqv = r8(rv) / 8;
    return r;
}

__device__ inline u32x4 bld16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
constexpr uint32_t kOOB = 0x80000000u;   // an offset past any resource: the load returns zero

__device__ inline void q4_issue_key_loads(Q4Key &f, const Q4Res &r, int n, int q) {
    // R~_K rows: lane-varying row and section start, so rows past the rank
    // fall outside the resource
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) f.bkc[rt] = bld16(r.k, r.bkc + 64u * rank_row(rt, n) + 16u * q, 0u);
#pragma unroll
    for (int s = 0; s < 4; ++s) f.bks[s] = bld16(r.k, 64u * q + 16u * s, r.bks);
    f.akc = bld16(r.k, q < r.kqk ? 16u * (16 * q + n) : kOOB, 0u);
#pragma unroll
    for (int u = 0; u < 2; ++u) f.aks[u] = bld16(r.k, q < r.kqk ? 32u * q + 16u * u + r.aks : kOOB, 0u);
}
// Value words past the rank read the pad (zero codes): A_V^T rank rows at or
// past r8(r_V), and B_V^T groups of 8 ranks at or past r8(r_V).
__device__ inline void q4_issue_y_loads(Q4ValY &f, const Q4Res &r, int n, int q) {
    f.avc = bld16(r.v, n < 4 * r.kqv ? r.avc + 16u * (4 * n + q) : r.pad, 0u);
#pragma unroll
    for (int k = 0; k < 2; ++k) f.avs[k] = bld16(r.v, 32u * q + 16u * k, r.avs);
}
__device__ inline void q4_issue_o_loads(Q4ValO &f, const Q4Res &r, int n, int q) {
#pragma unroll
    for (int h = 0; h < 2; ++h) f.bvc[h] = bld16(r.v, (q < r.kqv ? 32u * (16 * q + n) : r.pad) + 16u * h, 0u);
#pragma unroll
    for (int k = 0; k < 4; ++k) f.bvs[k] = bld16(r.v, 64u * q + 16u * k, r.bvs);
}

// The INT4 kernel's exp weights, l and O^T are in units of 2^-4, and its
// running max is raised once a score passes it by 2^4: every weight is then
// at most 1 (unit), so E x s and Y stay far inside fp16 range for row scales
// below ~140, while the weights of the page holding the current maximum stay
// at or above 1/16 and keep the fp16 hi/lo splits out of the subnormal range.
constexpr float kQ4UnitLog2 = 4.f;
constexpr float kQ4Unit = 16.f;

// Running state of one wave of the INT4 kernel: the lane's share of the
// normalizer and the running max (log2 units) in registers, the O^T
// accumulators in LDS (the wave's block of the merge buffer, rows of D + 4
// floats): lane (n, q) owns o[16 dt + 4q .. +3] of row n, at ol + 16 dt.
struct Q4State {
    float *ol;
    float l, m_run;
};
__device__ inline f32x4 lds_ld4(const float *p) { return *(const f32x4 *)p; }
__device__ inline void lds_st4(float *p, const f32x4 &v) { *(f32x4 *)p = v; }

// Online softmax over one page's raw scores (Eq. (5) state update) with a
// lazy running max: it is raised (and O^T, l rescaled) only when a score
// exceeds it by 2^4, so the exp weights, in units of 2^-4, stay at most 1.
// Rows at or past `rows` are masked (dense pages).
template <int D, int P, bool MASK, bool FOLD>
__device__ inline void q4_exp(Q4State &w, f32x4 (&st)[P / 16], int rows, int q, float c2) {
    constexpr int TT = P / 16;
    float pm = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            if (MASK && token_row<P>(tt, 4 * q + v) >= rows) st[tt][v] = -INFINITY;
            pm = fmaxf(pm, st[tt][v]);
        }
    if constexpr (FOLD) pm = row_hi_from_lo(pm, pm);   // lanes n + 8 follow query n's max
    if (__builtin_amdgcn_ballot_w64(pm * c2 > w.m_run + kLazyLog2Q4) != 0) {
        pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
        const float m_new = fmaxf(w.m_run, pm * c2);
        const float alpha = w.m_run == -INFINITY ? 0.f : exp2f(w.m_run - m_new);
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) lds_st4(w.ol + 16 * dt, lds_ld4(w.ol + 16 * dt) * alpha);
        w.l *= alpha;
        w.m_run = m_new;
    }
    // weights in units of 2^-4 (an exponent offset); l and O^T share the unit
    const float nm = -(w.m_run + kQ4UnitLog2);
    float sum = 0.f;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) st[tt][v] = __builtin_amdgcn_exp2f(fmaf(st[tt][v], c2, nm));
        sum += (st[tt][0] + st[tt][1]) + (st[tt][2] + st[tt][3]);
    }
    w.l += sum;
}

// The same update for factor-page scores that arrive already in log2 units
// and shifted: st = s c2 - (m_run + 2^4 units), or s c2 while the running max
// is still -inf (the wave's first page). The shift came in through the score
// accumulators' start, so the exponent needs no fma.
template <int D, bool FOLD>
__device__ inline void q4_exp_shifted(Q4State &w, f32x4 (&st)[4]) {
    float pm = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) pm = fmaxf(pm, st[tt][v]);
    if constexpr (FOLD) pm = row_hi_from_lo(pm, pm);   // lanes n + 8 follow query n's max
    const bool first = w.m_run == -INFINITY;           // the same in every lane
    // lazy max: raised only when a score passes it by 2^4 (kLazyLog2Q4 = kQ4UnitLog2)
    if (first || __builtin_amdgcn_ballot_w64(pm > kLazyLog2Q4 - kQ4UnitLog2) != 0) {
        pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
        const float top = first ? pm : w.m_run + kQ4UnitLog2 + pm;   // the page's largest s c2
        const float m_new = fmaxf(w.m_run, top);
        if (!first) {
            const float alpha = exp2f(w.m_run - m_new);
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) lds_st4(w.ol + 16 * dt, lds_ld4(w.ol + 16 * dt) * alpha);
            w.l *= alpha;
        }
        const float sh = first ? -(m_new + kQ4UnitLog2) : w.m_run - m_new;
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int v = 0; v < 4; ++v) st[tt][v] += sh;
        w.m_run = m_new;
    }
    float sum = 0.f;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) st[tt][v] = __builtin_amdgcn_exp2f(st[tt][v]);
        sum += (st[tt][0] + st[tt][1]) + (st[tt][2] + st[tt][3]);
    }
    w.l += sum;
}

// Scores of an INT4 factor page: Z^T, then S^T into st (fp32, log2 units,
// started from `shift` per query). qh16 (LDS, [s][lane]): the query group
// times c2 as fp16 B operands, elements of pairs 1 and 3 divided by 16.
__device__ inline void q4_scores(const Q4Key &f, const f16x8 (&qh16)[4][64], int lane, f32x4 (&st)[4],
                                 const Q4Consts &k, float shift) {
    f16x8 qs[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) qs[s] = qh16[s][lane] * __builtin_bit_cast(f16x8, f.bks[s]);
    // the raw words' offset (1032 per code of pairs 0, 2; 1152 / 16 per code
    // of pairs 1, 3) is removed by starting both rank tiles from -beta x B
    const f16x8 nbeta = f16x8{-1032, -1032, -1152, -1152, -1032, -1032, -1152, -1152};
    f32x4 z0 = zero_f4();
#pragma unroll
    for (int s = 0; s < 4; ++s) z0 = mfma_f16(nbeta, qs[s], z0);
    f32x4 z[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        z[rt] = z0;
#pragma unroll
        for (int s = 0; s < 4; ++s) z[rt] = mfma_f16(q4_frag_raw(f.bkc[rt][s], k), qs[s], z[rt]);
    }
    // S^T = L~_K Z^T with the L~_K scale (per 32-token run u and rank) folded
    // into Z in fp32: Z_u = s_u o Z, split into fp16 hi/lo (ranks of pairs 1
    // and 3 also / 16, through the scale), and A = raw code words, each token
    // tile started from -beta x Z_u of its run. Every product is then exact.
    float zero = 0.f;
    asm("" : "+v"(zero));
    f16x8 zh[2], zl[2];
    f32x4 sb[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const u32x4 sc = q4_scale_div16(f.aks[u]);
        f32x4 zs[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int v = 0; v < 4; v += 2) {
                const uint32_t pair = sc[2 * rt + (v >> 1)];
                const f16x2 s2 = __builtin_bit_cast(f16x2, pair);
                zs[rt][v] = fmaf(z[rt][v], (float)s2[0], zero);
                zs[rt][v + 1] = fmaf(z[rt][v + 1], (float)s2[1], zero);
            }
        split_tiles_f16(zs[0], zs[1], zh[u], zl[u]);
        sb[u] = mfma_f16(nbeta, zh[u], f32x4{shift, shift, shift, shift});
        sb[u] = mfma_f16(nbeta, zl[u], sb[u]);
    }
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
        const f16x8 a = q4_frag_raw(f.akc[tt], k);
        st[tt] = mfma_f16(a, zh[tt >> 1], sb[tt >> 1]);
        st[tt] = mfma_f16(a, zl[tt >> 1], st[tt]);
    }
}

// Y^T of an INT4 factor page from its exp weights st (units of 2^-4):
// E' = E x (row scale of L~_V) in fp16, then L~_V^T E'^T from raw code words;
// returned as the fp16 hi/lo B operands of O^T, with the rows of ranks 2 and
// 3 mod 4 (elements e = 2, 3, 6, 7 of each lane) divided by 16 for the raw
// R~_V words, by the magic 64.0 in those lanes' A operand.
template <bool FOLD>
__device__ inline void q4_values_y(const Q4ValY &f, const f32x4 (&st)[4], f16x8 &yh, f16x8 &yl,
                                   const Q4Consts &k) {
    // E' (fp16): token 32 ks + 8q + e in element e of eb[ks]; tokens whose
    // code nibble sits at bits 4-7 of the L~_V^T word (e = 2, 3, 6, 7, i.e.
    // v = 2, 3) take the scale / 16
    // The product E x s is formed in fp32 (one mixed-precision fma with s as
    // its fp16 operand; the zero addend is kept opaque so the fma stays) and
    // rounded to fp16 once.
    const u32x4 sv[2] = {q4_scale_div16(f.avs[0]), q4_scale_div16(f.avs[1])};
    float z0 = 0.f;
    asm("" : "+v"(z0));
    f16x8 eb[2];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int v = 0; v < 4; v += 2) {
            const uint32_t pair = sv[tt >> 1][2 * (tt & 1) + (v >> 1)];
            const f16x2 sc = __builtin_bit_cast(f16x2, pair);
            const f32x2 e = f32x2{fmaf(st[tt][v], (float)sc[0], z0), fmaf(st[tt][v + 1], (float)sc[1], z0)};
            const f16x2 h = __builtin_convertvector(e, f16x2);
            eb[tt >> 1][4 * (tt & 1) + v] = h[0];
            eb[tt >> 1][4 * (tt & 1) + v + 1] = h[1];
        }
    // started from -beta x E' (divided by 16 in the lanes that divide their row)
    f32x4 y0 = zero_f4();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) y0 = mfma_f16(k.nbeta_y, eb[ks], y0);
    f32x4 y[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        y[rt] = y0;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
            y[rt] = mfma_f16(q4_frag_raw(f.avc[2 * rt + ks], k, k.h16y), eb[ks], y[rt]);
    }
    split_tiles_f16(y[0], y[1], yh, yl);
    if constexpr (FOLD) yh = fold_hi_lo(yh, yl);
}

// O^T += s .* (R~_V^T Y^T) from raw R~_V^T code words, each dim tile started
// from -beta x Y so the product is the codes' alone; output row c scaled by
// the column scale of R~_V.
// With FOLD, yh is the folded operand (hi | lo by lane half) and yl unused.
template <int D, bool FOLD>
__device__ inline void q4_values_o(Q4State &w, const Q4ValO &f, const f16x8 &yh, const f16x8 &yl,
                                   const Q4Consts &k) {
    const f16x8 nbeta = f16x8{-1032, -1032, -1152, -1152, -1032, -1032, -1152, -1152};
    f32x4 ob = mfma_f16(nbeta, yh, zero_f4());
    if constexpr (!FOLD) ob = mfma_f16(nbeta, yl, ob);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
        const f16x8 a = q4_frag_raw(f.bvc[dt >> 2][dt & 3], k);
        f32x4 pr = mfma_f16(a, yh, ob);
        if constexpr (!FOLD) pr = mfma_f16(a, yl, pr);
        f32x4 o = lds_ld4(w.ol + 16 * dt);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint32_t pair = f.bvs[dt >> 1][2 * (dt & 1) + (v >> 1)];
            const float sc = (float)__builtin_bit_cast(f16x2, pair)[v & 1];
            o[v] = fmaf(sc, pr[v], o[v]);
        }
        lds_st4(w.ol + 16 * dt, o);
    }
}

// A dense page, loaded and computed in place in units of 32 tokens (used for
// the few dense pages after the INT4 stream).
template <int D, bool FOLD>
__device__ inline void q4_dense_page(Q4State &w, const bf16x8 (&qb)[D / 32], const char *dense,
                                     int64_t slot_bytes, int slot, int rows_page, int n, int q, float c2) {
    const uint16_t *K = (const uint16_t *)(dense + slot * slot_bytes);
    const uint16_t *Vt = K + (int64_t)64 * D;
    for (int half = 0; half * 32 < rows_page; ++half) {
        const int rows = min(32, rows_page - 32 * half);
        f32x4 st[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
            st[tt] = zero_f4();
            const uint16_t *kp = K + (int64_t)(32 * half + rank_row(tt, n)) * D + 8 * q;
#pragma unroll
            for (int s = 0; s < D / 32; ++s) st[tt] = mfma_bf16(ld_b8(kp + 32 * s), qb[s], st[tt]);
        }
        q4_exp<D, 32, true, FOLD>(w, st, rows, q, c2);
        bf16x8 eh, el;
        split_tiles(st[0], st[1], eh, el);
        if (FOLD && n >= 8) {   // rows 8-15 of O^T hold the factor pages' lo parts
            eh = zero8();
            el = zero8();
        }
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
            bf16x8 vv = ld_b8(Vt + (int64_t)(16 * dt + n) * 64 + 32 * half + 8 * q);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (8 * q + u >= rows) vv[u] = (__bf16)0.f;
            f32x4 o = lds_ld4(w.ol + 16 * dt);
            o = mfma_bf16(vv, eh, o);
            o = mfma_bf16(vv, el, o);
            lds_st4(w.ol + 16 * dt, o);
        }
    }
}

}  // namespace pkv
