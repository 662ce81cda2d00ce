// Mixed-page decode attention over INT4 factor pages (Section 4.3): the
// balanced factors L~ = U Sigma^(1/2), R~ = Sigma^(1/2) W^T are stored as
// 4-bit codes with fp16 scales (layout: int4_layout). Per factor page the
// four products of Eq. (4) run on the matrix cores with the codes turned
// into exact small integers in registers, and every scale applied where it
// is a diagonal of the product:
//   Z^T = R~_K Q^T       fp16 MFMA, A = code x scale (one rounding), B = q
//   S^T = L~_K Z^T       fp16 MFMA, A = code x scale, B = Z as fp16 hi/lo
//   Y^T = L~_V^T E'^T    bf16 MFMA, A = 136 + code (exact), B = E' hi/lo with
//                        E' = E x (row scale of L~_V); the 136 x sum(E')
//                        offset is removed with a ones x E' product
//   O^T += s .* (R~_V^T Y^T)  bf16 MFMA, A = 136 + code, B = Y hi/lo, output
//                        row c scaled by the column scale of R~_V (offset
//                        removed the same way)
// Unpacking a word of eight codes: XOR 0x88888888 maps a two's-complement
// nibble c to c + 8 in [1, 15]. Masked into the low mantissa bits of 1024.0
// (fp16, quantum 1) that is 1032 + c; minus 1032 it is c exactly, and one
// multiply by the scale rounds c x s once. Masked into the mantissa of 128.0
// (bf16, quantum 1) it is 136 + c. Dense pages (bf16) are queued and done
// after the stream. Included by attention_mfma.inl.

namespace pkv {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ inline f32x4 mfma_f16(const f16x8 &a, const f16x8 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Eight codes -> fp16 (code x scale); sc: the scales of the eight elements
// as four fp16 pairs. In the low mantissa bits of 1024.0 (quantum 1) the
// biased nibble c + 8 gives 1032 + c exactly; subtracting 1032 leaves c
// exactly, and its product with the scale is rounded once.
__device__ inline f16x8 q4_frag_scaled(uint32_t word, const u32x4 &sc) {
    const uint32_t x = word ^ 0x88888888u;
    const f16x2 bias = f16x2{(_Float16)-1032.f, (_Float16)-1032.f};
    f16x2 r[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t p = ((x >> (4 * k)) & 0x000f000fu) | 0x64006400u;
        // the element goes through a scalar first: a bit_cast of a vector
        // element expression reads element 0 whatever the index
        const uint32_t s = sc[k];
        r[k] = (__builtin_bit_cast(f16x2, p) + bias) * __builtin_bit_cast(f16x2, s);
    }
    return f16x8{r[0][0], r[0][1], r[1][0], r[1][1], r[2][0], r[2][1], r[3][0], r[3][1]};
}
// Eight codes -> bf16 (136 + code), exact.
__device__ inline bf16x8 q4_frag_offset(uint32_t word) {
    const uint32_t x = word ^ 0x88888888u;
    u32x4 p;
    p[0] = (x & 0x000f000fu) | 0x43004300u;
    p[1] = ((x >> 4) & 0x000f000fu) | 0x43004300u;
    p[2] = ((x >> 8) & 0x000f000fu) | 0x43004300u;
    p[3] = ((x >> 12) & 0x000f000fu) | 0x43004300u;
    return __builtin_bit_cast(bf16x8, p);
}

// fp32 pair -> fp16 hi (toward zero) and lo (the remainder), as packed words.
__device__ inline void split2_f16(float a, float b, uint32_t &hi, uint32_t &lo) {
    const f16x2 h = __builtin_bit_cast(f16x2, __builtin_amdgcn_cvt_pkrtz(a, b));
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(a - (float)h[0], b - (float)h[1]));
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

// Operand words of one INT4 factor page held by one lane.
struct Q4Key {
    u32x4 bkc[2];   // R~_K codes, rank row rank_row(rt, n): word s = dims 32s + 8q .. +7
    u32x4 bks[4];   // R~_K scales of those dims: [s] -> 4 fp16 pairs
    u32x4 akc;      // L~_K codes, word tt = token row token_row(tt, n), ranks 8q .. +7
    u32x4 aks[2];   // L~_K scales of those ranks, run 0 (tiles 0, 1) and run 1 (tiles 2, 3)
};
struct Q4Val {
    u32x4 bvc[2];   // R~_V^T codes, word dt = dim 16 dt + n, ranks 8q .. +7
    u32x4 bvs[4];   // R~_V scales of the lane's output rows 16 dt + 4q + v: word (2 dt + v/2)
    u32x4 avc;      // L~_V^T codes, word 2 rt + ks = rank row rank_row(rt, n), tokens 32 ks + 8q .. +7
    u32x4 avs[2];   // L~_V scales of the lane's score rows token_row(tt, 4q + v): word (2 tt + v/2)
};

// Per page: one resource for the key half and one for the value half (each
// ends with the section whose rows can pass the rank), and section offsets.
struct Q4Res {
    __amdgpu_buffer_rsrc_t k, v;
    uint32_t bkc, bks, aks;        // key half (akc starts at 0)
    uint32_t bvs, avs, avc;        // value half (bvc starts at 0)
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
__device__ inline void q4_issue_value_loads(Q4Val &f, const Q4Res &r, int n, int q) {
#pragma unroll
    for (int h = 0; h < 2; ++h) f.bvc[h] = bld16(r.v, q < r.kqv ? 32u * (16 * q + n) + 16u * h : kOOB, 0u);
#pragma unroll
    for (int k = 0; k < 4; ++k) f.bvs[k] = bld16(r.v, 64u * q + 16u * k, r.bvs);
    f.avc = bld16(r.v, r.avc + 16u * (4 * n + q), 0u);
#pragma unroll
    for (int k = 0; k < 2; ++k) f.avs[k] = bld16(r.v, 32u * q + 16u * k, r.avs);
}

// Phase 1 of an INT4 factor page: Z^T, S^T, softmax; the exp weights stay in
// st (fp32) for phase 2, which folds the L~_V row scales into them.
template <int D>
__device__ inline void q4_phase1(WaveState<D> &w, const Q4Key &f, const f16x8 (&qh)[4], f32x4 (&st)[4], int q,
                                 float c2) {
    f32x4 z[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        z[rt] = zero_f4();
#pragma unroll
        for (int s = 0; s < 4; ++s) z[rt] = mfma_f16(q4_frag_scaled(f.bkc[rt][s], f.bks[s]), qh[s], z[rt]);
    }
    f16x8 zh, zl;
    split_tiles_f16(z[0], z[1], zh, zl);
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
        const f16x8 a = q4_frag_scaled(f.akc[tt], tt < 2 ? f.aks[0] : f.aks[1]);
        st[tt] = mfma_f16(a, zh, zero_f4());
        st[tt] = mfma_f16(a, zl, st[tt]);
    }
    page_softmax_exp<D, 64, false>(w, st, 64, q, c2);
}

// Phase 2 of an INT4 factor page: E' = E x row scale, Y^T, O^T.
template <int D>
__device__ inline void q4_phase2(WaveState<D> &w, const Q4Val &f, const f32x4 (&st)[4]) {
    const bf16x8 ones = bf16x8{1, 1, 1, 1, 1, 1, 1, 1};
    f32x4 ep[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint32_t pair = f.avs[tt >> 1][2 * (tt & 1) + (v >> 1)];
            const float sc = (float)__builtin_bit_cast(f16x2, pair)[v & 1];
            ep[tt][v] = st[tt][v] * sc;
        }
    bf16x8 eh[2], el[2];
    split_tiles(ep[0], ep[1], eh[0], el[0]);
    split_tiles(ep[2], ep[3], eh[1], el[1]);
    f32x4 cse = zero_f4();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        cse = mfma_bf16(ones, eh[ks], cse);
        cse = mfma_bf16(ones, el[ks], cse);
    }
    f32x4 y[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        y[rt] = zero_f4();
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 a = q4_frag_offset(f.avc[2 * rt + ks]);
            y[rt] = mfma_bf16(a, eh[ks], y[rt]);
            y[rt] = mfma_bf16(a, el[ks], y[rt]);
        }
        y[rt] -= 136.f * cse;
    }
    bf16x8 yh, yl;
    split_tiles(y[0], y[1], yh, yl);
    f32x4 csy = mfma_bf16(ones, yh, zero_f4());
    csy = mfma_bf16(ones, yl, csy);
    const f32x4 off = 136.f * csy;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
        const bf16x8 a = q4_frag_offset(f.bvc[dt >> 2][dt & 3]);
        f32x4 pr = mfma_bf16(a, yh, zero_f4());
        pr = mfma_bf16(a, yl, pr);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint32_t pair = f.bvs[dt >> 1][2 * (dt & 1) + (v >> 1)];
            const float sc = (float)__builtin_bit_cast(f16x2, pair)[v & 1];
            w.o[dt][v] = fmaf(sc, pr[v] - off[v], w.o[dt][v]);
        }
    }
}

// A dense page, loaded and computed in place in units of 32 tokens (used for
// the few dense pages after the INT4 stream).
template <int D>
__device__ inline void q4_dense_page(WaveState<D> &w, const bf16x8 (&qb)[D / 32], const char *dense,
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
        page_softmax_exp<D, 32, true>(w, st, rows, q, c2);
        bf16x8 eh, el;
        split_tiles(st[0], st[1], eh, el);
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
            bf16x8 vv = ld_b8(Vt + (int64_t)(16 * dt + n) * 64 + 32 * half + 8 * q);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (8 * q + u >= rows) vv[u] = (__bf16)0.f;
            w.o[dt] = mfma_bf16(vv, eh, w.o[dt]);
            w.o[dt] = mfma_bf16(vv, el, w.o[dt]);
        }
    }
}

}  // namespace pkv
