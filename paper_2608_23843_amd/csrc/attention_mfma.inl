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
//
// Latency hiding: factor pages are read with buffer loads through a per-page
// resource whose size is the page's byte count; slices a lane does not need
// (rank rows past r) use an out-of-range offset and return zero without a
// memory access, so the loads carry no branches. Each wave keeps its loads
// half a page ahead of its math (see k_attn_mfma), so every wave always has
// part of a page in flight, with one operand set in registers.
// Included by pkv_kernels.hip.

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kMfmaWaves = 4;
constexpr float kRescaleLog2 = 8.0f;      // keep the running max until a page exceeds it by 2^8
constexpr uint32_t kOutOfRange = 0x80000000u;
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

__device__ inline __amdgpu_buffer_rsrc_t page_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kBufferDword3);
}
// Buffer loads: per-lane byte offset `voff` (an out-of-range value returns
// zero), wave-uniform byte offset `soff` (scalar operand).
__device__ inline bf16x8 bld8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ inline bf16x4 bld4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

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

// Operand slices of one factor page held by one lane, in two halves: the key
// factors feed phase 1 (scores and softmax), the value factors phase 2.
template <int D, int P>
struct KeyOps {
    bf16x8 bk[2][D / 32];  // R_K rows 16*rt + n, d-chunk s
    bf16x8 ak[P / 16];     // L_K row 16*tt + n, ranks {4 j4 .. +3} and {16 + 4 j4 .. +3}
};
template <int D, int P>
struct ValueOps {
    bf16x8 av[2][(P + 31) / 32];  // L_V^T row 16*rt + n, tokens of K-step ks in accumulator order
    bf16x8 bv[D / 16];            // R_V^T row 16*dt + n, ranks as for ak
};

// Per page: the buffer resource and section offsets (scalars) and the lane's
// byte offsets into each section (one value per operand half; out of range
// where the lane's slice lies past the page's rank). A page that is not a
// factor page gets a zero-size resource, so all its loads return zero.
struct PageRes {
    __amdgpu_buffer_rsrc_t rs;
    uint32_t oBk, oAvt, oBvt;     // section starts (bytes)
    int rk, rv, rk4, rv4;
    uint32_t v_bk[2], v_av[2];    // R_K / L_V^T rows of rank tile rt
    uint32_t v_ak_lo, v_ak_hi;    // L_K ranks {4 j4..} / {16 + 4 j4..} (before the tile offset)
    uint32_t v_bv_lo, v_bv_hi;    // R_V^T likewise
};

template <int D, int P>
__device__ inline PageRes page_res(const char *factor, int64_t slot_bytes, const pkv_page &e, int n, int j4) {
    PageRes r;
    const bool is_f = e.kind == PKV_FACTOR;
    r.rk = is_f ? e.rank_k : 0;
    r.rv = is_f ? e.rank_v : 0;
    r.rk4 = r4(r.rk);
    r.rv4 = r4(r.rv);
    const uint32_t bytes = (uint32_t)(2 * (P * r.rk4 + r.rk * D + r.rv * P + D * r.rv4));
    r.rs = page_rsrc(factor + (is_f ? e.slot : 0) * slot_bytes, bytes);
    r.oBk = 2u * P * r.rk4;
    r.oAvt = r.oBk + 2u * r.rk * D;
    r.oBvt = r.oAvt + 2u * r.rv * P;
    const uint32_t lb_bk = 2u * (n * D + 8 * j4), lb_av = 2u * (n * P + 4 * j4);
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        r.v_bk[rt] = 16 * rt + n < r.rk ? lb_bk : kOutOfRange;
        r.v_av[rt] = 16 * rt + n < r.rv ? lb_av : kOutOfRange;
    }
    const uint32_t lb_ak = 2u * n * r.rk4 + 8u * j4, lb_bv = 2u * n * r.rv4 + 8u * j4;
    r.v_ak_lo = 4 * j4 < r.rk4 ? lb_ak : kOutOfRange;
    r.v_ak_hi = 16 + 4 * j4 < r.rk4 ? lb_ak + 32u : kOutOfRange;
    r.v_bv_lo = 4 * j4 < r.rv4 ? lb_bv : kOutOfRange;
    r.v_bv_hi = 16 + 4 * j4 < r.rv4 ? lb_bv + 32u : kOutOfRange;
    return r;
}

template <int D, int P>
__device__ inline void issue_key_loads(KeyOps<D, P> &f, const PageRes &r) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int s = 0; s < D / 32; ++s) f.bk[rt][s] = bld8(r.rs, r.v_bk[rt] + 64u * s, r.oBk + 32u * rt * D);
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) {
        const uint32_t so = 32u * tt * r.rk4;
        f.ak[tt] = cat4(bld4(r.rs, r.v_ak_lo, so), bld4(r.rs, r.v_ak_hi, so));
    }
}

template <int D, int P>
__device__ inline void issue_value_loads(ValueOps<D, P> &f, const PageRes &r) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ks = 0; ks < (P + 31) / 32; ++ks) {
            const uint32_t so = r.oAvt + 32u * rt * P;
            f.av[rt][ks] = cat4(bld4(r.rs, r.v_av[rt] + 64u * ks, so),
                                32 * ks + 16 < P ? bld4(r.rs, r.v_av[rt] + 64u * ks + 32u, so) : zero4());
        }
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
        const uint32_t so = r.oBvt + 32u * dt * r.rv4;
        f.bv[dt] = cat4(bld4(r.rs, r.v_bv_lo, so), bld4(r.rs, r.v_bv_hi, so));
    }
}

// Running softmax state of one wave: O^T tiles, max (log2 units) and the
// lane's share of the normalizer.
template <int D>
struct WaveState {
    f32x4 o[D / 16];
    float m_run, l_part;
};

// Online softmax over one page's scores st (raw, unscaled on entry); leaves
// the exp weights as hi/lo B operands of the token contraction. Rows at or
// past `rows` are masked (dense pages only; factor pages are complete).
template <int D, int P, bool MASK>
__device__ inline void page_softmax(WaveState<D> &w, f32x4 (&st)[P / 16], bf16x8 (&eh)[(P + 31) / 32],
                                    bf16x8 (&el)[(P + 31) / 32], int rows, int j4, float c2) {
    constexpr int TT = P / 16, KS = (P + 31) / 32, DT = D / 16;
    float pm = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            float s = st[tt][v] * c2;
            if (MASK && 16 * tt + 4 * j4 + v >= rows) s = -INFINITY;
            st[tt][v] = s;
            pm = fmaxf(pm, s);
        }
    pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
    pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
    if (pm > w.m_run + kRescaleLog2 || w.m_run == -INFINITY) {
        const float alpha = w.m_run == -INFINITY ? 0.f : exp2f(w.m_run - pm);
#pragma unroll
        for (int t = 0; t < DT; ++t) w.o[t] *= alpha;
        w.l_part *= alpha;
        w.m_run = pm;
    }
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float ex = exp2f(st[tt][v] - w.m_run);
            st[tt][v] = ex;
            w.l_part += ex;
        }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
        split_hi_lo(st[2 * ks], 2 * ks + 1 < TT ? st[2 * ks + 1] : zero_f4(), eh[ks], el[ks]);
}

// Phase 1 of a factor page: Z^T = R_K Q^T, S^T = L_K Z^T, softmax.
template <int D, int P>
__device__ inline void factor_phase1(WaveState<D> &w, const KeyOps<D, P> &f, const bf16x8 (&qb)[D / 32], int rk,
                                     bf16x8 (&eh)[(P + 31) / 32], bf16x8 (&el)[(P + 31) / 32], int j4, float c2) {
    f32x4 z[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        z[rt] = zero_f4();
        if (rk > 16 * rt)
#pragma unroll
            for (int s = 0; s < D / 32; ++s) z[rt] = mfma_bf16(f.bk[rt][s], qb[s], z[rt]);
    }
    bf16x8 zh, zl;
    z[0] *= c2;  // scores come out in log2 units
    z[1] *= c2;
    split_hi_lo(z[0], z[1], zh, zl);
    f32x4 st[P / 16];
#pragma unroll
    for (int tt = 0; tt < P / 16; ++tt) {
        st[tt] = mfma_bf16(f.ak[tt], zh, zero_f4());
        st[tt] = mfma_bf16(f.ak[tt], zl, st[tt]);
    }
    page_softmax<D, P, false>(w, st, eh, el, P, j4, 1.0f);
}

// Phase 2 of a factor page: Y^T = L_V^T E^T, O^T += R_V^T Y^T.
template <int D, int P>
__device__ inline void factor_phase2(WaveState<D> &w, const ValueOps<D, P> &f, int rv,
                                     const bf16x8 (&eh)[(P + 31) / 32], const bf16x8 (&el)[(P + 31) / 32]) {
    f32x4 y[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
        y[rt] = zero_f4();
        if (rv > 16 * rt)
#pragma unroll
            for (int ks = 0; ks < (P + 31) / 32; ++ks) {
                y[rt] = mfma_bf16(f.av[rt][ks], eh[ks], y[rt]);
                y[rt] = mfma_bf16(f.av[rt][ks], el[ks], y[rt]);
            }
    }
    bf16x8 yh, yl;
    split_hi_lo(y[0], y[1], yh, yl);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
        w.o[dt] = mfma_bf16(f.bv[dt], yh, w.o[dt]);
        w.o[dt] = mfma_bf16(f.bv[dt], yl, w.o[dt]);
    }
}

// Dense page (sink, window, partial last page): loads and computes in place.
template <int D, int P>
__device__ inline void dense_page(WaveState<D> &w, const bf16x8 (&qb)[D / 32], const char *dense,
                                  int64_t slot_bytes, int slot, int rows, int n, int j4, float c2) {
    constexpr int KD = D / 32, DT = D / 16, TT = P / 16, KS = (P + 31) / 32;
    const uint16_t *K = (const uint16_t *)(dense + slot * slot_bytes);
    const uint16_t *Vt = K + (int64_t)P * D;
    f32x4 st[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
        st[tt] = zero_f4();
#pragma unroll
        for (int s = 0; s < KD; ++s)
            st[tt] = mfma_bf16(ld_b8(K + (int64_t)(16 * tt + n) * D + 32 * s + 8 * j4), qb[s], st[tt]);
    }
    bf16x8 eh[KS], el[KS];
    page_softmax<D, P, true>(w, st, eh, el, rows, j4, c2);
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
            const bf16x8 vv = cat4(lo, hi);
            w.o[dt] = mfma_bf16(vv, eh[ks], w.o[dt]);
            w.o[dt] = mfma_bf16(vv, el[ks], w.o[dt]);
        }
    }
}

// Entry `sl` of the lane-distributed batch, read with readlane so the slot and
// ranks are wave-uniform scalars (the page's buffer resource then lives in
// scalar registers and its loads need no per-lane resource handling).
__device__ inline pkv_page unpack_entry(uint2 ent, int sl) {
    pkv_page e;
    e.slot = (int32_t)__builtin_amdgcn_readlane((int)ent.x, sl);
    const unsigned int meta = (unsigned int)__builtin_amdgcn_readlane((int)ent.y, sl);
    e.kind = (uint8_t)(meta & 0xffu);
    e.rank_k = (uint8_t)((meta >> 8) & 0xffu);
    e.rank_v = (uint8_t)((meta >> 16) & 0xffu);
    e.flags = 0;
    return e;
}

// Four wavefronts per workgroup take the chunk's pages round-robin, each with
// its own running state; the states are merged in LDS at the end. Per wave
// the loads run half a page ahead of the math: phase 1 of page i reads the
// key operands, which are then refilled with page i+1's while phase 2 of
// page i reads the value operands, refilled in turn with page i+1's. One
// operand set per wave keeps the register budget at two waves per SIMD.
template <int D, int P>
__global__ __launch_bounds__(64 * kMfmaWaves, 2) void k_attn_mfma(Geo g, const pkv_page *table, const char *dense,
                                                                  const char *factor, const uint16_t *q, SeqArgs seq,
                                                                  int ppc, int n_chunks, Partials pp, float *out,
                                                                  float *lse) {
    constexpr int KD = D / 32, DT = D / 16, KS = (P + 31) / 32;
    const int chunk = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    const int G = g.g;
    // wave index as a scalar: everything derived from it (page indices, the
    // page resources) stays wave-uniform
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int lane = threadIdx.x % 64;
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

    WaveState<D> w;
#pragma unroll
    for (int t = 0; t < DT; ++t) w.o[t] = zero_f4();
    w.m_run = -INFINITY;
    w.l_part = 0.f;

    // This wave's pages: j = first + kMfmaWaves * i, i < n_mine. Their
    // page-table entries come 64 at a time, one per lane, broadcast per page.
    const int64_t first = j0 + wave;
    const int n_mine = first < j1 ? (int)ceil_div(j1 - first, kMfmaWaves) : 0;
    const uint2 *tab = (const uint2 *)(table + head * g.max_pages);
    uint2 batch = make_uint2(0u, 0u);
    auto entry_of = [&](int i) -> pkv_page {
        if ((i & 63) == 0) {
            const int64_t jl = first + (int64_t)kMfmaWaves * (i + lane);
            batch = (i + lane < n_mine) ? tab[jl] : make_uint2(0u, 0u);
        }
        return unpack_entry(batch, i & 63);
    };

    KeyOps<D, P> ko;
    ValueOps<D, P> vo;
    pkv_page cur;
    cur.kind = PKV_EMPTY;
    if (n_mine > 0) cur = entry_of(0);
    PageRes res = page_res<D, P>(factor, g.factor_slot_bytes, cur, n, j4);
    issue_key_loads<D, P>(ko, res);
    issue_value_loads<D, P>(vo, res);
    for (int i = 0; i < n_mine; ++i) {
        pkv_page nxt;
        nxt.kind = PKV_EMPTY;
        if (i + 1 < n_mine) nxt = entry_of(i + 1);
        const PageRes nres = page_res<D, P>(factor, g.factor_slot_bytes, nxt, n, j4);
        bf16x8 eh[KS], el[KS];
        if (cur.kind == PKV_FACTOR) factor_phase1<D, P>(w, ko, qb, res.rk, eh, el, j4, c2);
        issue_key_loads<D, P>(ko, nres);
        if (cur.kind == PKV_FACTOR) factor_phase2<D, P>(w, vo, res.rv, eh, el);
        issue_value_loads<D, P>(vo, nres);
        cur = nxt;
        res = nres;
    }
    // Dense pages (a few per sequence: sink, window, last) after the stream,
    // when the operand registers are free.
    for (int i = 0; i < n_mine; ++i) {
        const pkv_page e = entry_of(i);
        if (e.kind == PKV_DENSE) {
            const int64_t j = first + (int64_t)kMfmaWaves * i;
            dense_page<D, P>(w, qb, dense, g.dense_slot_bytes, e.slot, (int)min<int64_t>(P, T - j * P), n, j4, c2);
        } else if (e.kind != PKV_FACTOR && lane == 0) {
            raise_status(PKV_DEV_BAD_PAGE);
        }
    }

    // ---- merge the wave states (Eq. (5)) into the chunk's partial ---------
    __shared__ float s_m[kMfmaWaves][16], s_l[kMfmaWaves][16];
    __shared__ float s_o[kMfmaWaves][16][D];
    float l_part = w.l_part;
    l_part += __shfl_xor(l_part, 16, 64);
    l_part += __shfl_xor(l_part, 32, 64);
    if (j4 == 0) {
        s_m[wave][n] = w.m_run;
        s_l[wave][n] = l_part;
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int v = 0; v < 4; ++v) s_o[wave][n][16 * dt + 4 * j4 + v] = w.o[dt][v];
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * D; idx += 64 * kMfmaWaves) {
        const int qi = idx / D, k = idx % D;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kMfmaWaves; ++ww) M = fmaxf(M, s_m[ww][qi]);
        float acc = 0.f, l = 0.f;
#pragma unroll
        for (int ww = 0; ww < kMfmaWaves; ++ww) {
            const float sc = s_m[ww][qi] == -INFINITY ? 0.f : exp2f(s_m[ww][qi] - M);
            acc = fmaf(sc, s_o[ww][qi][k], acc);
            l = fmaf(sc, s_l[ww][qi], l);
        }
        pp.o[pp.oi(head, qi, k, chunk)] = acc;
        if (k == 0) {
            pp.m[pp.mi(head, qi, chunk)] = M;
            pp.l[pp.mi(head, qi, chunk)] = l;
        }
    }
    publish_and_merge(g, head, pp, out, lse, T);
}

inline bool mfma_supported(const Geo &g) {
    return g.dense_dtype == PKV_BF16 && g.factor_dtype == PKV_BF16 && (g.d == 64 || g.d == 128) &&
           (g.P == 16 || g.P == 32 || g.P == 64) && g.max_rank <= 32 && g.g <= 16;
}

hipError_t launch_attn_mfma(const LaunchCtx &L, const AttnPlan &plan, const uint16_t *q, const SeqArgs &seq,
                            const Partials &pp, float *out, float *lse) {
    LayerPtrs p = layer_ptrs(L);
    const Geo &g = L.geo;
    dim3 grid(plan.n_chunks, g.B * g.Hkv);
#define PKV_LAUNCH_MFMA(DD, PP)                                                                         \
    hipLaunchKernelGGL((k_attn_mfma<DD, PP>), grid, dim3(64 * kMfmaWaves), 0, L.stream, g, p.table, p.dense, \
                       p.factor, q, seq, plan.pages_per_chunk, plan.n_chunks, pp, out, lse)
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
