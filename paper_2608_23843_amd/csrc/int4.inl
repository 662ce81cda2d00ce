// INT4 factor pages (Section 4.3 "Quantization Compatibility"): where each
// code and scale of the balanced factors lives in a slot, the quantizer used
// by page compression, and import / export between slots and the canonical
// blob. The slot layout is described with int4_layout in pkv_internal.h.
// Included by pkv_kernels.hip.

namespace pkv {

constexpr int kQ4Max = 7;      // codes are symmetric in [-7, 7]
constexpr int kQ4Run = 32;     // elements per scale run

// ---- positions (P = 64, d = 128, so TT = 4 token tiles, S = 4 d-steps, DT = 8 dim tiles)

struct Q4Pos {
    int64_t byte;  // offset of the 32-bit word within the slot
    int shift;     // bit position of the nibble
};

__host__ __device__ inline Q4Pos q4_lk(const Int4Layout &f, int t, int a) {   // L~_K[t][a]
    const int tt = 2 * (t >> 5) + ((t >> 2) & 1), i = 4 * ((t >> 3) & 3) + (t & 3);
    return {f.akc + 4LL * (((a >> 3) * 16 + i) * 4 + tt), int4_nib(a & 7)};
}
__host__ __device__ inline int64_t q4_lk_scale(const Int4Layout &f, int u, int a) {
    return f.aks + 2LL * (((a >> 3) * 2 + u) * 8 + (a & 7));
}
__host__ __device__ inline Q4Pos q4_rk(const Int4Layout &f, int d, int a, int c) {   // R~_K[a][c]
    const int s = c >> 5, kq = (c >> 3) & 3;
    return {f.bkc + (int64_t)a * (d / 2) + 4LL * (kq * 4 + s), int4_nib(c & 7)};
}
__host__ __device__ inline int64_t q4_rk_scale(const Int4Layout &f, int c) {
    return f.bks + 2LL * ((((c >> 3) & 3) * 4 + (c >> 5)) * 8 + (c & 7));
}
__host__ __device__ inline Q4Pos q4_rv(const Int4Layout &f, int a, int c) {   // R~_V[a][c]
    const int dt = c >> 4, i = c & 15;
    return {f.bvc + 4LL * (((a >> 3) * 16 + i) * 8 + dt), int4_nib(a & 7)};
}
__host__ __device__ inline int64_t q4_rv_scale(const Int4Layout &f, int c) {
    return f.bvs + 2LL * ((((c >> 2) & 3) * 8 + (c >> 4)) * 4 + (c & 3));
}
__host__ __device__ inline Q4Pos q4_lv(const Int4Layout &f, int t, int a) {   // L~_V[t][a]
    const int rt = (a >> 2) & 1, i = 4 * (a >> 3) + (a & 3), ks = t >> 5, kq = (t >> 3) & 3;
    return {f.avc + 4LL * (((i * 4 + kq) * 2 + rt) * 2 + ks), int4_nib(t & 7)};
}
__host__ __device__ inline int64_t q4_lv_scale(const Int4Layout &f, int t) {
    const int tt = 2 * (t >> 5) + ((t >> 2) & 1);
    return f.avs + 2LL * ((((t >> 3) & 3) * 4 + tt) * 4 + (t & 3));
}

// Canonical blob offsets (bytes): codes as int8, then fp16 scales.
struct Int4Blob {
    int64_t clk, crk, clv, crv, slk, srk, slv, srv, end;
};
__host__ __device__ inline Int4Blob int4_blob(int P, int d, int rk, int rv) {
    Int4Blob b;
    b.clk = 0;
    b.crk = (int64_t)P * rk;
    b.clv = b.crk + (int64_t)rk * d;
    b.crv = b.clv + (int64_t)P * rv;
    b.slk = b.crv + (int64_t)rv * d;
    b.srk = b.slk + 2LL * (P / 32) * rk;
    b.slv = b.srk + 2LL * d;
    b.srv = b.slv + 2LL * P;
    b.end = b.srv + 2LL * d;
    return b;
}

__device__ inline float half_bits_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// fp16 round-to-nearest-even of a non-negative double (the quantizer's scale
// rule), without passing through fp32 (which could round twice).
__device__ inline uint16_t f16_rne(double x) {
    if (!(x > 0.0)) return 0;
    int e;
    (void)frexp(x, &e);                        // x in [2^(e-1), 2^e)
    const int q = (e - 1 < -14 ? -14 : e - 1) - 10;   // quantum 2^q (subnormals: 2^-24)
    const double r = rint(ldexp(x, -q)) * ldexp(1.0, q);
    if (r > 65504.0) return 0x7c00;
    return __builtin_bit_cast(uint16_t, (_Float16)(float)r);   // r is an fp16 value: exact
}
// code = x / s rounded half to even (the division in fp64, so the decision is
// the exact quotient's), clamped to [-7, 7]; s = 0 gives 0.
__device__ inline int q4_code(float x, float s) {
    if (!(s > 0.f)) return 0;
    const double qv = rint((double)x / (double)s);
    return (int)fmax(-kQ4Max, fmin((double)kQ4Max, qv));
}
// Offset-binary nibbles: code c is stored as c + 8.
__device__ inline uint32_t q4_nib(int code) { return (uint32_t)(code + 8) & 0xfu; }
__device__ inline int q4_nibble(uint32_t word, int shift) { return (int)((word >> shift) & 0xfu) - 8; }
constexpr uint32_t kQ4ZeroWord = 0x88888888u;   // eight zero codes

// ---- quantizer (page compression) -------------------------------------------
//
// Called by one wave after the balanced factors of one page half are staged:
// sL[t * 32 + a] = L~[t][a] (a < r) in LDS, R~ already quantized by the
// caller (its scales, one per column of ranks, stored in the slot; its codes
// in sRc: K as sRc[a * d + c], V as sRc[c * 32 + a], zero past rank r);
// `which` = 0 for K, 1 for V. L~'s scales first (one run per lane at a time),
// then every 32-bit word of codes is assembled by one lane from its eight
// elements.
__device__ void q4_store_codes(char *slot, const Int4Layout &f, int P, int d, int r, int which, const float *sL,
                               const int8_t *sRc, float *sScale, int lane) {
    // scales: K -> L~_K runs (run, a); V -> L~_V rows
    const int n_lruns = which == 0 ? (P / kQ4Run) * r8(r) : P;
    for (int idx = lane; idx < n_lruns; idx += 64) {
        float amax = 0.f;
        int64_t pos;
        if (which == 0) {
            const int u = idx / r8(r), a = idx % r8(r);
            if (a < r)
                for (int t = u * kQ4Run; t < (u + 1) * kQ4Run; ++t) amax = fmaxf(amax, fabsf(sL[t * 32 + a]));
            pos = q4_lk_scale(f, u, a);
        } else {
            const int t = idx;
            for (int a = 0; a < r; ++a) amax = fmaxf(amax, fabsf(sL[t * 32 + a]));
            pos = q4_lv_scale(f, t);
        }
        const uint16_t h = f16_rne((double)amax / (double)kQ4Max);
        *(uint16_t *)(slot + pos) = h;
        sScale[idx] = half_bits_to_f32(h);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): scale stores to LDS done
    __builtin_amdgcn_wave_barrier();
    // eight codes of R~ held contiguously in sRc -> one word
    auto pack8 = [](const int8_t *p8) -> uint32_t {
        const uint64_t v = *(const uint64_t *)p8;
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) word |= q4_nib((int)(int8_t)(v >> (8 * e))) << int4_nib(e);
        return word;
    };
    if (which == 0) {
        // L~_K words: [kq][i][tt], 16 * 4 words per kq
        const int n_lk = (r8(r) / 8) * 64;
        for (int w = lane; w < n_lk; w += 64) {
            const int kq = w / 64, i = (w / 4) % 16, tt = w % 4;
            const int t = tile_token_row(tt, i), u = t / kQ4Run;
            uint32_t word = 0;
            for (int e = 0; e < 8; ++e) {
                const int a = 8 * kq + e;
                const int code = a < r ? q4_code(sL[t * 32 + a], sScale[u * r8(r) + a]) : 0;
                word |= q4_nib(code) << int4_nib(e);
            }
            *(uint32_t *)(slot + f.akc + 4LL * w) = word;
        }
        // R~_K words: [a][kq][s], d / 8 words per row, dims 32 s + 8 kq + e
        for (int w = lane; w < r * (d / 8); w += 64) {
            const int a = w / (d / 8), kq = (w % (d / 8)) / 4, s = w % 4;
            *(uint32_t *)(slot + f.bkc + 4LL * w) = pack8(sRc + a * d + 32 * s + 8 * kq);
        }
    } else {
        // R~_V^T words: [kq][i][dt], 16 * 8 words per kq, ranks 8 kq + e of dim 16 dt + i
        const int n_rv = (r8(r) / 8) * 128;
        for (int w = lane; w < n_rv; w += 64) {
            const int kq = w / 128, i = (w / 8) % 16, dt = w % 8;
            *(uint32_t *)(slot + f.bvc + 4LL * w) = pack8(sRc + (16 * dt + i) * 32 + 8 * kq);
        }
        // L~_V^T words: [i][kq][rt][ks], 16 words per i, i < r8 / 2
        const int n_lv = (r8(r) / 2) * 16;
        for (int w = lane; w < n_lv; w += 64) {
            const int i = w / 16, kq = (w / 4) % 4, rt = (w / 2) % 2, ks = w % 2;
            const int a = tile_rank_row(rt, i);
            uint32_t word = 0;
            for (int e = 0; e < 8; ++e) {
                const int t = 32 * ks + 8 * kq + e;
                word |= q4_nib(a < r ? q4_code(sL[t * 32 + a], sScale[t]) : 0) << int4_nib(e);
            }
            *(uint32_t *)(slot + f.avc + 4LL * w) = word;
        }
        for (int w = lane; w < kInt4Pad / 4; w += 64) *(uint32_t *)(slot + f.pad + 4LL * w) = kQ4ZeroWord;
    }
}

// ---- import: canonical blob -> slot -------------------------------------------

__device__ void q4_import_page(char *slot, const char *blob, int P, int d, int rk, int rv) {
    const Int4Layout f = int4_layout(P, d, rk, rv);
    const Int4Blob b = int4_blob(P, d, rk, rv);
    const int8_t *clk = (const int8_t *)(blob + b.clk), *crk = (const int8_t *)(blob + b.crk);
    const int8_t *clv = (const int8_t *)(blob + b.clv), *crv = (const int8_t *)(blob + b.crv);
    const uint16_t *slk = (const uint16_t *)(blob + b.slk), *srk = (const uint16_t *)(blob + b.srk);
    const uint16_t *slv = (const uint16_t *)(blob + b.slv), *srv = (const uint16_t *)(blob + b.srv);
    // scales
    for (int idx = threadIdx.x; idx < 2 * r8(rk); idx += blockDim.x) {
        const int u = idx / r8(rk), a = idx % r8(rk);
        *(uint16_t *)(slot + q4_lk_scale(f, u, a)) = a < rk ? slk[u * rk + a] : (uint16_t)0;
    }
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        *(uint16_t *)(slot + q4_rk_scale(f, c)) = srk[c];
        *(uint16_t *)(slot + q4_rv_scale(f, c)) = srv[c];
    }
    for (int t = threadIdx.x; t < P; t += blockDim.x) *(uint16_t *)(slot + q4_lv_scale(f, t)) = slv[t];
    // codes, word by word
    for (int w = threadIdx.x; w < (r8(rk) / 8) * 64; w += blockDim.x) {
        const int kq = w / 64, i = (w / 4) % 16, tt = w % 4;
        const int t = tile_token_row(tt, i);
        uint32_t word = 0;
        for (int e = 0; e < 8; ++e) {
            const int a = 8 * kq + e;
            word |= q4_nib(a < rk ? clk[t * rk + a] : 0) << int4_nib(e);
        }
        *(uint32_t *)(slot + f.akc + 4LL * w) = word;
    }
    for (int w = threadIdx.x; w < rk * (d / 8); w += blockDim.x) {
        const int a = w / (d / 8), kq = (w % (d / 8)) / 4, s = w % 4;
        uint32_t word = 0;
        for (int e = 0; e < 8; ++e) word |= q4_nib(crk[a * d + 32 * s + 8 * kq + e]) << int4_nib(e);
        *(uint32_t *)(slot + f.bkc + 4LL * w) = word;
    }
    for (int w = threadIdx.x; w < (r8(rv) / 8) * 128; w += blockDim.x) {
        const int kq = w / 128, i = (w / 8) % 16, dt = w % 8;
        const int c = 16 * dt + i;
        uint32_t word = 0;
        for (int e = 0; e < 8; ++e) {
            const int a = 8 * kq + e;
            word |= q4_nib(a < rv ? crv[a * d + c] : 0) << int4_nib(e);
        }
        *(uint32_t *)(slot + f.bvc + 4LL * w) = word;
    }
    for (int w = threadIdx.x; w < (r8(rv) / 2) * 16; w += blockDim.x) {
        const int i = w / 16, kq = (w / 4) % 4, rt = (w / 2) % 2, ks = w % 2;
        const int a = tile_rank_row(rt, i);
        uint32_t word = 0;
        for (int e = 0; e < 8; ++e) word |= q4_nib(a < rv ? clv[(32 * ks + 8 * kq + e) * rv + a] : 0) << int4_nib(e);
        *(uint32_t *)(slot + f.avc + 4LL * w) = word;
    }
    for (int w = threadIdx.x; w < kInt4Pad / 4; w += blockDim.x) *(uint32_t *)(slot + f.pad + 4LL * w) = kQ4ZeroWord;
}

// ---- export: slot -> canonical blob, or dequantized fp32 block ---------------

__device__ void q4_export_blob(const char *slot, char *blob, int P, int d, int rk, int rv) {
    const Int4Layout f = int4_layout(P, d, rk, rv);
    const Int4Blob b = int4_blob(P, d, rk, rv);
    int8_t *clk = (int8_t *)(blob + b.clk), *crk = (int8_t *)(blob + b.crk);
    int8_t *clv = (int8_t *)(blob + b.clv), *crv = (int8_t *)(blob + b.crv);
    uint16_t *slk = (uint16_t *)(blob + b.slk), *srk = (uint16_t *)(blob + b.srk);
    uint16_t *slv = (uint16_t *)(blob + b.slv), *srv = (uint16_t *)(blob + b.srv);
    auto nib = [&](Q4Pos p) { return (int8_t)q4_nibble(*(const uint32_t *)(slot + p.byte), p.shift); };
    for (int x = threadIdx.x; x < P * rk; x += blockDim.x) clk[x] = nib(q4_lk(f, x / rk, x % rk));
    for (int x = threadIdx.x; x < rk * d; x += blockDim.x) crk[x] = nib(q4_rk(f, d, x / d, x % d));
    for (int x = threadIdx.x; x < P * rv; x += blockDim.x) clv[x] = nib(q4_lv(f, x / rv, x % rv));
    for (int x = threadIdx.x; x < rv * d; x += blockDim.x) crv[x] = nib(q4_rv(f, x / d, x % d));
    for (int x = threadIdx.x; x < 2 * rk; x += blockDim.x)
        slk[x] = *(const uint16_t *)(slot + q4_lk_scale(f, x / rk, x % rk));
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        srk[c] = *(const uint16_t *)(slot + q4_rk_scale(f, c));
        srv[c] = *(const uint16_t *)(slot + q4_rv_scale(f, c));
    }
    for (int t = threadIdx.x; t < P; t += blockDim.x) slv[t] = *(const uint16_t *)(slot + q4_lv_scale(f, t));
}

// Dequantized balanced factors in the fp32 export block: L_K (P x R), R_K
// (R x d), L_V (P x R), R_V (R x d), R = max rank, entries past the ranks 0.
__device__ void q4_export_dequant(const char *slot, float *o, int P, int d, int R, int rk, int rv) {
    const Int4Layout f = int4_layout(P, d, rk, rv);
    float *Lk = o, *Rk = Lk + P * R, *Lv = Rk + R * d, *Rv = Lv + P * R;
    auto nib = [&](Q4Pos p) { return q4_nibble(*(const uint32_t *)(slot + p.byte), p.shift); };
    auto scl = [&](int64_t pos) { return half_bits_to_f32(*(const uint16_t *)(slot + pos)); };
    for (int i = threadIdx.x; i < P * R; i += blockDim.x) {
        const int t = i / R, a = i % R;
        Lk[i] = a < rk ? nib(q4_lk(f, t, a)) * scl(q4_lk_scale(f, t / kQ4Run, a)) : 0.f;
        Lv[i] = a < rv ? nib(q4_lv(f, t, a)) * scl(q4_lv_scale(f, t)) : 0.f;
    }
    for (int i = threadIdx.x; i < R * d; i += blockDim.x) {
        const int a = i / d, c = i % d;
        Rk[i] = a < rk ? nib(q4_rk(f, d, a, c)) * scl(q4_rk_scale(f, c)) : 0.f;
        Rv[i] = a < rv ? nib(q4_rv(f, a, c)) * scl(q4_rv_scale(f, c)) : 0.f;
    }
}

__global__ __launch_bounds__(256) void k_export_int4(Geo g, const pkv_page *table, const char *factor, char *dst,
                                                     CopyItems items, int64_t block) {
    const CopyItem it = items.it[blockIdx.x];
    const pkv_page e = table[g.head_index(it.b, it.h) * g.max_pages + it.j];
    char *o = dst + it.src_off;
    if (e.kind != PKV_FACTOR) {
        for (int64_t i = threadIdx.x; i < block; i += blockDim.x) o[i] = 0;
        return;
    }
    q4_export_blob(factor + e.slot * g.factor_slot_bytes, o, g.P, g.d, e.rank_k, e.rank_v);
}

// Import for caches with INT4 factors: dense pages as bf16 blocks (offsets in
// elements), factor pages as canonical blobs (offsets in bytes).
__global__ __launch_bounds__(256) void k_import_q4(Geo g, pkv_page *table, char *dense, char *factor,
                                                   const char *src, CopyItems items) {
    const CopyItem it = items.it[blockIdx.x];
    const int64_t head = g.head_index(it.b, it.h);
    pkv_page *e = table + head * g.max_pages + it.j;
    if (it.kind == PKV_DENSE) {
        if (dense_slot_taken(g, table, head, it.j)) {
            if (threadIdx.x == 0) raise_status(PKV_DEV_RING_OVERRUN);
            return;
        }
        const uint16_t *s = (const uint16_t *)src + it.src_off;
        const int slot = (int)(head * g.dslots + g.dense_ring_slot(it.j));
        copy_dense_page<uint16_t>(g, s, s + (int64_t)g.P * g.d, g.d, g.P,
                                  (uint16_t *)(dense + slot * g.dense_slot_bytes));
        if (threadIdx.x == 0) write_entry(e, slot, PKV_DENSE, 0, 0, g.P);
        return;
    }
    const int slot = (int)(head * g.max_pages + it.j);
    q4_import_page(factor + slot * g.factor_slot_bytes, src + it.src_off, g.P, g.d, it.rk, it.rv);
    __syncthreads();
    if (threadIdx.x == 0) write_entry(e, slot, PKV_FACTOR, it.rk, it.rv);
}

// Export for caches with INT4 factors: dense pages as K, V; factor pages
// dequantized (balanced factors); empty pages as zeros.
__global__ __launch_bounds__(256) void k_export_dq4(Geo g, const pkv_page *table, const char *dense,
                                                    const char *factor, float *dst, CopyItems items,
                                                    int64_t block) {
    const CopyItem it = items.it[blockIdx.x];
    const pkv_page e = table[g.head_index(it.b, it.h) * g.max_pages + it.j];
    float *o = dst + it.src_off;
    const int P = g.P, d = g.d, R = g.max_rank;
    if (e.kind == PKV_DENSE) {
        const uint16_t *K = (const uint16_t *)(dense + e.slot * g.dense_slot_bytes);
        const uint16_t *Vt = K + (int64_t)P * d;
        for (int i = threadIdx.x; i < P * d; i += blockDim.x) {
            const int t = i / d, k = i % d;
            o[i] = bf16_to_f32(K[i]);
            o[P * d + i] = bf16_to_f32(Vt[(int64_t)k * P + t]);
        }
        for (int i = 2 * P * d + threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
        return;
    }
    if (e.kind != PKV_FACTOR) {
        for (int i = threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
        return;
    }
    q4_export_dequant(factor + e.slot * g.factor_slot_bytes, o, P, d, R, e.rank_k, e.rank_v);
    for (int i = 2 * (P + d) * R + threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
}

hipError_t launch_import_q4(const LaunchCtx &L, const CopyItems &items, const void *src) {
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL(k_import_q4, dim3(items.n), dim3(256), 0, L.stream, L.geo, p.table, p.dense, p.factor,
                       (const char *)src, items);
    return hipGetLastError();
}

hipError_t launch_export_dq4(const LaunchCtx &L, const CopyItems &items, float *dst, int64_t block) {
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL(k_export_dq4, dim3(items.n), dim3(256), 0, L.stream, L.geo, p.table, p.dense, p.factor,
                       dst, items, block);
    return hipGetLastError();
}

hipError_t launch_export_int4(const LaunchCtx &L, const CopyItems &items, char *dst, int64_t block) {
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL(k_export_int4, dim3(items.n), dim3(256), 0, L.stream, L.geo, p.table, p.factor, dst, items,
                       block);
    return hipGetLastError();
}

}  // namespace pkv
