// Internal definitions shared by the host side and the kernels of the
// PuzzleKV library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "puzzlekv.h"

namespace pkv {

constexpr int kMaxBatchArgs = 256;   // sequences whose lengths travel in kernel arguments
constexpr int kCompressItemsPerLaunch = 96;
constexpr int kCopyItemsPerLaunch = 64;

__host__ __device__ inline int r4(int r) { return (r + 3) & ~3; }
__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Elements of a packed factor page pair at ranks (rk, rv). kt: R_K stored
// transposed, d x r4(rk) (caches of pre-RoPE keys).
__host__ __device__ inline int64_t factor_page_elems(int P, int d, int rk, int rv, bool kt = false) {
    return (int64_t)P * r4(rk) + (int64_t)(kt ? r4(rk) : rk) * d + (int64_t)rv * P + (int64_t)d * r4(rv);
}

// Section starts (in elements) of a factor slot holding ranks (rk, rv):
// A_K = L_K (P x r4(rk)), B_K = R_K (rk x d) or, with kt, B_Kt = R_K^T
// (d x r4(rk)), B_Vt = R_V^T (d x r4(rv)), A_Vt = L_V^T (rv x P), packed in
// that order. A_Vt comes last because its reads past rank rv are the ones
// that must stop at the page's end.
struct FactorLayout {
    int64_t ak, bk, bvt, avt, end;
};
__host__ __device__ inline FactorLayout factor_layout(int P, int d, int rk, int rv, bool kt = false) {
    FactorLayout f;
    f.ak = 0;
    f.bk = (int64_t)P * r4(rk);
    f.bvt = f.bk + (int64_t)(kt ? r4(rk) : rk) * d;
    f.avt = f.bvt + (int64_t)d * r4(rv);
    f.end = f.avt + (int64_t)rv * P;
    return f;
}

// INT4 factor slot (factor dtype PKV_INT4; P = 64, d = 128, ranks <= 32).
// Codes c in [-7, 7] are stored offset-binary (nibble c + 8), eight to a
// dword with element e at bit int4_nib(e); scales are fp16. Byte offsets of
// the sections, in order:
//   akc  A_K codes      [kq][i][tt] dwords: token row tau(tt, i), ranks 8kq + e
//   aks  A_K scales     [kq][run][e]: column-wise runs of 32 tokens, rank 8kq + e
//   bks  B_K scales     [kq][s][e]: dim 32s + 8kq + e (column-wise, one run)
//   bkc  B_K codes      [a][kq][s] dwords: rank row a, dims 32s + 8kq + e
//   bvc  B_V^T codes    [kq][i][dt] dwords: dim 16dt + i, ranks 8kq + e
//   bvs  B_V scales     [q][dt][v]: dim 16dt + 4q + v (column-wise, one run)
//   avs  A_V scales     [q][tt][v]: token tau(tt, 4q + v) (row-wise, one run)
//   avc  A_V^T codes    [i][kq][rt][ks] dwords: rank row pi(rt, i), tokens 32ks + 8kq + e
//   pad  32 bytes of 0x88 (eight zero codes per dword)
// where pi and tau are the attention kernel's tile row maps. Each section is
// ordered so that one lane of that kernel reads its operand slice as one
// 16-byte piece. Reads of key rows past the rank fall outside the key half
// and return zero words; value reads past the rank are pointed at the pad,
// so they decode as zero codes.
__host__ __device__ inline int r8(int r) { return (r + 7) & ~7; }
__host__ __device__ inline int int4_nib(int e) { return 4 * (e >> 1) + 16 * (e & 1); }
struct Int4Layout {
    int64_t akc, aks, bks, bkc, keys_end, bvc, bvs, avs, avc, pad, end;
};
constexpr int kInt4Pad = 32;
__host__ __device__ inline Int4Layout int4_layout(int P, int d, int rk, int rv) {
    Int4Layout f;
    f.akc = 0;
    f.aks = f.akc + (int64_t)r8(rk) * P / 2;
    f.bks = f.aks + (int64_t)r8(rk) * (P / 32) * 2;
    f.bkc = f.bks + 2LL * d;
    f.keys_end = f.bkc + (int64_t)rk * d / 2;
    f.bvc = f.keys_end;
    f.bvs = f.bvc + (int64_t)r8(rv) * d / 2;
    f.avs = f.bvs + 2LL * d;
    f.avc = f.avs + 2LL * P;
    f.pad = f.avc + (int64_t)r8(rv) * P / 2;
    f.end = f.pad + kInt4Pad;
    return f;
}
// Tile row maps shared by the INT4 layout and the attention kernel: rank tile
// rt, row m -> rank 8(m/4) + 4rt + m%4; token tile tt, row m -> token
// 32(tt/2) + 8(m/4) + 4(tt%2) + m%4 (P >= 32).
__host__ __device__ inline int tile_rank_row(int rt, int m) { return 8 * (m >> 2) + 4 * rt + (m & 3); }
__host__ __device__ inline int tile_token_row(int tt, int m) {
    return 32 * (tt >> 1) + 8 * (m >> 2) + 4 * (tt & 1) + (m & 3);
}

// Kind of logical page j of a sequence of T tokens (sink S, window W tokens).
__host__ __device__ inline int plan_kind(int64_t T, int P, int S, int W, int64_t j) {
    if (j < 0 || j * P >= T) return PKV_EMPTY;
    const bool complete = (j + 1) * P <= T;
    const bool in_sink = j < ceil_div(S, P);
    const bool in_window = (j + 1) * P > T - W;
    return (complete && !in_sink && !in_window) ? PKV_FACTOR : PKV_DENSE;
}

// Flattened geometry, passed to kernels by value.
struct Geo {
    int B, Hkv, Hq, g, d, P, max_pages, max_rank;
    float rank_err;                           // adaptive ranks: eps, or 0 (off)
    float rope_base;                          // keys stored before RoPE: its base, or 0 (off)
    int key_t;                                // R_K stored transposed (rope_base > 0)
    int S, W, sink_pages, ring_len, dslots;   // dslots = dense slots per head
    int dense_es, factor_es;                  // element sizes in bytes
    int dense_dtype, factor_dtype;
    int64_t dense_slot_bytes, factor_slot_bytes;
    // per-layer strides
    int64_t layer_entries;       // page-table entries per layer
    int64_t layer_dense_bytes;   // dense pool bytes per layer
    int64_t layer_factor_bytes;  // factor pool bytes per layer

    __host__ __device__ int dense_ring_slot(int j) const {
        return j < sink_pages ? j : sink_pages + (j - sink_pages) % ring_len;
    }
    __host__ __device__ int64_t head_index(int b, int h) const { return (int64_t)b * Hkv + h; }
};

// bf16 <-> fp32 with round-to-nearest-even (NaN kept quiet).
__host__ __device__ inline float bf16_to_f32(uint16_t v) {
    union { uint32_t u; float f; } x;
    x.u = (uint32_t)v << 16;
    return x.f;
}
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
    union { uint32_t u; float f; } x;
    x.f = f;
    if ((x.u & 0x7f800000u) == 0x7f800000u && (x.u & 0x007fffffu)) return (uint16_t)((x.u >> 16) | 0x40);
    uint32_t r = x.u + 0x7fffu + ((x.u >> 16) & 1u);
    return (uint16_t)(r >> 16);
}

// Storage element access: float or bf16 (uint16_t).
template <typename T> __device__ inline float ld(const T *p, int64_t i);
template <> __device__ inline float ld<float>(const float *p, int64_t i) { return p[i]; }
template <> __device__ inline float ld<uint16_t>(const uint16_t *p, int64_t i) { return bf16_to_f32(p[i]); }
__device__ inline float to_f32(float x) { return x; }
__device__ inline float to_f32(uint16_t x) { return bf16_to_f32(x); }
template <typename T> __device__ inline void st(T *p, int64_t i, float v);
template <> __device__ inline void st<float>(float *p, int64_t i, float v) { p[i] = v; }
template <> __device__ inline void st<uint16_t>(uint16_t *p, int64_t i, float v) { p[i] = f32_to_bf16(v); }

// Reads and clears the sticky device status word of the current device.
hipError_t status_read_clear(unsigned int *bits);
// Reads and clears the device's count of executed Jacobi sweeps.
hipError_t sweeps_read_clear(unsigned long long *n);

// ---- launchers (defined in the .hip files) --------------------------------

struct LaunchCtx {
    const pkv_cache *c;
    Geo geo;
    int layer;
    hipStream_t stream;
};

// Compress work item (one logical page: K and V decompositions).
struct CompressItem {
    int32_t b, h, j;
    uint8_t rk, rv, pad0, pad1;
};
struct CompressItems {
    int32_t n;
    CompressItem it[kCompressItemsPerLaunch];
};

struct CopyItem {
    int32_t b, h, j;
    uint8_t kind, rk, rv, pad;
    int64_t src_off;
};
struct CopyItems {
    int32_t n;
    CopyItem it[kCopyItemsPerLaunch];
};

struct SeqArgs {
    int32_t n;  // batch
    int32_t len[kMaxBatchArgs];
};

hipError_t launch_reset(const LaunchCtx &L, int64_t first_entry, int64_t n_entries);
hipError_t launch_prefill_pages(const LaunchCtx &L, const void *k, const void *v, int64_t src_tokens,
                                const SeqArgs &seq, const uint8_t *rank_k, const uint8_t *rank_v,
                                int def_rk, int def_rv, int max_pages_in_batch, int glob_r = 0);
hipError_t launch_prefill_compress(const LaunchCtx &L, const void *k, const void *v,
                                   int64_t src_tokens, const int32_t *item_offsets, int64_t n_items,
                                   const uint8_t *rank_k, const uint8_t *rank_v, int def_rk, int def_rv);
hipError_t launch_append(const LaunchCtx &L, const void *k_new, const void *v_new, const SeqArgs &pos);
hipError_t launch_compress(const LaunchCtx &L, const CompressItems &items);
hipError_t launch_compress_commit(const LaunchCtx &L, const CompressItems &items);
// The same with the n items in device memory, in one launch each.
hipError_t launch_compress_list(const LaunchCtx &L, const CompressItem *list, int64_t n);
hipError_t launch_compress_commit_list(const LaunchCtx &L, const CompressItem *list, int64_t n);
hipError_t launch_import(const LaunchCtx &L, const CopyItems &items, const void *src);
hipError_t launch_export(const LaunchCtx &L, const CopyItems &items, float *dst, int64_t block);
hipError_t launch_export_int4(const LaunchCtx &L, const CopyItems &items, char *dst, int64_t block_bytes);
hipError_t launch_import_q4(const LaunchCtx &L, const CopyItems &items, const void *src);
hipError_t launch_export_dq4(const LaunchCtx &L, const CopyItems &items, float *dst, int64_t block);
// Canonical INT4 page blob (import and code export): int8 codes L_K [P][rk],
// R_K [rk][d], L_V [P][rv], R_V [rv][d], then fp16 scales L_K [P/32][rk],
// R_K [d], L_V [P], R_V [d].
__host__ __device__ inline int64_t int4_blob_bytes(int P, int d, int rk, int rv) {
    return (int64_t)P * rk + (int64_t)rk * d + (int64_t)P * rv + (int64_t)rv * d +
           2LL * ((P / 32) * rk + d + P + d);
}

// Global SVD factors beside a cache: rank, padded rank, coefficient rows per head.
struct GlobalGeo {
    int r, r8, max_tokens;
};
struct GlobalLayer {
    char *basis, *coef;   // this layer's factors
};
int global_gram_chunks(const Geo &g, int64_t max_T);
int64_t global_prefill_workspace_bytes(const Geo &g, int64_t max_T);
int global_attention_chunks(const Geo &g, int64_t max_T);
int64_t global_attention_workspace_bytes(const Geo &g, int64_t max_T);
hipError_t launch_global_prefill(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, const void *k,
                                 const void *v, int64_t src_tokens, const SeqArgs &seq, int64_t max_T, void *ws);
hipError_t launch_global_attention(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, const void *q,
                                   const SeqArgs &seq, int64_t max_T, float *out, float *lse, void *ws);
hipError_t launch_global_export(const LaunchCtx &L, const GlobalGeo &gg, const pkv_global *gl, int b, int h,
                                int64_t n_rows, float *bk, float *bv, float *ak, float *av);

hipError_t bandwidth_probe(const void *src, void *dst, int64_t bytes, int mode, int reps, int blocks, int threads,
                           double *gbps, hipStream_t stream);

struct AttnPlan {
    int pages_per_chunk;
    int n_chunks;
    int use_mfma;
    int sched;   // matrix-core kernel: kSched* bits
};
// Page schedule of the matrix-core kernel: pages claimed per wave rather
// than per workgroup round; pages handed out last to first.
constexpr int kSchedWaveClaims = 1, kSchedReverse = 2;
AttnPlan attention_plan(const Geo &g, int64_t max_T);
int64_t attention_workspace_bytes(const Geo &g, int64_t max_T);
// Partial-state bytes the calls without a workspace can use, and the bytes
// such a call needs for its geometry and longest sequence.
int64_t scratch_state_bytes();
int64_t attention_state_bytes(const Geo &g, int64_t max_T);
hipError_t launch_attention_noalloc(const LaunchCtx &L, const AttnPlan &plan, const void *q, const SeqArgs &seq,
                                    float *out, float *lse);
hipError_t launch_attention(const LaunchCtx &L, const AttnPlan &plan, const void *q, const SeqArgs &seq,
                            float *out, float *lse, void *ws);

}  // namespace pkv
