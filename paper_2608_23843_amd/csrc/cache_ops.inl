// Cache maintenance kernels: page-table reset, prefill of dense pages and
// table entries, token append, page import / export, compress commit.
// Included by pkv_kernels.hip (single device translation unit).

namespace pkv {

__device__ unsigned int g_status;
__device__ inline void raise_status(unsigned int bits) { atomicOr(&g_status, bits); }

// Jacobi sweeps executed by decompositions since the last read (diagnostic).
__device__ unsigned long long g_sweeps;
__device__ inline void count_sweeps(int n) { atomicAdd(&g_sweeps, (unsigned long long)n); }

hipError_t sweeps_read_clear(unsigned long long *n) {
    unsigned long long zero = 0;
    hipError_t e = hipMemcpyFromSymbol(n, HIP_SYMBOL(g_sweeps), sizeof(zero), 0, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return e;
    return hipMemcpyToSymbol(HIP_SYMBOL(g_sweeps), &zero, sizeof(zero), 0, hipMemcpyHostToDevice);
}

hipError_t status_read_clear(unsigned int *bits) {
    unsigned int zero = 0;
    hipError_t e = hipMemcpyFromSymbol(bits, HIP_SYMBOL(g_status), sizeof(unsigned int), 0,
                                       hipMemcpyDeviceToHost);
    if (e != hipSuccess) return e;
    return hipMemcpyToSymbol(HIP_SYMBOL(g_status), &zero, sizeof(unsigned int), 0,
                             hipMemcpyHostToDevice);
}

struct LayerPtrs {
    pkv_page *table;  // this layer's entries
    char *dense;      // this layer's dense slots
    char *factor;     // this layer's factor slots
};

inline LayerPtrs layer_ptrs(const LaunchCtx &L) {
    LayerPtrs p;
    p.table = L.c->page_table + (int64_t)L.layer * L.geo.layer_entries;
    p.dense = (char *)L.c->dense_pool + (int64_t)L.layer * L.geo.layer_dense_bytes;
    p.factor = (char *)L.c->factor_pool + (int64_t)L.layer * L.geo.layer_factor_bytes;
    return p;
}

// rows: tokens a DENSE page holds (1..P); 0 for other kinds.
__device__ inline void write_entry(pkv_page *e, int slot, int kind, int rk, int rv, int rows = 0) {
    pkv_page v;
    v.slot = slot;
    v.kind = (uint8_t)kind;
    v.rank_k = (uint8_t)rk;
    v.rank_v = (uint8_t)rv;
    v.rows = (uint8_t)rows;
    *e = v;
}

// Whether logical page j of (sequence, KV head) `head` may be factorized now
// (Section 3.3, "Incremental Cache Update": a page is converted once, when it
// is complete and has left the local window; sink pages stay dense). It must
// be DENSE and hold P rows, lie outside the sink, and the cache must already
// hold token (j + 1) P + W - 1, i.e. at least W tokens past the page. Returns
// 0, or the status bit that refuses it.
__device__ inline unsigned int compress_refusal(const Geo &g, const pkv_page *table, int64_t head, int j) {
    const pkv_page e = table[head * g.max_pages + j];
    if (e.kind != PKV_DENSE) return PKV_DEV_NOT_DENSE;
    if (j < g.sink_pages || e.rows < g.P) return PKV_DEV_NOT_ELIGIBLE;
    const int64_t m = (int64_t)(j + 1) * g.P + g.W - 1;
    const int64_t jm = m / g.P;
    if (jm >= g.max_pages) return PKV_DEV_NOT_ELIGIBLE;
    const pkv_page em = table[head * g.max_pages + jm];
    const bool held = em.kind == PKV_FACTOR || (em.kind == PKV_DENSE && (int64_t)em.rows > m % g.P);
    return held ? 0u : PKV_DEV_NOT_ELIGIBLE;
}

// Whether the dense slot of page j is held by another DENSE page of the head
// (a page that maps to the same ring position). Every thread of the
// workgroup scans a share of those pages; the result is the workgroup's.
__device__ inline bool dense_slot_taken(const Geo &g, const pkv_page *table, int64_t head, int j) {
    __shared__ int s_taken;
    if (threadIdx.x == 0) s_taken = 0;
    __syncthreads();
    if (j >= g.sink_pages) {
        const int first = g.sink_pages + (j - g.sink_pages) % g.ring_len;
        for (int jj = first + (int)threadIdx.x * g.ring_len; jj < g.max_pages; jj += (int)blockDim.x * g.ring_len)
            if (jj != j && table[head * g.max_pages + jj].kind == PKV_DENSE) s_taken = 1;
    }
    __syncthreads();
    return s_taken != 0;
}

// ---- reset ------------------------------------------------------------------

__global__ void k_reset(pkv_page *table, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        write_entry(table + i, 0, PKV_EMPTY, 0, 0);
}

hipError_t launch_reset(const LaunchCtx &L, int64_t first_entry, int64_t n_entries) {
    if (n_entries <= 0) return hipSuccess;
    int blocks = (int)std::min<int64_t>(ceil_div(n_entries, 256), 4096);
    hipLaunchKernelGGL(k_reset, dim3(blocks), dim3(256), 0, L.stream, L.c->page_table + first_entry,
                       n_entries);
    return hipGetLastError();
}

// ---- dense page copy: source rows (row-major) -> slot (K row-major, V^T) ----

template <typename T>
__device__ void copy_dense_page(const Geo &g, const T *srcK, const T *srcV, int64_t src_row_stride,
                                int rows, T *slot) {
    const int P = g.P, d = g.d;
    T *K = slot;
    T *Vt = slot + (int64_t)P * d;
    for (int i = threadIdx.x; i < P * d; i += blockDim.x) {
        int t = i / d, k = i % d;
        K[i] = t < rows ? srcK[t * src_row_stride + k] : T(0);
    }
    for (int i = threadIdx.x; i < P * d; i += blockDim.x) {
        int k = i / P, t = i % P;
        Vt[i] = t < rows ? srcV[t * src_row_stride + k] : T(0);
    }
}

// ---- prefill: table entries and dense pages --------------------------------

template <typename TE>
__global__ __launch_bounds__(256) void k_prefill_pages(Geo g, pkv_page *table, char *dense,
                                                       const TE *k, const TE *v, int64_t src_tokens,
                                                       SeqArgs seq, const uint8_t *rank_k,
                                                       const uint8_t *rank_v, int def_rk, int def_rv,
                                                       int glob_r) {
    const int j = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int64_t T = seq.len[b];
    const int64_t head = g.head_index(b, h);
    pkv_page *e = table + head * g.max_pages + j;
    const int kind = plan_kind(T, g.P, g.S, g.W, j);
    if (kind == PKV_EMPTY) {
        if (threadIdx.x == 0) write_entry(e, 0, PKV_EMPTY, 0, 0);
        return;
    }
    if (kind == PKV_FACTOR && glob_r > 0) {
        // Global SVD cache: the page's tokens are rows of the head's
        // coefficients; slot = the row of its first token
        if (threadIdx.x == 0) write_entry(e, (j - g.sink_pages) * g.P, PKV_GLOBAL, glob_r, glob_r);
        return;
    }
    if (kind == PKV_FACTOR) {
        if (threadIdx.x == 0) {
            const int rmax = min(g.max_rank, min(g.P, g.d));
            int rk = def_rk, rv = def_rv;
            if (rank_k) {
                rk = rank_k[head * g.max_pages + j];
                rv = rank_v[head * g.max_pages + j];
                // 0 with adaptive ranks: chosen by the decomposition, which
                // writes it into this entry
                const int rmin = g.rank_err > 0.f ? 0 : 1;
                if (rk < rmin || rk > rmax || rv < rmin || rv > rmax) raise_status(PKV_DEV_BAD_RANK);
                rk = max(rmin, min(rk, rmax));
                rv = max(rmin, min(rv, rmax));
            }
            write_entry(e, (int)(head * g.max_pages + j), PKV_FACTOR, rk, rv);
        }
        return;
    }
    const int slot = (int)(head * g.dslots + g.dense_ring_slot(j));
    const int64_t t0 = (int64_t)j * g.P;
    const int rows = (int)min<int64_t>(g.P, T - t0);
    const TE *sK = k + (head * src_tokens + t0) * g.d;
    const TE *sV = v + (head * src_tokens + t0) * g.d;
    copy_dense_page<TE>(g, sK, sV, g.d, rows, (TE *)(dense + slot * g.dense_slot_bytes));
    if (threadIdx.x == 0) write_entry(e, slot, PKV_DENSE, 0, 0, rows);
}

hipError_t launch_prefill_pages(const LaunchCtx &L, const void *k, const void *v, int64_t src_tokens,
                                const SeqArgs &seq, const uint8_t *rank_k, const uint8_t *rank_v,
                                int def_rk, int def_rv, int max_pages_in_batch, int glob_r) {
    LayerPtrs p = layer_ptrs(L);
    dim3 grid(max_pages_in_batch, L.geo.Hkv, L.geo.B);
    if (L.geo.dense_dtype == PKV_BF16)
        hipLaunchKernelGGL(k_prefill_pages<uint16_t>, grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, (const uint16_t *)k, (const uint16_t *)v, src_tokens, seq, rank_k,
                           rank_v, def_rk, def_rv, glob_r);
    else
        hipLaunchKernelGGL(k_prefill_pages<float>, grid, dim3(256), 0, L.stream, L.geo, p.table, p.dense,
                           (const float *)k, (const float *)v, src_tokens, seq, rank_k, rank_v, def_rk,
                           def_rv, glob_r);
    return hipGetLastError();
}

// ---- append ------------------------------------------------------------------

template <typename T>
__global__ void k_append(Geo g, pkv_page *table, char *dense, const T *k_new, const T *v_new,
                         SeqArgs pos) {
    const int h = blockIdx.x, b = blockIdx.y;
    const int64_t p = pos.len[b];
    if (p < 0) return;
    const int64_t head = g.head_index(b, h);
    const int j = (int)(p / g.P), row = (int)(p % g.P);
    pkv_page *e = table + head * g.max_pages + j;
    int slot;
    if (row == 0) {
        // a new page starts; its ring position must not hold a page still dense
        const int jprev = j - g.ring_len;
        if (j >= g.sink_pages && jprev >= g.sink_pages) {
            pkv_page old = table[head * g.max_pages + jprev];
            if (old.kind == PKV_DENSE) {
                if (threadIdx.x == 0) raise_status(PKV_DEV_RING_OVERRUN);
                return;
            }
        }
        slot = (int)(head * g.dslots + g.dense_ring_slot(j));
    } else {
        pkv_page cur = *e;
        if (cur.kind != PKV_DENSE) {
            if (threadIdx.x == 0) raise_status(PKV_DEV_BAD_PAGE);
            return;
        }
        slot = cur.slot;
    }
    T *K = (T *)(dense + slot * g.dense_slot_bytes);
    T *Vt = K + (int64_t)g.P * g.d;
    const T *kn = k_new + head * g.d;
    const T *vn = v_new + head * g.d;
    for (int i = threadIdx.x; i < g.d; i += blockDim.x) {
        K[(int64_t)row * g.d + i] = kn[i];
        Vt[(int64_t)i * g.P + row] = vn[i];
    }
    if (threadIdx.x == 0) {
        if (row == 0) write_entry(e, slot, PKV_DENSE, 0, 0, 1);
        else e->rows = (uint8_t)(row + 1);
    }
}

hipError_t launch_append(const LaunchCtx &L, const void *k_new, const void *v_new, const SeqArgs &pos) {
    LayerPtrs p = layer_ptrs(L);
    dim3 grid(L.geo.Hkv, L.geo.B);
    int threads = std::min(256, L.geo.d);
    if (L.geo.dense_dtype == PKV_BF16)
        hipLaunchKernelGGL(k_append<uint16_t>, grid, dim3(threads), 0, L.stream, L.geo, p.table, p.dense,
                           (const uint16_t *)k_new, (const uint16_t *)v_new, pos);
    else
        hipLaunchKernelGGL(k_append<float>, grid, dim3(threads), 0, L.stream, L.geo, p.table, p.dense,
                           (const float *)k_new, (const float *)v_new, pos);
    return hipGetLastError();
}

// ---- compress commit: DENSE -> FACTOR entries after the decompositions ------

// list: the items in device memory (n of them), or null for the launch's items.
__global__ void k_compress_commit(Geo g, pkv_page *table, CompressItems items, const CompressItem *list,
                                  int64_t n) {
    const int64_t i = threadIdx.x + (int64_t)blockIdx.x * blockDim.x;
    if (i >= (list ? n : (int64_t)items.n)) return;
    const CompressItem it = list ? list[i] : items.it[i];
    const int64_t idx = g.head_index(it.b, it.h) * g.max_pages + it.j;
    // the same test the decompositions made: a refused page stays as it is
    if (compress_refusal(g, table, g.head_index(it.b, it.h), it.j) == 0u) {
        // a requested rank of 0 was chosen by the decomposition and stored in the entry
        const pkv_page cur = table[idx];
        write_entry(table + idx, (int)idx, PKV_FACTOR, it.rk ? it.rk : cur.rank_k, it.rv ? it.rv : cur.rank_v);
    }
}

hipError_t launch_compress_commit(const LaunchCtx &L, const CompressItems &items) {
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL(k_compress_commit, dim3(1), dim3(128), 0, L.stream, L.geo, p.table, items,
                       (const CompressItem *)nullptr, (int64_t)0);
    return hipGetLastError();
}

hipError_t launch_compress_commit_list(const LaunchCtx &L, const CompressItem *list, int64_t n) {
    if (n <= 0) return hipSuccess;
    LayerPtrs p = layer_ptrs(L);
    hipLaunchKernelGGL(k_compress_commit, dim3((unsigned)ceil_div(n, 128)), dim3(128), 0, L.stream, L.geo, p.table,
                       CompressItems{}, list, n);
    return hipGetLastError();
}

// ---- import (logical layout -> slots) ---------------------------------------

template <typename TD, typename TF>
__global__ __launch_bounds__(256) void k_import(Geo g, pkv_page *table, char *dense, char *factor,
                                                const char *src, CopyItems items) {
    const CopyItem it = items.it[blockIdx.x];
    const int64_t head = g.head_index(it.b, it.h);
    pkv_page *e = table + head * g.max_pages + it.j;
    const int P = g.P, d = g.d;
    if (it.kind == PKV_DENSE) {
        if (dense_slot_taken(g, table, head, it.j)) {
            if (threadIdx.x == 0) raise_status(PKV_DEV_RING_OVERRUN);
            return;
        }
        const TD *s = (const TD *)src + it.src_off;
        const int slot = (int)(head * g.dslots + g.dense_ring_slot(it.j));
        copy_dense_page<TD>(g, s, s + (int64_t)P * d, d, P, (TD *)(dense + slot * g.dense_slot_bytes));
        if (threadIdx.x == 0) write_entry(e, slot, PKV_DENSE, 0, 0, P);
        return;
    }
    const int rk = it.rk, rv = it.rv, rk4 = r4(rk), rv4 = r4(rv);
    const TF *Lk = (const TF *)src + it.src_off;
    const TF *Rk = Lk + (int64_t)P * rk;
    const TF *Lv = Rk + (int64_t)rk * d;
    const TF *Rv = Lv + (int64_t)P * rv;
    const int slot = (int)(head * g.max_pages + it.j);
    const FactorLayout fl = factor_layout(P, d, rk, rv, g.key_t != 0);
    TF *Ak = (TF *)(factor + slot * g.factor_slot_bytes);
    TF *Bk = Ak + fl.bk, *Bvt = Ak + fl.bvt, *Avt = Ak + fl.avt;
    for (int i = threadIdx.x; i < P * rk4; i += blockDim.x) {
        int t = i / rk4, a = i % rk4;
        Ak[i] = a < rk ? Lk[t * rk + a] : TF(0);
    }
    if (g.key_t) {   // R_K^T, d x r4(rk)
        for (int i = threadIdx.x; i < d * rk4; i += blockDim.x) {
            int k = i / rk4, a = i % rk4;
            Bk[i] = a < rk ? Rk[(int64_t)a * d + k] : TF(0);
        }
    } else {
        for (int i = threadIdx.x; i < rk * d; i += blockDim.x) Bk[i] = Rk[i];
    }
    for (int i = threadIdx.x; i < rv * P; i += blockDim.x) {
        int a = i / P, t = i % P;
        Avt[i] = Lv[t * rv + a];
    }
    for (int i = threadIdx.x; i < d * rv4; i += blockDim.x) {
        int k = i / rv4, a = i % rv4;
        Bvt[i] = a < rv ? Rv[(int64_t)a * d + k] : TF(0);
    }
    if (threadIdx.x == 0) write_entry(e, slot, PKV_FACTOR, rk, rv);
}

hipError_t launch_import(const LaunchCtx &L, const CopyItems &items, const void *src) {
    if (L.geo.factor_dtype == PKV_INT4) return launch_import_q4(L, items, src);
    LayerPtrs p = layer_ptrs(L);
    dim3 grid(items.n);
    const bool db = L.geo.dense_dtype == PKV_BF16, fb = L.geo.factor_dtype == PKV_BF16;
    if (db && fb)
        hipLaunchKernelGGL((k_import<uint16_t, uint16_t>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, (const char *)src, items);
    else if (db)
        hipLaunchKernelGGL((k_import<uint16_t, float>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, (const char *)src, items);
    else if (fb)
        hipLaunchKernelGGL((k_import<float, uint16_t>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, (const char *)src, items);
    else
        hipLaunchKernelGGL((k_import<float, float>), grid, dim3(256), 0, L.stream, L.geo, p.table, p.dense,
                           p.factor, (const char *)src, items);
    return hipGetLastError();
}

// ---- export (slots -> logical fp32 blocks) ----------------------------------

template <typename TD, typename TF>
__global__ __launch_bounds__(256) void k_export(Geo g, const pkv_page *table, const char *dense,
                                                const char *factor, float *dst, CopyItems items,
                                                int64_t block) {
    const CopyItem it = items.it[blockIdx.x];
    const int64_t head = g.head_index(it.b, it.h);
    const pkv_page e = table[head * g.max_pages + it.j];
    float *o = dst + it.src_off;
    const int P = g.P, d = g.d, R = g.max_rank;
    if (e.kind == PKV_DENSE) {
        const TD *K = (const TD *)(dense + e.slot * g.dense_slot_bytes);
        const TD *Vt = K + (int64_t)P * d;
        for (int i = threadIdx.x; i < P * d; i += blockDim.x) {
            int t = i / d, k = i % d;
            o[i] = ld(K, i);
            o[P * d + i] = ld(Vt, (int64_t)k * P + t);
        }
        for (int i = 2 * P * d + threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
        return;
    }
    if (e.kind != PKV_FACTOR) {
        for (int i = threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
        return;
    }
    const int rk = e.rank_k, rv = e.rank_v, rk4 = r4(rk), rv4 = r4(rv);
    const FactorLayout fl = factor_layout(P, d, rk, rv, g.key_t != 0);
    const TF *Ak = (const TF *)(factor + e.slot * g.factor_slot_bytes);
    const TF *Bk = Ak + fl.bk, *Bvt = Ak + fl.bvt, *Avt = Ak + fl.avt;
    float *Lk = o, *Rk = Lk + P * R, *Lv = Rk + R * d, *Rv = Lv + P * R;
    for (int i = threadIdx.x; i < P * R; i += blockDim.x) {
        int t = i / R, a = i % R;
        Lk[i] = a < rk ? ld(Ak, t * rk4 + a) : 0.f;
        Lv[i] = a < rv ? ld(Avt, (int64_t)a * P + t) : 0.f;
    }
    for (int i = threadIdx.x; i < R * d; i += blockDim.x) {
        int a = i / d, k = i % d;
        Rk[i] = a < rk ? ld(Bk, g.key_t ? (int64_t)k * rk4 + a : (int64_t)i) : 0.f;
        Rv[i] = a < rv ? ld(Bvt, (int64_t)k * rv4 + a) : 0.f;
    }
    for (int i = 2 * (P + d) * R + threadIdx.x; i < block; i += blockDim.x) o[i] = 0.f;
}

hipError_t launch_export(const LaunchCtx &L, const CopyItems &items, float *dst, int64_t block) {
    if (L.geo.factor_dtype == PKV_INT4) return launch_export_dq4(L, items, dst, block);
    LayerPtrs p = layer_ptrs(L);
    dim3 grid(items.n);
    const bool db = L.geo.dense_dtype == PKV_BF16, fb = L.geo.factor_dtype == PKV_BF16;
    if (db && fb)
        hipLaunchKernelGGL((k_export<uint16_t, uint16_t>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, dst, items, block);
    else if (db)
        hipLaunchKernelGGL((k_export<uint16_t, float>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, dst, items, block);
    else if (fb)
        hipLaunchKernelGGL((k_export<float, uint16_t>), grid, dim3(256), 0, L.stream, L.geo, p.table,
                           p.dense, p.factor, dst, items, block);
    else
        hipLaunchKernelGGL((k_export<float, float>), grid, dim3(256), 0, L.stream, L.geo, p.table, p.dense,
                           p.factor, dst, items, block);
    return hipGetLastError();
}

}  // namespace pkv
