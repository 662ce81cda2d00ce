// Host side of the PuzzleKV C ABI: argument and state validation, page
// planning (integer), work lists, and kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pkv_internal.h"

using namespace pkv;

namespace {

thread_local std::string g_err;

pkv_status fail(pkv_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

pkv_status hip_fail(hipError_t e, const char *what) {
    return fail(PKV_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

int elem_size(int dt) { return dt == PKV_F32 ? 4 : dt == PKV_BF16 ? 2 : 0; }

pkv_status check_geometry(const pkv_cache *c) {
    if (!c) return fail(PKV_E_ARG, "cache descriptor is NULL");
    if (c->n_layers <= 0 || c->batch <= 0 || c->n_kv_heads <= 0 || c->n_q_heads <= 0)
        return fail(PKV_E_SHAPE, "layers, batch and head counts must be positive");
    if (c->batch > kMaxBatchArgs - 1)
        return fail(PKV_E_SHAPE, "batch %d above the supported %d", c->batch, kMaxBatchArgs - 1);
    if (c->n_q_heads % c->n_kv_heads)
        return fail(PKV_E_SHAPE, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)",
                    c->n_q_heads, c->n_kv_heads);
    if (c->n_q_heads / c->n_kv_heads > 16)
        return fail(PKV_E_SHAPE, "query group %d above 16", c->n_q_heads / c->n_kv_heads);
    if (c->head_dim <= 0 || c->head_dim % 32 || c->head_dim > 256)
        return fail(PKV_E_SHAPE, "head_dim %d: must be a multiple of 32 and <= 256", c->head_dim);
    if (c->page_size != 16 && c->page_size != 32 && c->page_size != 64)
        return fail(PKV_E_SHAPE, "page_size %d: must be 16, 32 or 64", c->page_size);
    if (c->max_pages <= 0) return fail(PKV_E_SHAPE, "max_pages must be positive");
    if (c->max_rank <= 0 || c->max_rank > std::min(c->page_size, c->head_dim) || c->max_rank > 255)
        return fail(PKV_E_RANK, "max_rank %d outside 1..min(P, d)", c->max_rank);
    if (c->sink_tokens < 0 || c->window_tokens < 0)
        return fail(PKV_E_SHAPE, "sink and window must be non-negative");
    if (elem_size(c->dense_dtype) == 0) return fail(PKV_E_UNSUPPORTED, "dense dtype %d", c->dense_dtype);
    if (!(c->adaptive_rank_error >= 0.f && c->adaptive_rank_error < 1.f))
        return fail(PKV_E_ARG, "adaptive_rank_error %g outside [0, 1)", (double)c->adaptive_rank_error);
    if (c->adaptive_rank_error > 0.f && (c->dense_dtype != PKV_BF16 || (c->page_size != 32 && c->page_size != 64)))
        return fail(PKV_E_UNSUPPORTED, "adaptive ranks need bf16 dense pages with P = 32 or 64");
    if (!(c->key_rope_base >= 0.f && c->key_rope_base < INFINITY))
        return fail(PKV_E_ARG, "key_rope_base %g: must be 0 (off) or a positive finite base", (double)c->key_rope_base);
    if (c->key_rope_base > 0.f) {
        if (c->dense_dtype != PKV_BF16 || c->factor_dtype != PKV_BF16 || (c->page_size != 32 && c->page_size != 64) ||
            (c->head_dim != 64 && c->head_dim != 128) || c->max_rank > 32)
            return fail(PKV_E_UNSUPPORTED, "pre-RoPE keys need bf16 dense pages and factors, P = 32 or 64, "
                                           "head_dim = 64 or 128 and max_rank <= 32");
        if ((int64_t)c->max_pages * c->page_size > (1 << 24))
            return fail(PKV_E_UNSUPPORTED, "pre-RoPE keys: positions must stay below 2^24");
    }
    if (c->factor_dtype == PKV_INT4) {
        if (c->dense_dtype != PKV_BF16 || c->page_size != 64 || c->head_dim != 128 || c->max_rank > 32)
            return fail(PKV_E_UNSUPPORTED,
                        "INT4 factors need bf16 dense pages, P = 64, head_dim = 128 and max_rank <= 32");
        if (ceil_div(c->sink_tokens, c->page_size) + ceil_div(c->window_tokens, c->page_size) + 2 > 256)
            return fail(PKV_E_UNSUPPORTED, "INT4 factors need at most 256 dense slots per head");
        return PKV_OK;
    }
    if (elem_size(c->factor_dtype) == 0)
        return fail(PKV_E_UNSUPPORTED, "factor dtype %d", c->factor_dtype);
    return PKV_OK;
}

// Stored bytes of one factor page pair (codes and scales for INT4); a slot
// adds the INT4 pad.
int64_t factor_page_bytes_of(int dtype, int P, int d, int rk, int rv, bool kt) {
    if (dtype == PKV_INT4) return int4_layout(P, d, rk, rv).pad;
    return factor_page_elems(P, d, rk, rv, kt) * elem_size(dtype);
}
int64_t factor_slot_bytes_of(int dtype, int P, int d, int r, bool kt) {
    if (dtype == PKV_INT4) return int4_layout(P, d, r, r).end;
    return factor_page_bytes_of(dtype, P, d, r, r, kt);
}

Geo make_geo(const pkv_cache *c) {
    Geo g{};
    g.B = c->batch;
    g.Hkv = c->n_kv_heads;
    g.Hq = c->n_q_heads;
    g.g = c->n_q_heads / c->n_kv_heads;
    g.d = c->head_dim;
    g.P = c->page_size;
    g.max_pages = c->max_pages;
    g.max_rank = c->max_rank;
    g.rank_err = c->adaptive_rank_error;
    g.rope_base = c->key_rope_base;
    g.key_t = c->key_rope_base > 0.f ? 1 : 0;
    g.S = c->sink_tokens;
    g.W = c->window_tokens;
    g.sink_pages = (int)ceil_div(c->sink_tokens, c->page_size);
    g.ring_len = (int)ceil_div(c->window_tokens, c->page_size) + 2;
    g.dslots = g.sink_pages + g.ring_len;
    g.dense_es = elem_size(c->dense_dtype);
    g.factor_es = elem_size(c->factor_dtype);
    g.dense_dtype = c->dense_dtype;
    g.factor_dtype = c->factor_dtype;
    g.dense_slot_bytes = 2LL * g.P * g.d * g.dense_es;
    int64_t fb = factor_slot_bytes_of(c->factor_dtype, g.P, g.d, g.max_rank, g.key_t != 0);
    g.factor_slot_bytes = (fb + 255) / 256 * 256;
    g.layer_entries = (int64_t)g.B * g.Hkv * g.max_pages;
    g.layer_dense_bytes = (int64_t)g.B * g.Hkv * g.dslots * g.dense_slot_bytes;
    g.layer_factor_bytes = g.layer_entries * g.factor_slot_bytes;
    return g;
}

pkv_status check_cache(const pkv_cache *c, bool need_pools) {
    pkv_status s = check_geometry(c);
    if (s != PKV_OK) return s;
    if (!c->page_table) return fail(PKV_E_ARG, "page_table is NULL");
    if (need_pools && (!c->dense_pool || !c->factor_pool))
        return fail(PKV_E_ARG, "dense_pool or factor_pool is NULL");
    return PKV_OK;
}

pkv_status check_layer(const pkv_cache *c, int32_t layer) {
    if (layer < 0 || layer >= c->n_layers)
        return fail(PKV_E_ARG, "layer %d outside 0..%d", layer, c->n_layers - 1);
    return PKV_OK;
}

pkv_status check_ws(void *ws, size_t have, size_t need) {
    if (need == 0) return PKV_OK;
    if (!ws) return fail(PKV_E_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
    if (have < need) return fail(PKV_E_WORKSPACE, "workspace of %zu bytes, %zu needed", have, need);
    return PKV_OK;
}

pkv_status check_launch(hipError_t e, const char *what) {
    if (e != hipSuccess) return hip_fail(e, what);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, what);
    return PKV_OK;
}

LaunchCtx ctx(const pkv_cache *c, int layer, pkv_stream s) {
    LaunchCtx L;
    L.c = c;
    L.geo = make_geo(c);
    L.layer = layer;
    L.stream = (hipStream_t)s;
    return L;
}

}  // namespace

extern "C" {

const char *pkv_last_error(void) { return g_err.c_str(); }
const char *pkv_version(void) { return "puzzlekv-mi355x 0.1 (gfx950)"; }

pkv_status pkv_cache_check(const pkv_cache *c) { return check_cache(c, true); }

int64_t pkv_dense_slots_per_head(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return -1;
    return make_geo(c).dslots;
}
size_t pkv_dense_slot_bytes(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return 0;
    return (size_t)make_geo(c).dense_slot_bytes;
}
size_t pkv_factor_slot_bytes(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return 0;
    return (size_t)make_geo(c).factor_slot_bytes;
}
size_t pkv_dense_pool_bytes(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return 0;
    return (size_t)(make_geo(c).layer_dense_bytes * c->n_layers);
}
size_t pkv_factor_pool_bytes(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return 0;
    return (size_t)(make_geo(c).layer_factor_bytes * c->n_layers);
}
size_t pkv_page_table_bytes(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return 0;
    return (size_t)(make_geo(c).layer_entries * c->n_layers * (int64_t)sizeof(pkv_page));
}
size_t pkv_factor_page_bytes(const pkv_cache *c, int32_t rank_k, int32_t rank_v) {
    if (check_geometry(c) != PKV_OK) return 0;
    if (rank_k < 1 || rank_v < 1 || rank_k > c->max_rank || rank_v > c->max_rank) return 0;
    return (size_t)factor_page_bytes_of(c->factor_dtype, c->page_size, c->head_dim, rank_k, rank_v,
                                        c->key_rope_base > 0.f);
}
int64_t pkv_int4_blob_bytes(const pkv_cache *c, int32_t rank_k, int32_t rank_v) {
    if (check_geometry(c) != PKV_OK || c->factor_dtype != PKV_INT4) return -1;
    if (rank_k < 1 || rank_v < 1 || rank_k > c->max_rank || rank_v > c->max_rank) return -1;
    return int4_blob_bytes(c->page_size, c->head_dim, rank_k, rank_v);
}
int64_t pkv_export_block_elems(const pkv_cache *c) {
    if (check_geometry(c) != PKV_OK) return -1;
    int64_t dense = 2LL * c->page_size * c->head_dim;
    int64_t fact = 2LL * (c->page_size + c->head_dim) * c->max_rank;
    return std::max(dense, fact);
}

size_t pkv_workspace_bytes(const pkv_cache *c, int32_t op, int64_t n) {
    if (check_geometry(c) != PKV_OK || n < 0) return 0;
    Geo g = make_geo(c);
    switch (op) {
    case PKV_OP_ATTENTION: return (size_t)attention_workspace_bytes(g, n);
    case PKV_OP_COMPRESS: return (size_t)((n * (int64_t)sizeof(CompressItem) + 255) / 256 * 256);
    case PKV_OP_PREFILL: return 0;
    case PKV_OP_IMPORT: return 0;
    case PKV_OP_GLOBAL_PREFILL: return (size_t)global_prefill_workspace_bytes(g, n);
    case PKV_OP_GLOBAL_ATTENTION: return (size_t)global_attention_workspace_bytes(g, n);
    default: return 0;
    }
}

// ---- page plan -------------------------------------------------------------

pkv_status pkv_plan_pages(int64_t T, int32_t P, int32_t S, int32_t W, uint8_t *kind, int64_t n,
                          int64_t *n_pages) {
    if (P <= 0 || T < 0 || S < 0 || W < 0 || n < 0) return fail(PKV_E_ARG, "negative or zero argument");
    if (n > 0 && !kind) return fail(PKV_E_ARG, "kind is NULL");
    for (int64_t j = 0; j < n; ++j) kind[j] = (uint8_t)plan_kind(T, P, S, W, j);
    if (n_pages) *n_pages = T > 0 ? ceil_div(T, P) : 0;
    return PKV_OK;
}

pkv_status pkv_eligible_pages(int64_t T_prev, int64_t T_new, int32_t P, int32_t S, int32_t W,
                              int32_t *pages, int64_t cap, int64_t *count) {
    if (P <= 0 || T_prev < 0 || T_new < 0 || S < 0 || W < 0 || cap < 0)
        return fail(PKV_E_ARG, "negative or zero argument");
    if (cap > 0 && !pages) return fail(PKV_E_ARG, "pages is NULL");
    // Factor pages form the range [sink_pages, floor((T - W) / P) - 1]; a
    // length increase only extends it upward.
    int64_t cnt = 0;
    int64_t n_new = T_new > 0 ? ceil_div(T_new, P) : 0;
    for (int64_t j = 0; j < n_new; ++j) {
        if (plan_kind(T_new, P, S, W, j) == PKV_FACTOR && plan_kind(T_prev, P, S, W, j) != PKV_FACTOR) {
            if (cnt < cap) pages[cnt] = (int32_t)j;
            ++cnt;
        }
    }
    if (count) *count = cnt;
    return PKV_OK;
}

// ---- cache maintenance ---------------------------------------------------------

pkv_status pkv_cache_reset(const pkv_cache *c, int32_t layer, pkv_stream s) {
    pkv_status st = check_cache(c, false);
    if (st != PKV_OK) return st;
    if (layer >= c->n_layers) return fail(PKV_E_ARG, "layer %d outside 0..%d", layer, c->n_layers - 1);
    LaunchCtx L = ctx(c, layer < 0 ? 0 : layer, s);
    int64_t first = layer < 0 ? 0 : layer * L.geo.layer_entries;
    int64_t n = layer < 0 ? L.geo.layer_entries * c->n_layers : L.geo.layer_entries;
    return check_launch(launch_reset(L, first, n), "pkv_cache_reset");
}

pkv_status pkv_prefill(const pkv_cache *c, int32_t layer, const void *k, const void *v,
                       int64_t src_tokens, const int32_t *seq_len, const uint8_t *rank_k,
                       const uint8_t *rank_v, int32_t default_rank_k, int32_t default_rank_v,
                       void *ws, size_t ws_bytes, pkv_stream s) {
    (void)ws; (void)ws_bytes;
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!k || !v || !seq_len) return fail(PKV_E_ARG, "k, v or seq_len is NULL");
    if ((rank_k == nullptr) != (rank_v == nullptr))
        return fail(PKV_E_ARG, "rank_k and rank_v must both be given or both be NULL");
    const int rmax = std::min(c->max_rank, std::min(c->page_size, c->head_dim));
    const int rmin = c->adaptive_rank_error > 0.f ? 0 : 1;   // 0: chosen per page
    if (!rank_k && (default_rank_k < rmin || default_rank_v < rmin || default_rank_k > rmax ||
                    default_rank_v > rmax))
        return fail(PKV_E_RANK, "default ranks (%d, %d) outside %d..%d", default_rank_k, default_rank_v, rmin,
                    rmax);
    SeqArgs seq{};
    seq.n = c->batch;
    int max_np = 0;
    for (int b = 0; b < c->batch; ++b) {
        if (seq_len[b] < 0 || seq_len[b] > src_tokens ||
            (int64_t)seq_len[b] > (int64_t)c->max_pages * c->page_size)
            return fail(PKV_E_SHAPE, "seq_len[%d] = %d outside 0..min(src_tokens, max_pages * P)", b,
                        seq_len[b]);
        seq.len[b] = seq_len[b];
        max_np = std::max(max_np, (int)ceil_div(seq_len[b], c->page_size));
    }
    LaunchCtx L = ctx(c, layer, s);
    const Geo &g = L.geo;
    // Factor pages of sequence b are j in [sink_pages, floor((T - W) / P) - 1];
    // items are numbered b-major, then KV head, then page.
    SeqArgs off{};
    off.n = c->batch + 1;
    int64_t total = 0;
    for (int b = 0; b < c->batch; ++b) {
        off.len[b] = (int32_t)total;
        int64_t T = seq_len[b];
        int64_t jmax = T - g.W >= 0 ? (T - g.W) / g.P - 1 : -1;
        int64_t nf = std::max<int64_t>(0, jmax - g.sink_pages + 1);
        total += nf * g.Hkv;
    }
    off.len[c->batch] = (int32_t)total;
    if (total > INT32_MAX / 2) return fail(PKV_E_SHAPE, "too many pages in one prefill");
    hipError_t e = launch_prefill_pages(L, k, v, src_tokens, seq, rank_k, rank_v, default_rank_k,
                                        default_rank_v, c->max_pages);
    if ((st = check_launch(e, "pkv_prefill (pages)")) != PKV_OK) return st;
    if (total > 0) {
        e = launch_prefill_compress(L, k, v, src_tokens, off.len, total, rank_k, rank_v, default_rank_k,
                                    default_rank_v);
        if ((st = check_launch(e, "pkv_prefill (compress)")) != PKV_OK) return st;
    }
    return PKV_OK;
}

pkv_status pkv_append_kv(const pkv_cache *c, int32_t layer, const void *k_new, const void *v_new,
                         const int32_t *pos, pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!k_new || !v_new || !pos) return fail(PKV_E_ARG, "k_new, v_new or pos is NULL");
    SeqArgs a{};
    a.n = c->batch;
    for (int b = 0; b < c->batch; ++b) {
        if (pos[b] >= (int64_t)c->max_pages * c->page_size)
            return fail(PKV_E_SHAPE, "pos[%d] = %d beyond max_pages * P", b, pos[b]);
        a.len[b] = pos[b];
    }
    LaunchCtx L = ctx(c, layer, s);
    return check_launch(launch_append(L, k_new, v_new, a), "pkv_append_kv");
}

pkv_status pkv_compress_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                              const int32_t *kv_head, const int32_t *page, const uint8_t *rank_k,
                              const uint8_t *rank_v, void *ws, size_t ws_bytes, pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (n < 0) return fail(PKV_E_ARG, "n < 0");
    if (n == 0) return PKV_OK;
    if (!b || !kv_head || !page || !rank_k || !rank_v) return fail(PKV_E_ARG, "NULL page list");
    const int rmax = std::min(c->max_rank, std::min(c->page_size, c->head_dim));
    const int rmin = c->adaptive_rank_error > 0.f ? 0 : 1;   // 0: chosen per page
    std::vector<int64_t> keys((size_t)n);
    for (int i = 0; i < n; ++i) {
        if (b[i] < 0 || b[i] >= c->batch || kv_head[i] < 0 || kv_head[i] >= c->n_kv_heads ||
            page[i] < 0 || page[i] >= c->max_pages)
            return fail(PKV_E_ARG, "page ref %d (b=%d, h=%d, j=%d) out of range", i, b[i], kv_head[i], page[i]);
        if (rank_k[i] < rmin || rank_v[i] < rmin || rank_k[i] > rmax || rank_v[i] > rmax)
            return fail(PKV_E_RANK, "page ref %d: ranks (%d, %d) outside %d..%d", i, rank_k[i], rank_v[i], rmin,
                        rmax);
        if (page[i] < ceil_div(c->sink_tokens, c->page_size))
            return fail(PKV_E_STATE, "page ref %d: page %d is a sink page, which stays dense", i, page[i]);
        keys[i] = ((int64_t)b[i] * c->n_kv_heads + kv_head[i]) * c->max_pages + page[i];
    }
    std::vector<int64_t> sorted = keys;
    std::sort(sorted.begin(), sorted.end());
    if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
        return fail(PKV_E_ARG, "duplicate page in one compress call");
    LaunchCtx L = ctx(c, layer, s);
    if (ws && ws_bytes >= (size_t)n * sizeof(CompressItem)) {
        // the item list in the workspace: every page in one launch
        std::vector<CompressItem> list((size_t)n);
        for (int i = 0; i < n; ++i) {
            CompressItem &it = list[(size_t)i];
            it = CompressItem{};
            it.b = b[i];
            it.h = kv_head[i];
            it.j = page[i];
            it.rk = rank_k[i];
            it.rv = rank_v[i];
        }
        const CompressItem *dl = (const CompressItem *)ws;
        if ((st = check_launch(hipMemcpyAsync(ws, list.data(), (size_t)n * sizeof(CompressItem),
                                              hipMemcpyHostToDevice, L.stream),
                               "pkv_compress_pages (item list)")) != PKV_OK)
            return st;
        if ((st = check_launch(launch_compress_list(L, dl, n), "pkv_compress_pages")) != PKV_OK) return st;
        return check_launch(launch_compress_commit_list(L, dl, n), "pkv_compress_pages (commit)");
    }
    for (int base = 0; base < n; base += kCompressItemsPerLaunch) {
        CompressItems items{};
        items.n = std::min(kCompressItemsPerLaunch, n - base);
        for (int i = 0; i < items.n; ++i) {
            CompressItem &it = items.it[i];
            it.b = b[base + i];
            it.h = kv_head[base + i];
            it.j = page[base + i];
            it.rk = rank_k[base + i];
            it.rv = rank_v[base + i];
        }
        if ((st = check_launch(launch_compress(L, items), "pkv_compress_pages")) != PKV_OK) return st;
        if ((st = check_launch(launch_compress_commit(L, items), "pkv_compress_pages (commit)")) != PKV_OK)
            return st;
    }
    return PKV_OK;
}

pkv_status pkv_mixed_decode_attention(const pkv_cache *c, int32_t layer, const void *q,
                                      const int32_t *seq_len, float *out, float *lse, void *ws,
                                      size_t ws_bytes, pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!q || !seq_len || !out) return fail(PKV_E_ARG, "q, seq_len or out is NULL");
    SeqArgs seq{};
    seq.n = c->batch;
    int64_t max_T = 0;
    for (int b = 0; b < c->batch; ++b) {
        if (seq_len[b] < 0 || (int64_t)seq_len[b] > (int64_t)c->max_pages * c->page_size)
            return fail(PKV_E_SHAPE, "seq_len[%d] = %d outside 0..max_pages * P", b, seq_len[b]);
        seq.len[b] = seq_len[b];
        max_T = std::max<int64_t>(max_T, seq_len[b]);
    }
    LaunchCtx L = ctx(c, layer, s);
    size_t need = (size_t)attention_workspace_bytes(L.geo, max_T);
    if ((st = check_ws(ws, ws_bytes, need)) != PKV_OK) return st;
    AttnPlan plan = attention_plan(L.geo, max_T);
    return check_launch(launch_attention(L, plan, q, seq, out, lse, ws), "pkv_mixed_decode_attention");
}

pkv_status pkv_mixed_decode_attention_noalloc(const pkv_cache *c, int32_t layer, const void *q,
                                              const int32_t *seq_len, float *out, float *lse, pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!q || !seq_len || !out) return fail(PKV_E_ARG, "q, seq_len or out is NULL");
    SeqArgs seq{};
    seq.n = c->batch;
    int64_t max_T = 0;
    for (int b = 0; b < c->batch; ++b) {
        if (seq_len[b] < 0 || (int64_t)seq_len[b] > (int64_t)c->max_pages * c->page_size)
            return fail(PKV_E_SHAPE, "seq_len[%d] = %d outside 0..max_pages * P", b, seq_len[b]);
        seq.len[b] = seq_len[b];
        max_T = std::max<int64_t>(max_T, seq_len[b]);
    }
    LaunchCtx L = ctx(c, layer, s);
    const int64_t heads = (int64_t)c->batch * c->n_kv_heads;
    if (heads > PKV_NOALLOC_MAX_HEADS)
        return fail(PKV_E_WORKSPACE, "batch * n_kv_heads = %lld above the static scratch's %d heads; use "
                    "pkv_mixed_decode_attention with a workspace", (long long)heads, PKV_NOALLOC_MAX_HEADS);
    const int64_t need = attention_state_bytes(L.geo, max_T);
    if (need > scratch_state_bytes())
        return fail(PKV_E_WORKSPACE, "partial states of %lld bytes above the static scratch's %lld; use "
                    "pkv_mixed_decode_attention with a workspace", (long long)need, (long long)scratch_state_bytes());
    AttnPlan plan = attention_plan(L.geo, max_T);
    return check_launch(launch_attention_noalloc(L, plan, q, seq, out, lse), "pkv_mixed_decode_attention_noalloc");
}

// ---- import / export ---------------------------------------------------------

pkv_status pkv_import_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                            const int32_t *kv_head, const int32_t *page, const uint8_t *kind,
                            const uint8_t *rank_k, const uint8_t *rank_v, const void *src,
                            const int64_t *src_offset, void *ws, size_t ws_bytes, pkv_stream s) {
    (void)ws; (void)ws_bytes;
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (n < 0) return fail(PKV_E_ARG, "n < 0");
    if (n == 0) return PKV_OK;
    if (!b || !kv_head || !page || !kind || !rank_k || !rank_v || !src || !src_offset)
        return fail(PKV_E_ARG, "NULL argument");
    const int rmax = std::min(c->max_rank, std::min(c->page_size, c->head_dim));
    LaunchCtx L = ctx(c, layer, s);
    // two dense pages of one head on one ring slot in this call: the kernels
    // of one launch cannot see each other's entries, so this is checked here
    {
        std::vector<int64_t> slots;
        for (int x = 0; x < n; ++x) {
            if (kind[x] != PKV_DENSE || b[x] < 0 || b[x] >= c->batch || kv_head[x] < 0 ||
                kv_head[x] >= c->n_kv_heads || page[x] < 0 || page[x] >= c->max_pages)
                continue;   // reported below
            slots.push_back(L.geo.head_index(b[x], kv_head[x]) * L.geo.dslots + L.geo.dense_ring_slot(page[x]));
        }
        std::sort(slots.begin(), slots.end());
        if (std::adjacent_find(slots.begin(), slots.end()) != slots.end())
            return fail(PKV_E_ARG, "two dense pages of one head map to the same dense slot in one import");
    }
    for (int base = 0; base < n; base += kCopyItemsPerLaunch) {
        CopyItems items{};
        items.n = std::min(kCopyItemsPerLaunch, n - base);
        for (int i = 0; i < items.n; ++i) {
            int x = base + i;
            if (b[x] < 0 || b[x] >= c->batch || kv_head[x] < 0 || kv_head[x] >= c->n_kv_heads ||
                page[x] < 0 || page[x] >= c->max_pages)
                return fail(PKV_E_ARG, "page ref %d out of range", x);
            if (kind[x] != PKV_DENSE && kind[x] != PKV_FACTOR)
                return fail(PKV_E_ARG, "page ref %d: kind %d", x, kind[x]);
            if (kind[x] == PKV_FACTOR &&
                (rank_k[x] < 1 || rank_v[x] < 1 || rank_k[x] > rmax || rank_v[x] > rmax))
                return fail(PKV_E_RANK, "page ref %d: ranks (%d, %d) outside 1..%d", x, rank_k[x], rank_v[x], rmax);
            if (src_offset[x] < 0) return fail(PKV_E_ARG, "page ref %d: negative offset", x);
            CopyItem &it = items.it[i];
            it.b = b[x];
            it.h = kv_head[x];
            it.j = page[x];
            it.kind = kind[x];
            it.rk = kind[x] == PKV_FACTOR ? rank_k[x] : 0;
            it.rv = kind[x] == PKV_FACTOR ? rank_v[x] : 0;
            it.src_off = src_offset[x];
        }
        if ((st = check_launch(launch_import(L, items, src), "pkv_import_pages")) != PKV_OK) return st;
    }
    return PKV_OK;
}

pkv_status pkv_export_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                            const int32_t *kv_head, const int32_t *page, float *dst, void *ws,
                            size_t ws_bytes, pkv_stream s) {
    (void)ws; (void)ws_bytes;
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (n < 0) return fail(PKV_E_ARG, "n < 0");
    if (n == 0) return PKV_OK;
    if (!b || !kv_head || !page || !dst) return fail(PKV_E_ARG, "NULL argument");
    LaunchCtx L = ctx(c, layer, s);
    int64_t block = pkv_export_block_elems(c);
    for (int base = 0; base < n; base += kCopyItemsPerLaunch) {
        CopyItems items{};
        items.n = std::min(kCopyItemsPerLaunch, n - base);
        for (int i = 0; i < items.n; ++i) {
            int x = base + i;
            if (b[x] < 0 || b[x] >= c->batch || kv_head[x] < 0 || kv_head[x] >= c->n_kv_heads ||
                page[x] < 0 || page[x] >= c->max_pages)
                return fail(PKV_E_ARG, "page ref %d out of range", x);
            CopyItem &it = items.it[i];
            it.b = b[x];
            it.h = kv_head[x];
            it.j = page[x];
            it.src_off = (int64_t)x * block;
        }
        if ((st = check_launch(launch_export(L, items, dst, block), "pkv_export_pages")) != PKV_OK) return st;
    }
    return PKV_OK;
}

pkv_status pkv_export_int4_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                                 const int32_t *kv_head, const int32_t *page, void *dst, pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if (c->factor_dtype != PKV_INT4) return fail(PKV_E_ARG, "the cache's factor dtype is not PKV_INT4");
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (n < 0) return fail(PKV_E_ARG, "n < 0");
    if (n == 0) return PKV_OK;
    if (!b || !kv_head || !page || !dst) return fail(PKV_E_ARG, "NULL argument");
    LaunchCtx L = ctx(c, layer, s);
    const int64_t block = int4_blob_bytes(c->page_size, c->head_dim, c->max_rank, c->max_rank);
    for (int base = 0; base < n; base += kCopyItemsPerLaunch) {
        CopyItems items{};
        items.n = std::min(kCopyItemsPerLaunch, n - base);
        for (int i = 0; i < items.n; ++i) {
            int x = base + i;
            if (b[x] < 0 || b[x] >= c->batch || kv_head[x] < 0 || kv_head[x] >= c->n_kv_heads ||
                page[x] < 0 || page[x] >= c->max_pages)
                return fail(PKV_E_ARG, "page ref %d out of range", x);
            CopyItem &it = items.it[i];
            it.b = b[x];
            it.h = kv_head[x];
            it.j = page[x];
            it.src_off = (int64_t)x * block;
        }
        if ((st = check_launch(launch_export_int4(L, items, (char *)dst, block), "pkv_export_int4_pages")) !=
            PKV_OK)
            return st;
    }
    return PKV_OK;
}

// ---- Global SVD baseline ------------------------------------------------------

namespace {

pkv_status check_global(const pkv_cache *c, const pkv_global *gl, bool need_buffers) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if (!gl) return fail(PKV_E_ARG, "global descriptor is NULL");
    if (c->dense_dtype != PKV_BF16 || c->head_dim != 128 || (c->page_size != 32 && c->page_size != 64))
        return fail(PKV_E_UNSUPPORTED, "Global SVD needs bf16 dense pages, head_dim 128 and P = 32 or 64");
    if (gl->rank < 1 || gl->rank > 128) return fail(PKV_E_RANK, "global rank %d outside 1..128", gl->rank);
    if (gl->max_tokens <= 0 || gl->max_tokens % 32)
        return fail(PKV_E_SHAPE, "max_tokens %d: must be a positive multiple of 32", gl->max_tokens);
    if (need_buffers && (!gl->basis || !gl->coef)) return fail(PKV_E_ARG, "basis or coef is NULL");
    return PKV_OK;
}

GlobalGeo global_geo(const pkv_global *gl) {
    GlobalGeo gg;
    gg.r = gl->rank;
    gg.r8 = (gl->rank + 7) & ~7;
    gg.max_tokens = gl->max_tokens;
    return gg;
}

int64_t region_rows(const Geo &g, int64_t T) {
    const int64_t t0 = (int64_t)g.sink_pages * g.P;
    const int64_t t1 = T - g.W >= 0 ? (T - g.W) / g.P * g.P : 0;
    return std::max<int64_t>(0, t1 - t0);
}

pkv_status global_seq(const pkv_cache *c, const pkv_global *gl, const int32_t *seq_len, int64_t src_cap, SeqArgs &seq,
                      int64_t &max_T) {
    if (!seq_len) return fail(PKV_E_ARG, "seq_len is NULL");
    const Geo g = make_geo(c);
    seq = SeqArgs{};
    seq.n = c->batch;
    max_T = 0;
    for (int b = 0; b < c->batch; ++b) {
        if (seq_len[b] < 0 || seq_len[b] > src_cap || (int64_t)seq_len[b] > (int64_t)c->max_pages * c->page_size)
            return fail(PKV_E_SHAPE, "seq_len[%d] = %d outside 0..max_pages * P (and the source)", b, seq_len[b]);
        if (region_rows(g, seq_len[b]) > gl->max_tokens)
            return fail(PKV_E_SHAPE, "sequence %d: %lld region rows above max_tokens %d", b,
                        (long long)region_rows(g, seq_len[b]), gl->max_tokens);
        seq.len[b] = seq_len[b];
        max_T = std::max<int64_t>(max_T, seq_len[b]);
    }
    return PKV_OK;
}

}  // namespace

size_t pkv_global_basis_bytes(const pkv_cache *c, const pkv_global *gl) {
    if (check_global(c, gl, false) != PKV_OK) return 0;
    const GlobalGeo gg = global_geo(gl);
    return (size_t)c->n_layers * c->batch * c->n_kv_heads * 3 * gg.r8 * c->head_dim * 2;
}

size_t pkv_global_coef_bytes(const pkv_cache *c, const pkv_global *gl) {
    if (check_global(c, gl, false) != PKV_OK) return 0;
    const GlobalGeo gg = global_geo(gl);
    return (size_t)c->n_layers * c->batch * c->n_kv_heads * 2 * gg.r8 * (int64_t)gg.max_tokens * 2;
}

int32_t pkv_global_rank(int64_t T, int32_t P, int32_t S, int32_t W, int32_t d, double rho) {
    if (T < 0 || P <= 0 || S < 0 || W < 0 || d <= 0 || !(rho > 0.0)) return -1;
    int64_t n_dense = 0, n_fact = 0;
    for (int64_t j = 0; j * P < T; ++j) {
        const int64_t rows = std::min<int64_t>(P, T - j * P);
        if (plan_kind(T, P, S, W, j) == PKV_FACTOR) n_fact += rows;
        else n_dense += rows;
    }
    const double budget = rho * 2.0 * (double)T * d;
    int32_t best = 0;
    for (int64_t r = 1; r <= std::min<int64_t>(n_fact, d); ++r)
        if (2.0 * n_dense * d + 2.0 * r * (n_fact + d) <= budget) best = (int32_t)r;
    return best;
}

pkv_status pkv_global_prefill(const pkv_cache *c, const pkv_global *gl, int32_t layer, const void *k, const void *v,
                              int64_t src_tokens, const int32_t *seq_len, void *ws, size_t ws_bytes, pkv_stream s) {
    pkv_status st = check_global(c, gl, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!k || !v) return fail(PKV_E_ARG, "k or v is NULL");
    SeqArgs seq;
    int64_t max_T = 0;
    if ((st = global_seq(c, gl, seq_len, src_tokens, seq, max_T)) != PKV_OK) return st;
    LaunchCtx L = ctx(c, layer, s);
    const size_t need = (size_t)global_prefill_workspace_bytes(L.geo, max_T);
    if ((st = check_ws(ws, ws_bytes, need)) != PKV_OK) return st;
    hipError_t e = launch_prefill_pages(L, k, v, src_tokens, seq, nullptr, nullptr, 1, 1, c->max_pages, gl->rank);
    if ((st = check_launch(e, "pkv_global_prefill (pages)")) != PKV_OK) return st;
    return check_launch(launch_global_prefill(L, global_geo(gl), gl, k, v, src_tokens, seq, max_T, ws),
                        "pkv_global_prefill");
}

pkv_status pkv_global_attention(const pkv_cache *c, const pkv_global *gl, int32_t layer, const void *q,
                                const int32_t *seq_len, float *out, float *lse, void *ws, size_t ws_bytes,
                                pkv_stream s) {
    pkv_status st = check_global(c, gl, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (!q || !out) return fail(PKV_E_ARG, "q or out is NULL");
    SeqArgs seq;
    int64_t max_T = 0;
    if ((st = global_seq(c, gl, seq_len, INT64_MAX, seq, max_T)) != PKV_OK) return st;
    LaunchCtx L = ctx(c, layer, s);
    const size_t need = (size_t)global_attention_workspace_bytes(L.geo, max_T);
    if ((st = check_ws(ws, ws_bytes, need)) != PKV_OK) return st;
    return check_launch(launch_global_attention(L, global_geo(gl), gl, q, seq, max_T, out, lse, ws),
                        "pkv_global_attention");
}

pkv_status pkv_global_export(const pkv_cache *c, const pkv_global *gl, int32_t layer, int32_t b, int32_t h,
                             int64_t n_rows, float *basis_k, float *basis_v, float *coef_k, float *coef_v,
                             pkv_stream s) {
    pkv_status st = check_global(c, gl, true);
    if (st != PKV_OK) return st;
    if ((st = check_layer(c, layer)) != PKV_OK) return st;
    if (b < 0 || b >= c->batch || h < 0 || h >= c->n_kv_heads) return fail(PKV_E_ARG, "head (%d, %d) out of range", b, h);
    if (n_rows < 0 || n_rows > gl->max_tokens) return fail(PKV_E_ARG, "n_rows %lld outside 0..max_tokens", (long long)n_rows);
    if (!basis_k || !basis_v || (n_rows > 0 && (!coef_k || !coef_v))) return fail(PKV_E_ARG, "NULL output");
    LaunchCtx L = ctx(c, layer, s);
    return check_launch(launch_global_export(L, global_geo(gl), gl, b, h, n_rows, basis_k, basis_v, coef_k, coef_v),
                        "pkv_global_export");
}

pkv_status pkv_compress_sweeps(pkv_stream s, uint64_t *sweeps) {
    if (!sweeps) return fail(PKV_E_ARG, "sweeps is NULL");
    hipError_t e = hipStreamSynchronize((hipStream_t)s);
    if (e != hipSuccess) return hip_fail(e, "pkv_compress_sweeps (sync)");
    unsigned long long v = 0;
    e = sweeps_read_clear(&v);
    if (e != hipSuccess) return hip_fail(e, "pkv_compress_sweeps (read)");
    *sweeps = (uint64_t)v;
    return PKV_OK;
}

pkv_status pkv_cache_bytes(const pkv_cache *c, int32_t layer, const int32_t *seq_len, pkv_footprint *out,
                           pkv_stream s) {
    pkv_status st = check_cache(c, true);
    if (st != PKV_OK) return st;
    if (!seq_len || !out) return fail(PKV_E_ARG, "seq_len and out must not be NULL");
    if (layer >= c->n_layers) return fail(PKV_E_ARG, "layer %d outside 0..%d", layer, c->n_layers - 1);
    const Geo g = make_geo(c);
    for (int b = 0; b < g.B; ++b)
        if (seq_len[b] < 0 || (int64_t)seq_len[b] > (int64_t)g.max_pages * g.P)
            return fail(PKV_E_SHAPE, "seq_len[%d] = %d outside 0..max_pages * P", b, seq_len[b]);
    const int64_t P = g.P, d = g.d, ed = g.dense_es;
    const bool kt = g.key_t != 0;
    // logical bytes of a factor page pair at ranks (rk, rv)
    auto logical = [&](int64_t rk, int64_t rv) -> int64_t {
        if (g.factor_dtype == PKV_INT4) {
            auto runs = [](int64_t n) { return (n + 31) / 32; };
            const int64_t scales = rk * runs(P) + d * runs(rk) + P * runs(rv) + d * runs(rv);
            return (rk + rv) * (P + d) / 2 + 2 * scales;
        }
        return (rk + rv) * (P + d) * g.factor_es;
    };
    pkv_footprint f{};
    std::vector<pkv_page> tab((size_t)g.layer_entries);
    const int l0 = layer < 0 ? 0 : layer, l1 = layer < 0 ? c->n_layers : layer + 1;
    for (int l = l0; l < l1; ++l) {
        hipError_t e = hipMemcpyAsync(tab.data(), c->page_table + (int64_t)l * g.layer_entries,
                                      sizeof(pkv_page) * (size_t)g.layer_entries, hipMemcpyDeviceToHost,
                                      (hipStream_t)s);
        if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)s);
        if (e != hipSuccess) return hip_fail(e, "pkv_cache_bytes (page table copy)");
        for (int b = 0; b < g.B; ++b) {
            const int64_t T = seq_len[b];
            for (int h = 0; h < g.Hkv; ++h) {
                f.raw_bytes += 2 * T * d * ed;
                const pkv_page *row = tab.data() + g.head_index(b, h) * g.max_pages;
                for (int64_t j = 0; j * P < T; ++j) {
                    const pkv_page ent = row[j];
                    if (ent.kind == PKV_DENSE) {
                        ++f.dense_pages;
                        f.dense_bytes += 2 * std::min<int64_t>(P, T - j * P) * d * ed;
                    } else if (ent.kind == PKV_FACTOR) {
                        ++f.factor_pages;
                        f.factor_bytes += logical(ent.rank_k, ent.rank_v);
                        f.factor_slot_bytes +=
                            factor_page_bytes_of(g.factor_dtype, (int)P, (int)d, ent.rank_k, ent.rank_v, kt);
                    } else {
                        return fail(PKV_E_STATE, "layer %d, sequence %d, KV head %d: page %lld holds tokens but is "
                                    "empty", l, b, h, (long long)j);
                    }
                }
            }
        }
    }
    *out = f;
    return PKV_OK;
}

pkv_status pkv_bandwidth_probe(const void *src, void *dst, int64_t bytes, int32_t mode, int32_t reps,
                               int32_t blocks, int32_t threads, double *gbps, pkv_stream s) {
    if (!src || !dst || !gbps) return fail(PKV_E_ARG, "src, dst or gbps is NULL");
    if (bytes <= 0 || bytes % 16 || ((uintptr_t)src | (uintptr_t)dst) % 16)
        return fail(PKV_E_ARG, "bytes must be a positive multiple of 16 and the buffers 16-byte aligned");
    if (mode < 0 || mode > 3 || reps < 1 || blocks < 1 || blocks > (1 << 20) || threads < 64 || threads > 512 ||
        threads % 64)
        return fail(PKV_E_ARG, "mode %d, reps %d, blocks %d or threads %d out of range", mode, reps, blocks, threads);
    hipError_t e = bandwidth_probe(src, dst, bytes, mode, reps, blocks, threads, gbps, (hipStream_t)s);
    if (e != hipSuccess) return hip_fail(e, "pkv_bandwidth_probe");
    return PKV_OK;
}

pkv_status pkv_device_status(pkv_stream s, uint32_t *bits) {
    if (!bits) return fail(PKV_E_ARG, "bits is NULL");
    hipError_t e = hipStreamSynchronize((hipStream_t)s);
    if (e != hipSuccess) return hip_fail(e, "pkv_device_status (sync)");
    unsigned int v = 0;
    e = status_read_clear(&v);
    if (e != hipSuccess) return hip_fail(e, "pkv_device_status (read)");
    *bits = v;
    return PKV_OK;
}

}  // extern "C"
