/*
 * puzzlekv.h -- C ABI of the PuzzleKV hot path on MI355X (gfx950).
 *
 * PuzzleKV keeps every token of a KV cache: each (layer, KV head) is cut into
 * pages of P tokens; a sink page and a local window stay dense, every other
 * completed page is stored as an independent rank-r factor pair
 * K_p ~ L_K R_K, V_p ~ L_V R_V (Section 3.3, Eq. (2)). Decode attention reads
 * the mixed cache directly (Eq. (4), Eq. (5)); pages that leave the window are
 * factorized during decoding (Section 3.3, "Incremental Cache Update").
 *
 * Conventions for every call:
 *   - Ownership: the caller allocates and frees every buffer (pools, page
 *     table, queries, outputs, workspace). The library allocates no device
 *     memory. Pointers marked "device" are HIP device pointers, "host" are
 *     ordinary host pointers; host arrays may be reused once the call returns.
 *   - Streams: work is enqueued on the given stream (a hipStream_t; NULL is the
 *     null stream) with no implicit synchronization, except where noted.
 *   - Errors: every call returns a pkv_status. Argument and state errors that
 *     the host can see are reported before anything is enqueued;
 *     pkv_last_error() then holds a message (thread-local). Errors only the
 *     device can see (for example, compressing a page that is not dense) set a
 *     sticky per-device status word, read and cleared by pkv_device_status().
 *   - Page-table entries, page kinds and eligible-page lists are integers and
 *     are deterministic.
 *   - Nothing here falls back to a CPU implementation.
 */
#ifndef PUZZLEKV_H
#define PUZZLEKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *pkv_stream; /* hipStream_t */

typedef enum {
    PKV_OK = 0,
    PKV_E_ARG = 1,         /* null pointer, bad enum value, negative count */
    PKV_E_SHAPE = 2,       /* geometry inconsistent or out of the supported range */
    PKV_E_RANK = 3,        /* rank 0 or above min(P, d, max_rank) */
    PKV_E_STATE = 4,       /* page not in a state that allows the operation */
    PKV_E_WORKSPACE = 5,   /* workspace pointer null or smaller than required */
    PKV_E_UNSUPPORTED = 6, /* valid request that this build does not implement */
    PKV_E_HIP = 7          /* HIP runtime error; pkv_last_error() has its text */
} pkv_status;

/* Element types. PKV_INT4 is a factor storage type only (see below). */
typedef enum { PKV_F32 = 0, PKV_BF16 = 1, PKV_INT4 = 2 } pkv_dtype;

/* Kind of a logical page. PKV_GLOBAL: the page's tokens are rows of the
 * head's Global SVD coefficients (pkv_global_prefill). */
typedef enum { PKV_EMPTY = 0, PKV_DENSE = 1, PKV_FACTOR = 2, PKV_GLOBAL = 3 } pkv_kind;

/* Device status bits (pkv_device_status). */
#define PKV_DEV_NOT_DENSE     0x1u /* compress_pages found a page that is not dense   */
#define PKV_DEV_BAD_PAGE      0x2u /* attention met an empty page below the length,   */
                                   /* or more dense pages per head than dense slots  */
#define PKV_DEV_RING_OVERRUN  0x4u /* append or import would overwrite a page still  */
                                   /* dense (two dense pages on one ring slot)       */
#define PKV_DEV_NO_CONVERGE   0x8u /* a decomposition hit the sweep cap (result kept)  */
#define PKV_DEV_BAD_RANK      0x10u /* prefill met a rank outside 1..max_rank (clamped) */
#define PKV_DEV_NOT_ELIGIBLE  0x20u /* compress_pages found a dense page that is       */
                                    /* incomplete or still inside the window           */

/*
 * Page-table entry, 8 bytes. slot is relative to the layer:
 *   DENSE : index into the layer's dense slots
 *           ((b * n_kv_heads + h) * dense_slots_per_head + ring position)
 *   FACTOR: index into the layer's factor slots ((b * n_kv_heads + h) * max_pages + j)
 * The page table is laid out [n_layers][batch][n_kv_heads][max_pages].
 */
typedef struct {
    int32_t slot;
    uint8_t kind;   /* pkv_kind */
    uint8_t rank_k; /* factor pages: r_K, else 0 */
    uint8_t rank_v; /* factor pages: r_V, else 0 */
    uint8_t rows;   /* dense pages: tokens written (1..P; P for imported pages), else 0 */
} pkv_page;

/*
 * Cache descriptor. Geometry plus three caller-owned device buffers whose
 * sizes come from pkv_dense_pool_bytes / pkv_factor_pool_bytes /
 * pkv_page_table_bytes.
 *
 * Dense pool: [n_layers][batch][n_kv_heads][dense_slots_per_head] slots of
 * pkv_dense_slot_bytes. A slot holds K as P x d row-major, then V transposed
 * (d x P row-major), both in dense_dtype. The first ceil(sink/P) slots of a
 * head hold the sink pages; the rest form a ring of ceil(window/P) + 2 slots
 * in which page j sits at position (j - sink_pages) mod ring length.
 *
 * Factor pool: [n_layers][batch][n_kv_heads][max_pages] slots of
 * pkv_factor_slot_bytes (sized for max_rank). With e the factor element size
 * and r4(x) = x rounded up to a multiple of 4, a slot holding ranks (rk, rv)
 * stores, packed from its start:
 *   A_K  = L_K          P  x r4(rk) row-major (columns >= rk are zero)
 *   B_K  = R_K          rk x d      row-major
 *   B_Vt = R_V^T        d  x r4(rv) row-major (columns >= rv are zero)
 *   A_Vt = L_V^T        rv x P      row-major
 * for e * (P r4(rk) + rk d + rv P + d r4(rv)) bytes (pkv_factor_page_bytes).
 * A cache of pre-RoPE keys (key_rope_base > 0) stores B_Kt = R_K^T,
 * d x r4(rk) row-major (columns >= rk zero), in place of B_K, for
 * e * (P r4(rk) + d r4(rk) + rv P + d r4(rv)) bytes.
 * Every operand is stored with its contraction index contiguous, the order
 * the attention kernel streams it in.
 *
 * INT4 factors (factor_dtype PKV_INT4; Section 4.3 "Quantization
 * Compatibility"): a factor page stores the balanced factors
 * L~ = U Sigma^(1/2) and R~ = Sigma^(1/2) W^T of K and V, each quantized to
 * symmetric 4-bit codes in [-7, 7] with one fp16 scale per run of up to 32
 * consecutive elements along the paper's direction: column-wise for L~_K,
 * R~_K and R~_V, row-wise for L~_V. Scale = fp16(max|x| / 7) rounded to
 * nearest even; code = x / scale rounded half to even (exactly, as in fp64);
 * a zero scale gives zero codes. Needs bf16 dense pages, P = 64,
 * head_dim = 128 and max_rank <= 32; the slot layout is internal (codes
 * packed eight to a 32-bit word in the order the attention kernel reads
 * them), pkv_factor_page_bytes gives its size (5,344 bytes at ranks 24/24).
 * Pages enter and leave in the canonical blob of pkv_int4_blob_bytes.
 */
typedef struct {
    int32_t n_layers;
    int32_t batch;
    int32_t n_kv_heads;
    int32_t n_q_heads;     /* multiple of n_kv_heads; query head i reads KV head i / g */
    int32_t head_dim;      /* d: multiple of 32, <= 256 */
    int32_t page_size;     /* P: 16, 32 or 64 */
    int32_t max_pages;     /* logical pages per (layer, b, kv head) */
    int32_t max_rank;      /* 1 .. min(P, d) */
    int32_t sink_tokens;   /* S >= 0 */
    int32_t window_tokens; /* W >= 0 */
    int32_t dense_dtype;   /* PKV_F32 or PKV_BF16 (also the query dtype) */
    int32_t factor_dtype;  /* PKV_F32, PKV_BF16 or PKV_INT4 */
    void *dense_pool;      /* device */
    void *factor_pool;     /* device */
    pkv_page *page_table;  /* device */
    /* Adaptive page ranks: 0 (off) or eps in (0, 1). When set, a rank request
     * of 0 (a page's entry in pkv_prefill's rank tables, its default ranks, or
     * pkv_compress_pages' rank arrays) asks the decomposition for the smallest
     * r with |X - X_r|_F <= eps |X|_F, X the stored page, capped at
     * min(P, d, max_rank): the rank a page needs for a reconstruction accuracy
     * of 1 - eps (the criterion behind the paper's Figure 2; 80% is
     * eps = 0.2). K and V choose independently; the chosen ranks are written
     * to the page table. Needs bf16 dense pages with P = 32 or 64. */
    float adaptive_rank_error;
    /* Keys stored before RoPE: 0 (off: keys are used as stored, the usual
     * post-RoPE cache) or the RoPE base. When set, every cached key (k rows
     * given to pkv_prefill and pkv_append_kv, dense pages, and the pages
     * pkv_compress_pages factorizes) is the pre-RoPE key, and attention
     * rotates key t of a sequence to position t before its score, with the
     * rotate-half pairing: dims i < d/2 and i + d/2 form a pair rotated by
     * t * base^(-2i/d). Queries are given already rotated. The paper
     * factorizes post-RoPE keys and compares factorizing pre-RoPE keys with
     * RoPE applied at cache access (Section 4.2 "Main Results"; Appendix
     * "RoPE Key Analysis"). Factor slots then hold R_K transposed (B_Kt
     * above). Needs bf16 dense pages and factors, P = 32 or 64, head_dim =
     * 64 or 128, max_rank <= 32 and positions below 2^24. The score product
     * takes the rotated keys as fp16 hi/lo pairs (about 22 bits) and the
     * queries in fp16, so query and rotated-key entries must stay below
     * 65504 in magnitude; query entries below fp16's normal range (2^-14)
     * keep an absolute error under 2^-25. */
    float key_rope_base;
} pkv_cache;

/* ---- geometry and sizing (host only, no device work) -------------------- */

/* Checks the descriptor's geometry and pointers. */
pkv_status pkv_cache_check(const pkv_cache *c);
int64_t pkv_dense_slots_per_head(const pkv_cache *c);
size_t pkv_dense_slot_bytes(const pkv_cache *c);
size_t pkv_factor_slot_bytes(const pkv_cache *c);
size_t pkv_dense_pool_bytes(const pkv_cache *c);
size_t pkv_factor_pool_bytes(const pkv_cache *c);
size_t pkv_page_table_bytes(const pkv_cache *c);
/* Bytes of one factor page pair at ranks (rk, rv): what attention reads for it. */
size_t pkv_factor_page_bytes(const pkv_cache *c, int32_t rank_k, int32_t rank_v);

/* Workspace sizes. op PKV_OP_ATTENTION: n = longest sequence length passed to
 * pkv_mixed_decode_attention (a workspace sized for n serves every call with
 * sequences up to n tokens); PKV_OP_COMPRESS: n = pages per call;
 * PKV_OP_PREFILL: n = longest prompt length; PKV_OP_GLOBAL_PREFILL and
 * PKV_OP_GLOBAL_ATTENTION: n = longest sequence of pkv_global_prefill and
 * pkv_global_attention. */
enum { PKV_OP_ATTENTION = 0, PKV_OP_COMPRESS = 1, PKV_OP_PREFILL = 2, PKV_OP_IMPORT = 3,
       PKV_OP_GLOBAL_PREFILL = 4, PKV_OP_GLOBAL_ATTENTION = 5 };
size_t pkv_workspace_bytes(const pkv_cache *c, int32_t op, int64_t n);

/* ---- page plan (host, integer; Section 3.3 and Section 4.1) ---------------
 * Page j of a sequence of T tokens is FACTOR iff it is complete
 * ((j+1) P <= T), outside the sink (j >= ceil(S / P)) and entirely older than
 * the W-token window ((j+1) P <= T - W); pages holding a token but not
 * factorized are DENSE; pages past the last token are EMPTY. With S = W = P
 * this is the paper's default dense region: one sink page, the most recently
 * completed page and the current incomplete page.
 * pkv_plan_pages writes kind[0..n) and the page count ceil(T/P) to *n_pages.
 * pkv_eligible_pages lists, ascending, the pages FACTOR at T_new but not at
 * T_prev (at most cap of them; *count gets the full number). */
pkv_status pkv_plan_pages(int64_t T, int32_t P, int32_t S, int32_t W, uint8_t *kind /*host*/,
                          int64_t n, int64_t *n_pages);
pkv_status pkv_eligible_pages(int64_t T_prev, int64_t T_new, int32_t P, int32_t S, int32_t W,
                              int32_t *pages /*host*/, int64_t cap, int64_t *count);

/* ---- cache construction and maintenance --------------------------------- */

/* Marks every page of `layer` (all layers if layer < 0) EMPTY. */
pkv_status pkv_cache_reset(const pkv_cache *c, int32_t layer, pkv_stream s);

/* Builds one layer from the dense prompt cache (Section 3.3, steps 1-3 of the
 * workflow: pages, dense sink/window, every other completed page factorized).
 * k, v: device [batch][n_kv_heads][src_tokens][d] in dense_dtype.
 * seq_len: host [batch], 0 <= seq_len[b] <= min(src_tokens, max_pages * P).
 * rank_k, rank_v: device [batch][n_kv_heads][max_pages] ranks of factor pages,
 * or NULL to use default_rank_k / default_rank_v for every page; a device rank
 * outside 1..max_rank is clamped and raises PKV_DEV_BAD_RANK. With adaptive
 * ranks enabled (adaptive_rank_error > 0) a rank of 0 is chosen per page.
 * Pages of the plan for seq_len[b] are written: dense pages copied, factor
 * pages decomposed by the same kernel as pkv_compress_pages; pages past the
 * sequence become EMPTY. Workspace: pkv_workspace_bytes(PKV_OP_PREFILL, max T). */
pkv_status pkv_prefill(const pkv_cache *c, int32_t layer, const void *k, const void *v,
                       int64_t src_tokens, const int32_t *seq_len, const uint8_t *rank_k,
                       const uint8_t *rank_v, int32_t default_rank_k, int32_t default_rank_v,
                       void *ws, size_t ws_bytes, pkv_stream s);

/* Appends one token per sequence to `layer` (Section 3.3, "Incremental Cache
 * Update": the new pair joins the most recent dense page).
 * k_new, v_new: device [batch][n_kv_heads][d] in dense_dtype.
 * pos: host [batch], the token index being written (the sequence length before
 * the append); pos[b] < 0 skips sequence b. When pos[b] is a multiple of P a
 * new dense page starts in the ring; if the ring position still holds a dense
 * page the row is not written and PKV_DEV_RING_OVERRUN is raised. */
pkv_status pkv_append_kv(const pkv_cache *c, int32_t layer, const void *k_new, const void *v_new,
                         const int32_t *pos, pkv_stream s);

/* Factorizes n dense pages of `layer` (Section 3.3: Gram matrix G = X X^T,
 * L = its top-r eigenvectors, R = L^T X, which are the rank-r truncated-SVD
 * factors of Eq. (2)); K and V of a page are decomposed independently.
 * b, kv_head, page: host [n]; rank_k, rank_v: host [n], 1 <= r <= min(P, d,
 * max_rank), or 0 for a rank chosen per page when adaptive ranks are enabled
 * (adaptive_rank_error > 0). A page is factorized once, when it has left the
 * window (Section 3.3, "Incremental Cache Update"): it must be DENSE and
 * complete (P rows written), outside the sink, and the cache must hold at
 * least window_tokens tokens after it. The entry then becomes FACTOR with its
 * ranks and its dense slot is free for reuse. A sink page is refused on the
 * host (PKV_E_STATE, nothing enqueued). Other refusals are seen on the device:
 * the page is left untouched and PKV_DEV_NOT_DENSE (already factorized or
 * empty) or PKV_DEV_NOT_ELIGIBLE (incomplete, or still inside the window) is
 * raised. Duplicate pages in one call are rejected (PKV_E_ARG).
 * Workspace: optional. With ws (device) of at least
 * pkv_workspace_bytes(PKV_OP_COMPRESS, n) bytes, the page list is copied
 * there (an asynchronous host-to-device copy on s) and all n pages are
 * factorized in one launch; calls that share a workspace must be ordered
 * (one stream). With ws NULL or smaller, the pages go in launches of 96. */
pkv_status pkv_compress_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                              const int32_t *kv_head, const int32_t *page, const uint8_t *rank_k,
                              const uint8_t *rank_v, void *ws, size_t ws_bytes, pkv_stream s);

/* Single-query grouped-query decode attention over the mixed cache of `layer`
 * (Eq. (4) per factor page, the same state from K and V on dense pages,
 * merged by Eq. (5)); factor pages are never rebuilt into K or V.
 * q: device [batch][n_q_heads][d] in dense_dtype. seq_len: host [batch], the
 * tokens each sequence attends to (1 <= seq_len[b] <= max_pages * P; 0 gives
 * out = 0 and lse = -inf). out: device fp32 [batch][n_q_heads][d], normalized.
 * lse: device fp32 [batch][n_q_heads] log-sum-exp of the scaled scores, or NULL.
 * Softmax scale 1/sqrt(d); query head i uses KV head i / (n_q_heads / n_kv_heads).
 * Workspace: pkv_workspace_bytes(PKV_OP_ATTENTION, max seq_len) bytes. It
 * begins with two counters per (sequence, KV head): 4 * batch * n_kv_heads
 * bytes rounded up to a multiple of 256, then 256 * batch * n_kv_heads bytes;
 * per-chunk partial states follow. The counters must be zero before the first
 * use; every call returns them to zero and writes every partial it reads, so
 * a workspace sized for the longest sequence serves calls of any shorter
 * length. Calls that share a workspace must not overlap. One kernel launch per call. With bf16 storage the pages of a head
 * are handed to the GPU's waves dynamically, so the order of the fp32 sums,
 * and with it the last bits of out and lse, can differ from call to call. */
pkv_status pkv_mixed_decode_attention(const pkv_cache *c, int32_t layer, const void *q,
                                      const int32_t *seq_len, float *out, float *lse, void *ws,
                                      size_t ws_bytes, pkv_stream s);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * attention as pkv_mixed_decode_attention, same arguments and results, with
 * no workspace argument. Its counters and partial states live in a static
 * device array of PKV_NOALLOC_SCRATCH_BYTES bytes that the library holds on
 * each GPU it runs on until the process ends; it calls no allocator. The
 * array keeps the last call's contents: its counter region (laid out for
 * PKV_NOALLOC_MAX_HEADS (sequence, KV head) pairs) is cleared by a kernel on
 * the caller's stream at the first call on a device, and every call returns
 * it to zero. All calls on one GPU share the array, so calls that overlap on
 * one GPU (different streams, or different threads without ordering) race
 * and must not be made. Returns PKV_E_WORKSPACE, before anything is
 * enqueued, when batch * n_kv_heads exceeds PKV_NOALLOC_MAX_HEADS or the
 * call's partial states do not fit beside the counters (then use
 * pkv_mixed_decode_attention with a workspace). */
#define PKV_NOALLOC_SCRATCH_BYTES (16ll << 20)
#define PKV_NOALLOC_MAX_HEADS 2048
pkv_status pkv_mixed_decode_attention_noalloc(const pkv_cache *c, int32_t layer, const void *q,
                                              const int32_t *seq_len, float *out, float *lse, pkv_stream s);

/* ---- import / export of pages in the logical layout ---------------------
 * Logical page block, row-major:
 *   DENSE : K (P x d), V (P x d)
 *   FACTOR: L_K (P x rk), R_K (rk x d), L_V (P x rv), R_V (rv x d)
 * pkv_import_pages writes n pages of `layer`: b, kv_head, page, kind, rank_k,
 * rank_v, src_offset are host [n]; src is a device array in the destination
 * dtype (dense_dtype for dense pages, factor_dtype for factor pages) and page
 * i's block starts src_offset[i] elements into it (for INT4 factor pages the
 * block is the canonical INT4 blob and src_offset[i] counts bytes). The
 * page-table entry is set; a dense page counts as complete (rows = P). A
 * dense page goes to its ring slot: two dense pages of one head on the same
 * slot in one call are rejected (PKV_E_ARG), and a dense page whose slot
 * already holds another dense page of the head is not written and raises
 * PKV_DEV_RING_OVERRUN. Workspace: pkv_workspace_bytes(PKV_OP_IMPORT, n). */
pkv_status pkv_import_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                            const int32_t *kv_head, const int32_t *page, const uint8_t *kind,
                            const uint8_t *rank_k, const uint8_t *rank_v, const void *src,
                            const int64_t *src_offset, void *ws, size_t ws_bytes, pkv_stream s);

/* pkv_export_pages reads n pages of `layer` as fp32 into dst (device), page i
 * at dst + i * pkv_export_block_elems(c): DENSE as K, V (P x d each); FACTOR as
 * L_K (P x max_rank), R_K (max_rank x d), L_V (P x max_rank), R_V (max_rank x d)
 * with entries past the page's ranks zero; EMPTY as zeros. INT4 factor pages
 * come out dequantized (code x scale) as the balanced factors L~, R~. */
int64_t pkv_export_block_elems(const pkv_cache *c);
pkv_status pkv_export_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                            const int32_t *kv_head, const int32_t *page, float *dst, void *ws,
                            size_t ws_bytes, pkv_stream s);

/* Canonical INT4 page blob (import and pkv_export_int4_pages): int8 codes
 * L~_K [P][rk], R~_K [rk][d], L~_V [P][rv], R~_V [rv][d] (row-major), then
 * fp16 scales L~_K [P/32][rk] (run u covers tokens 32u..32u+31 of column a),
 * R~_K [d], L~_V [P], R~_V [d] (one run per line since ranks are <= 32).
 * Returns its size in bytes, or -1 if the cache is not INT4 or the ranks are
 * outside 1..max_rank. For INT4 factor pages pkv_import_pages reads this blob
 * at src + src_offset[i] bytes (dense pages keep element offsets). */
int64_t pkv_int4_blob_bytes(const pkv_cache *c, int32_t rank_k, int32_t rank_v);
/* Writes the blobs of n INT4 factor pages to dst (device), page i at
 * dst + i * pkv_int4_blob_bytes(c, max_rank, max_rank); a page that is not a
 * factor page gives zeros. */
pkv_status pkv_export_int4_pages(const pkv_cache *c, int32_t layer, int32_t n, const int32_t *b,
                                 const int32_t *kv_head, const int32_t *page, void *dst, pkv_stream s);

/* ---- Global SVD baseline ----------------------------------------------------
 * The paper's controlled baseline for compression granularity (Section 4.1
 * "Baselines"; Section 4.2 "Main Results"; Appendix "Baseline
 * Configurations"): for each (layer, sequence, KV head) and each of K and V,
 * one rank-r basis shared by every token of the compressible region, which
 * is the run of pages the plan factorizes; the sink and window pages stay
 * dense exactly as in PuzzleKV. The region X (N x d) is stored as X ~ A B with
 * B = W_r^T (r x d), the top-r right singular vectors of X (eigenvectors of
 * its Gram matrix X^T X), and A = X B^T (N x r), one coefficient row per
 * token (A = U_r Sigma_r). The dense pages and the page table live in a
 * pkv_cache (bf16 dense pages, head_dim 128, P = 32 or 64); the factorized
 * pages' entries get kind PKV_GLOBAL (slot = the coefficient row of the
 * page's first token, rank_k = rank_v = r). The baseline is built from a
 * prompt and attended at that length (append and compress_pages do not apply
 * to it), and pkv_cache_bytes refuses its layers (PKV_E_STATE).
 *
 * Layout, bf16, r8 = r rounded up to a multiple of 8, per (layer, sequence,
 * KV head) in [n_layers][batch][n_kv_heads] order:
 *   basis: B_K (r8 x d), B_V (r8 x d), B_V^T (d x r8), row-major, entries
 *          past rank r zero
 *   coef:  A_K (max_tokens x r8) token-major, then A_V^T as max_tokens / 32
 *          blocks of r8 x 32, one per 32-token unit, each rank-major (A_V^T
 *          entry (a, t) at element (t - t mod 32) r8 + 32 a + t mod 32); row
 *          t of A_K and column t of A_V^T are token t0 + t of the region,
 *          t0 = ceil(S / P) P; entries past rank r zero
 */
typedef struct {
    int32_t rank;        /* r: 1 .. 128 */
    int32_t max_tokens;  /* coefficient rows per (layer, sequence, KV head): a positive multiple of 32 */
    void *basis;         /* device, pkv_global_basis_bytes */
    void *coef;          /* device, pkv_global_coef_bytes */
} pkv_global;
size_t pkv_global_basis_bytes(const pkv_cache *c, const pkv_global *gl);
size_t pkv_global_coef_bytes(const pkv_cache *c, const pkv_global *gl);
/* The rank matched to a storage budget (host, integer): the largest r in
 * 1..min(N, d) with 2 n d + 2 r (N + d) <= rho 2 T d, where a head of T tokens
 * keeps n of them dense (sink and window pages of the plan for T, P, S, W) and
 * N = T - n in the region: the dense tokens count against the budget as the
 * paper's appendix describes; with n = 0 it is the paper's
 * rho_global = r (S + d) / (S d) <= rho. Returns 0 if no rank fits, -1 for an
 * invalid argument. */
int32_t pkv_global_rank(int64_t T, int32_t P, int32_t S, int32_t W, int32_t d, double rho);
/* Builds one layer from the dense prompt cache, as pkv_prefill does for
 * PuzzleKV: dense pages copied, and for each (sequence, KV head) and each of
 * K and V the Gram matrix of the region on the matrix cores, its eigenvectors
 * by one-sided Jacobi (fp32), the basis rounded to bf16 and the coefficients
 * A = X B^T projected with that rounded basis. k, v: device
 * [batch][n_kv_heads][src_tokens][d] bf16; seq_len: host [batch], each at
 * most src_tokens and max_pages * P, with its region at most max_tokens rows.
 * Workspace: pkv_workspace_bytes(PKV_OP_GLOBAL_PREFILL, max seq_len) (fp32
 * Gram partials of 4,096-token chunks). PKV_DEV_NO_CONVERGE if an
 * eigen-solve reaches its sweep cap (result kept). */
pkv_status pkv_global_prefill(const pkv_cache *c, const pkv_global *gl, int32_t layer, const void *k, const void *v,
                              int64_t src_tokens, const int32_t *seq_len, void *ws, size_t ws_bytes, pkv_stream s);
/* Single-query GQA decode attention over a layer built by pkv_global_prefill,
 * at the prefill lengths: per (sequence, KV head) Z = B_K q once, scores from
 * A_K Z, Y = sum_t p_t A_V[t] in the rank space and O = Y B_V, plus the dense
 * pages, merged by Eq. (5); coefficients are never rebuilt into K or V.
 * Arguments, outputs and workspace conventions as pkv_mixed_decode_attention,
 * with pkv_workspace_bytes(PKV_OP_GLOBAL_ATTENTION, max seq_len). A page the
 * plan keeps dense that is not DENSE, or a region whose last page is not
 * PKV_GLOBAL, raises PKV_DEV_BAD_PAGE. */
pkv_status pkv_global_attention(const pkv_cache *c, const pkv_global *gl, int32_t layer, const void *q,
                                const int32_t *seq_len, float *out, float *lse, void *ws, size_t ws_bytes,
                                pkv_stream s);
/* Reads one (sequence b, KV head h)'s factors as fp32 (device outputs):
 * basis_k, basis_v (r x d) and coef_k, coef_v (n_rows x r, rows 0..n_rows-1
 * of the region), n_rows <= max_tokens. */
pkv_status pkv_global_export(const pkv_cache *c, const pkv_global *gl, int32_t layer, int32_t b, int32_t h,
                             int64_t n_rows, float *basis_k, float *basis_v, float *coef_k, float *coef_v,
                             pkv_stream s);

/* ---- accounting ----------------------------------------------------------- */

/* Live KV footprint of one layer (layer >= 0) or of every layer (layer < 0),
 * read from the page table: the logical live cache against the raw,
 * uncompressed one (Section 4.5, "Memory Footprint"; Eq. (3) for a factor
 * page). seq_len: host [batch], the tokens each sequence holds. Sums over
 * the selected layers and every (sequence, KV head):
 *   raw_bytes          K and V of every live token in dense_dtype (2 T d e)
 *   dense_bytes        K and V of the tokens held on dense pages
 *   factor_bytes       factor pages at their ranks, logical: (r_K + r_V)(P + d)
 *                      elements of factor_dtype (Eq. (3)); INT4: half a byte
 *                      per code plus 2 bytes per fp16 scale, one scale per run
 *                      of up to 32 elements along the paper's directions
 *   factor_slot_bytes  what those pages' slots hold, padding included (the
 *                      sum of pkv_factor_page_bytes)
 *   dense_pages, factor_pages
 * (dense_bytes + factor_bytes) / raw_bytes is the footprint ratio the paper
 * reports. The page table is copied to the host on stream s, which is
 * synchronized; no kernel runs. A page inside a sequence that is neither
 * dense nor factorized gives PKV_E_STATE. */
typedef struct {
    int64_t raw_bytes;
    int64_t dense_bytes;
    int64_t factor_bytes;
    int64_t factor_slot_bytes;
    int64_t dense_pages;
    int64_t factor_pages;
} pkv_footprint;
pkv_status pkv_cache_bytes(const pkv_cache *c, int32_t layer, const int32_t *seq_len, pkv_footprint *out,
                           pkv_stream s);

/* ---- diagnostics --------------------------------------------------------- */

/* Bandwidth calibration: the best rate (GB/s, bytes moved per second) of
 * `reps` timed launches (after one untimed) of a plain streaming kernel over
 * `bytes` bytes of src (device, 16-byte aligned, bytes a multiple of 16),
 * with `blocks` workgroups of `threads` (64..512, a multiple of 64) threads,
 * 16-byte loads, four in flight per thread. mode 0: read, one grid-stride
 * sweep; mode 2: read, each workgroup taking contiguous 64 KB chunks (dst
 * receives one 4-byte word per thread in both); modes 1 and 3: copy src to
 * dst with the same two patterns (bytes moved = 2 * bytes). Synchronizes the
 * stream. It states the attention rates against what the chip's HBM gives a
 * simple stream. */
pkv_status pkv_bandwidth_probe(const void *src, void *dst, int64_t bytes, int32_t mode, int32_t reps,
                               int32_t blocks, int32_t threads, double *gbps, pkv_stream s);

/* Synchronizes the stream, then returns (and clears) the current device's
 * sticky status bits (PKV_DEV_*) in *bits. */
pkv_status pkv_device_status(pkv_stream s, uint32_t *bits);
/* Synchronizes the stream, then returns (and clears) the number of Jacobi
 * sweeps that decompositions on the current device have executed since the
 * last call, summed over decompositions (a page's K and V count as two).
 * With the number of decompositions it gives the work a pkv_prefill or
 * pkv_compress_pages call actually executed; the factors do not depend on it. */
pkv_status pkv_compress_sweeps(pkv_stream s, uint64_t *sweeps);
/* Message of the last error on this thread ("" if none). */
const char *pkv_last_error(void);
const char *pkv_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PUZZLEKV_H */
