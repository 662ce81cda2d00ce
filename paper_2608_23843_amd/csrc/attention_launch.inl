// Attention planning (kernel choice, pages per chunk) and launch.
// Included by pkv_kernels.hip.

namespace pkv {

// The split kernel keeps one workgroup per (sequence, KV head, chunk of pages).
// Chunks are sized so the grid holds about `target` workgroups: for the
// matrix-core kernel 256 eight-wave workgroups, one per CU (its register
// budget allows two waves per SIMD), each wave streaming many pages; fewer
// chunks also keep the final merge short.
AttnPlan attention_plan(const Geo &g, int64_t max_T) {
    AttnPlan p{};
    const int64_t n_pages = std::max<int64_t>(1, ceil_div(max_T, g.P));
    const int64_t heads = (int64_t)g.B * g.Hkv;
    p.use_mfma = mfma_supported(g) ? 1 : 0;
    const int64_t target = p.use_mfma ? 256 : 1024;
    p.pages_per_chunk = (int)std::max<int64_t>(1, ceil_div(n_pages * heads, target));
    p.n_chunks = (int)ceil_div(n_pages, p.pages_per_chunk);
    // Measured on one MI355X, each choice against the other:
    // - per-wave page claims (no round barrier) for pre-RoPE caches and for
    //   streams of at most two 64-token pages per wave: pre-RoPE 128K layers
    //   248 -> 221 us, a batch-1 32K layer (two pages per wave) 29.2 -> 27.1
    //   us; one GPU's tensor-parallel share of the 128K layers (four pages
    //   per wave) loses (46.3 -> 52.3 us), as do the 128K bf16 layers (32
    //   pages per wave) and 32-token pages (no two-unit dense pages);
    // - pages handed out last to first, except for short streams with
    //   per-wave claims: 128K layers 209.2 -> 204.9 us (adaptive ranks 187.8
    //   -> 182.9, pre-RoPE 223.5 -> 221.7), the tensor-parallel share with
    //   block claims 46.3 -> 42.4 us; the batch-1 32K layer (per-wave claims)
    //   loses (27.9 -> 29.3 us), where the static first round gives the dense
    //   pages to a few waves.
    const bool short_stream = p.pages_per_chunk <= 8 * kMfmaWaves;
    const bool wave_claims = g.key_t || (g.P == 64 && p.pages_per_chunk <= 2 * kMfmaWaves);
    p.sched = (wave_claims ? kSchedWaveClaims : 0) | (short_stream && wave_claims ? 0 : kSchedReverse);
    return p;
}

int64_t attention_workspace_bytes(const Geo &g, int64_t max_T) {
    const AttnPlan p = attention_plan(g, max_T);
    return partials_bytes((int64_t)g.B * g.Hkv, p.n_chunks, g.g, g.d);
}

int64_t attention_state_bytes(const Geo &g, int64_t max_T) {
    const AttnPlan p = attention_plan(g, max_T);
    return partial_state_bytes((int64_t)g.B * g.Hkv, p.n_chunks, g.g, g.d);
}

template <typename TD, typename TF>
static void launch_generic(const LaunchCtx &L, const LayerPtrs &p, const AttnPlan &plan, const void *q,
                           const SeqArgs &seq, const Partials &pp, float *out, float *lse) {
    const Geo &g = L.geo;
    dim3 grid(plan.n_chunks, g.B * g.Hkv);
    hipLaunchKernelGGL((k_attn_generic<TD, TF>), grid, dim3(kGenThreads), 0, L.stream, g, p.table, p.dense,
                       p.factor, (const TD *)q, seq, plan.pages_per_chunk, plan.n_chunks, pp, out, lse);
}

static hipError_t launch_attention_pp(const LaunchCtx &L, const AttnPlan &plan, const void *q, const SeqArgs &seq,
                                      float *out, float *lse, const Partials &pp) {
    LayerPtrs p = layer_ptrs(L);
    const Geo &g = L.geo;
    if (plan.use_mfma) return launch_attn_mfma(L, plan, (const uint16_t *)q, seq, pp, out, lse);
    if (g.key_t) return hipErrorInvalidValue;   // pre-RoPE keys: matrix-core kernel only
    const bool db = g.dense_dtype == PKV_BF16, fb = g.factor_dtype == PKV_BF16;
    if (db && fb) launch_generic<uint16_t, uint16_t>(L, p, plan, q, seq, pp, out, lse);
    else if (db) launch_generic<uint16_t, float>(L, p, plan, q, seq, pp, out, lse);
    else if (fb) launch_generic<float, uint16_t>(L, p, plan, q, seq, pp, out, lse);
    else launch_generic<float, float>(L, p, plan, q, seq, pp, out, lse);
    return hipGetLastError();
}

hipError_t launch_attention(const LaunchCtx &L, const AttnPlan &plan, const void *q, const SeqArgs &seq,
                            float *out, float *lse, void *ws) {
    const Geo &g = L.geo;
    return launch_attention_pp(L, plan, q, seq, out, lse,
                               make_partials(ws, (int64_t)g.B * g.Hkv, plan.n_chunks, g.g, g.d));
}

// ---- attention without a caller workspace -----------------------------------
//
// For callers that cannot allocate (graph capture, serving loops): the
// counters and partial states live in one static device array per GPU. Its
// counter region is laid out for kScratchHeads heads whatever the call's
// geometry, so calls of different batch sizes, head counts and lengths find
// their counters at the same addresses; it is cleared once per device (first
// call on the device, by a kernel on the caller's stream) and every call
// returns the counters it used to zero. The partial states that follow are
// written by each call before they are read. Calls that overlap on one GPU
// race on this memory.
constexpr int64_t kScratchBytes = PKV_NOALLOC_SCRATCH_BYTES;
constexpr int64_t kScratchHeads = PKV_NOALLOC_MAX_HEADS;
constexpr int kScratchDevices = 64;
static_assert(kScratchBytes % 256 == 0, "scratch size");

static __device__ __align__(256) char scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static void *g_scratch_ptr[kScratchDevices];   // device address of `scratch`, per device

__global__ void k_zero_words(unsigned int *p, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

int64_t scratch_state_bytes() { return kScratchBytes - counter_bytes(kScratchHeads); }

// The device address of this GPU's scratch array (set up on first use).
static hipError_t scratch_on_device(hipStream_t stream, char **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        const int64_t words = counter_bytes(kScratchHeads) / 4;
        hipLaunchKernelGGL(k_zero_words, dim3((unsigned)ceil_div(words, 256)), dim3(256), 0, stream,
                           (unsigned int *)p, words);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = (char *)g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_attention_noalloc(const LaunchCtx &L, const AttnPlan &plan, const void *q, const SeqArgs &seq,
                                    float *out, float *lse) {
    const Geo &g = L.geo;
    char *base = nullptr;
    hipError_t e = scratch_on_device(L.stream, &base);
    if (e != hipSuccess) return e;
    const Partials pp = make_partials(base, kScratchHeads, base + counter_bytes(kScratchHeads), (int64_t)g.B * g.Hkv,
                                      plan.n_chunks, g.g, g.d);
    return launch_attention_pp(L, plan, q, seq, out, lse, pp);
}

}  // namespace pkv
