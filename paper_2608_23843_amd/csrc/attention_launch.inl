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
    return p;
}

int64_t attention_workspace_bytes(const Geo &g, int64_t max_T) {
    const AttnPlan p = attention_plan(g, max_T);
    return partials_bytes((int64_t)g.B * g.Hkv, p.n_chunks, g.g, g.d);
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

}  // namespace pkv
