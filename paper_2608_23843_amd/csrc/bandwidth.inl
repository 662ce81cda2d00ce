// Bandwidth calibration: plain streaming read and copy kernels, used to state
// the attention kernels' rates against what this chip's HBM delivers to a
// simple stream (beside the 8 TB/s of the specification).
// Included by pkv_kernels.hip.

namespace pkv {

constexpr int kChunk16 = 4096;   // 64 KB contiguous per workgroup visit (chunked modes)

// Streaming read of n 16-byte words, four loads in flight per thread. CHUNK:
// workgroup w reads contiguous 64 KB chunks w, w + grid, ...; otherwise one
// grid-stride sweep. Each thread folds what it read into one word so the
// loads are kept.
template <bool CHUNK>
__global__ __launch_bounds__(512) void k_stream_read(const uint4 *__restrict__ src, int64_t n, uint32_t *sink) {
    uint32_t acc = 0u;
    auto fold = [&](const uint4 &a) { acc ^= a.x ^ a.y ^ a.z ^ a.w; };
    if (CHUNK) {
        const int bd = blockDim.x;
        for (int64_t base = (int64_t)blockIdx.x * kChunk16; base < n; base += (int64_t)gridDim.x * kChunk16) {
            const int64_t end = min<int64_t>(n, base + kChunk16);
            int64_t i = base + threadIdx.x;
            for (; i + 3 * bd < end; i += 4 * bd) {
                const uint4 a = src[i], b = src[i + bd], c = src[i + 2 * bd], d = src[i + 3 * bd];
                fold(a); fold(b); fold(c); fold(d);
            }
            for (; i < end; i += bd) fold(src[i]);
        }
    } else {
        const int64_t stride = (int64_t)gridDim.x * blockDim.x;
        int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        for (; i + 3 * stride < n; i += 4 * stride) {
            const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
            fold(a); fold(b); fold(c); fold(d);
        }
        for (; i < n; i += stride) fold(src[i]);
    }
    sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

template <bool CHUNK>
__global__ __launch_bounds__(512) void k_stream_copy(const uint4 *__restrict__ src, uint4 *__restrict__ dst, int64_t n) {
    if (CHUNK) {
        const int bd = blockDim.x;
        for (int64_t base = (int64_t)blockIdx.x * kChunk16; base < n; base += (int64_t)gridDim.x * kChunk16) {
            const int64_t end = min<int64_t>(n, base + kChunk16);
            int64_t i = base + threadIdx.x;
            for (; i + 3 * bd < end; i += 4 * bd) {
                const uint4 a = src[i], b = src[i + bd], c = src[i + 2 * bd], d = src[i + 3 * bd];
                dst[i] = a; dst[i + bd] = b; dst[i + 2 * bd] = c; dst[i + 3 * bd] = d;
            }
            for (; i < end; i += bd) dst[i] = src[i];
        }
    } else {
        const int64_t stride = (int64_t)gridDim.x * blockDim.x;
        int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        for (; i + 3 * stride < n; i += 4 * stride) {
            const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
            dst[i] = a; dst[i + stride] = b; dst[i + 2 * stride] = c; dst[i + 3 * stride] = d;
        }
        for (; i < n; i += stride) dst[i] = src[i];
    }
}

// mode 0 / 2: read `bytes` of src, grid-stride / in 64 KB chunks per
// workgroup (dst receives one word per thread); mode 1 / 3: copy src to dst,
// the same two patterns. Returns the best rate of `reps` launches in GB/s
// (bytes moved: read, or read + written).
hipError_t bandwidth_probe(const void *src, void *dst, int64_t bytes, int mode, int reps, int blocks, int threads,
                           double *gbps, hipStream_t stream) {
    const int64_t n = bytes / 16;
    hipEvent_t e0, e1;
    hipError_t e = hipEventCreate(&e0);
    if (e != hipSuccess) return e;
    e = hipEventCreate(&e1);
    if (e != hipSuccess) {
        (void)hipEventDestroy(e0);   // the creation error is the one reported
        return e;
    }
    double best = 0.0;
    for (int r = 0; r < reps + 1 && e == hipSuccess; ++r) {
        e = hipEventRecord(e0, stream);
        if (e != hipSuccess) break;
        const dim3 grid(blocks), block(threads);
        switch (mode) {
        case 0: hipLaunchKernelGGL(k_stream_read<false>, grid, block, 0, stream, (const uint4 *)src, n, (uint32_t *)dst); break;
        case 1: hipLaunchKernelGGL(k_stream_copy<false>, grid, block, 0, stream, (const uint4 *)src, (uint4 *)dst, n); break;
        case 2: hipLaunchKernelGGL(k_stream_read<true>, grid, block, 0, stream, (const uint4 *)src, n, (uint32_t *)dst); break;
        default: hipLaunchKernelGGL(k_stream_copy<true>, grid, block, 0, stream, (const uint4 *)src, (uint4 *)dst, n); break;
        }
        e = hipGetLastError();
        if (e != hipSuccess) break;
        e = hipEventRecord(e1, stream);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        if (e == hipSuccess && r > 0 && ms > 0.f) {   // the first launch warms up
            const double moved = (double)n * 16.0 * ((mode & 1) ? 2.0 : 1.0);
            best = std::max(best, moved / (ms * 1e-3) / 1e9);
        }
    }
    // a failure to release the events does not change the measurement
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    *gbps = best;
    return e;
}

}  // namespace pkv
