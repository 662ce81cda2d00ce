// Mixed-page decode attention (Eq. (4) for factor pages, the same state from
// K and V for dense pages, Eq. (5) to merge) -- split phase and combine.
//
// Work is split flash-decoding style: each workgroup owns one (sequence, KV
// head) and a contiguous chunk of pages, keeps the running (m, l, O) state
// of the g query heads of that KV head, and writes it as a partial; the
// combine kernel merges the partials of a head with the Eq. (5) rescaling.
// Scores are kept in the base-2 domain (s * log2(e) / sqrt(d)) so every
// exponential is one exp2.
// Included by pkv_kernels.hip.

namespace pkv {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Partials: [B*Hkv][n_chunks][g][d + 2] floats, slot layout {m2, l, O[0..d)}.
__host__ __device__ inline int64_t partial_index(int64_t head, int chunk, int n_chunks, int qi, int g,
                                                 int d) {
    return ((head * n_chunks + chunk) * g + qi) * (int64_t)(d + 2);
}

// ---- combine: Eq. (5) across the chunks of one head, then normalize -----------
//
// Fused into the split kernels: every workgroup publishes its partial, then
// bumps the head's counter; the workgroup that brings it to n_chunks merges
// the head (one wavefront) and resets the counter to zero for the next call.
// No workgroup ever waits on another, so the pattern cannot stall.

// Workspace: partials, then one uint32 counter per (sequence, KV head).
__host__ __device__ inline int64_t counters_offset(int64_t heads, int n_chunks, int g, int d) {
    const int64_t bytes = heads * n_chunks * g * (int64_t)(d + 2) * (int64_t)sizeof(float);
    return (bytes + 255) / 256 * 256;
}

__device__ inline float wave_max(float v) {
    for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
    return v;
}
__device__ inline float wave_sum(float v) {
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// Called by all lanes of one wavefront of every workgroup after its partial
// stores. Returns after the merge (last workgroup) or immediately.
__device__ void publish_and_merge(const Geo &g, int64_t head, int n_chunks, float *part,
                                  unsigned int *counters, float *out, float *lse, int64_t T, int lane) {
    __threadfence();  // partial stores visible device-wide before the count
    unsigned int prev = 0;
    if (lane == 0) prev = atomicAdd(&counters[head], 1u);
    prev = __shfl(prev, 0, 64);
    if (prev != (unsigned int)(n_chunks - 1)) return;
    __threadfence();  // see every other workgroup's partial

    const int G = g.g, d = g.d;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    for (int qi = 0; qi < G; ++qi) {
        float M = -INFINITY;
        for (int c = lane; c < n_chunks; c += 64) M = fmaxf(M, part[partial_index(head, c, n_chunks, qi, G, d)]);
        M = wave_max(M);
        float l = 0.f;
        for (int c = lane; c < n_chunks; c += 64) {
            const int64_t p = partial_index(head, c, n_chunks, qi, G, d);
            const float m = part[p];
            if (m != -INFINITY) l += exp2f(m - M) * part[p + 1];
        }
        l = wave_sum(l);
        const bool empty = T <= 0 || M == -INFINITY || !(l > 0.f);
        const float inv = empty ? 0.f : 1.f / l;
        const int qh = h * G + qi;
        float *o = out + ((int64_t)b * g.Hq + qh) * d;
        for (int k = lane; k < d; k += 64) {
            float acc = 0.f;
            if (!empty)
                for (int c = 0; c < n_chunks; ++c) {
                    const int64_t p = partial_index(head, c, n_chunks, qi, G, d);
                    const float m = part[p];
                    if (m != -INFINITY) acc = fmaf(exp2f(m - M), part[p + 2 + k], acc);
                }
            o[k] = acc * inv;
        }
        if (lse && lane == 0) lse[(int64_t)b * g.Hq + qh] = empty ? -INFINITY : (M + log2f(l)) * kLn2;
    }
    if (lane == 0) atomicExch(&counters[head], 0u);
}

// ---- generic kernel: any supported geometry, fp32 or bf16 storage ----------
//
// 256 threads. Per page: Z = Q R_K^T (g x rk), S = Z L_K^T (g x P), online
// softmax over the page, Y = E L_V (g x rv), O = O * alpha + Y R_V. Dense
// pages: S = Q K^T, O = O * alpha + E V. All contractions in fp32 from the
// stored values; each thread keeps its own slice of O in registers.

constexpr int kGenThreads = 256;
constexpr int kGenMaxOut = 16;  // g * d / 256 <= 16 for g <= 16, d <= 256

template <typename TD, typename TF>
__global__ __launch_bounds__(kGenThreads) void k_attn_generic(Geo g, const pkv_page *table,
                                                              const char *dense, const char *factor,
                                                              const TD *q, SeqArgs seq, int ppc,
                                                              int n_chunks, float *part,
                                                              unsigned int *counters, float *out,
                                                              float *lse) {
    __shared__ float sq[16 * 256];
    __shared__ float sZ[16 * 64];
    __shared__ float sS[16 * 64];
    __shared__ float sM[16], sL[16], sAlpha[16];

    const int chunk = blockIdx.x;
    const int64_t head = blockIdx.y;
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    const int G = g.g, d = g.d, P = g.P;
    const int tid = threadIdx.x;
    const int64_t T = seq.len[b];
    const int64_t n_pages = ceil_div(T, P);
    const int64_t j0 = (int64_t)chunk * ppc;
    const int64_t j1 = min<int64_t>(j0 + ppc, n_pages);
    const float c2 = kLog2e / sqrtf((float)d);

    for (int i = tid; i < G * d; i += kGenThreads) {
        const int qi = i / d, k = i % d;
        sq[qi * 256 + k] = to_f32(q[((int64_t)b * g.Hq + (int64_t)h * G + qi) * d + k]);
    }
    if (tid < G) { sM[tid] = -INFINITY; sL[tid] = 0.f; sAlpha[tid] = 1.f; }
    float o[kGenMaxOut];
#pragma unroll
    for (int i = 0; i < kGenMaxOut; ++i) o[i] = 0.f;
    const int n_out = G * d;
    __syncthreads();

    const int wave = tid / 64, lane = tid % 64;
    for (int64_t j = j0; j < j1; ++j) {
        const pkv_page e = table[head * g.max_pages + j];
        const int rows = (int)min<int64_t>(P, T - j * P);
        if (e.kind == PKV_FACTOR) {
            const int rk = e.rank_k, rv = e.rank_v, rk4 = r4(rk), rv4 = r4(rv);
            const TF *Ak = (const TF *)(factor + e.slot * g.factor_slot_bytes);
            const TF *Bk = Ak + (int64_t)P * rk4;
            const TF *Avt = Bk + (int64_t)rk * d;
            const TF *Bvt = Avt + (int64_t)rv * P;
            for (int i = tid; i < G * rk; i += kGenThreads) {
                const int qi = i / rk, a = i % rk;
                float z = 0.f;
                for (int k = 0; k < d; ++k) z = fmaf(sq[qi * 256 + k], ld(Bk, (int64_t)a * d + k), z);
                sZ[qi * 64 + a] = z;
            }
            __syncthreads();
            for (int i = tid; i < G * P; i += kGenThreads) {
                const int qi = i / P, t = i % P;
                float s = 0.f;
                for (int a = 0; a < rk; ++a) s = fmaf(sZ[qi * 64 + a], ld(Ak, (int64_t)t * rk4 + a), s);
                sS[qi * 64 + t] = t < rows ? s * c2 : -INFINITY;
            }
            __syncthreads();
            // online softmax over the page, one wave per query
            for (int qi = wave; qi < G; qi += kGenThreads / 64) {
                const float s = lane < P ? sS[qi * 64 + lane] : -INFINITY;
                float pm = s;
                for (int m = 32; m >= 1; m >>= 1) pm = fmaxf(pm, __shfl_xor(pm, m, 64));
                const float m_old = sM[qi];
                const float m_new = fmaxf(m_old, pm);
                const float ex = (lane < P && s != -INFINITY) ? exp2f(s - m_new) : 0.f;
                float sum = ex;
                for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
                if (lane < P) sS[qi * 64 + lane] = ex;
                if (lane == 0) {
                    const float alpha = m_old == -INFINITY ? 0.f : exp2f(m_old - m_new);
                    sL[qi] = sL[qi] * alpha + sum;
                    sM[qi] = m_new;
                    sAlpha[qi] = alpha;
                }
            }
            __syncthreads();
            // Y = E L_V (reuse sZ)
            for (int i = tid; i < G * rv; i += kGenThreads) {
                const int qi = i / rv, a = i % rv;
                float y = 0.f;
                for (int t = 0; t < P; ++t) y = fmaf(sS[qi * 64 + t], ld(Avt, (int64_t)a * P + t), y);
                sZ[qi * 64 + a] = y;
            }
            __syncthreads();
            for (int i = 0; i < kGenMaxOut; ++i) {
                const int idx = tid + i * kGenThreads;
                if (idx >= n_out) break;
                const int qi = idx / d, k = idx % d;
                float acc = o[i] * sAlpha[qi];
                for (int a = 0; a < rv; ++a) acc = fmaf(sZ[qi * 64 + a], ld(Bvt, (int64_t)k * rv4 + a), acc);
                o[i] = acc;
            }
            __syncthreads();
        } else if (e.kind == PKV_DENSE) {
            const TD *K = (const TD *)(dense + e.slot * g.dense_slot_bytes);
            const TD *Vt = K + (int64_t)P * d;
            for (int i = tid; i < G * P; i += kGenThreads) {
                const int qi = i / P, t = i % P;
                float s = 0.f;
                if (t < rows)
                    for (int k = 0; k < d; ++k) s = fmaf(sq[qi * 256 + k], ld(K, (int64_t)t * d + k), s);
                sS[qi * 64 + t] = t < rows ? s * c2 : -INFINITY;
            }
            __syncthreads();
            for (int qi = wave; qi < G; qi += kGenThreads / 64) {
                const float s = lane < P ? sS[qi * 64 + lane] : -INFINITY;
                float pm = s;
                for (int m = 32; m >= 1; m >>= 1) pm = fmaxf(pm, __shfl_xor(pm, m, 64));
                const float m_old = sM[qi];
                const float m_new = fmaxf(m_old, pm);
                const float ex = (lane < P && s != -INFINITY) ? exp2f(s - m_new) : 0.f;
                float sum = ex;
                for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
                if (lane < P) sS[qi * 64 + lane] = ex;
                if (lane == 0) {
                    const float alpha = m_old == -INFINITY ? 0.f : exp2f(m_old - m_new);
                    sL[qi] = sL[qi] * alpha + sum;
                    sM[qi] = m_new;
                    sAlpha[qi] = alpha;
                }
            }
            __syncthreads();
            for (int i = 0; i < kGenMaxOut; ++i) {
                const int idx = tid + i * kGenThreads;
                if (idx >= n_out) break;
                const int qi = idx / d, k = idx % d;
                float acc = o[i] * sAlpha[qi];
                for (int t = 0; t < rows; ++t) acc = fmaf(sS[qi * 64 + t], ld(Vt, (int64_t)k * P + t), acc);
                o[i] = acc;
            }
            __syncthreads();
        } else {
            if (tid == 0) raise_status(PKV_DEV_BAD_PAGE);
        }
    }

    // partial state of this chunk
    for (int i = 0; i < kGenMaxOut; ++i) {
        const int idx = tid + i * kGenThreads;
        if (idx >= n_out) break;
        const int qi = idx / d, k = idx % d;
        part[partial_index(head, chunk, n_chunks, qi, G, d) + 2 + k] = o[i];
    }
    if (tid < G) {
        const int64_t p = partial_index(head, chunk, n_chunks, tid, G, d);
        part[p] = sM[tid];
        part[p + 1] = sL[tid];
    }
    __syncthreads();
    if (wave == 0) publish_and_merge(g, head, n_chunks, part, counters, out, lse, T, lane);
}

}  // namespace pkv
