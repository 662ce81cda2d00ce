// Mixed-page decode attention (Eq. (4) for factor pages, the same state from
// K and V for dense pages, Eq. (5) to merge) -- split phase and combine.
//
// Work is split flash-decoding style: each workgroup owns one (sequence, KV
// head) and a contiguous chunk of pages, keeps the running (m, l, O) state
// of the g query heads of that KV head, and writes it as a partial; the last
// workgroup of a head merges its partials with the Eq. (5) rescaling.
// Scores are kept in the base-2 domain (s * log2(e) / sqrt(d)) so every
// exponential is one exp2.
// Included by pkv_kernels.hip.

namespace pkv {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Workspace of one call. It starts with the per-head words that must be zero
// when a call begins and that every call returns to zero: one merge counter
// per (sequence, KV head) `head`, then one page-claim word per head on its
// own 256-byte line. Their offsets depend only on the number of heads, so a
// workspace sized for the longest sequence can be shared by calls of any
// length. The partial states follow, for each head, chunk c and query qi of
// the group: O[head][c][qi][k], the max M[head][c][qi] (log2 units) and the
// normalizer L[head][c][qi], so that each workgroup's partial is one
// contiguous block (whole cache lines written, no line shared between
// workgroups) and the merge reads one chunk per load across consecutive
// lanes. The partials are fully written by every call before they are read.
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct Partials {
    float *o, *m, *l;
    unsigned int *counters;  // chunks published, per head
    unsigned int *claims;    // pages handed out, per head (streaming kernel), one per 256 bytes
    __host__ __device__ unsigned int *claim(int64_t head) const { return claims + head * 64; }
    int nc, nc4, g, d;
    __host__ __device__ int64_t oi(int64_t head, int qi, int k, int c) const {
        return ((head * nc4 + c) * g + qi) * d + k;
    }
    __host__ __device__ int64_t mi(int64_t head, int qi, int c) const { return (head * nc4 + c) * g + qi; }
};

__host__ __device__ inline int64_t round256(int64_t b) { return (b + 255) / 256 * 256; }

// Bytes of the zero-on-entry words for `heads` heads.
__host__ __device__ inline int64_t counter_bytes(int64_t heads) { return round256(heads * 4) + heads * 256; }
// Bytes of the partial states.
__host__ __device__ inline int64_t partial_state_bytes(int64_t heads, int n_chunks, int g, int d) {
    const int64_t nc4 = (n_chunks + 3) / 4 * 4;
    return round256(heads * g * d * nc4 * 4) + 2 * round256(heads * g * nc4 * 4);
}
__host__ __device__ inline int64_t partials_bytes(int64_t heads, int n_chunks, int g, int d) {
    return counter_bytes(heads) + partial_state_bytes(heads, n_chunks, g, d);
}

// counters: a region of counter_bytes(heads_cap) bytes (heads_cap >= heads)
// laid out as the counters of heads_cap heads; states: the partial states.
__host__ __device__ inline Partials make_partials(void *counters, int64_t heads_cap, void *states, int64_t heads,
                                                  int n_chunks, int g, int d) {
    Partials p;
    p.nc = n_chunks;
    p.nc4 = (n_chunks + 3) / 4 * 4;
    p.g = g;
    p.d = d;
    p.counters = (unsigned int *)counters;
    p.claims = (unsigned int *)((char *)counters + round256(heads_cap * 4));
    char *c = (char *)states;
    p.o = (float *)c;
    c += round256(heads * g * d * p.nc4 * 4);
    p.m = (float *)c;
    c += round256(heads * g * p.nc4 * 4);
    p.l = (float *)c;
    return p;
}
// A caller's workspace: the counters of `heads` heads, then the states.
__host__ __device__ inline Partials make_partials(void *ws, int64_t heads, int n_chunks, int g, int d) {
    return make_partials(ws, heads, (char *)ws + counter_bytes(heads), heads, n_chunks, g, d);
}

// ---- combine: Eq. (5) across the chunks of one head, then normalize -----------
//
// Fused into the split kernels: every workgroup publishes its partial, then
// bumps the head's counter; the workgroup that brings it to n_chunks merges
// the head and resets the counter to zero for the next call. No workgroup
// ever waits on another, so the pattern cannot stall.
//
// Partials and counters are written and read with device-scope atomic
// accesses (relaxed), which the caches keep coherent across the chip's
// L2 slices one access at a time. A device-scope fence would instead write
// back and invalidate a whole L2 per workgroup, stalling every other
// workgroup's stream on that slice. Order comes from waiting for the
// workgroup's own stores to complete before the counter is bumped.
__device__ inline void st_dev(float *p, float v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
__device__ inline float ld_dev(const float *p) {
    return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Called by every thread of an NT-thread workgroup after its partial stores.
// The workgroup that completes the head merges all of its chunks (Eq. (5)).
// Chunks are folded in groups of kMergeGroup. A group's maxima and
// normalizers are read once, one or two per thread, and passed through LDS;
// each thread's kMergeGroup partial outputs are in flight with them, so a
// group costs one round trip to memory (kMergeGroup + 2 loads stay within a
// wave's 63 outstanding vector loads). The loads are unconditional (a chunk
// past the end reads the last one and is masked), which keeps this code
// short: it runs once per launch, from a cold instruction cache.
constexpr int kMergeGroup = 32;

// The fold of the last workgroup with 16-byte partial loads, for shapes whose
// F = G d / 4 groups of four outputs divide the workgroup into R lanes each:
// thread (f, r) folds chunks r, r + R, ... of output group f (one coherent
// 16-byte load per chunk, J per group of kMergeGroup chunks, loads past the
// last chunk read it again and are masked), every lane of a query uses the
// same running max (the group's maxima through LDS), and the R partial sums
// of an output group are added through LDS at the end. s_mg, s_lg: the
// group maxima and normalizers (16 x kMergeGroup floats each); red: 5 NT
// floats of LDS for the sums, 16-byte aligned.
template <int NT, int R>
__device__ void merge_vec(const Geo &g, int64_t head, const Partials &pp, float *out, float *lse, int64_t T,
                          float *s_mg, float *s_lg, float *red) {
    constexpr int J = (kMergeGroup + R - 1) / R;
    constexpr int MLT = (16 * kMergeGroup + NT - 1) / NT;
    f32x4 *s_ra = (f32x4 *)red;
    float *s_rl = red + 4 * NT;
    const int tid = threadIdx.x;
    const int nc = pp.nc, G = g.g, d = g.d;
    const int F = NT / R;
    const int f = tid % F, r = tid / F;
    const int q = (4 * f) / d, k = (4 * f) % d;
    const uint32_t cs = (uint32_t)(G * d) * 4u;   // chunk stride in bytes
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        pp.o + pp.oi(head, 0, 0, 0), (short)0, (int)((uint32_t)pp.nc4 * cs), 0x00020000);
    float M = -INFINITY, L = 0.f;
    f32x4 A = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nc; c0 += kMergeGroup) {
        float mreg[MLT], lreg[MLT];
#pragma unroll
        for (int i = 0; i < MLT; ++i) {
            const int t = tid + i * NT;
            const int qm = min(t / kMergeGroup, G - 1), cu = min(c0 + t % kMergeGroup, nc - 1);
            mreg[i] = ld_dev(pp.m + pp.mi(head, qm, cu));
            lreg[i] = ld_dev(pp.l + pp.mi(head, qm, cu));
        }
        f32x4 ov[J];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const uint32_t c = (uint32_t)min(c0 + r + R * j, nc - 1);
            ov[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ro, c * cs + 16u * (uint32_t)f, 0, 16));
        }
        __syncthreads();   // the previous group's maxima have been read
#pragma unroll
        for (int i = 0; i < MLT; ++i) {
            const int t = tid + i * NT;
            if (t < 16 * kMergeGroup) {
                s_mg[t] = (t % kMergeGroup) < nc - c0 ? mreg[i] : -INFINITY;
                s_lg[t] = lreg[i];
            }
        }
        __syncthreads();
        const float *mg = s_mg + q * kMergeGroup, *lg = s_lg + q * kMergeGroup;
        float Mg = M;
        for (int u = 0; u < kMergeGroup; u += 4) {
            const f32x4 m4 = *(const f32x4 *)(mg + u);
            Mg = fmaxf(Mg, fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3])));
        }
        if (Mg == -INFINITY) continue;   // no tokens in any chunk so far
        const float sc = __builtin_amdgcn_exp2f(M - Mg);
        L *= sc;
        A *= sc;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int u = r + R * j;   // chunk c0 + u; at or past nc its maximum is -inf
            const float wgt = u < kMergeGroup ? __builtin_amdgcn_exp2f(mg[u] - Mg) : 0.f;
            if (u < kMergeGroup) L = fmaf(wgt, lg[u], L);
            A += wgt * ov[j];
        }
        M = Mg;
    }
    s_ra[tid] = A;
    s_rl[tid] = L;
    __syncthreads();
    if (r == 0) {
#pragma unroll
        for (int i = 1; i < R; ++i) {
            A += s_ra[i * F + f];
            L += s_rl[i * F + f];
        }
        const bool empty = T <= 0 || !(L > 0.f);
        const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
        float *o = out + ((int64_t)b * g.Hq + h * G + q) * d + k;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = empty ? 0.f : A[i] / L;
        if (lse && k == 0) lse[(int64_t)b * g.Hq + h * G + q] = empty ? -INFINITY : (M + log2f(L)) * kLn2;
    }
}

// red: at least 5 NT floats of LDS the caller no longer needs (16-byte
// aligned), or null: the fold with 16-byte loads needs them.
template <int NT>
__device__ void publish_and_merge(const Geo &g, int64_t head, const Partials &pp, float *out, float *lse,
                                  int64_t T, float *red = nullptr) {
    constexpr int kMaxG = 16;                                      // the kernels' query-group limit
    constexpr int MLT = (kMaxG * kMergeGroup + NT - 1) / NT;       // group maxima per thread
    __shared__ unsigned int s_prev;
    __shared__ float s_mg[kMaxG * kMergeGroup], s_lg[kMaxG * kMergeGroup];
    const int tid = threadIdx.x;
    const int nc = pp.nc;
    __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this thread's partial stores have completed
    __syncthreads();
    if (tid == 0) s_prev = __hip_atomic_fetch_add(&pp.counters[head], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (s_prev != (unsigned int)(nc - 1)) return;

    const int G = g.g, d = g.d;
    bool done = false;
    // only where the per-output fold below would take several passes (G d >
    // NT, so two or three lanes per output group): at batch 1 (G d = NT, 32
    // chunks) that fold measured faster
    if (red && G * d > NT && (G * d) % 4 == 0 && NT % (G * d / 4) == 0) {
        switch (NT / (G * d / 4)) {
        case 2: merge_vec<NT, 2>(g, head, pp, out, lse, T, s_mg, s_lg, red); done = true; break;
        case 3: merge_vec<NT, 3>(g, head, pp, out, lse, T, s_mg, s_lg, red); done = true; break;
        default: break;
        }
    }
    if (done) {
        if (tid == 0) {
            __hip_atomic_store(&pp.counters[head], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(pp.claim(head), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
    }
    const int b = (int)(head / g.Hkv), h = (int)(head % g.Hkv);
    // the same trip counts in every thread: the group loop holds barriers
    for (int base = 0; base < G * d; base += NT) {
        const int idx = min(base + tid, G * d - 1);   // threads past the end redo the last output, unstored
        const int qi = idx / d, k = idx % d;
        const float *op = pp.o + pp.oi(head, qi, k, 0);
        const int co = G * d;   // chunk stride of the outputs
        float M = -INFINITY, L = 0.f, A = 0.f;
        for (int c0 = 0; c0 < nc; c0 += kMergeGroup) {
            float mreg[MLT], lreg[MLT];
#pragma unroll
            for (int i = 0; i < MLT; ++i) {
                const int t = tid + i * NT;
                const int qm = min(t / kMergeGroup, G - 1), cu = min(c0 + t % kMergeGroup, nc - 1);
                mreg[i] = ld_dev(pp.m + pp.mi(head, qm, cu));
                lreg[i] = ld_dev(pp.l + pp.mi(head, qm, cu));
            }
            float ov[kMergeGroup];
#pragma unroll
            for (int u = 0; u < kMergeGroup; ++u) ov[u] = ld_dev(op + (uint32_t)(min(c0 + u, nc - 1) * co));
            __syncthreads();   // the previous group's maxima have been read
#pragma unroll
            for (int i = 0; i < MLT; ++i) {
                const int t = tid + i * NT;
                if (t < kMaxG * kMergeGroup) {
                    s_mg[t] = (t % kMergeGroup) < nc - c0 ? mreg[i] : -INFINITY;
                    s_lg[t] = lreg[i];
                }
            }
            __syncthreads();
            const float *mg = s_mg + qi * kMergeGroup, *lg = s_lg + qi * kMergeGroup;
            float Mg = M;
#pragma unroll
            for (int u = 0; u < kMergeGroup; ++u) Mg = fmaxf(Mg, mg[u]);
            if (Mg == -INFINITY) continue;   // no tokens in any chunk so far
            // arguments <= 0 with Mg finite: the hardware exp2 gives 0 for -inf
            // (an empty chunk, or no state yet) and needs no range fix-up
            const float sc = __builtin_amdgcn_exp2f(M - Mg);
            L *= sc;
            A *= sc;
#pragma unroll
            for (int u = 0; u < kMergeGroup; ++u) {
                const float wgt = __builtin_amdgcn_exp2f(mg[u] - Mg);
                L = fmaf(wgt, lg[u], L);
                A = fmaf(wgt, ov[u], A);
            }
            M = Mg;
        }
        if (base + tid < G * d) {
            const bool empty = T <= 0 || !(L > 0.f);
            out[((int64_t)b * g.Hq + h * G + qi) * d + k] = empty ? 0.f : A / L;
            if (lse && k == 0) lse[(int64_t)b * g.Hq + h * G + qi] = empty ? -INFINITY : (M + log2f(L)) * kLn2;
        }
    }
    if (tid == 0) {
        __hip_atomic_store(&pp.counters[head], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(pp.claim(head), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
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
                                                              int n_chunks, Partials pp, float *out,
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
            const FactorLayout fl = factor_layout(P, d, rk, rv);
            const TF *Ak = (const TF *)(factor + e.slot * g.factor_slot_bytes);
            const TF *Bk = Ak + fl.bk, *Bvt = Ak + fl.bvt, *Avt = Ak + fl.avt;
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
        st_dev(&pp.o[pp.oi(head, qi, k, chunk)], o[i]);
    }
    if (tid < G) {
        st_dev(&pp.m[pp.mi(head, tid, chunk)], sM[tid]);
        st_dev(&pp.l[pp.mi(head, tid, chunk)], sL[tid]);
    }
    publish_and_merge<kGenThreads>(g, head, pp, out, lse, T);
}

}  // namespace pkv
