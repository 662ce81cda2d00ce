/*
 * PuzzleKV CPU oracle, fp64.
 *
 * TEST INFRASTRUCTURE ONLY. The product library never includes, links or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark load it. It shares no source with the HIP path.
 *
 * Every routine is the plain, slow definition of what the method computes:
 *
 *   orc_page_kind / orc_plan_pages / orc_eligible_pages
 *       which logical pages are dense and which are factorized
 *       (Section 3.3, "Page-Wise Low-Rank KV Cache Construction" and
 *       "Incremental Cache Update"; Section 4.1 "Implementation" for the
 *       default dense region of one sink page, the last completed page and
 *       the current incomplete page).
 *   orc_svd_rows / orc_truncated_factors / orc_adaptive_rank
 *       rank-r truncated SVD of one P x d page, computed without the Gram
 *       matrix by one-sided (Hestenes) Jacobi on the page rows, and the
 *       factor pair L = U_r, R = Sigma_r W_r^T (Section 3.2 "Truncated SVD";
 *       Section 3.3, Eq. (2)).
 *   orc_attention
 *       textbook softmax(q K^T / sqrt(d)) V over the cache rebuilt page by
 *       page from its stored form (Section 3.2, Eq. (1)); for a cache that
 *       stores keys before RoPE, every rebuilt key row is first rotated to
 *       its absolute position (orc_rope_rows).
 *   orc_rope_rows
 *       rotary position embedding of key rows, rotate-half pairing: the
 *       paper factorizes post-RoPE keys by default and compares factorizing
 *       pre-RoPE keys with RoPE applied at cache access (Section 4.2 "Main
 *       Results"; Appendix "RoPE Key Analysis").
 *   orc_attention_pagewise
 *       the page-local softmax state of Eq. (4) evaluated directly from the
 *       factors, merged by the online-softmax reduction of Eq. (5) in a caller
 *       chosen page order and grouping. It exists to pin the re-association
 *       that the GPU kernel relies on against orc_attention.
 *
 * Page kinds: 0 = empty (holds no token), 1 = dense, 2 = factorized.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_EMPTY = 0, ORC_DENSE = 1, ORC_FACTOR = 2 };

static long long ceil_div_ll(long long a, long long b) { return (a + b - 1) / b; }

/* ------------------------------------------------------------------------ */
/* Page plan (Section 3.3; Section 4.1 "Implementation").                    */
/*                                                                           */
/* T tokens are cut into pages of P tokens. The first ceil(S/P) pages form   */
/* the sink and stay dense. The local window holds the most recent W tokens; */
/* any page that overlaps it stays dense, and so does the incomplete last    */
/* page. Every other page is complete, outside the sink and entirely older   */
/* than the window, and is factorized. With S = W = P this is exactly the    */
/* paper's default dense region (one sink page, the most recently completed  */
/* page and the current incomplete page).                                    */
/* ------------------------------------------------------------------------ */
int orc_page_kind(long long T, int P, int S, int W, long long j)
{
    if (P <= 0 || j < 0 || j * P >= T) return ORC_EMPTY;
    int complete = (j + 1) * P <= T;
    int in_sink = j < ceil_div_ll(S, P);
    int in_window = (j + 1) * P > T - W;
    return (complete && !in_sink && !in_window) ? ORC_FACTOR : ORC_DENSE;
}

/* Fills kind[0..n) and returns the number of non-empty pages, ceil(T/P). */
long long orc_plan_pages(long long T, int P, int S, int W, uint8_t *kind, long long n)
{
    for (long long j = 0; j < n; ++j) kind[j] = (uint8_t)orc_page_kind(T, P, S, W, j);
    return T > 0 ? ceil_div_ll(T, P) : 0;
}

/* Pages that are factorized at T_new but were not at T_prev (Section 3.3,
 * "Incremental Cache Update": a page is converted once, when it leaves the
 * window). Writes at most cap indices to out and returns the full count. */
long long orc_eligible_pages(long long T_prev, long long T_new, int P, int S, int W,
                             long long *out, long long cap)
{
    long long count = 0;
    long long n_new = T_new > 0 ? ceil_div_ll(T_new, P) : 0;
    for (long long j = 0; j < n_new; ++j) {
        if (orc_page_kind(T_new, P, S, W, j) == ORC_FACTOR &&
            orc_page_kind(T_prev, P, S, W, j) != ORC_FACTOR) {
            if (count < cap) out[count] = j;
            ++count;
        }
    }
    return count;
}

/* ------------------------------------------------------------------------ */
/* Truncated SVD of a page (Section 3.2 "Truncated SVD"; Eq. (2)).           */
/*                                                                           */
/* One-sided Jacobi on the n rows of X (n x d): rows y_i, y_j are rotated    */
/* until every pair is orthogonal to working precision. Then X = J Y with J  */
/* orthogonal, the rows of Y are sigma_i w_i^T and the columns of J are the  */
/* left singular vectors u_i.                                                */
/*                                                                           */
/* Outputs, sorted by sigma descending (ties keep the lower index):          */
/*   U   n x n row-major, column k = u_k                                     */
/*   sig n values                                                            */
/*   Rf  n x d row-major, row k = sig_k w_k^T                                */
/* Returns the number of sweeps used, or -1 if max_sweeps was reached       */
/* without a sweep free of rotations. A pair is rotated while              */
/* |y_i . y_j| > n 2^-53 |y_i| |y_j|; rows below n 2^-53 |X|_F count as zero. */
/* ------------------------------------------------------------------------ */
static double dot(const double *a, const double *b, int n)
{
    double s = 0.0;
    for (int k = 0; k < n; ++k) s += a[k] * b[k];
    return s;
}

int orc_svd_rows(int n, int d, const double *X, double *U, double *sig, double *Rf,
                 int max_sweeps)
{
    double *Y = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *J = (double *)malloc(sizeof(double) * (size_t)n * n);
    double *nrm = (double *)malloc(sizeof(double) * (size_t)n);
    int *perm = (int *)malloc(sizeof(int) * (size_t)n);
    if (!Y || !J || !nrm || !perm) {
        free(Y); free(J); free(nrm); free(perm);
        return -2;
    }
    memcpy(Y, X, sizeof(double) * (size_t)n * d);
    for (int a = 0; a < n; ++a)
        for (int b = 0; b < n; ++b) J[(size_t)a * n + b] = (a == b) ? 1.0 : 0.0;

    const double tol = (double)n * (DBL_EPSILON / 2.0); /* n * 2^-53 */
    /* A row whose norm is below tol * |X|_F is zero to working precision; it
     * is left alone (otherwise, with more rows than columns, rounding residue
     * rows could never be made orthogonal to the rows spanning the space). */
    double fro2 = 0.0;
    for (size_t e = 0; e < (size_t)n * d; ++e) fro2 += X[e] * X[e];
    const double tiny2 = tol * tol * fro2;
    int sweeps = 0, converged = 0;
    while (sweeps < max_sweeps) {
        ++sweeps;
        int rotated = 0;
        for (int i = 0; i < n; ++i) {
            for (int j = i + 1; j < n; ++j) {
                double *yi = Y + (size_t)i * d, *yj = Y + (size_t)j * d;
                double alpha = dot(yi, yi, d);
                double beta = dot(yj, yj, d);
                double gamma = dot(yi, yj, d);
                if (alpha <= tiny2 || beta <= tiny2) continue;
                if (!(fabs(gamma) > tol * sqrt(alpha * beta))) continue;
                /* Rotation that makes the two rows orthogonal (smaller angle). */
                double zeta = (beta - alpha) / (2.0 * gamma);
                double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                double c = 1.0 / sqrt(1.0 + t * t);
                double s = c * t;
                for (int k = 0; k < d; ++k) {
                    double a = yi[k], b = yj[k];
                    yi[k] = c * a - s * b;
                    yj[k] = s * a + c * b;
                }
                /* Keep X = J Y: J <- J * rot^T, the same update on columns. */
                for (int r = 0; r < n; ++r) {
                    double a = J[(size_t)r * n + i], b = J[(size_t)r * n + j];
                    J[(size_t)r * n + i] = c * a - s * b;
                    J[(size_t)r * n + j] = s * a + c * b;
                }
                ++rotated;
            }
        }
        if (!rotated) { converged = 1; break; }
    }

    for (int i = 0; i < n; ++i) {
        nrm[i] = sqrt(dot(Y + (size_t)i * d, Y + (size_t)i * d, d));
        perm[i] = i;
    }
    /* Insertion sort by sigma descending; stable, so ties keep the lower index. */
    for (int i = 1; i < n; ++i) {
        int p = perm[i];
        int k = i - 1;
        while (k >= 0 && nrm[perm[k]] < nrm[p]) { perm[k + 1] = perm[k]; --k; }
        perm[k + 1] = p;
    }
    for (int k = 0; k < n; ++k) {
        int src = perm[k];
        sig[k] = nrm[src];
        for (int r = 0; r < n; ++r) U[(size_t)r * n + k] = J[(size_t)r * n + src];
        memcpy(Rf + (size_t)k * d, Y + (size_t)src * d, sizeof(double) * (size_t)d);
    }
    free(Y); free(J); free(nrm); free(perm);
    return converged ? sweeps : -1;
}

/* Rank-r factor pair of one page, Eq. (2): L = U_r (P x r), R = Sigma_r W_r^T
 * (r x d). sig receives all P singular values (descending). Returns the
 * sweep count of orc_svd_rows. */
int orc_truncated_factors(int P, int d, int r, const double *X, double *L, double *R,
                          double *sig, int max_sweeps)
{
    double *U = (double *)malloc(sizeof(double) * (size_t)P * P);
    double *Rf = (double *)malloc(sizeof(double) * (size_t)P * d);
    if (!U || !Rf) { free(U); free(Rf); return -2; }
    int sw = orc_svd_rows(P, d, X, U, sig, Rf, max_sweeps);
    for (int t = 0; t < P; ++t)
        for (int k = 0; k < r; ++k) L[(size_t)t * r + k] = U[(size_t)t * P + k];
    memcpy(R, Rf, sizeof(double) * (size_t)r * d);
    free(U); free(Rf);
    return sw;
}

/* Adaptive page rank. The paper sizes ranks by reconstruction accuracy
 * (Figure 2: the rank a page needs for 80% reconstruction accuracy), read
 * here as the relative Frobenius error of the rank-r truncation: the rank is
 * the smallest r >= 1 with |X - X_r|_F <= eps |X|_F, i.e. with
 * sum_{i >= r} sig_i^2 <= eps^2 sum_i sig_i^2 (Eckart-Young), capped at cap.
 * sig: the n singular values in descending order. */
int orc_adaptive_rank(int n, const double *sig, double eps, int cap)
{
    double total = 0.0;
    for (int i = 0; i < n; ++i) total += sig[i] * sig[i];
    const double budget = eps * eps * total;
    for (int r = 1; r <= cap && r <= n; ++r) {
        double tail = 0.0;
        for (int i = r; i < n; ++i) tail += sig[i] * sig[i];
        if (tail <= budget) return r;
    }
    return cap < n ? cap : n;
}

/* Batched form over n pages for the CPU baseline and large test sweeps; page
 * p reads X + p*P*d and writes L + p*P*r, R + p*r*d, sig + p*P, sweeps[p]. */
void orc_truncated_factors_batch(int n, int P, int d, const int *rank, const double *X,
                                 double *L, double *R, int ldr_max, double *sig, int *sweeps,
                                 int max_sweeps)
{
    #pragma omp parallel for schedule(dynamic, 4)
    for (int p = 0; p < n; ++p) {
        sweeps[p] = orc_truncated_factors(P, d, rank[p], X + (size_t)p * P * d,
                                          L + (size_t)p * P * ldr_max,
                                          R + (size_t)p * ldr_max * d,
                                          sig + (size_t)p * P, max_sweeps);
    }
}

/* ------------------------------------------------------------------------ */
/* Attention over the rebuilt cache (Eq. (1)).                               */
/*                                                                           */
/* One KV head holding T tokens in n_pages pages, attended by g query heads. */
/* Page j stores rows j*P .. min(T,(j+1)*P)-1. Its data starts at            */
/* data + off[j]:                                                            */
/*   dense  : K (P x d) then V (P x d), row-major                            */
/*   factor : L_K (P x rk), R_K (rk x d), L_V (P x rv), R_V (rv x d)         */
/* Each page is rebuilt (K = L_K R_K, V = L_V R_V for factor pages) and the   */
/* softmax is the textbook one: s = K q / sqrt(d), p = exp(s - max) / sum,   */
/* out = p^T V, lse = max + log(sum).                                        */
/* ------------------------------------------------------------------------ */
static void rebuild_page(int P, int d, int kind, int rk, int rv, const double *src,
                         int rows, double *Kout, double *Vout)
{
    if (kind == ORC_DENSE) {
        memcpy(Kout, src, sizeof(double) * (size_t)rows * d);
        memcpy(Vout, src + (size_t)P * d, sizeof(double) * (size_t)rows * d);
        return;
    }
    const double *Lk = src;
    const double *Rk = Lk + (size_t)P * rk;
    const double *Lv = Rk + (size_t)rk * d;
    const double *Rv = Lv + (size_t)P * rv;
    for (int t = 0; t < rows; ++t) {
        for (int k = 0; k < d; ++k) {
            double sk = 0.0, sv = 0.0;
            for (int a = 0; a < rk; ++a) sk += Lk[(size_t)t * rk + a] * Rk[(size_t)a * d + k];
            for (int a = 0; a < rv; ++a) sv += Lv[(size_t)t * rv + a] * Rv[(size_t)a * d + k];
            Kout[(size_t)t * d + k] = sk;
            Vout[(size_t)t * d + k] = sv;
        }
    }
}

/* Rotary position embedding in place, rotate-half pairing. Row t of X (an   */
/* n x d matrix) is the key at position pos[t]. Dimension i < d/2 pairs with */
/* i + d/2, at frequency theta_i = base^(-2i/d): the pair (x_i, x_{i+d/2})    */
/* is rotated by the angle pos * theta_i,                                    */
/*   x_i       <- x_i cos(a) - x_{i+d/2} sin(a)                              */
/*   x_{i+d/2} <- x_{i+d/2} cos(a) + x_i sin(a).                             */
/* Angles, sines and cosines in fp64 (libm).                                 */
int orc_rope_rows(int n, int d, const long long *pos, double base, double *X)
{
    if (d % 2 != 0 || !(base > 0.0)) return -1;
    const int h = d / 2;
    for (int t = 0; t < n; ++t) {
        double *x = X + (size_t)t * d;
        for (int i = 0; i < h; ++i) {
            const double theta = pow(base, -2.0 * (double)i / (double)d);
            const double a = (double)pos[t] * theta;
            const double c = cos(a), s = sin(a);
            const double x0 = x[i], x1 = x[i + h];
            x[i] = x0 * c - x1 * s;
            x[i + h] = x1 * c + x0 * s;
        }
    }
    return 0;
}

/* key_rope_base > 0: the stored keys are pre-RoPE; each rebuilt key row t   */
/* is rotated to position t (orc_rope_rows) before the scores. 0: keys are   */
/* used as stored.                                                           */
int orc_attention(long long T, int P, int d, int g, int n_pages, const int *kind,
                  const int *rank_k, const int *rank_v, const long long *off,
                  const double *data, const double *q, double key_rope_base,
                  double *out, double *lse)
{
    if (T <= 0) return -1;
    double *Kh = (double *)malloc(sizeof(double) * (size_t)T * d);
    double *Vh = (double *)malloc(sizeof(double) * (size_t)T * d);
    double *s = (double *)malloc(sizeof(double) * (size_t)T);
    if (!Kh || !Vh || !s) { free(Kh); free(Vh); free(s); return -2; }

    int bad = 0;
    #pragma omp parallel for schedule(dynamic, 8) reduction(|:bad)
    for (int j = 0; j < n_pages; ++j) {
        long long t0 = (long long)j * P;
        if (t0 >= T) continue;
        int rows = (int)((T - t0) < P ? (T - t0) : P);
        if (kind[j] != ORC_DENSE && kind[j] != ORC_FACTOR) { bad |= 1; continue; }
        rebuild_page(P, d, kind[j], rank_k[j], rank_v[j], data + off[j], rows,
                     Kh + (size_t)t0 * d, Vh + (size_t)t0 * d);
    }
    if (bad || (long long)n_pages * P < T) { free(Kh); free(Vh); free(s); return -3; }
    if (key_rope_base > 0.0) {
        int rbad = 0;
        #pragma omp parallel for schedule(static) reduction(|:rbad)
        for (long long t = 0; t < T; ++t) {
            const long long pos = t;
            rbad |= orc_rope_rows(1, d, &pos, key_rope_base, Kh + (size_t)t * d) != 0;
        }
        if (rbad) { free(Kh); free(Vh); free(s); return -4; }
    }

    const double scale = 1.0 / sqrt((double)d);
    for (int i = 0; i < g; ++i) {
        const double *qi = q + (size_t)i * d;
        #pragma omp parallel for schedule(static)
        for (long long t = 0; t < T; ++t) s[t] = dot(Kh + (size_t)t * d, qi, d) * scale;
        double m = -INFINITY;
        for (long long t = 0; t < T; ++t) m = s[t] > m ? s[t] : m;
        double Z = 0.0;
        for (long long t = 0; t < T; ++t) { s[t] = exp(s[t] - m); Z += s[t]; }
        #pragma omp parallel for schedule(static)
        for (int k = 0; k < d; ++k) {
            double acc = 0.0;
            for (long long t = 0; t < T; ++t) acc += s[t] * Vh[(size_t)t * d + k];
            out[(size_t)i * d + k] = acc / Z;
        }
        if (lse) lse[i] = m + log(Z);
    }
    free(Kh); free(Vh); free(s);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Page-wise state and merge (Eq. (4) and Eq. (5)).                          */
/*                                                                           */
/* Same page description as orc_attention. Pages are visited in the order    */
/* given by `order` (NULL = natural); consecutive runs of `group` visited     */
/* pages are first merged into one unnormalized state with the Eq. (5)      */
/* rescaling, and the group states are merged the same way at the end.      */
/* For a factor page the score is (q R_K^T) L_K^T / sqrt(d) and the          */
/* unnormalized output is (exp(s - m_p) L_V) R_V, contracted in that order.  */
/* ------------------------------------------------------------------------ */
static void page_state(long long T, int P, int d, int kind, int rk, int rv, const double *src,
                       long long t0, const double *q, double *m_p, double *l_p, double *o_p)
{
    int rows = (int)((T - t0) < P ? (T - t0) : P);
    const double scale = 1.0 / sqrt((double)d);
    double s[1024];
    if (kind == ORC_DENSE) {
        const double *K = src, *V = src + (size_t)P * d;
        for (int t = 0; t < rows; ++t) s[t] = dot(K + (size_t)t * d, q, d) * scale;
        double m = -INFINITY;
        for (int t = 0; t < rows; ++t) m = s[t] > m ? s[t] : m;
        double l = 0.0;
        for (int k = 0; k < d; ++k) o_p[k] = 0.0;
        for (int t = 0; t < rows; ++t) {
            double e = exp(s[t] - m);
            l += e;
            for (int k = 0; k < d; ++k) o_p[k] += e * V[(size_t)t * d + k];
        }
        *m_p = m; *l_p = l;
        return;
    }
    const double *Lk = src;
    const double *Rk = Lk + (size_t)P * rk;
    const double *Lv = Rk + (size_t)rk * d;
    const double *Rv = Lv + (size_t)P * rv;
    double u[256], y[256];
    for (int a = 0; a < rk; ++a) u[a] = dot(Rk + (size_t)a * d, q, d);         /* q R_K^T */
    for (int t = 0; t < rows; ++t) s[t] = dot(Lk + (size_t)t * rk, u, rk) * scale; /* ... L_K^T */
    double m = -INFINITY;
    for (int t = 0; t < rows; ++t) m = s[t] > m ? s[t] : m;
    double l = 0.0;
    for (int a = 0; a < rv; ++a) y[a] = 0.0;
    for (int t = 0; t < rows; ++t) {
        double e = exp(s[t] - m);
        l += e;
        for (int a = 0; a < rv; ++a) y[a] += e * Lv[(size_t)t * rv + a];      /* e^T L_V */
    }
    for (int k = 0; k < d; ++k) {
        double acc = 0.0;
        for (int a = 0; a < rv; ++a) acc += y[a] * Rv[(size_t)a * d + k];       /* ... R_V */
        o_p[k] = acc;
    }
    *m_p = m; *l_p = l;
}

/* Merge of unnormalized states (m_i, l_i, o_i), i < n, into one (Eq. (5)). */
static void merge_states(int n, int d, const double *m, const double *l, const double *o,
                         double *m_out, double *l_out, double *o_out)
{
    double mm = -INFINITY;
    for (int i = 0; i < n; ++i) mm = m[i] > mm ? m[i] : mm;
    double ll = 0.0;
    for (int k = 0; k < d; ++k) o_out[k] = 0.0;
    for (int i = 0; i < n; ++i) {
        double w = exp(m[i] - mm);
        ll += w * l[i];
        for (int k = 0; k < d; ++k) o_out[k] += w * o[(size_t)i * d + k];
    }
    *m_out = mm; *l_out = ll;
}

int orc_attention_pagewise(long long T, int P, int d, int g, int n_pages, const int *kind,
                           const int *rank_k, const int *rank_v, const long long *off,
                           const double *data, const double *q, const int *order, int group,
                           double *out, double *lse)
{
    if (T <= 0 || P > 1024) return -1;
    for (int j = 0; j < n_pages; ++j)
        if (kind[j] == ORC_FACTOR && (rank_k[j] > 256 || rank_v[j] > 256)) return -1;
    int np = 0;
    for (int j = 0; j < n_pages; ++j) if ((long long)j * P < T) ++np;
    if (group <= 0) group = np;
    int ng = (np + group - 1) / group;
    double *pm = (double *)malloc(sizeof(double) * (size_t)np);
    double *pl = (double *)malloc(sizeof(double) * (size_t)np);
    double *po = (double *)malloc(sizeof(double) * (size_t)np * d);
    double *gm = (double *)malloc(sizeof(double) * (size_t)ng);
    double *gl = (double *)malloc(sizeof(double) * (size_t)ng);
    double *go = (double *)malloc(sizeof(double) * (size_t)ng * d);
    if (!pm || !pl || !po || !gm || !gl || !go) {
        free(pm); free(pl); free(po); free(gm); free(gl); free(go);
        return -2;
    }
    for (int i = 0; i < g; ++i) {
        const double *qi = q + (size_t)i * d;
        for (int v = 0; v < np; ++v) {
            int j = order ? order[v] : v;
            page_state(T, P, d, kind[j], rank_k[j], rank_v[j], data + off[j], (long long)j * P,
                       qi, pm + v, pl + v, po + (size_t)v * d);
        }
        for (int c = 0; c < ng; ++c) {
            int a = c * group, n = (np - a) < group ? (np - a) : group;
            merge_states(n, d, pm + a, pl + a, po + (size_t)a * d, gm + c, gl + c,
                         go + (size_t)c * d);
        }
        double m, l;
        double *o = out + (size_t)i * d;
        merge_states(ng, d, gm, gl, go, &m, &l, o);
        for (int k = 0; k < d; ++k) o[k] /= l;
        if (lse) lse[i] = m + log(l);
    }
    free(pm); free(pl); free(po); free(gm); free(gl); free(go);
    return 0;
}

/* Number of OpenMP threads the parallel loops above use (1 without OpenMP). */
int orc_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sets the number of OpenMP threads of the parallel loops above (for timing
 * the oracle on one core and on all of them); no effect without OpenMP. */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
