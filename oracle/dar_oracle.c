/*
 * DAR attention oracle: plain fp64 loops, written from the paper
 * "Dual Dimensionality for Local and Global Attention" (arXiv 2606.18587).
 *
 * TEST INFRASTRUCTURE ONLY. Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library. It shares no code,
 * header, table or helper with the HIP path, and the HIP path never calls it.
 *
 * What is computed, per KV head g (query heads h with g = h / (Hq/Hkv)):
 *
 *   Eq. 1   c_j  = x_j W_down           down-projection of a token (d -> d_down)
 *   Eq. 2   x'_j = c_j W_up             lift back to d (W_up = W_down^T if absent)
 *   Eq. 3   for query position i, token j <= i is used at full dimension when
 *           i - j < w (the window, which includes the token itself), and in
 *           lifted form otherwise; this applies to keys and to values.
 *   Eq. 4   o_i = softmax_j( q_i . key_j / sqrt(d_k) ) . value_j, one softmax
 *           over all j in [0, i]; d_k is the full per-head key dimension d for
 *           both regions, since the lifted key has dimension d.
 *
 * The method's readings taken here (bottleneck per KV head acting on k and v,
 * no rotary embedding inside the boundary, 0-based positions) are listed in
 * the design notes of the repository.
 *
 * Parallelism: OpenMP over independent query rows only; every row is the
 * plain sequential definition above.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Eq. 1: out[n][dd] = x[n][d] . wd[d][dd] */
void dar_oracle_down(int n, int d, int dd, const double* x, const double* wd, double* out)
{
    for (int t = 0; t < n; ++t)
        for (int c = 0; c < dd; ++c) {
            double acc = 0.0;
            for (int e = 0; e < d; ++e) acc += x[(size_t)t * d + e] * wd[(size_t)e * dd + c];
            out[(size_t)t * dd + c] = acc;
        }
}

/* Eq. 2: out[n][d] = h[n][dd] . wu[dd][d]; a NULL wu means wu = wd^T. */
void dar_oracle_up(int n, int d, int dd, const double* h, const double* wd, const double* wu,
                   double* out)
{
    for (int t = 0; t < n; ++t)
        for (int e = 0; e < d; ++e) {
            double acc = 0.0;
            for (int c = 0; c < dd; ++c) {
                double u = wu ? wu[(size_t)c * d + e] : wd[(size_t)e * dd + c];
                acc += h[(size_t)t * dd + c] * u;
            }
            out[(size_t)t * d + e] = acc;
        }
}

/* The lifted token x'_j = (x_j W_down) W_up for tokens [0, n). */
static double* lift_all(int n, int d, int dd, const double* x, const double* wd, const double* wu)
{
    double* h = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * dd);
    double* out = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * d);
    if (!h || !out) { free(h); free(out); return NULL; }
    dar_oracle_down(n, d, dd, x, wd, h);
    dar_oracle_up(n, d, dd, h, wd, wu, out);
    free(h);
    return out;
}

/* One query row of Eq. 3-4 against tokens [0, i] of one head.
 * k, v, kl, vl are [>= i+1][d]: original and lifted keys and values.
 * p (optional) receives the softmax weights for j in [0, i]. */
static void one_row(int d, int w, int i, const double* qi, const double* k, const double* v,
                    const double* kl, const double* vl, double* s, double* oi, double* p)
{
    const double scale = 1.0 / sqrt((double)d);
    double m = -INFINITY;
    for (int j = 0; j <= i; ++j) {
        const double* key = (i - j < w) ? k + (size_t)j * d : kl + (size_t)j * d;
        double acc = 0.0;
        for (int e = 0; e < d; ++e) acc += qi[e] * key[e];
        s[j] = acc * scale;
        if (s[j] > m) m = s[j];
    }
    double sum = 0.0;
    for (int j = 0; j <= i; ++j) { s[j] = exp(s[j] - m); sum += s[j]; }
    for (int e = 0; e < d; ++e) oi[e] = 0.0;
    for (int j = 0; j <= i; ++j) {
        const double pj = s[j] / sum;
        if (p) p[j] = pj;
        const double* val = (i - j < w) ? v + (size_t)j * d : vl + (size_t)j * d;
        for (int e = 0; e < d; ++e) oi[e] += pj * val[e];
    }
}

/*
 * Query rows of one head against one KV head's tokens.
 *   k, v  [T][d]     keys and values of tokens 0..T-1 (full dimension)
 *   wd    [d][dd], wu [dd][d] or NULL (tied: W_up = W_down^T)
 *   pos   [n_rows]   query positions, each in [0, T)
 *   qr    [n_rows][d]
 *   o     [n_rows][d]  output
 *   p     optional [n_rows][T]: softmax weights, zero for j > pos
 * Returns 0, or -1 on a bad argument / allocation failure.
 */
int dar_oracle_rows(int T, int d, int dd, int w, const double* k, const double* v,
                    const double* wd, const double* wu, int n_rows, const int* pos,
                    const double* qr, double* o, double* p)
{
    if (T < 1 || d < 1 || dd < 1 || w < 0 || n_rows < 0) return -1;
    for (int r = 0; r < n_rows; ++r)
        if (pos[r] < 0 || pos[r] >= T) return -1;
    double* kl = lift_all(T, d, dd, k, wd, wu);
    double* vl = lift_all(T, d, dd, v, wd, wu);
    if (!kl || !vl) { free(kl); free(vl); return -1; }
    int bad = 0;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)T);
        if (!s) {
#pragma omp atomic write
            bad = 1;
        } else {
#pragma omp for schedule(dynamic, 4)
            for (int r = 0; r < n_rows; ++r) {
                double* pr = p ? p + (size_t)r * T : NULL;
                if (pr) for (int j = 0; j < T; ++j) pr[j] = 0.0;
                one_row(d, w, pos[r], qr + (size_t)r * d, k, v, kl, vl, s, o + (size_t)r * d, pr);
            }
            free(s);
        }
    }
    free(kl);
    free(vl);
    return bad ? -1 : 0;
}

/*
 * Full causal prefill of a batch: every row i of every query head.
 *   q [B][Hq][T][d], k, v [B][Hkv][T][d], wd [Hkv][d][dd], wu [Hkv][dd][d] or NULL
 *   o [B][Hq][T][d]
 * nthreads > 0 sets the OpenMP thread count (0 keeps the default).
 */
int dar_oracle_prefill(int B, int Hq, int Hkv, int T, int d, int dd, int w, const double* q,
                       const double* k, const double* v, const double* wd, const double* wu,
                       double* o, int nthreads)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || T < 1 || d < 1 || dd < 1 || w < 0)
        return -1;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    const int group = Hq / Hkv;
    int* pos = (int*)malloc(sizeof(int) * (size_t)T);
    if (!pos) return -1;
    for (int i = 0; i < T; ++i) pos[i] = i;
    int rc = 0;
    for (int b = 0; b < B && rc == 0; ++b)
        for (int h = 0; h < Hq && rc == 0; ++h) {
            const int g = h / group;
            const size_t kv_off = ((size_t)b * Hkv + g) * (size_t)T * d;
            const size_t q_off = ((size_t)b * Hq + h) * (size_t)T * d;
            rc = dar_oracle_rows(T, d, dd, w, k + kv_off, v + kv_off, wd + (size_t)g * d * dd,
                                 wu ? wu + (size_t)g * dd * d : NULL, T, pos, q + q_off,
                                 o + q_off, NULL);
        }
    free(pos);
    return rc;
}

int dar_oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
