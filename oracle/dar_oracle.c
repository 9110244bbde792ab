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
 * 0-based positions) are listed in the design notes of the repository. The
 * functions without "rope" in their name leave rotary position embedding to
 * the caller; dar_oracle_rows_rope / dar_oracle_prefill_rope put it where
 * Eq. 3 does (after the lift on the distant path).
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
 * p (optional) receives the softmax weights for j in [0, i]; lse (optional)
 * the log of the softmax denominator, log sum_j exp(S_ij). */
static void one_row(int d, int w, int i, const double* qi, const double* k, const double* v,
                    const double* kl, const double* vl, double* s, double* oi, double* p,
                    double* lse)
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
    if (lse) *lse = m + log(sum);
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
 *   lse   optional [n_rows]: log sum_j exp(S_ij) of each row (natural log)
 * Returns 0, or -1 on a bad argument / allocation failure.
 */
int dar_oracle_rows(int T, int d, int dd, int w, const double* k, const double* v,
                    const double* wd, const double* wu, int n_rows, const int* pos,
                    const double* qr, double* o, double* p, double* lse)
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
                one_row(d, w, pos[r], qr + (size_t)r * d, k, v, kl, vl, s, o + (size_t)r * d, pr,
                        lse ? lse + r : NULL);
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
 *   o [B][Hq][T][d]; lse optional [B][Hq][T]: log sum_j exp(S_ij) of each row
 * nthreads > 0 sets the OpenMP thread count (0 keeps the default).
 */
int dar_oracle_prefill(int B, int Hq, int Hkv, int T, int d, int dd, int w, const double* q,
                       const double* k, const double* v, const double* wd, const double* wu,
                       double* o, double* lse, int nthreads)
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
                                 o + q_off, NULL, lse ? lse + ((size_t)b * Hq + h) * T : NULL);
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

/*
 * Backward of the causal prefill (the training setting of the paper's
 * Section 2.3, Eq. 5): gradients of L = sum(dO * O) with respect to Q, K, V,
 * W_down and W_up, by the chain rule applied to the definition above:
 *
 *   S_ij = q_i . key_ij / sqrt(d),  P_i = softmax_j(S_i),  O_i = sum_j P_ij val_ij
 *   with key_ij = k_j (i - j < w) or k'_j = (k_j W_down) W_up, and the same for
 *   val_ij (Eq. 3).
 *   dP_ij = dO_i . val_ij,  dS_ij = P_ij (dP_ij - sum_l P_il dP_il)
 *   dq_i = sum_j dS_ij key_ij / sqrt(d)
 *   window pairs:  dk_j += dS_ij q_i / sqrt(d),  dv_j += P_ij dO_i
 *   lifted pairs:  dk'_j += dS_ij q_i / sqrt(d),  dv'_j += P_ij dO_i, then
 *   through x' = (x W_down) W_up (Eq. 1-2):
 *     dx_j += dx'_j (W_down W_up)^T,
 *     dW_down += x_j^T (dx'_j W_up^T),  dW_up += (x_j W_down)^T dx'_j.
 *   Tied (wu NULL, W_up = W_down^T): dwd receives dW_down + dW_up^T and dwu
 *   is not written.
 *
 *   q, dout, dq [B][Hq][T][d]; k, v, dk, dv [B][Hkv][T][d];
 *   wd, dwd [Hkv][d][dd]; wu, dwu [Hkv][dd][d] (both NULL when tied).
 * dk, dv, dwd, dwu are overwritten (not accumulated into).
 * Returns 0, or -1 on a bad argument / allocation failure.
 */
int dar_oracle_backward(int B, int Hq, int Hkv, int T, int d, int dd, int w, const double* q,
                        const double* k, const double* v, const double* wd, const double* wu,
                        const double* dout, double* dq, double* dk, double* dv, double* dwd,
                        double* dwu, int nthreads)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || T < 1 || d < 1 || dd < 1 || w < 0)
        return -1;
    if ((wu == NULL) != (dwu == NULL)) return -1;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    const int group = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)d);
    const size_t wsz = (size_t)d * dd;
    /* per (b, g) partial weight gradients, summed over b afterwards in order */
    double* pwd = (double*)calloc((size_t)B * Hkv * wsz, sizeof(double));
    double* pwu = (double*)calloc((size_t)B * Hkv * wsz, sizeof(double));
    if (!pwd || !pwu) { free(pwd); free(pwu); return -1; }
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bg = 0; bg < B * Hkv; ++bg) {
        const int b = bg / Hkv, g = bg % Hkv;
        const double* kb = k + (size_t)bg * T * d;
        const double* vb = v + (size_t)bg * T * d;
        const double* wdg = wd + (size_t)g * wsz;
        const double* wug = wu ? wu + (size_t)g * wsz : NULL;
        double* dkb = dk + (size_t)bg * T * d;
        double* dvb = dv + (size_t)bg * T * d;
        double* kl = lift_all(T, d, dd, kb, wdg, wug);
        double* vl = lift_all(T, d, dd, vb, wdg, wug);
        double* dkl = (double*)calloc((size_t)T * d, sizeof(double));  /* dk'_j */
        double* dvl = (double*)calloc((size_t)T * d, sizeof(double));  /* dv'_j */
        double* p = (double*)malloc(sizeof(double) * (size_t)T);
        double* s = (double*)malloc(sizeof(double) * (size_t)T);
        double* dp = (double*)malloc(sizeof(double) * (size_t)T);
        double* oi = (double*)malloc(sizeof(double) * (size_t)d);
        if (!kl || !vl || !dkl || !dvl || !p || !s || !dp || !oi) {
#pragma omp atomic write
            bad = 1;
        } else {
            for (size_t x = 0; x < (size_t)T * d; ++x) { dkb[x] = 0.0; dvb[x] = 0.0; }
            for (int hh = 0; hh < group; ++hh) {
                const int h = g * group + hh;
                const double* qh = q + ((size_t)b * Hq + h) * T * d;
                const double* doh = dout + ((size_t)b * Hq + h) * T * d;
                double* dqh = dq + ((size_t)b * Hq + h) * T * d;
                for (int i = 0; i < T; ++i) {
                    const double* qi = qh + (size_t)i * d;
                    const double* doi = doh + (size_t)i * d;
                    one_row(d, w, i, qi, kb, vb, kl, vl, s, oi, p, NULL);
                    double delta = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        const double* val = (i - j < w) ? vb + (size_t)j * d : vl + (size_t)j * d;
                        double acc = 0.0;
                        for (int e = 0; e < d; ++e) acc += doi[e] * val[e];
                        dp[j] = acc;
                        delta += p[j] * acc;
                    }
                    double* dqi = dqh + (size_t)i * d;
                    for (int e = 0; e < d; ++e) dqi[e] = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        const double ds = p[j] * (dp[j] - delta);
                        const int local = i - j < w;
                        const double* key = local ? kb + (size_t)j * d : kl + (size_t)j * d;
                        double* dkey = local ? dkb + (size_t)j * d : dkl + (size_t)j * d;
                        double* dval = local ? dvb + (size_t)j * d : dvl + (size_t)j * d;
                        for (int e = 0; e < d; ++e) {
                            dqi[e] += ds * key[e] * scale;
                            dkey[e] += ds * qi[e] * scale;
                            dval[e] += p[j] * doi[e];
                        }
                    }
                }
            }
            /* through the lift x' = (x W_down) W_up, for keys and for values */
            double* pwdg = pwd + (size_t)bg * wsz;
            double* pwug = pwu + (size_t)bg * wsz;
            for (int which = 0; which < 2; ++which) {
                const double* xb = which ? vb : kb;
                const double* dxl = which ? dvl : dkl;
                double* dxb = which ? dvb : dkb;
                for (int j = 0; j < T; ++j) {
                    const double* xj = xb + (size_t)j * d;
                    const double* gj = dxl + (size_t)j * d;
                    for (int c = 0; c < dd; ++c) {
                        /* u_c = (dx'_j W_up^T)[c], h_c = (x_j W_down)[c] */
                        double u = 0.0, hc = 0.0;
                        for (int e = 0; e < d; ++e) {
                            const double wup = wug ? wug[(size_t)c * d + e] : wdg[(size_t)e * dd + c];
                            u += gj[e] * wup;
                            hc += xj[e] * wdg[(size_t)e * dd + c];
                        }
                        for (int e = 0; e < d; ++e) {
                            dxb[(size_t)j * d + e] += u * wdg[(size_t)e * dd + c];
                            pwdg[(size_t)e * dd + c] += xj[e] * u;
                            pwug[(size_t)c * d + e] += hc * gj[e];
                        }
                    }
                }
            }
        }
        free(kl); free(vl); free(dkl); free(dvl); free(p); free(s); free(dp); free(oi);
    }
    if (!bad) {
        for (int g = 0; g < Hkv; ++g) {
            double* dwdg = dwd + (size_t)g * wsz;
            double* dwug = dwu ? dwu + (size_t)g * wsz : NULL;
            for (size_t x = 0; x < wsz; ++x) {
                dwdg[x] = 0.0;
                if (dwug) dwug[x] = 0.0;
            }
            for (int b = 0; b < B; ++b) {
                const double* a = pwd + ((size_t)b * Hkv + g) * wsz;
                const double* u = pwu + ((size_t)b * Hkv + g) * wsz;
                for (int e = 0; e < d; ++e)
                    for (int c = 0; c < dd; ++c) {
                        dwdg[(size_t)e * dd + c] += a[(size_t)e * dd + c];
                        if (dwug) dwug[(size_t)c * d + e] += u[(size_t)c * d + e];
                        else dwdg[(size_t)e * dd + c] += u[(size_t)c * d + e];  /* tied: + dW_up^T */
                    }
            }
        }
    }
    free(pwd);
    free(pwu);
    return bad ? -1 : 0;
}

/*
 * Rotary position embedding inside Eq. 3 (the paper applies RoPE to the key
 * of both paths: to the token's own key in the window, and to the key
 * computed from the lifted representation beyond it; values are not
 * rotated, and the query is rotated at its own position as usual).
 *
 * Pairing: rotate-half (the GPT-NeoX convention of the Pythia models the
 * paper trains): for m < r/2 the pair (x[m], x[m + r/2]) of a row at
 * position p is turned by the angle p * base^(-2m/r); elements r..d-1 are
 * left unchanged (a partial rotary dimension, r < d, is allowed).
 *
 * out[t][.] = RoPE(x[t][.], pos[t]) for t < n. r even, 0 <= r <= d.
 */
void dar_oracle_rope(int n, int d, int r, double base, const int* pos, const double* x,
                     double* out)
{
    const int half = r / 2;
    for (int t = 0; t < n; ++t) {
        const double* xr = x + (size_t)t * d;
        double* yr = out + (size_t)t * d;
        for (int e = 0; e < d; ++e) yr[e] = xr[e];
        for (int m = 0; m < half; ++m) {
            const double ang = (double)pos[t] * pow(base, -2.0 * m / r);
            const double c = cos(ang), s = sin(ang);
            yr[m] = xr[m] * c - xr[m + half] * s;
            yr[m + half] = xr[m + half] * c + xr[m] * s;
        }
    }
}

/* The angle table: tab[p][m] = cos(p * base^(-2m/r)), tab[p][r/2 + m] = the
 * sine, for p < n_pos and m < r/2. */
void dar_oracle_rope_table(int r, double base, int n_pos, double* tab)
{
    const int half = r / 2;
    for (int p = 0; p < n_pos; ++p)
        for (int m = 0; m < half; ++m) {
            const double ang = (double)p * pow(base, -2.0 * m / r);
            tab[(size_t)p * r + m] = cos(ang);
            tab[(size_t)p * r + half + m] = sin(ang);
        }
}

/*
 * Query rows of one head with RoPE inside Eq. 3. Token j sits at position
 * pos0 + j; the query of row r at position pos0 + pos[r].
 *   window key    RoPE(k_j)                    value v_j
 *   distant key   RoPE((k_j W_down) W_up)      value (v_j W_down) W_up
 * Other arguments as for dar_oracle_rows (k, v, qr are un-rotated).
 */
int dar_oracle_rows_rope(int T, int d, int dd, int w, int r, double base, int pos0,
                         const double* k, const double* v, const double* wd, const double* wu,
                         int n_rows, const int* pos, const double* qr, double* o, double* lse)
{
    if (T < 1 || d < 1 || dd < 1 || w < 0 || n_rows < 0 || r < 0 || r > d || (r & 1) ||
        pos0 < 0 || !(base > 0.0))
        return -1;
    for (int i = 0; i < n_rows; ++i)
        if (pos[i] < 0 || pos[i] >= T) return -1;
    int* tpos = (int*)malloc(sizeof(int) * (size_t)T);
    int* qpos = (int*)malloc(sizeof(int) * (size_t)(n_rows > 0 ? n_rows : 1));
    double* kr = (double*)malloc(sizeof(double) * (size_t)T * d);
    double* klr = (double*)malloc(sizeof(double) * (size_t)T * d);
    double* qrr = (double*)malloc(sizeof(double) * (size_t)(n_rows > 0 ? n_rows : 1) * d);
    double* kl = lift_all(T, d, dd, k, wd, wu);
    double* vl = lift_all(T, d, dd, v, wd, wu);
    int bad = !tpos || !qpos || !kr || !klr || !qrr || !kl || !vl;
    if (!bad) {
        for (int j = 0; j < T; ++j) tpos[j] = pos0 + j;
        for (int i = 0; i < n_rows; ++i) qpos[i] = pos0 + pos[i];
        dar_oracle_rope(T, d, r, base, tpos, k, kr);      /* window keys */
        dar_oracle_rope(T, d, r, base, tpos, kl, klr);    /* distant keys, after the lift */
        dar_oracle_rope(n_rows, d, r, base, qpos, qr, qrr);
#pragma omp parallel
        {
            double* s = (double*)malloc(sizeof(double) * (size_t)T);
            if (!s) {
#pragma omp atomic write
                bad = 1;
            } else {
#pragma omp for schedule(dynamic, 4)
                for (int i = 0; i < n_rows; ++i)
                    one_row(d, w, pos[i], qrr + (size_t)i * d, kr, v, klr, vl, s,
                            o + (size_t)i * d, NULL, lse ? lse + i : NULL);
                free(s);
            }
        }
    }
    free(tpos);
    free(qpos);
    free(kr);
    free(klr);
    free(qrr);
    free(kl);
    free(vl);
    return bad ? -1 : 0;
}

/*
 * Backward of the causal prefill with RoPE inside Eq. 3 (Section 2.3 trains
 * through it): gradients of L = sum(dO * O) with respect to the un-rotated
 * q, k, v and W_down, W_up, for tokens at positions pos0 .. pos0+T-1.
 * With R_p the rotation of position p (an orthogonal map, R_p^T = R_{-p}):
 *
 *   query       qr_i = R_i q_i
 *   window      key kr_j = R_j k_j,                value v_j
 *   distant     key kd_j = R_j ((k_j W_down) W_up), value (v_j W_down) W_up
 *   S, P, dP, dS as for dar_oracle_backward, with these keys and values;
 *   dqr_i = sum_j dS_ij key_ij / sqrt(d),  dq_i = R_i^T dqr_i
 *   window pairs:  dkr_j += dS_ij qr_i / sqrt(d),  dv_j += P_ij dO_i
 *   distant pairs: dkd_j += dS_ij qr_i / sqrt(d),  dv'_j += P_ij dO_i
 *   dk_j += R_j^T dkr_j; the lifted key k'_j = (k_j W_down) W_up receives
 *   R_j^T dkd_j and the lifted value dv'_j, both taken back through the lift
 *   exactly as in dar_oracle_backward.
 * Arguments as for dar_oracle_backward, plus r (even, 0 <= r <= d), base > 0
 * and pos0 >= 0. With r = 0 the result is dar_oracle_backward's.
 */
int dar_oracle_backward_rope(int B, int Hq, int Hkv, int T, int d, int dd, int w, int r,
                             double base, int pos0, const double* q, const double* k,
                             const double* v, const double* wd, const double* wu,
                             const double* dout, double* dq, double* dk, double* dv, double* dwd,
                             double* dwu, int nthreads)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || T < 1 || d < 1 || dd < 1 || w < 0)
        return -1;
    if (r < 0 || r > d || (r & 1) || pos0 < 0 || !(base > 0.0)) return -1;
    if ((wu == NULL) != (dwu == NULL)) return -1;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    const int group = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)d);
    const size_t wsz = (size_t)d * dd;
    const size_t td = (size_t)T * d;
    double* pwd = (double*)calloc((size_t)B * Hkv * wsz, sizeof(double));
    double* pwu = (double*)calloc((size_t)B * Hkv * wsz, sizeof(double));
    int* tpos = (int*)malloc(sizeof(int) * (size_t)T);
    int* npos = (int*)malloc(sizeof(int) * (size_t)T);
    if (!pwd || !pwu || !tpos || !npos) {
        free(pwd); free(pwu); free(tpos); free(npos);
        return -1;
    }
    for (int j = 0; j < T; ++j) {
        tpos[j] = pos0 + j;
        npos[j] = -(pos0 + j);
    }
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bg = 0; bg < B * Hkv; ++bg) {
        const int b = bg / Hkv, g = bg % Hkv;
        const double* kb = k + (size_t)bg * td;
        const double* vb = v + (size_t)bg * td;
        const double* wdg = wd + (size_t)g * wsz;
        const double* wug = wu ? wu + (size_t)g * wsz : NULL;
        double* dkb = dk + (size_t)bg * td;
        double* dvb = dv + (size_t)bg * td;
        double* kl = lift_all(T, d, dd, kb, wdg, wug);
        double* vl = lift_all(T, d, dd, vb, wdg, wug);
        double* kr = (double*)malloc(sizeof(double) * td);     /* window keys R_j k_j */
        double* kdr = (double*)malloc(sizeof(double) * td);    /* distant keys R_j k'_j */
        double* qr = (double*)malloc(sizeof(double) * td);     /* one head's rotated queries */
        double* dqr = (double*)malloc(sizeof(double) * td);
        double* dkr = (double*)calloc(td, sizeof(double));     /* window key grads, rotated */
        double* dkd = (double*)calloc(td, sizeof(double));     /* distant key grads, rotated */
        double* dkl = (double*)malloc(sizeof(double) * td);    /* dk'_j = R_j^T dkd_j */
        double* dvl = (double*)calloc(td, sizeof(double));     /* dv'_j */
        double* p = (double*)malloc(sizeof(double) * (size_t)T);
        double* s = (double*)malloc(sizeof(double) * (size_t)T);
        double* dp = (double*)malloc(sizeof(double) * (size_t)T);
        double* oi = (double*)malloc(sizeof(double) * (size_t)d);
        if (!kl || !vl || !kr || !kdr || !qr || !dqr || !dkr || !dkd || !dkl || !dvl || !p || !s ||
            !dp || !oi) {
#pragma omp atomic write
            bad = 1;
        } else {
            dar_oracle_rope(T, d, r, base, tpos, kb, kr);
            dar_oracle_rope(T, d, r, base, tpos, kl, kdr);
            for (size_t x = 0; x < td; ++x) dvb[x] = 0.0;
            for (int hh = 0; hh < group; ++hh) {
                const int h = g * group + hh;
                const double* qh = q + ((size_t)b * Hq + h) * td;
                const double* doh = dout + ((size_t)b * Hq + h) * td;
                dar_oracle_rope(T, d, r, base, tpos, qh, qr);
                for (size_t x = 0; x < td; ++x) dqr[x] = 0.0;
                for (int i = 0; i < T; ++i) {
                    const double* qi = qr + (size_t)i * d;
                    const double* doi = doh + (size_t)i * d;
                    one_row(d, w, i, qi, kr, vb, kdr, vl, s, oi, p, NULL);
                    double delta = 0.0;
                    for (int j = 0; j <= i; ++j) {
                        const double* val = (i - j < w) ? vb + (size_t)j * d : vl + (size_t)j * d;
                        double acc = 0.0;
                        for (int e = 0; e < d; ++e) acc += doi[e] * val[e];
                        dp[j] = acc;
                        delta += p[j] * acc;
                    }
                    double* dqi = dqr + (size_t)i * d;
                    for (int j = 0; j <= i; ++j) {
                        const double ds = p[j] * (dp[j] - delta);
                        const int local = i - j < w;
                        const double* key = local ? kr + (size_t)j * d : kdr + (size_t)j * d;
                        double* dkey = local ? dkr + (size_t)j * d : dkd + (size_t)j * d;
                        double* dval = local ? dvb + (size_t)j * d : dvl + (size_t)j * d;
                        for (int e = 0; e < d; ++e) {
                            dqi[e] += ds * key[e] * scale;
                            dkey[e] += ds * qi[e] * scale;
                            dval[e] += p[j] * doi[e];
                        }
                    }
                }
                /* dq = R^T dqr */
                dar_oracle_rope(T, d, r, base, npos, dqr, dq + ((size_t)b * Hq + h) * td);
            }
            /* window keys: dk = R^T dkr; distant keys: dk' = R^T dkd */
            dar_oracle_rope(T, d, r, base, npos, dkr, dkb);
            dar_oracle_rope(T, d, r, base, npos, dkd, dkl);
            /* through the lift x' = (x W_down) W_up, for keys and for values */
            double* pwdg = pwd + (size_t)bg * wsz;
            double* pwug = pwu + (size_t)bg * wsz;
            for (int which = 0; which < 2; ++which) {
                const double* xb = which ? vb : kb;
                const double* dxl = which ? dvl : dkl;
                double* dxb = which ? dvb : dkb;
                for (int j = 0; j < T; ++j) {
                    const double* xj = xb + (size_t)j * d;
                    const double* gj = dxl + (size_t)j * d;
                    for (int c = 0; c < dd; ++c) {
                        double u = 0.0, hc = 0.0;
                        for (int e = 0; e < d; ++e) {
                            const double wup = wug ? wug[(size_t)c * d + e] : wdg[(size_t)e * dd + c];
                            u += gj[e] * wup;
                            hc += xj[e] * wdg[(size_t)e * dd + c];
                        }
                        for (int e = 0; e < d; ++e) {
                            dxb[(size_t)j * d + e] += u * wdg[(size_t)e * dd + c];
                            pwdg[(size_t)e * dd + c] += xj[e] * u;
                            pwug[(size_t)c * d + e] += hc * gj[e];
                        }
                    }
                }
            }
        }
        free(kl); free(vl); free(kr); free(kdr); free(qr); free(dqr); free(dkr); free(dkd);
        free(dkl); free(dvl); free(p); free(s); free(dp); free(oi);
    }
    if (!bad) {
        for (int g = 0; g < Hkv; ++g) {
            double* dwdg = dwd + (size_t)g * wsz;
            double* dwug = dwu ? dwu + (size_t)g * wsz : NULL;
            for (size_t x = 0; x < wsz; ++x) {
                dwdg[x] = 0.0;
                if (dwug) dwug[x] = 0.0;
            }
            for (int b = 0; b < B; ++b) {
                const double* a = pwd + ((size_t)b * Hkv + g) * wsz;
                const double* u = pwu + ((size_t)b * Hkv + g) * wsz;
                for (int e = 0; e < d; ++e)
                    for (int c = 0; c < dd; ++c) {
                        dwdg[(size_t)e * dd + c] += a[(size_t)e * dd + c];
                        if (dwug) dwug[(size_t)c * d + e] += u[(size_t)c * d + e];
                        else dwdg[(size_t)e * dd + c] += u[(size_t)c * d + e];
                    }
            }
        }
    }
    free(pwd);
    free(pwu);
    free(tpos);
    free(npos);
    return bad ? -1 : 0;
}

/* Causal prefill with RoPE inside Eq. 3: positions pos0 .. pos0+T-1.
 * Shapes as for dar_oracle_prefill. */
int dar_oracle_prefill_rope(int B, int Hq, int Hkv, int T, int d, int dd, int w, int r,
                            double base, int pos0, const double* q, const double* k,
                            const double* v, const double* wd, const double* wu, double* o,
                            double* lse, int nthreads)
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
            rc = dar_oracle_rows_rope(T, d, dd, w, r, base, pos0, k + kv_off, v + kv_off,
                                      wd + (size_t)g * d * dd, wu ? wu + (size_t)g * dd * d : NULL,
                                      T, pos, q + q_off, o + q_off,
                                      lse ? lse + ((size_t)b * Hq + h) * T : NULL);
        }
    free(pos);
    return rc;
}

/*
 * Single shared latent (the cache the Limitations section proposes: one
 * d_down vector per token, from which both the key and the value of the
 * distant path are computed). With the latent c_j = h_j W_down of Eq. 1 and
 * the lift of Eq. 2 followed by the key and value projections, the distant
 * key is c_j (W_up W_K) and the distant value c_j (W_up W_V); per KV head
 * these products are the matrices U_K, U_V [d_down][d]. The latent is an
 * input here (a projection of the hidden state, like q, k, v).
 *
 * Query rows of one head:
 *   window (i - j < w)   key k_j,        value v_j
 *   distant              key c_j U_K,    value c_j U_V
 * c [T][dd], uk, uv [dd][d]; other arguments as for dar_oracle_rows.
 */
int dar_oracle_rows_shared(int T, int d, int dd, int w, const double* k, const double* v,
                           const double* c, const double* uk, const double* uv, int n_rows,
                           const int* pos, const double* qr, double* o, double* lse)
{
    if (T < 1 || d < 1 || dd < 1 || w < 0 || n_rows < 0) return -1;
    for (int i = 0; i < n_rows; ++i)
        if (pos[i] < 0 || pos[i] >= T) return -1;
    double* kl = (double*)malloc(sizeof(double) * (size_t)T * d);
    double* vl = (double*)malloc(sizeof(double) * (size_t)T * d);
    int bad = !kl || !vl;
    if (!bad) {
        /* Eq. 2 with the key / value projection folded in: x'_j = c_j U */
        for (int j = 0; j < T; ++j)
            for (int e = 0; e < d; ++e) {
                double ak = 0.0, av = 0.0;
                for (int cc = 0; cc < dd; ++cc) {
                    ak += c[(size_t)j * dd + cc] * uk[(size_t)cc * d + e];
                    av += c[(size_t)j * dd + cc] * uv[(size_t)cc * d + e];
                }
                kl[(size_t)j * d + e] = ak;
                vl[(size_t)j * d + e] = av;
            }
#pragma omp parallel
        {
            double* s = (double*)malloc(sizeof(double) * (size_t)T);
            if (!s) {
#pragma omp atomic write
                bad = 1;
            } else {
#pragma omp for schedule(dynamic, 4)
                for (int i = 0; i < n_rows; ++i)
                    one_row(d, w, pos[i], qr + (size_t)i * d, k, v, kl, vl, s, o + (size_t)i * d,
                            NULL, lse ? lse + i : NULL);
                free(s);
            }
        }
    }
    free(kl);
    free(vl);
    return bad ? -1 : 0;
}

/* Causal prefill with the shared latent: q [B][Hq][T][d], k, v [B][Hkv][T][d],
 * c [B][Hkv][T][dd], uk, uv [Hkv][dd][d], o [B][Hq][T][d], lse optional. */
int dar_oracle_prefill_shared(int B, int Hq, int Hkv, int T, int d, int dd, int w,
                              const double* q, const double* k, const double* v, const double* c,
                              const double* uk, const double* uv, double* o, double* lse,
                              int nthreads)
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
            const size_t c_off = ((size_t)b * Hkv + g) * (size_t)T * dd;
            const size_t q_off = ((size_t)b * Hq + h) * (size_t)T * d;
            rc = dar_oracle_rows_shared(T, d, dd, w, k + kv_off, v + kv_off, c + c_off,
                                        uk + (size_t)g * dd * d, uv + (size_t)g * dd * d, T, pos,
                                        q + q_off, o + q_off,
                                        lse ? lse + ((size_t)b * Hq + h) * T : NULL);
        }
    free(pos);
    return rc;
}
