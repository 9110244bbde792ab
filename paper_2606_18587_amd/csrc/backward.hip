// Backward of the causal DAR prefill on the vector ALUs (every shape and
// dtype), plus the preparation and weight-gradient kernels that the
// matrix-core backward shares.
//
// For L = sum(dO * O) (the training objective's attention part, Section 2.3)
// with S_ij = q_i . key_ij / sqrt(d), P = softmax(S) row by row and
// dP_ij = dO_i . val_ij, the softmax Jacobian gives
//   dS_ij = P_ij (dP_ij - delta_i),  delta_i = sum_j P_ij dP_ij = dO_i . O_i.
// Window pairs (i - j < w) use the token itself; distant pairs use the lifted
// token x' = (x W_down) W_up (Eq. 1-3), and all their products stay in d_down
// space through the absorption of W_up:
//   distant score  q_i . k'_j = q~_i . c^K_j        q~ = q W_up^T
//   distant dP     dO_i . v'_j = dO~_i . c^V_j       dO~ = dO W_up^T
//   dq_i  = s (sum_win dS_ij k_j + h_i W_up),        h_i = sum_dist dS_ij c^K_j
//   dk_j  = s (sum_win dS_ij q_i + gK_j W_down^T),   gK_j = sum_dist dS_ij q~_i
//   dv_j  = sum_win P_ij dO_i + gV_j W_down^T,       gV_j = sum_dist P_ij dO~_i
//   dW_down = sum_j (k_j^T s gK_j + v_j^T gV_j)
//   dW_up   = sum_i (s h_i^T q_i + ol_i^T dO_i),     ol_i = sum_dist P_ij c^V_j
// (s = 1/sqrt(d)); tied W_up = W_down^T receives dW_down + dW_up^T. Only
// pairs whose query takes the distant path reach the bottleneck weights,
// which is how the paper describes their training.
//
// The softmax statistics are not recomputed: each row's log-sum-exp comes
// from the forward call.
//
// Kernels, in launch order:
//   bwd_latent_kernel   c^K, c^V for every token (fp32)
//   bwd_rowprep_kernel  q~, dO~ and delta for every query row
//   bwd_rows_valu_kernel   one wave per query row: dq, h, ol
//   bwd_cols_valu_kernel   one wave per key: dk, dv, gK, gV
//   bwd_wpart_kernel / bwd_wreduce_kernel  weight gradients, split over row
//                          chunks then summed in a fixed order (deterministic)
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

namespace {
constexpr float kLog2e = 1.4426950408889634f;
}

BwdWs bwd_ws_layout(int B, int Hq, int Hkv, int T, int d, int dd, bool mfma) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    BwdWs L{};
    // token counts padded to a multiple of 64 (the matrix-core path reads whole
    // 64-token tiles and keeps two bf16 arrays where this path keeps one fp32)
    const size_t Tr = (size_t)round_up(T, 64);
    const size_t rows = (size_t)B * Hq * Tr;
    const size_t toks = (size_t)B * Hkv * Tr;
    // operand arrays: fp32 [n][dd] here; on the matrix-core path bf16 [n][dd]
    // followed by the transposed 32-token blocks padded to 32 latent rows
    const size_t opw = mfma ? (size_t)(dd + 32) * 2 : (size_t)dd * 4;
    size_t off = 0;
    L.lse_off = off;   off += al(rows * 4);
    L.delta_off = off; off += al(rows * 4);
    L.qt_off = off;    off += al(rows * opw);
    L.dot_off = off;   off += al(rows * opw);
    L.rc_off = off;    off += mfma ? al(rows * 16 * 2) : 0;
    L.hk_off = off;    off += al(rows * dd * 4);
    L.ol_off = off;    off += al(rows * dd * 4);
    L.ck_off = off;    off += al(toks * opw);
    L.cv_off = off;    off += al(toks * opw);
    L.gk_off = off;    off += al(toks * dd * 4);
    L.gv_off = off;    off += al(toks * dd * 4);
    const int G = Hq / Hkv;
    if (mfma) {  // one share per workgroup of 128 keys / 128 query rows
        const int nblk = (T + 127) / 128;
        L.nchunk_d = B * nblk;
        L.nchunk_u = B * G * nblk;
    } else {
        L.nchunk_d = bwd_nchunk((long long)B * T);
        L.nchunk_u = bwd_nchunk((long long)B * G * T);
    }
    L.nchunk = L.nchunk_d > L.nchunk_u ? L.nchunk_d : L.nchunk_u;
    L.wpart_off = off; off += al((size_t)2 * Hkv * L.nchunk * d * dd * 4);
    L.bytes = off;
    return L;
}

// ---------------------------------------------------------------- preparation

// c^K_j = k_j W_down and c^V_j = v_j W_down (Eq. 1) in fp32, one thread per
// (token, column). Grid: (ceil(T * dd / 256), B * Hkv).
template <typename T>
__global__ __launch_bounds__(256) void bwd_latent_kernel(const T* __restrict__ k,
                                                         const T* __restrict__ v,
                                                         const T* __restrict__ wd,
                                                         float* __restrict__ ck,
                                                         float* __restrict__ cv, int Hkv, int T_,
                                                         int d, int dd) {
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    const long long idx = (long long)wg_id_x() * 256 + lane_id_x();
    if (idx >= (long long)T_ * dd) return;
    const int j = (int)(idx / dd), c = (int)(idx % dd);
    const size_t row = (size_t)bg * T_ + j;
    const T* wdg = wd + (size_t)g * d * dd;
    ck[row * dd + c] = project_col(k + row * d, wdg, d, dd, c);
    cv[row * dd + c] = project_col(v + row * d, wdg, d, dd, c);
}

// Per query row: q~ = q W_up^T and dO~ = dO W_up^T (unscaled, fp32) and
// delta = dO . O. One wave per (row, batch * query head).
template <typename T>
__global__ __launch_bounds__(64) void bwd_rowprep_kernel(
    const T* __restrict__ q, const T* __restrict__ o, const T* __restrict__ dout,
    const T* __restrict__ wd, const T* __restrict__ wu, float* __restrict__ qt,
    float* __restrict__ dot, float* __restrict__ delta, int Hq, int Hkv, int T_, int d, int dd) {
    const int lane = lane_id_x();
    const int i = wg_id_x();
    const int bh = wg_id_y();
    const int g = (bh % Hq) / (Hq / Hkv);
    const size_t row = (size_t)bh * T_ + i;
    const T* qr = q + row * d;
    const T* orow = o + row * d;
    const T* dr = dout + row * d;
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    float dl = 0.f;
    for (int e = lane; e < d; e += 64)
        dl = __builtin_fmaf(elem<T>::load(dr + e), elem<T>::load(orow + e), dl);
    dl = wave_sum(dl);
    if (lane == 0) delta[row] = dl;
    for (int c = lane; c < dd; c += 64) {
        float aq = 0.f, ad = 0.f;
        for (int e = 0; e < d; ++e) {
            const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                : elem<T>::load(wdg + (size_t)e * dd + c);
            aq = __builtin_fmaf(elem<T>::load(qr + e), u, aq);
            ad = __builtin_fmaf(elem<T>::load(dr + e), u, ad);
        }
        qt[row * dd + c] = aq;
        dot[row * dd + c] = ad;
    }
}

// ---------------------------------------------------------------- rows (dq)

// One wave per query row i of one (batch, query head): recomputes P of the
// single softmax (Eq. 4) from the forward's log-sum-exp, forms dP and dS and
// accumulates dq (window keys, d wide), h = sum dS c^K and ol = sum P c^V
// (distant keys, d_down wide). Scores are kept in the log2 domain
// (log2(e) / sqrt(d) folded into the query).
template <typename T>
__global__ __launch_bounds__(64) void bwd_rows_valu_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const T* __restrict__ wd, const T* __restrict__ wu,
    const float* __restrict__ ck, const float* __restrict__ cv, const float* __restrict__ qt,
    const float* __restrict__ dot, const float* __restrict__ delta, const float* __restrict__ lse,
    float* __restrict__ hk, float* __restrict__ ol, T* __restrict__ dq, int Hq, int Hkv, int T_,
    int d, int dd, int w, float scale) {
    __shared__ float qs[256];
    __shared__ float dos[256];
    __shared__ float qts[256];
    __shared__ float dots[256];
    __shared__ float hs[256];
    __shared__ float ps[64];
    __shared__ float dss[64];
    const int lane = lane_id_x();
    const int i = (T_ - 1) - wg_id_x();  // longest rows first
    const int bh = wg_id_y();
    const int b = bh / Hq, h = bh % Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    const size_t row = (size_t)bh * T_ + i;
    const float qscale = scale * kLog2e;
    for (int e = lane; e < d; e += 64) {
        qs[e] = elem<T>::load(q + row * d + e) * qscale;
        dos[e] = elem<T>::load(dout + row * d + e);
    }
    for (int c = lane; c < dd; c += 64) {
        qts[c] = qt[row * dd + c] * qscale;
        dots[c] = dot[row * dd + c];
    }
    __syncthreads();
    const float dl = delta[row];
    const int n_dist = imax(0, i - w + 1);  // distant keys j in [0, i - w]
    const float* ckg = ck + (size_t)bg * T_ * dd;
    const float* cvg = cv + (size_t)bg * T_ * dd;
    const T* kg = k + (size_t)bg * T_ * d;
    const T* vg = v + (size_t)bg * T_ * d;

    auto score = [&](int j) -> float {  // log2-domain score of key j (j <= i)
        float acc = 0.f;
        if (j < n_dist) {
            for (int c = 0; c < dd; ++c) acc = __builtin_fmaf(qts[c], ckg[(size_t)j * dd + c], acc);
        } else {
            for (int e = 0; e < d; ++e)
                acc = __builtin_fmaf(qs[e], elem<T>::load(kg + (size_t)j * d + e), acc);
        }
        return acc;
    };

    const float L2 = lse[row] * kLog2e;  // the forward's log-sum-exp, log2 units

    // gradients
    float dql[4] = {0.f, 0.f, 0.f, 0.f};
    float ha[4] = {0.f, 0.f, 0.f, 0.f};
    float oa[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 <= i; j0 += 64) {
        const int j = j0 + lane;
        float p = 0.f, ds = 0.f;
        if (j <= i) {
            p = exp2f(score(j) - L2);
            float dp = 0.f;
            if (j < n_dist) {
                for (int c = 0; c < dd; ++c)
                    dp = __builtin_fmaf(dots[c], cvg[(size_t)j * dd + c], dp);
            } else {
                for (int e = 0; e < d; ++e)
                    dp = __builtin_fmaf(dos[e], elem<T>::load(vg + (size_t)j * d + e), dp);
            }
            ds = p * (dp - dl);
        }
        ps[lane] = p;
        dss[lane] = ds;
        __syncthreads();
        const int cnt = imin(64, i + 1 - j0);
        for (int jj = 0; jj < cnt; ++jj) {
            const int jx = j0 + jj;
            const float pj = ps[jj], dsj = dss[jj];
            if (jx < n_dist) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int c = lane + 64 * r;
                    if (c < dd) {
                        ha[r] = __builtin_fmaf(dsj, ckg[(size_t)jx * dd + c], ha[r]);
                        oa[r] = __builtin_fmaf(pj, cvg[(size_t)jx * dd + c], oa[r]);
                    }
                }
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int e = lane + 64 * r;
                    if (e < d) dql[r] = __builtin_fmaf(dsj, elem<T>::load(kg + (size_t)jx * d + e),
                                                       dql[r]);
                }
            }
        }
        __syncthreads();
    }

    // dq = s (dq_win + h W_up); h and ol go to the workspace for dW_up
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int c = lane + 64 * r;
        if (c < dd) {
            hs[c] = ha[r];
            hk[row * dd + c] = ha[r];
            ol[row * dd + c] = oa[r];
        }
    }
    __syncthreads();
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int e = lane + 64 * r;
        if (e < d) {
            float acc = dql[r];
            if (n_dist > 0)
                for (int c = 0; c < dd; ++c) {
                    const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                        : elem<T>::load(wdg + (size_t)e * dd + c);
                    acc = __builtin_fmaf(hs[c], u, acc);
                }
            dq[row * d + e] = elem<T>::from_f32(acc * scale);
        }
    }
}

// ---------------------------------------------------------------- columns (dk, dv)

// One wave per key j of one (batch, KV head): loops over the query heads of
// the group and over the rows that see key j, window rows j <= i < j + w at
// full d and distant rows i >= j + w in d_down space.
template <typename T>
__global__ __launch_bounds__(64) void bwd_cols_valu_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const T* __restrict__ wd, const float* __restrict__ ck,
    const float* __restrict__ cv, const float* __restrict__ qt, const float* __restrict__ dot,
    const float* __restrict__ delta, const float* __restrict__ lse, float* __restrict__ gk,
    float* __restrict__ gv, T* __restrict__ dk, T* __restrict__ dv, int Hq, int Hkv, int T_,
    int d, int dd, int w, float scale) {
    __shared__ float ks[256];
    __shared__ float vs[256];
    __shared__ float cks[256];
    __shared__ float cvs[256];
    __shared__ float gks[256];
    __shared__ float gvs[256];
    __shared__ float ps[64];
    __shared__ float dss[64];
    const int lane = lane_id_x();
    const int j = wg_id_x();
    const int bg = wg_id_y();
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const size_t tok = (size_t)bg * T_ + j;
    const float qscale = scale * kLog2e;
    for (int e = lane; e < d; e += 64) {
        ks[e] = elem<T>::load(k + tok * d + e) * qscale;
        vs[e] = elem<T>::load(v + tok * d + e);
    }
    for (int c = lane; c < dd; c += 64) {
        cks[c] = ck[tok * dd + c] * qscale;
        cvs[c] = cv[tok * dd + c];
    }
    __syncthreads();
    float dka[4] = {0.f, 0.f, 0.f, 0.f};
    float dva[4] = {0.f, 0.f, 0.f, 0.f};
    float gka[4] = {0.f, 0.f, 0.f, 0.f};
    float gva[4] = {0.f, 0.f, 0.f, 0.f};
    const int i_far = j + w;  // first distant row (may exceed T - 1)
    for (int hh = 0; hh < G; ++hh) {
        const size_t bh = (size_t)b * Hq + g * G + hh;
        const T* qh = q + bh * T_ * d;
        const T* dh = dout + bh * T_ * d;
        const float* qth = qt + bh * T_ * dd;
        const float* dth = dot + bh * T_ * dd;
        const float* lh = lse + bh * T_;
        const float* delh = delta + bh * T_;
        for (int i0 = j; i0 < T_; i0 += 64) {
            const int i = i0 + lane;
            float p = 0.f, ds = 0.f;
            if (i < T_) {
                float s = 0.f, dp = 0.f;
                if (i >= i_far) {
                    for (int c = 0; c < dd; ++c) {
                        s = __builtin_fmaf(qth[(size_t)i * dd + c], cks[c], s);
                        dp = __builtin_fmaf(dth[(size_t)i * dd + c], cvs[c], dp);
                    }
                } else {
                    for (int e = 0; e < d; ++e) {
                        s = __builtin_fmaf(elem<T>::load(qh + (size_t)i * d + e), ks[e], s);
                        dp = __builtin_fmaf(elem<T>::load(dh + (size_t)i * d + e), vs[e], dp);
                    }
                }
                p = exp2f(s - lh[i] * kLog2e);
                ds = p * (dp - delh[i]);
            }
            ps[lane] = p;
            dss[lane] = ds;
            __syncthreads();
            const int cnt = imin(64, T_ - i0);
            for (int ii = 0; ii < cnt; ++ii) {
                const int ix = i0 + ii;
                const float pi = ps[ii], dsi = dss[ii];
                if (ix >= i_far) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int c = lane + 64 * r;
                        if (c < dd) {
                            gka[r] = __builtin_fmaf(dsi, qth[(size_t)ix * dd + c], gka[r]);
                            gva[r] = __builtin_fmaf(pi, dth[(size_t)ix * dd + c], gva[r]);
                        }
                    }
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int e = lane + 64 * r;
                        if (e < d) {
                            dka[r] = __builtin_fmaf(dsi, elem<T>::load(qh + (size_t)ix * d + e),
                                                    dka[r]);
                            dva[r] = __builtin_fmaf(pi, elem<T>::load(dh + (size_t)ix * d + e),
                                                    dva[r]);
                        }
                    }
                }
            }
            __syncthreads();
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int c = lane + 64 * r;
        if (c < dd) {
            gks[c] = gka[r];
            gvs[c] = gva[r];
            gk[tok * dd + c] = gka[r];
            gv[tok * dd + c] = gva[r];
        }
    }
    __syncthreads();
    const T* wdg = wd + (size_t)g * d * dd;
    const bool any_far = i_far < T_;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int e = lane + 64 * r;
        if (e < d) {
            float ak = dka[r], av = dva[r];
            if (any_far)
                for (int c = 0; c < dd; ++c) {
                    const float u = elem<T>::load(wdg + (size_t)e * dd + c);
                    ak = __builtin_fmaf(gks[c], u, ak);
                    av = __builtin_fmaf(gvs[c], u, av);
                }
            dk[tok * d + e] = elem<T>::from_f32(ak * scale);
            dv[tok * d + e] = elem<T>::from_f32(av);
        }
    }
}

// ---------------------------------------------------------------- weights

// Partial weight gradients over one chunk of rows, stored [e][c] (d x dd):
//   z = 0: rows (b, j) of KV head g,  sum k_e (s gK_c) + v_e gV_c   -> dW_down
//   z = 1: rows (b, h, i), h in g,    sum q_e (s h_c) + dO_e ol_c   -> dW_up^T
// Grid: (nchunk, Hkv, 2), 256 threads, each owning outputs tid + 256 u.
template <typename T>
__global__ __launch_bounds__(256) void bwd_wpart_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ gk, const float* __restrict__ gv,
    const float* __restrict__ hk, const float* __restrict__ ol, float* __restrict__ part, int B,
    int Hq, int Hkv, int T_, int d, int dd, int nchunk_d, int nchunk_u, int nchunk, float scale) {
    const int chunk = wg_id_x(), g = wg_id_y(), z = wg_id_z();
    const int G = Hq / Hkv;
    const long long rows = z == 0 ? (long long)B * T_ : (long long)B * G * T_;
    const int nch = z == 0 ? nchunk_d : nchunk_u;
    if (chunk >= nch) return;
    const long long per = (rows + nch - 1) / nch;
    const long long r0 = (long long)chunk * per;
    const long long r1 = r0 + per < rows ? r0 + per : rows;
    float* out = part + (((size_t)z * Hkv + g) * nchunk + chunk) * (size_t)d * dd;
    const int n_out = d * dd;
    for (int o0 = 0; o0 < n_out; o0 += 256 * 8) {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (long long r = r0; r < r1; ++r) {
            size_t xrow, yrow;
            const T *x1, *x2;
            const float *y1, *y2;
            if (z == 0) {
                const long long b = r / T_, j = r % T_;
                xrow = ((size_t)b * Hkv + g) * T_ + j;
                yrow = xrow;
                x1 = k; x2 = v; y1 = gk; y2 = gv;
            } else {
                const long long b = r / ((long long)G * T_), rem = r % ((long long)G * T_);
                const long long hh = rem / T_, i = rem % T_;
                xrow = ((size_t)b * Hq + g * G + hh) * T_ + i;
                yrow = xrow;
                x1 = q; x2 = dout; y1 = hk; y2 = ol;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int o = o0 + lane_id_x() + 256 * u;
                if (o < n_out) {
                    const int e = o / dd, c = o % dd;
                    const float a = elem<T>::load(x1 + xrow * d + e) * (y1[yrow * dd + c] * scale);
                    acc[u] = __builtin_fmaf(elem<T>::load(x2 + xrow * d + e), y2[yrow * dd + c],
                                            acc[u] + a);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int o = o0 + lane_id_x() + 256 * u;
            if (o < n_out) out[o] = acc[u];
        }
    }
}

// Sum of the chunk partials; tied: dw_down = dW_down + dW_up^T. A workgroup
// takes 16 outputs of one KV head; its 16 thread groups each sum every 16th
// chunk in chunk order, and the 16 sums are added in group order, so the
// result is the same on every run. Grid: (ceil(d * dd / 16), Hkv).
__global__ __launch_bounds__(256) void bwd_wreduce_kernel(const float* __restrict__ part,
                                                          float* __restrict__ dwd,
                                                          float* __restrict__ dwu, int Hkv,
                                                          int d, int dd, int nchunk_d,
                                                          int nchunk_u, int nchunk) {
    __shared__ float red[2][16][16];
    const int g = wg_id_y();
    const int ol = lane_id_x() & 15, grp = lane_id_x() >> 4;
    const int o = wg_id_x() * 16 + ol;
    const int n_out = d * dd;
    float sd = 0.f, su = 0.f;
    if (o < n_out) {
        const float* pd = part + ((size_t)g * nchunk) * n_out + o;
        const float* pu = part + ((size_t)(Hkv + g) * nchunk) * n_out + o;
        // independent loads first, then the sums in chunk order
        constexpr int U = 8;
        for (int c0 = grp; c0 < nchunk_d; c0 += 16 * U) {
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = c0 + 16 * u;
                x[u] = c < nchunk_d ? pd[(size_t)c * n_out] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) sd += x[u];
        }
        for (int c0 = grp; c0 < nchunk_u; c0 += 16 * U) {
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = c0 + 16 * u;
                x[u] = c < nchunk_u ? pu[(size_t)c * n_out] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) su += x[u];
        }
    }
    red[0][grp][ol] = sd;
    red[1][grp][ol] = su;
    __syncthreads();
    if (grp != 0 || o >= n_out) return;
    sd = 0.f;
    su = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        sd += red[0][k][ol];
        su += red[1][k][ol];
    }
    const int e = o / dd, c = o % dd;
    if (dwu) {
        dwd[(size_t)g * n_out + o] = sd;
        dwu[(size_t)g * n_out + (size_t)c * d + e] = su;
    } else {
        dwd[(size_t)g * n_out + o] = sd + su;
    }
}

hipError_t launch_bwd_wreduce(const float* part, float* dwd, float* dwu, int Hkv, int d, int dd,
                              const BwdWs& L, hipStream_t st) {
    hipLaunchKernelGGL(bwd_wreduce_kernel, dim3((d * dd + 15) / 16, Hkv), dim3(256), 0, st, part,
                       dwd, dwu, Hkv, d, dd, L.nchunk_d, L.nchunk_u, L.nchunk);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_prep(const T* q, const T* k, const T* v, const T* o, const T* dout,
                           const T* wd, const T* wu, float* ck, float* cv, float* qt, float* dot,
                           float* delta, int B, int Hq, int Hkv, int T_, int d, int dd,
                           hipStream_t st) {
    const long long n = (long long)T_ * dd;
    hipLaunchKernelGGL(bwd_latent_kernel<T>, dim3((unsigned)((n + 255) / 256), B * Hkv),
                       dim3(256), 0, st, k, v, wd, ck, cv, Hkv, T_, d, dd);
    hipLaunchKernelGGL(bwd_rowprep_kernel<T>, dim3(T_, B * Hq), dim3(64), 0, st, q, o, dout, wd,
                       wu, qt, dot, delta, Hq, Hkv, T_, d, dd);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_weights(const T* q, const T* k, const T* v, const T* dout, const float* gk,
                              const float* gv, const float* hk, const float* ol, float* part,
                              float* dwd, float* dwu, int B, int Hq, int Hkv, int T_, int d,
                              int dd, const BwdWs& L, hipStream_t st) {
    const float scale = 1.f / sqrtf((float)d);
    hipLaunchKernelGGL(bwd_wpart_kernel<T>, dim3(L.nchunk, Hkv, 2), dim3(256), 0, st, q, k, v,
                       dout, gk, gv, hk, ol, part, B, Hq, Hkv, T_, d, dd, L.nchunk_d, L.nchunk_u,
                       L.nchunk, scale);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bwd_wreduce(part, dwd, dwu, Hkv, d, dd, L, st);
}

template <typename T>
hipError_t launch_bwd_valu(const T* q, const T* k, const T* v, const T* o, const float* lse,
                           const T* dout, const T* wd, const T* wu, T* dq, T* dk, T* dv,
                           float* dwd, float* dwu, char* ws, const BwdWs& L, int B, int Hq,
                           int Hkv, int T_, int d, int dd, int w, hipStream_t st) {
    float* delta = (float*)(ws + L.delta_off);
    float* qt = (float*)(ws + L.qt_off);
    float* dot = (float*)(ws + L.dot_off);
    float* hk = (float*)(ws + L.hk_off);
    float* ol = (float*)(ws + L.ol_off);
    float* ck = (float*)(ws + L.ck_off);
    float* cv = (float*)(ws + L.cv_off);
    float* gk = (float*)(ws + L.gk_off);
    float* gv = (float*)(ws + L.gv_off);
    float* part = (float*)(ws + L.wpart_off);
    const float scale = 1.f / sqrtf((float)d);
    hipError_t e = launch_bwd_prep<T>(q, k, v, o, dout, wd, wu, ck, cv, qt, dot, delta, B, Hq,
                                      Hkv, T_, d, dd, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_rows_valu_kernel<T>, dim3(T_, B * Hq), dim3(64), 0, st, q, k, v, dout,
                       wd, wu, (const float*)ck, (const float*)cv, (const float*)qt,
                       (const float*)dot, (const float*)delta, lse, hk, ol, dq, Hq, Hkv, T_, d,
                       dd, w, scale);
    hipLaunchKernelGGL(bwd_cols_valu_kernel<T>, dim3(T_, B * Hkv), dim3(64), 0, st, q, k, v, dout,
                       wd, (const float*)ck, (const float*)cv, (const float*)qt,
                       (const float*)dot, (const float*)delta, (const float*)lse, gk, gv, dk, dv,
                       Hq, Hkv, T_, d, dd, w, scale);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bwd_weights<T>(q, k, v, dout, gk, gv, hk, ol, part, dwd, dwu, B, Hq, Hkv, T_, d,
                                 dd, L, st);
}

#define DAR_BWD_INST(T)                                                                         \
    template hipError_t launch_bwd_prep<T>(const T*, const T*, const T*, const T*, const T*,   \
                                           const T*, const T*, float*, float*, float*, float*, \
                                           float*, int, int, int, int, int, int, hipStream_t); \
    template hipError_t launch_bwd_weights<T>(const T*, const T*, const T*, const T*,          \
                                              const float*, const float*, const float*,        \
                                              const float*, float*, float*, float*, int, int,  \
                                              int, int, int, int, const BwdWs&, hipStream_t);  \
    template hipError_t launch_bwd_valu<T>(const T*, const T*, const T*, const T*,             \
                                           const float*, const T*, const T*, const T*, T*, T*, \
                                           T*, float*, float*, char*, const BwdWs&, int, int,  \
                                           int, int, int, int, int, hipStream_t);
DAR_BWD_INST(float)
DAR_BWD_INST(bf16_t)
#undef DAR_BWD_INST

}  // namespace dar
