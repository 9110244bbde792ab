// Generic causal DAR prefill on the vector ALUs (fp32 path, and the fallback
// for bf16 head sizes the matrix-core kernel does not cover).
//
// One wavefront per (query row, batch * query head); row r is the query at
// position i = q0 + r (q0 = 0 for a whole sequence, the cache length for a
// chunk appended to a cache), and k/v row t holds position kv0 + t. For row i the keys
// j <= i - w are distant: their score is q~ . c^K_j with q~ = q W_up^T, their
// value contribution is accumulated in d_down space and lifted once at the
// end, (sum_j p_j c^V_j) W_up (Eq. 2 absorbed, Limitations section). The keys
// i - w < j <= i are local: q . k_j and p_j v_j at full d (Eq. 3). Both
// regions share one running max and one running sum, so the result is the
// single softmax of Eq. 4. Scores use scale 1/sqrt(d) for both regions;
// log2(e) is folded into the query so the exponentials are exp2.
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

template <typename T>
__global__ __launch_bounds__(64) void prefill_valu_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ wd, const T* __restrict__ wu, const T* __restrict__ cK,
    const T* __restrict__ cVt, T* __restrict__ o, float* __restrict__ lse, int Hq, int Hkv,
    int q0, int n_rows, int kv0, int Tkv, int d, int dd, int w, int Tp, float qscale,
    const T* __restrict__ wv, const int* __restrict__ seq_lens) {
    __shared__ float qs[256];
    __shared__ float qts[256];
    __shared__ float ps[64];
    __shared__ float lat[256];
    const int lane = lane_id_x();
    const int row = (n_rows - 1) - wg_id_x();  // longest rows are launched first
    const int i = q0 + row;                    // its position
    const int bh = wg_id_y();
    const int b = bh / Hq, h = bh - (bh / Hq) * Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    // a ragged batch: rows at or past this sequence's length are not computed
    if (seq_lens && i >= seq_lens[b]) return;
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    const T* wvg = wv ? wv + (size_t)g * dd * d : nullptr;  // value lift (shared latent), else W_up

    const T* qrow = q + ((size_t)bh * n_rows + row) * d;
    for (int e = lane; e < d; e += 64) qs[e] = elem<T>::load(qrow + e) * qscale;
    __syncthreads();

    const int n_dist = imax(0, i - w + 1);  // distant keys: j in [0, i - w]
    if (n_dist > 0) {
        for (int c = lane; c < dd; c += 64) {
            float acc = 0.f;
            for (int e = 0; e < d; ++e) {
                const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                    : elem<T>::load(wdg + (size_t)e * dd + c);
                acc = __builtin_fmaf(qs[e], u, acc);
            }
            qts[c] = acc;
        }
    }
    __syncthreads();

    float m = -INFINITY, l = 0.f;
    float aw[4] = {0.f, 0.f, 0.f, 0.f};
    float al[4] = {0.f, 0.f, 0.f, 0.f};

    // distant region, d_down wide
    const T* cKg = cK + (size_t)bg * Tp * dd;
    const T* cVg = cVt + (size_t)bg * Tp * dd;
    for (int j0 = 0; j0 < n_dist; j0 += 64) {
        const int j = j0 + lane;
        float s = -INFINITY;
        if (j < n_dist) {
            const T* kr = cKg + (size_t)j * dd;
            float acc = 0.f;
            for (int c = 0; c < dd; ++c) acc = __builtin_fmaf(qts[c], elem<T>::load(kr + c), acc);
            s = acc;
        }
        const float mn = fmaxf(m, wave_max(s));
        const float corr = exp2f(m - mn);
        const float p = (j < n_dist) ? exp2f(s - mn) : 0.f;
        l = l * corr + wave_sum(p);
#pragma unroll
        for (int r = 0; r < 4; ++r) { aw[r] *= corr; al[r] *= corr; }
        m = mn;
        ps[lane] = p;
        __syncthreads();
        const int cnt = imin(64, n_dist - j0);
        for (int jj = 0; jj < cnt; ++jj) {
            const float pj = ps[jj];
            const int jx = j0 + jj;
            const T* vb = cVg + (size_t)(jx >> 5) * 32 * dd + (jx & 31);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int c = lane + 64 * r;
                if (c < dd) al[r] = __builtin_fmaf(pj, elem<T>::load(vb + (size_t)c * 32), al[r]);
            }
        }
        __syncthreads();
    }

    // local region (the window, including the query's own token), d wide
    const int j_lo = imax(0, i - w + 1);
    const T* kg = k + (size_t)bg * Tkv * d;  // row of position j: j - kv0
    const T* vg = v + (size_t)bg * Tkv * d;
    for (int j0 = j_lo; j0 <= i; j0 += 64) {
        const int j = j0 + lane;
        float s = -INFINITY;
        if (j <= i) {
            const T* kr = kg + (size_t)(j - kv0) * d;
            float acc = 0.f;
            for (int e = 0; e < d; ++e) acc = __builtin_fmaf(qs[e], elem<T>::load(kr + e), acc);
            s = acc;
        }
        const float mn = fmaxf(m, wave_max(s));
        const float corr = exp2f(m - mn);
        const float p = (j <= i) ? exp2f(s - mn) : 0.f;
        l = l * corr + wave_sum(p);
#pragma unroll
        for (int r = 0; r < 4; ++r) { aw[r] *= corr; al[r] *= corr; }
        m = mn;
        ps[lane] = p;
        __syncthreads();
        const int cnt = imin(64, i + 1 - j0);
        for (int jj = 0; jj < cnt; ++jj) {
            const float pj = ps[jj];
            const T* vr = vg + (size_t)(j0 + jj - kv0) * d;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int e = lane + 64 * r;
                if (e < d) aw[r] = __builtin_fmaf(pj, elem<T>::load(vr + e), aw[r]);
            }
        }
        __syncthreads();
    }

    // epilogue: o = (o_win + o_lat W_up) / l
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int c = lane + 64 * r;
        if (c < dd) lat[c] = al[r];
    }
    __syncthreads();
    T* orow = o + ((size_t)bh * n_rows + row) * d;
    const float inv_l = 1.f / l;
    // log of the row's softmax denominator (natural log), for a backward pass
    if (lse && lane == 0) lse[(size_t)bh * n_rows + row] = (m + log2f(l)) * 0.6931471805599453f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int e = lane + 64 * r;
        if (e < d) {
            float acc = aw[r];
            if (n_dist > 0)
                for (int c = 0; c < dd; ++c) {
                    const float u = wvg ? elem<T>::load(wvg + (size_t)c * d + e)
                                  : wug ? elem<T>::load(wug + (size_t)c * d + e)
                                        : elem<T>::load(wdg + (size_t)e * dd + c);
                    acc = __builtin_fmaf(lat[c], u, acc);
                }
            orow[e] = elem<T>::from_f32(acc * inv_l);
        }
    }
}

template <typename T>
hipError_t launch_prefill_valu(const T* q, const T* k, const T* v, const T* wd, const T* wu,
                               const T* cK, const T* cVt, T* o, float* lse, int B, int Hq,
                               int Hkv, const PrefillGeo& geo, int d, int dd, int w,
                               hipStream_t st, const T* wv) {
    const int Tp = prefill_tp(geo.total(), w);
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    dim3 grid(geo.n_rows, B * Hq);
    hipLaunchKernelGGL(prefill_valu_kernel<T>, grid, dim3(64), 0, st, q, k, v, wd, wu, cK, cVt, o,
                       lse, Hq, Hkv, geo.q0, geo.n_rows, geo.kv0, geo.Tkv, d, dd, w, Tp, qscale, wv,
                       geo.seq_lens);
    return hipGetLastError();
}

template hipError_t launch_prefill_valu<float>(const float*, const float*, const float*,
                                               const float*, const float*, const float*,
                                               const float*, float*, float*, int, int, int,
                                               const PrefillGeo&, int, int, int, hipStream_t,
                                               const float*);
template hipError_t launch_prefill_valu<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                                const bf16_t*, const bf16_t*, const bf16_t*,
                                                const bf16_t*, bf16_t*, float*, int, int, int,
                                                const PrefillGeo&, int, int, int, hipStream_t,
                                                const bf16_t*);

}  // namespace dar
