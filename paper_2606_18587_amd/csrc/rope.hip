// Rotary position embedding (RoPE) where Eq. 3 applies it: the window key
// is RoPE(k_j), the distant key is RoPE of the lifted key, RoPE((k_j W_down)
// W_up), values are not rotated, and the query is rotated at its own
// position. The rotation does not commute with W_up, so the distant key can
// no longer be absorbed into the query as in the rotation-free path: the
// distant region is attended at full d here, from lifted and rotated keys.
//
// Rotate-half pairing (the GPT-NeoX convention of the Pythia models): for
// m < r/2 the pair (x[m], x[m + r/2]) at position p turns by the angle
// p * base^(-2m/r); elements r..d-1 pass through. The angles come from a
// table [n_pos][r] (cos of the r/2 angles, then their sin) in fp32, computed
// once in fp64 by rope_table_kernel.
//
// Prefill pre-pass (per (batch, KV head), 32-token blocks):
//   Qr = RoPE(q), Kr = RoPE(k)            every position
//   Kd = RoPE((k W_down) W_up), Vd = (v W_down) W_up   positions < T - w
// with the latent rounded to the storage type between the two projections
// (as the split cache stores it), and the largest L2 norm of each 32-row
// block of Kr and Kd (the matrix-core kernel's fixed softmax reference).
#include "../../include/dar.h"
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

// ---------------------------------------------------------------- angle table

// One thread per (position, pair): grid (ceil(r/2 / 64), n_pos), 64 threads.
__global__ __launch_bounds__(64) void rope_table_kernel(int r, double base,
                                                         float* __restrict__ tab) {
    const int half = r / 2;
    const int m = wg_id_x() * 64 + lane_id_x(), p = wg_id_y();
    if (m >= half) return;
    const double ang = (double)p * pow(base, -2.0 * m / r);
    double s, c;
    sincos(ang, &s, &c);
    tab[(size_t)p * r + m] = (float)c;
    tab[(size_t)p * r + half + m] = (float)s;
}

hipError_t launch_rope_table(int r, double base, int n_pos, float* tab, hipStream_t st) {
    hipLaunchKernelGGL(rope_table_kernel, dim3((r / 2 + 63) / 64, n_pos), dim3(64), 0, st, r, base,
                       tab);
    return hipGetLastError();
}

// ---------------------------------------------------------------- pre-pass

// Largest value over the 32 rows of a block: x is this thread's row value,
// the 8 threads of a row hold the same value; red is 32 floats of LDS.
__device__ __forceinline__ void block_norm_max(float row_sq, float* red, int row, int sub, float* out) {
    if (sub == 0) red[row] = row_sq;
    __syncthreads();
    if (lane_id_x() == 0) {
        float m = 0.f;
        for (int t = 0; t < 32; ++t) m = fmaxf(m, red[t]);
        *out = sqrtf(m);
    }
}

// Sum of squares over the 8 consecutive threads that share a row.
__device__ __forceinline__ float row_sum8(float x) {
    x += __shfl_xor(x, 1, 64);
    x += __shfl_xor(x, 2, 64);
    x += __shfl_xor(x, 4, 64);
    return x;
}

// One row's rotation, elements e = sub, sub + 8, ... (8 threads per row);
// x(e) reads element e of the input row. Returns the sum of squares of the
// stored (rounded) outputs.
template <typename T, typename X>
__device__ __forceinline__ float rotate_row(X x, T* out, const float* cs, int d, int r, int sub) {
    const int half = r / 2;
    float sq = 0.f;
    for (int e = sub; e < d; e += 8) {
        if (e < half) {
            const float c = cs[e], s = cs[half + e];
            const float a = x(e), b = x(e + half);
            const T ya = elem<T>::from_f32(__builtin_fmaf(a, c, -(b * s)));
            const T yb = elem<T>::from_f32(__builtin_fmaf(b, c, a * s));
            out[e] = ya;
            out[e + half] = yb;
            const float fa = elem<T>::to_f32(ya), fb = elem<T>::to_f32(yb);
            sq = __builtin_fmaf(fa, fa, __builtin_fmaf(fb, fb, sq));
        } else if (e >= r) {
            const T y = elem<T>::from_f32(x(e));
            out[e] = y;
            const float fy = elem<T>::to_f32(y);
            sq = __builtin_fmaf(fy, fy, sq);
        }
    }
    return sq;
}

// Qr / Kr: rows of n_seq sequences of T positions, rotated at pos0 + t.
// Grid (ceil(T/32), n_seq); 256 threads = 32 rows x 8. norm (optional):
// [n_seq][ceil(T/32)] largest L2 norm of the block's stored rows.
template <typename T>
__global__ __launch_bounds__(256) void rope_rows_kernel(const T* __restrict__ x, T* __restrict__ out,
                                                         float* __restrict__ norm,
                                                         const float* __restrict__ tab, int T_,
                                                         int d, int r, int pos0) {
    __shared__ float red[32];
    const int tid = lane_id_x();
    const int row = tid >> 3, sub = tid & 7;
    const int blk = wg_id_x(), seq = wg_id_y();
    const int t = blk * 32 + row;
    float sq = 0.f;
    if (t < T_) {
        const T* xr = x + ((size_t)seq * T_ + t) * d;
        sq = rotate_row<T>([=](int e) { return elem<T>::load(xr + e); },
                           out + ((size_t)seq * T_ + t) * d, tab + (size_t)(pos0 + t) * r, d, r, sub);
    }
    sq = row_sum8(sq);
    if (norm) block_norm_max(sq, red, row, sub, norm + (size_t)seq * ((T_ + 31) / 32) + blk);
}

// Kd / Vd for positions t < Td (= T - w) of each (batch, KV head): latent
// c = x W_down (project_col, rounded to T), lift x' = c W_up (fp32 FMAs in
// increasing latent column), keys rotated at pos0 + t. Grid (ceil(Td/32),
// B*Hkv); 256 threads. Dynamic LDS: 32 x d floats (rows) + 32 x dd floats
// (latents). dnorm: [B*Hkv][ceil(Td/32)].
template <typename T>
__global__ __launch_bounds__(256) void rope_lift_kernel(const T* __restrict__ k, const T* __restrict__ v,
                                                         const T* __restrict__ wd, const T* __restrict__ wu,
                                                         T* __restrict__ kd, T* __restrict__ vd,
                                                         float* __restrict__ dnorm,
                                                         const float* __restrict__ tab, int Hkv, int T_,
                                                         int Td, int d, int dd, int r, int pos0) {
    extern __shared__ float lsh[];
    float* xs = lsh;            // [32][d]
    float* cs = lsh + 32 * d;   // [32][dd]
    __shared__ float red[32];
    const int tid = lane_id_x();
    const int blk = wg_id_x(), bg = wg_id_y();
    const int g = bg % Hkv;
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    const int t0 = blk * 32;
    const int nrow = imin(32, Td - t0);
    const int row = tid >> 3, sub = tid & 7;
    for (int which = 0; which < 2; ++which) {
        const T* src = (which == 0 ? k : v) + ((size_t)bg * T_ + t0) * d;
        T* dst = (which == 0 ? kd : vd) + ((size_t)bg * Td + t0) * d;
        // Eq. 1 per token and latent column (project_col: the same arithmetic
        // as the cache's window-exit projection)
        for (int idx = tid; idx < nrow * dd; idx += 256) {
            const int tt = idx / dd, c = idx - (idx / dd) * dd;
            cs[tt * dd + c] = elem<T>::to_f32(elem<T>::from_f32(
                project_col<T>(src + (size_t)tt * d, wdg, d, dd, c)));
        }
        __syncthreads();
        // Eq. 2 per token and element
        for (int idx = tid; idx < nrow * d; idx += 256) {
            const int tt = idx / d, e = idx - (idx / d) * d;
            float acc = 0.f;
            for (int c = 0; c < dd; ++c) {
                const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                    : elem<T>::load(wdg + (size_t)e * dd + c);
                acc = __builtin_fmaf(cs[tt * dd + c], u, acc);
            }
            xs[tt * d + e] = acc;
        }
        __syncthreads();
        float sq = 0.f;
        if (row < nrow) {
            if (which == 0) {
                const float* xr = xs + row * d;
                sq = rotate_row<T>([=](int e) { return xr[e]; }, dst + (size_t)row * d,
                                   tab + (size_t)(pos0 + t0 + row) * r, d, r, sub);
            } else {
                for (int e = sub; e < d; e += 8) dst[(size_t)row * d + e] = elem<T>::from_f32(xs[row * d + e]);
            }
        }
        if (which == 0 && dnorm) {
            sq = row_sum8(sq);
            block_norm_max(sq, red, row, sub, dnorm + (size_t)bg * ((Td + 31) / 32) + blk);
        }
        __syncthreads();
    }
}

template <typename T>
hipError_t launch_rope_prepass(const T* q, const T* k, const T* v, const T* wd, const T* wu,
                               const float* tab, T* qr, T* kr, T* kd, T* vd, float* knorm,
                               float* dnorm, int B, int Hq, int Hkv, int T_, int d, int dd, int w,
                               int r, int pos0, hipStream_t st) {
    const int nb = (T_ + 31) / 32;
    hipLaunchKernelGGL(rope_rows_kernel<T>, dim3(nb, B * Hq), dim3(256), 0, st, q, qr,
                       (float*)nullptr, tab, T_, d, r, pos0);
    hipLaunchKernelGGL(rope_rows_kernel<T>, dim3(nb, B * Hkv), dim3(256), 0, st, k, kr, knorm, tab,
                       T_, d, r, pos0);
    const int Td = T_ - w;
    if (Td > 0) {
        const size_t lds = sizeof(float) * 32 * (d + dd);
        if (lds > 60000) {  // (plus the static reduction array)
            hipError_t e = hipFuncSetAttribute((const void*)rope_lift_kernel<T>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(rope_lift_kernel<T>, dim3((Td + 31) / 32, B * Hkv), dim3(256), lds, st, k,
                           v, wd, wu, kd, vd, dnorm, tab, Hkv, T_, Td, d, dd, r, pos0);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------- generic attention

// One wavefront per (row, batch * query head), as the rotation-free generic
// kernel, but both regions at full d: keys j <= i - w from (Kd, Vd), keys
// i - w < j <= i from (Kr, v); one online softmax (Eq. 4).
template <typename T>
__global__ __launch_bounds__(64) void prefill_rope_valu_kernel(
    const T* __restrict__ qr, const T* __restrict__ kr, const T* __restrict__ v,
    const T* __restrict__ kd, const T* __restrict__ vd, T* __restrict__ o,
    float* __restrict__ lse, int Hq, int Hkv, int T_, int d, int w, float qscale) {
    __shared__ float qs[256];
    __shared__ float ps[64];
    const int lane = lane_id_x();
    const int i = (T_ - 1) - wg_id_x();  // longest rows first
    const int bh = wg_id_y();
    const int b = bh / Hq, h = bh - (bh / Hq) * Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    const int Td = imax(T_ - w, 0);
    const T* qrow = qr + ((size_t)bh * T_ + i) * d;
    for (int e = lane; e < d; e += 64) qs[e] = elem<T>::load(qrow + e) * qscale;
    __syncthreads();
    float m = -INFINITY, l = 0.f;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 <= i; j0 += 64) {
        const int j = j0 + lane;
        float s = -INFINITY;
        if (j <= i) {
            const bool far = i - j >= w;
            const T* key = far ? kd + ((size_t)bg * Td + j) * d : kr + ((size_t)bg * T_ + j) * d;
            float a = 0.f;
            for (int e = 0; e < d; ++e) a = __builtin_fmaf(qs[e], elem<T>::load(key + e), a);
            s = a;
        }
        const float mn = fmaxf(m, wave_max(s));
        const float corr = exp2f(m - mn);
        const float p = (j <= i) ? exp2f(s - mn) : 0.f;
        l = l * corr + wave_sum(p);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] *= corr;
        m = mn;
        ps[lane] = p;
        __syncthreads();
        const int cnt = imin(64, i + 1 - j0);
        for (int jj = 0; jj < cnt; ++jj) {
            const float pj = ps[jj];
            const int jx = j0 + jj;
            const T* val = (i - jx >= w) ? vd + ((size_t)bg * Td + jx) * d : v + ((size_t)bg * T_ + jx) * d;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int e = lane + 64 * t;
                if (e < d) acc[t] = __builtin_fmaf(pj, elem<T>::load(val + e), acc[t]);
            }
        }
        __syncthreads();
    }
    if (lse && lane == 0) lse[(size_t)bh * T_ + i] = (m + log2f(l)) * 0.6931471805599453f;
    const float inv = 1.f / l;
    T* orow = o + ((size_t)bh * T_ + i) * d;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int e = lane + 64 * t;
        if (e < d) orow[e] = elem<T>::from_f32(acc[t] * inv);
    }
}

template <typename T>
hipError_t launch_prefill_rope_valu(const T* qr, const T* kr, const T* v, const T* kd, const T* vd,
                                    T* o, float* lse, int B, int Hq, int Hkv, int T_, int d, int w,
                                    hipStream_t st) {
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    hipLaunchKernelGGL(prefill_rope_valu_kernel<T>, dim3(T_, B * Hq), dim3(64), 0, st, qr, kr, v, kd,
                       vd, o, lse, Hq, Hkv, T_, d, w, qscale);
    return hipGetLastError();
}

#define DAR_ROPE_INST(T)                                                                            \
    template hipError_t launch_rope_prepass<T>(const T*, const T*, const T*, const T*, const T*,   \
                                               const float*, T*, T*, T*, T*, float*, float*, int,  \
                                               int, int, int, int, int, int, int, int, hipStream_t); \
    template hipError_t launch_prefill_rope_valu<T>(const T*, const T*, const T*, const T*,        \
                                                    const T*, T*, float*, int, int, int, int, int, \
                                                    int, hipStream_t);
DAR_ROPE_INST(float)
DAR_ROPE_INST(bf16_t)
#undef DAR_ROPE_INST

}  // namespace dar
