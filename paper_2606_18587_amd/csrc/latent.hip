// Window-exit down-projection (Eq. 1, applied per KV head to keys and values).
//
//  * prefill pre-pass: latents of every token that is distant for some query
//    of the sequence (tokens [0, T - w)), into the prefill workspace;
//  * cache append: each token that leaves the window is projected into its
//    latent slot, the newest tokens go to the ring.
//
// Both accumulate c[col] = sum_e x[e] * W_down[e][col] with fp32 fused
// multiply-adds in increasing e (the order of dar::project_col), so the two
// produce identical bits for identical inputs, however tokens are batched.
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

// One block = 64 tokens of one (batch, KV head). Lane = token; the 4 waves
// share the 2*dd output columns (K and V) in chunks of 8.
//   cK:  [B*Hkv][Tp][dd]               token-major (columns in latent_pos order
//                                       when perm is set)
//   cVt: [B*Hkv][Tp/64][dd][64]        64-token blocks, transposed inside
// Rows [Tl, Tp) are written as zeros.
template <typename T>
__global__ __launch_bounds__(256) void prefill_latent_kernel(
    const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ wd,
    T* __restrict__ cK, T* __restrict__ cVt, int Hkv, int T_, int d, int dd, int Tl, int Tp,
    int perm) {
    extern __shared__ float xs[];  // [2][64][d+1]
    const int bg = blockIdx.y;
    const int g = bg % Hkv;
    const int t0 = blockIdx.x * 64;
    const int ld = d + 1;
    const T* wdg = wd + (size_t)g * d * dd;
    for (int which = 0; which < 2; ++which) {
        const T* x = (which ? v : k) + (size_t)bg * T_ * d;
        float* dst = xs + which * 64 * ld;
        for (int idx = threadIdx.x; idx < 64 * d; idx += 256) {
            const int t = idx / d, e = idx - (idx / d) * d;
            dst[t * ld + e] = (t0 + t < Tl) ? elem<T>::load(x + (size_t)(t0 + t) * d + e) : 0.f;
        }
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int t = t0 + lane;
    const int nchunk = (dd + 7) / 8;
    for (int ch = wave; ch < 2 * nchunk; ch += 4) {
        const int which = ch / nchunk;
        const int c0 = (ch - which * nchunk) * 8;
        const float* xr = xs + which * 64 * ld + lane * ld;
        float acc[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = 0.f;
        for (int e = 0; e < d; ++e) {
            const float xv = xr[e];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (c0 + j < dd)
                    acc[j] = __builtin_fmaf(xv, elem<T>::load(wdg + (size_t)e * dd + c0 + j), acc[j]);
        }
        if (t < Tp) {
            if (which == 0) {
                T* out = cK + ((size_t)bg * Tp + t) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd)
                        out[perm ? latent_pos(c0 + j) : c0 + j] = elem<T>::from_f32(acc[j]);
            } else {
                T* out = cVt + ((size_t)bg * Tp + (size_t)(t >> 6) * 64) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd) out[(size_t)(c0 + j) * 64 + (t & 63)] = elem<T>::from_f32(acc[j]);
            }
        }
    }
}

// Cache append. One block = up to 64 new tokens of one (batch, KV head).
// New token t (position p = len + t) makes token e = p - w leave the window:
// its latent is projected from the ring (e < len) or from the new tokens
// (e >= len). Token t itself is written to ring slot p % w if it is still in
// the window after the whole append (t >= n - w).
// mode 0: project and write the ring (safe when n <= w: the slot a block
//         reads is only rewritten by the same block, after its barrier);
// mode 1: project only; mode 2: ring only (mode 1 then mode 2 when n > w).
template <typename T>
__global__ __launch_bounds__(256) void append_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, const T* __restrict__ wd,
    T* k_win, T* v_win, T* __restrict__ k_lat, T* __restrict__ v_lat, int Hkv, int d, int dd,
    int w, int cap, int len, int n, int mode) {
    extern __shared__ float xs[];  // [2][64][d+1]
    const int bg = blockIdx.y;
    const int g = bg % Hkv;
    const int t0 = blockIdx.x * 64;
    const int ld = d + 1;
    const size_t new_base = (size_t)bg * n * d;
    const size_t win_base = (size_t)bg * w * d;
    if (mode != 2) {
        for (int which = 0; which < 2; ++which) {
            const T* src_new = (which ? v_new : k_new) + new_base;
            const T* src_win = (which ? v_win : k_win) + win_base;
            float* dst = xs + which * 64 * ld;
            for (int idx = threadIdx.x; idx < 64 * d; idx += 256) {
                const int tl = idx / d, e = idx - (idx / d) * d;
                const int tt = t0 + tl;
                const int ex = len + tt - w;  // position leaving the window
                float val = 0.f;
                if (tt < n && ex >= 0) {
                    const T* row = (ex < len) ? src_win + (size_t)(ex % w) * d
                                              : src_new + (size_t)(ex - len) * d;
                    val = elem<T>::load(row + e);
                }
                dst[tl * ld + e] = val;
            }
        }
    }
    __syncthreads();  // every ring read of this block is done before any ring write
    if (mode != 2) {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int tt = t0 + lane;
        const int ex = len + tt - w;
        const int nchunk = (dd + 7) / 8;
        const T* wdg = wd + (size_t)g * d * dd;
        for (int ch = wave; ch < 2 * nchunk; ch += 4) {
            const int which = ch / nchunk;
            const int c0 = (ch - which * nchunk) * 8;
            const float* xr = xs + which * 64 * ld + lane * ld;
            float acc[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j] = 0.f;
            for (int e = 0; e < d; ++e) {
                const float xv = xr[e];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd)
                        acc[j] = __builtin_fmaf(xv, elem<T>::load(wdg + (size_t)e * dd + c0 + j), acc[j]);
            }
            if (tt < n && ex >= 0) {
                T* out = (which ? v_lat : k_lat) + ((size_t)bg * cap + ex) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd) out[c0 + j] = elem<T>::from_f32(acc[j]);
            }
        }
    }
    if (mode != 1 && w > 0) {
        for (int which = 0; which < 2; ++which) {
            const T* src = (which ? v_new : k_new) + new_base;
            T* ring = (which ? v_win : k_win) + win_base;
            for (int idx = threadIdx.x; idx < 64 * d; idx += 256) {
                const int tl = idx / d, e = idx - (idx / d) * d;
                const int tt = t0 + tl;
                if (tt < n && tt >= n - w)
                    ring[(size_t)((len + tt) % w) * d + e] = src[(size_t)tt * d + e];
            }
        }
    }
}

template <typename T>
hipError_t launch_prefill_latent(const T* k, const T* v, const T* wd, T* cK, T* cVt, int B,
                                 int Hkv, int T_, int d, int dd, int w, bool perm, hipStream_t st) {
    const int Tl = T_ - w;
    if (Tl <= 0) return hipSuccess;
    const int Tp = round_up(Tl, 64);
    dim3 grid(Tp / 64, B * Hkv);
    const size_t lds = sizeof(float) * 2 * 64 * (d + 1);
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)prefill_latent_kernel<T>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(prefill_latent_kernel<T>, grid, dim3(256), lds, st, k, v, wd, cK, cVt, Hkv,
                       T_, d, dd, Tl, Tp, perm ? 1 : 0);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_append(const T* k_new, const T* v_new, const T* wd, T* k_win, T* v_win,
                         T* k_lat, T* v_lat, int B, int Hkv, int d, int dd, int w, int cap, int len,
                         int n, hipStream_t st) {
    dim3 grid((n + 63) / 64, B * Hkv);
    const size_t lds = sizeof(float) * 2 * 64 * (d + 1);
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)append_kernel<T>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    if (n <= w || w == 0) {
        hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), lds, st, k_new, v_new, wd, k_win,
                           v_win, k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), lds, st, k_new, v_new, wd, k_win, v_win,
                       k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), 0, st, k_new, v_new, wd, k_win, v_win,
                       k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 2);
    return hipGetLastError();
}

template hipError_t launch_prefill_latent<float>(const float*, const float*, const float*, float*,
                                                 float*, int, int, int, int, int, int, bool,
                                                 hipStream_t);
template hipError_t launch_prefill_latent<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                                  bf16_t*, bf16_t*, int, int, int, int, int, int,
                                                  bool, hipStream_t);
template hipError_t launch_append<float>(const float*, const float*, const float*, float*, float*,
                                         float*, float*, int, int, int, int, int, int, int, int,
                                         hipStream_t);
template hipError_t launch_append<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*, bf16_t*,
                                          bf16_t*, bf16_t*, bf16_t*, int, int, int, int, int, int,
                                          int, int, hipStream_t);

}  // namespace dar
