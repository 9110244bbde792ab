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

// ---- vectorised pre-pass (d / 8 a power of two, r % 16 == 0): one thread
// per 8-element chunk; a rotated chunk is combined with its partner chunk
// (r / 16 chunks away) element by element.

template <typename T> struct vec8;
template <> struct vec8<bf16_t> {
    static __device__ __forceinline__ void load(const bf16_t* p, float (&x)[8]) {
        const uint4 u = *reinterpret_cast<const uint4*>(p);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            x[2 * j] = __uint_as_float(w4[j] << 16);
            x[2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
        }
    }
    // stores the rounded values; returns their sum of squares
    static __device__ __forceinline__ float store(bf16_t* p, const float (&y)[8]) {
        uint32_t w4[4];
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bf16_t a = f32_to_bf16(y[2 * j]), b = f32_to_bf16(y[2 * j + 1]);
            w4[j] = (uint32_t)a | ((uint32_t)b << 16);
            const float fa = bf16_to_f32(a), fb = bf16_to_f32(b);
            sq = __builtin_fmaf(fa, fa, __builtin_fmaf(fb, fb, sq));
        }
        *reinterpret_cast<uint4*>(p) = make_uint4(w4[0], w4[1], w4[2], w4[3]);
        return sq;
    }
};
template <> struct vec8<float> {
    static __device__ __forceinline__ void load(const float* p, float (&x)[8]) {
        const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    }
    static __device__ __forceinline__ float store(float* p, const float (&y)[8]) {
        *reinterpret_cast<float4*>(p) = make_float4(y[0], y[1], y[2], y[3]);
        *reinterpret_cast<float4*>(p + 4) = make_float4(y[4], y[5], y[6], y[7]);
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) sq = __builtin_fmaf(y[j], y[j], sq);
        return sq;
    }
};

// Chunk ch of a row after rotation: a = the chunk, b = its partner chunk
// (read only for rotated chunks), cs = the table row of the position.
__device__ __forceinline__ void rotate_chunk(int ch, int r, const float (&a)[8], const float (&b)[8],
                                             const float* cs, float (&y)[8]) {
    const int hc = r >> 4;
    if (ch < 2 * hc) {
        const bool first = ch < hc;
        const int m0 = (first ? ch : ch - hc) * 8;
        const float4 c0 = *reinterpret_cast<const float4*>(cs + m0);
        const float4 c1 = *reinterpret_cast<const float4*>(cs + m0 + 4);
        const float4 s0 = *reinterpret_cast<const float4*>(cs + (r >> 1) + m0);
        const float4 s1 = *reinterpret_cast<const float4*>(cs + (r >> 1) + m0 + 4);
        const float c8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        const float s8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j)
            y[j] = first ? __builtin_fmaf(a[j], c8[j], -(b[j] * s8[j])) : __builtin_fmaf(a[j], c8[j], b[j] * s8[j]);
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = a[j];
    }
}

// Sum over the nch consecutive lanes of a row (nch a power of two <= 32).
__device__ __forceinline__ float chunk_row_sum(float x, int nch) {
    for (int o = 1; o < nch; o <<= 1) x += __shfl_xor(x, o, 64);
    return x;
}

// Qr / Kr rows (vectorised): grid (ceil(T/32), n_seq), 32 * d/8 threads.
template <typename T>
__global__ __launch_bounds__(1024) void rope_rows_vec_kernel(const T* __restrict__ x, T* __restrict__ out,
                                                             float* __restrict__ norm,
                                                             const float* __restrict__ tab, int T_,
                                                             int d, int r, int pos0) {
    __shared__ float rsq[32];
    const int nch = d >> 3;
    const int tid = lane_id_x();
    const int row = tid / nch, ch = tid - (tid / nch) * nch;
    const int blk = wg_id_x(), seq = wg_id_y();
    const int t = blk * 32 + row;
    float sq = 0.f;
    if (t < T_) {
        const T* xr = x + ((size_t)seq * T_ + t) * d;
        const int hc = r >> 4;
        float a[8], b[8], y[8];
        vec8<T>::load(xr + ch * 8, a);
        if (ch < 2 * hc) vec8<T>::load(xr + (ch < hc ? ch + hc : ch - hc) * 8, b);
        rotate_chunk(ch, r, a, b, tab + (size_t)(pos0 + t) * r, y);
        sq = vec8<T>::store(out + ((size_t)seq * T_ + t) * d + ch * 8, y);
    }
    if (norm) {
        sq = chunk_row_sum(sq, nch);
        if (ch == 0) rsq[row] = sq;
        __syncthreads();
        if (tid == 0) {
            float m = 0.f;
            for (int i = 0; i < 32; ++i) m = fmaxf(m, rsq[i]);
            norm[(size_t)seq * ((T_ + 31) / 32) + blk] = sqrtf(m);
        }
    }
}

// Kd / Vd with W_down and W_up staged in LDS (fp32), rows read and written
// as 16-byte chunks. Same arithmetic as rope_lift_kernel: the latent by
// fp32 FMAs in increasing e (as project_col), rounded to T, the lift by fp32
// FMAs in increasing latent column. Grid (ceil(Td/32), B*Hkv), 256 threads;
// dynamic LDS (2 d dd + 32 d + 32 dd) floats.
template <typename T>
__global__ __launch_bounds__(256) void rope_lift_lds_kernel(const T* __restrict__ k, const T* __restrict__ v,
                                                            const T* __restrict__ wd, const T* __restrict__ wu,
                                                            T* __restrict__ kd, T* __restrict__ vd,
                                                            float* __restrict__ dnorm,
                                                            const float* __restrict__ tab, int Hkv,
                                                            int T_, int Td, int d, int dd, int r,
                                                            int pos0) {
    extern __shared__ float lsh[];
    float* wD = lsh;              // [d][dd]
    float* wU = wD + d * dd;      // [dd][d]
    float* xs = wU + dd * d;      // [32][d]: input rows, then lifted rows
    float* cs = xs + 32 * d;      // [32][dd]
    __shared__ float rsq[32];
    const int tid = lane_id_x();
    const int blk = wg_id_x(), bg = wg_id_y();
    const int g = bg % Hkv;
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    for (int idx = tid; idx < d * dd; idx += 256) {
        wD[idx] = elem<T>::load(wdg + idx);
        const int c = idx / d, e = idx - (idx / d) * d;  // wU[c][e]
        wU[idx] = wug ? elem<T>::load(wug + idx) : elem<T>::load(wdg + (size_t)e * dd + c);
    }
    const int t0 = blk * 32;
    const int nrow = imin(32, Td - t0);
    const int nch = d >> 3;
    for (int which = 0; which < 2; ++which) {
        const T* src = (which == 0 ? k : v) + ((size_t)bg * T_ + t0) * d;
        T* dst = (which == 0 ? kd : vd) + ((size_t)bg * Td + t0) * d;
        for (int idx = tid; idx < nrow * nch; idx += 256) {
            float a[8];
            vec8<T>::load(src + (size_t)idx * 8, a);
#pragma unroll
            for (int j = 0; j < 8; ++j) xs[idx * 8 + j] = a[j];
        }
        __syncthreads();
        // Eq. 1
        for (int idx = tid; idx < nrow * dd; idx += 256) {
            const int tt = idx / dd, c = idx - (idx / dd) * dd;
            float acc = 0.f;
            for (int e = 0; e < d; ++e) acc = __builtin_fmaf(xs[tt * d + e], wD[e * dd + c], acc);
            cs[idx] = elem<T>::to_f32(elem<T>::from_f32(acc));
        }
        __syncthreads();
        // Eq. 2 (the input rows are no longer needed: the lifted rows replace them)
        for (int idx = tid; idx < nrow * d; idx += 256) {
            const int tt = idx / d, e = idx - (idx / d) * d;
            float acc = 0.f;
            for (int c = 0; c < dd; ++c) acc = __builtin_fmaf(cs[tt * dd + c], wU[c * d + e], acc);
            xs[idx] = acc;
        }
        __syncthreads();
        // rotate (keys) and store
        for (int idx = tid; idx < 32 * nch; idx += 256) {
            const int row = idx / nch, ch = idx - (idx / nch) * nch;
            float sq = 0.f;
            if (row < nrow) {
                float a[8], b[8], y[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) a[j] = xs[row * d + ch * 8 + j];
                if (which == 0) {
                    const int hc = r >> 4;
                    if (ch < 2 * hc) {
                        const int pc = ch < hc ? ch + hc : ch - hc;
#pragma unroll
                        for (int j = 0; j < 8; ++j) b[j] = xs[row * d + pc * 8 + j];
                    }
                    rotate_chunk(ch, r, a, b, tab + (size_t)(pos0 + t0 + row) * r, y);
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) y[j] = a[j];
                }
                sq = vec8<T>::store(dst + (size_t)row * d + ch * 8, y);
            }
            if (which == 0 && dnorm) {
                sq = chunk_row_sum(sq, nch);
                if (ch == 0) rsq[row] = sq;
            }
        }
        __syncthreads();
        if (which == 0 && dnorm && tid == 0) {
            float m = 0.f;
            for (int i = 0; i < 32; ++i) m = fmaxf(m, rsq[i]);
            dnorm[(size_t)bg * ((Td + 31) / 32) + blk] = sqrtf(m);
        }
    }
}

// ---- matrix-core lift (bf16, d in {64, 128}, d_down in {16, 32}): one
// wavefront per 32-token tile, four tiles per workgroup, no barriers.
//   latent^T = W_down^T X^T   (A: W_down^T rows = latent columns, B: the
//                              token rows as read from memory)
//   lifted^T = W_up^T latent^T (B: the rounded latent accumulator registers
//                              taken as they are, A: W_up^T with its
//                              contraction index permuted to match them)
// The lifted tile goes through this wavefront's LDS (fp32, padded rows) to
// be rotated and stored as 16-byte row chunks.

typedef __bf16 rbf16x8 __attribute__((ext_vector_type(8)));
typedef float rf32x16 __attribute__((ext_vector_type(16)));
typedef float rf32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 rbf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ rf32x16 rmfma(rbf16x8 a, rbf16x8 b, rf32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t rpack2(float a, float b) {
    rf32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, rbf16x2));
}

template <int D, int DD>
__global__ __launch_bounds__(256) void rope_lift_mfma_kernel(const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
                                                             const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu,
                                                             bf16_t* __restrict__ kd, bf16_t* __restrict__ vd,
                                                             float* __restrict__ dnorm,
                                                             const float* __restrict__ tab, int Hkv,
                                                             int T_, int Td, int r, int pos0) {
    constexpr int KS = D / 16, NT = D / 32, DS = DD / 16, LDX = D + 4, NCH = D / 8;
    __shared__ __attribute__((aligned(16))) float xsh[4][32 * LDX];
    const int tid = lane_id_x();
    const int wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, hg = lane >> 5;
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    const int t0 = wg_id_x() * 128 + wave * 32;
    if (t0 >= Td) return;  // (no barrier in this kernel)
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
    // A operands: W_down^T (row = latent column `col`, k = e), and W_up^T
    // (row = e, k = the latent column the B operand's slot j holds)
    rbf16x8 aD[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        uint16_t e8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) e8[j] = col < DD ? wdg[(size_t)(16 * s + 8 * hg + j) * DD + col] : (uint16_t)0;
        aD[s] = __builtin_bit_cast(rbf16x8, e8);
    }
    rbf16x8 aU[NT][DS];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int s2 = 0; s2 < DS; ++s2) {
            uint16_t e8[8];
            const int e = 32 * t + col;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int c = 16 * s2 + (j < 4 ? 4 * hg + j : 8 + 4 * hg + (j - 4));
                e8[j] = wug ? wug[(size_t)c * D + e] : wdg[(size_t)e * DD + c];
            }
            aU[t][s2] = __builtin_bit_cast(rbf16x8, e8);
        }
    float* xs = xsh[wave];
    const int tok = imin(t0 + col, Td - 1);  // rows past the end are computed, never stored
    float nmax = 0.f;
    for (int which = 0; which < 2; ++which) {
        const bf16_t* xrow = (which == 0 ? k : v) + ((size_t)bg * T_ + tok) * D;
        rf32x16 c = {};
#pragma unroll
        for (int s = 0; s < KS; ++s)
            c = rmfma(aD[s], __builtin_bit_cast(rbf16x8, *reinterpret_cast<const uint4*>(xrow + 16 * s + 8 * hg)), c);
        // the latent rounded to bf16 (as the cache stores it): register 8 s2 + j
        // holds latent column 16 s2 + (j < 4 ? 4 hg + j : 8 + 4 hg + j - 4)
        rbf16x8 cb[DS];
#pragma unroll
        for (int s2 = 0; s2 < DS; ++s2)
            cb[s2] = __builtin_bit_cast(rbf16x8, make_uint4(rpack2(c[8 * s2 + 0], c[8 * s2 + 1]), rpack2(c[8 * s2 + 2], c[8 * s2 + 3]),
                                                            rpack2(c[8 * s2 + 4], c[8 * s2 + 5]), rpack2(c[8 * s2 + 6], c[8 * s2 + 7])));
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            rf32x16 x = {};
#pragma unroll
            for (int s2 = 0; s2 < DS; ++s2) x = rmfma(aU[t][s2], cb[s2], x);
            // register 4 m + i: element e = 32 t + 8 m + 4 hg + i of token `col`
#pragma unroll
            for (int m = 0; m < 4; ++m)
                *reinterpret_cast<float4*>(xs + col * LDX + 32 * t + 8 * m + 4 * hg) =
                    make_float4(x[4 * m], x[4 * m + 1], x[4 * m + 2], x[4 * m + 3]);
        }
        // rows of the tile: rotate (keys) and store as 16-byte chunks
        bf16_t* dst = (which == 0 ? kd : vd) + ((size_t)bg * Td + t0) * D;
        const int hc = r >> 4;
#pragma unroll
        for (int it = 0; it < 32 * NCH / 64; ++it) {
            const int idx = it * 64 + lane;
            const int row = idx / NCH, ch = idx % NCH;
            float a[8], b[8], y[8];
            const float* xr = xs + row * LDX;
#pragma unroll
            for (int j = 0; j < 8; ++j) a[j] = xr[ch * 8 + j];
            if (which == 0) {
                if (ch < 2 * hc) {
                    const int pc = ch < hc ? ch + hc : ch - hc;
#pragma unroll
                    for (int j = 0; j < 8; ++j) b[j] = xr[pc * 8 + j];
                }
                rotate_chunk(ch, r, a, b, tab + (size_t)(pos0 + imin(t0 + row, Td - 1)) * r, y);
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) y[j] = a[j];
            }
            float sq = 0.f;
            if (t0 + row < Td) sq = vec8<bf16_t>::store(dst + (size_t)row * D + ch * 8, y);
            if (which == 0) nmax = fmaxf(nmax, chunk_row_sum(sq, NCH));
        }
    }
    nmax = wave_max(nmax);
    if (dnorm && lane == 0) dnorm[(size_t)bg * ((Td + 31) / 32) + t0 / 32] = sqrtf(nmax);
}

static bool rope_vec_ok(int d, int r) {
    const int nch = d / 8;
    return d % 8 == 0 && d <= 256 && (nch & (nch - 1)) == 0 && r % 16 == 0;
}

template <typename T>
hipError_t launch_rope_prepass(const T* q, const T* k, const T* v, const T* wd, const T* wu,
                               const float* tab, T* qr, T* kr, T* kd, T* vd, float* knorm,
                               float* dnorm, int B, int Hq, int Hkv, int T_, int d, int dd, int w,
                               int r, int pos0, hipStream_t st) {
    const int nb = (T_ + 31) / 32;
    const bool vec = rope_vec_ok(d, r);
    if (vec) {
        const int nt = 32 * (d / 8);
        hipLaunchKernelGGL(rope_rows_vec_kernel<T>, dim3(nb, B * Hq), dim3(nt), 0, st, q, qr,
                           (float*)nullptr, tab, T_, d, r, pos0);
        hipLaunchKernelGGL(rope_rows_vec_kernel<T>, dim3(nb, B * Hkv), dim3(nt), 0, st, k, kr, knorm,
                           tab, T_, d, r, pos0);
    } else {
        hipLaunchKernelGGL(rope_rows_kernel<T>, dim3(nb, B * Hq), dim3(256), 0, st, q, qr,
                           (float*)nullptr, tab, T_, d, r, pos0);
        hipLaunchKernelGGL(rope_rows_kernel<T>, dim3(nb, B * Hkv), dim3(256), 0, st, k, kr, knorm,
                           tab, T_, d, r, pos0);
    }
    const int Td = T_ - w;
    const size_t lds_vec = sizeof(float) * (2 * (size_t)d * dd + 32 * (size_t)d + 32 * (size_t)dd);
    const bool mfma = sizeof(T) == 2 && (d == 64 || d == 128) && (dd == 16 || dd == 32) && r % 16 == 0;
    if (Td > 0 && mfma) {
        const dim3 grid((Td + 127) / 128, B * Hkv);
        const bf16_t *k16 = (const bf16_t*)k, *v16 = (const bf16_t*)v, *wd16 = (const bf16_t*)wd,
                     *wu16 = (const bf16_t*)wu;
        bf16_t *kd16 = (bf16_t*)kd, *vd16 = (bf16_t*)vd;
        if (d == 64 && dd == 16)
            hipLaunchKernelGGL((rope_lift_mfma_kernel<64, 16>), grid, dim3(256), 0, st, k16, v16, wd16, wu16, kd16, vd16, dnorm, tab, Hkv, T_, Td, r, pos0);
        else if (d == 64)
            hipLaunchKernelGGL((rope_lift_mfma_kernel<64, 32>), grid, dim3(256), 0, st, k16, v16, wd16, wu16, kd16, vd16, dnorm, tab, Hkv, T_, Td, r, pos0);
        else if (dd == 16)
            hipLaunchKernelGGL((rope_lift_mfma_kernel<128, 16>), grid, dim3(256), 0, st, k16, v16, wd16, wu16, kd16, vd16, dnorm, tab, Hkv, T_, Td, r, pos0);
        else
            hipLaunchKernelGGL((rope_lift_mfma_kernel<128, 32>), grid, dim3(256), 0, st, k16, v16, wd16, wu16, kd16, vd16, dnorm, tab, Hkv, T_, Td, r, pos0);
    } else if (Td > 0 && vec && lds_vec <= 60000) {
        hipLaunchKernelGGL(rope_lift_lds_kernel<T>, dim3((Td + 31) / 32, B * Hkv), dim3(256), lds_vec,
                           st, k, v, wd, wu, kd, vd, dnorm, tab, Hkv, T_, Td, d, dd, r, pos0);
    } else if (Td > 0) {
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

// ---- chunked prefill into a split cache with the rotary embedding

// Kd / Vd rows [out_row0, out_row0 + nrows) of each (batch, KV head), row =
// position, either from full-d rows (in_k / in_v row in_row0 + t, in_stride
// rows a head: the latent is projected as in rope_lift_lds_kernel) or, when
// lat_k is given, from the cache's latents (lat_k / lat_v row out_row0 + t,
// lat_stride rows a head); then lifted with W_up by fp32 FMAs in increasing
// latent column, and the keys rotated at their positions. Grid
// (ceil(nrows / 32), B*Hkv), 256 threads, dynamic LDS (2 d dd + 32 d +
// 32 dd) floats.
template <typename T>
__global__ __launch_bounds__(256) void rope_lift_span_kernel(
    const T* __restrict__ in_k, const T* __restrict__ in_v, int in_stride, int in_row0,
    const T* __restrict__ lat_k, const T* __restrict__ lat_v, int lat_stride,
    const T* __restrict__ wd, const T* __restrict__ wu, T* __restrict__ kd, T* __restrict__ vd,
    int out_stride, int out_row0, int nrows, const float* __restrict__ tab, int Hkv, int d, int dd,
    int r) {
    extern __shared__ float lsh[];
    float* wD = lsh;              // [d][dd]
    float* wU = wD + d * dd;      // [dd][d]
    float* xs = wU + dd * d;      // [32][d]: input rows, then lifted rows
    float* cs = xs + 32 * d;      // [32][dd]
    const int tid = lane_id_x();
    const int blk = wg_id_x(), bg = wg_id_y();
    const int g = bg % Hkv;
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    for (int idx = tid; idx < d * dd; idx += 256) {
        wD[idx] = elem<T>::load(wdg + idx);
        const int c = idx / d, e = idx - (idx / d) * d;  // wU[c][e]
        wU[idx] = wug ? elem<T>::load(wug + idx) : elem<T>::load(wdg + (size_t)e * dd + c);
    }
    const int t0 = blk * 32;
    const int nrow = imin(32, nrows - t0);
    const int nch = d >> 3;
    for (int which = 0; which < 2; ++which) {
        T* dst = (which == 0 ? kd : vd) + ((size_t)bg * out_stride + out_row0 + t0) * d;
        if (lat_k) {
            const T* lat = (which == 0 ? lat_k : lat_v) + ((size_t)bg * lat_stride + out_row0 + t0) * dd;
            for (int idx = tid; idx < nrow * dd; idx += 256) cs[idx] = elem<T>::load(lat + idx);
            __syncthreads();
        } else {
            const T* src = (which == 0 ? in_k : in_v) + ((size_t)bg * in_stride + in_row0 + t0) * d;
            for (int idx = tid; idx < nrow * nch; idx += 256) {
                float a[8];
                vec8<T>::load(src + (size_t)idx * 8, a);
#pragma unroll
                for (int j = 0; j < 8; ++j) xs[idx * 8 + j] = a[j];
            }
            __syncthreads();
            // Eq. 1
            for (int idx = tid; idx < nrow * dd; idx += 256) {
                const int tt = idx / dd, c = idx - (idx / dd) * dd;
                float acc = 0.f;
                for (int e = 0; e < d; ++e) acc = __builtin_fmaf(xs[tt * d + e], wD[e * dd + c], acc);
                cs[idx] = elem<T>::to_f32(elem<T>::from_f32(acc));
            }
            __syncthreads();
        }
        // Eq. 2
        for (int idx = tid; idx < nrow * d; idx += 256) {
            const int tt = idx / d, e = idx - (idx / d) * d;
            float acc = 0.f;
            for (int c = 0; c < dd; ++c) acc = __builtin_fmaf(cs[tt * dd + c], wU[c * d + e], acc);
            xs[idx] = acc;
        }
        __syncthreads();
        // rotate (keys) and store
        for (int idx = tid; idx < nrow * nch; idx += 256) {
            const int row = idx / nch, ch = idx - (idx / nch) * nch;
            float a[8], b[8], y[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) a[j] = xs[row * d + ch * 8 + j];
            if (which == 0) {
                const int hc = r >> 4;
                if (ch < 2 * hc) {
                    const int pc = ch < hc ? ch + hc : ch - hc;
#pragma unroll
                    for (int j = 0; j < 8; ++j) b[j] = xs[row * d + pc * 8 + j];
                }
                rotate_chunk(ch, r, a, b, tab + (size_t)(out_row0 + t0 + row) * r, y);
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) y[j] = a[j];
            }
            vec8<T>::store(dst + (size_t)row * d + ch * 8, y);
        }
        __syncthreads();
    }
}

// Largest L2 norm of the stored rows of each 32-position block (the
// matrix-core kernel's fixed softmax reference): row t of x (stride rows a
// head) holds position row_pos0 + t, t < nrows; block b covers positions
// [32 b, 32 b + 32) and lands in out[bg * out_blocks + b]. Grid
// (blocks met by the rows, B*Hkv), 256 threads = 32 rows x 8.
template <typename T>
__global__ __launch_bounds__(256) void block_norm_kernel(const T* __restrict__ x, int stride,
                                                         int row_pos0, int nrows, int d,
                                                         float* __restrict__ out, int out_blocks) {
    __shared__ float rsq[32];
    const int tid = lane_id_x();
    const int row = tid >> 3, sub = tid & 7;
    const int bg = wg_id_y();
    const int b = (row_pos0 >> 5) + wg_id_x();
    const int pos = 32 * b + row;
    float sq = 0.f;
    if (pos >= row_pos0 && pos < row_pos0 + nrows) {
        const T* xr = x + ((size_t)bg * stride + (pos - row_pos0)) * d;
        for (int e = sub; e < d; e += 8) {
            const float v = elem<T>::load(xr + e);
            sq = __builtin_fmaf(v, v, sq);
        }
    }
    sq += __shfl_xor(sq, 1, 64);
    sq += __shfl_xor(sq, 2, 64);
    sq += __shfl_xor(sq, 4, 64);
    if (sub == 0) rsq[row] = sq;
    __syncthreads();
    if (tid == 0) {
        float m = 0.f;
        for (int i = 0; i < 32; ++i) m = fmaxf(m, rsq[i]);
        out[(size_t)bg * out_blocks + b] = sqrtf(m);
    }
}

template <typename T>
hipError_t launch_rope_chunk_prepass(const T* q, const T* ctx_k, const T* ctx_v, const T* k_lat,
                                     const T* v_lat, int cap, const T* wd, const T* wu,
                                     const float* tab, T* qr, T* kr, T* kd, T* vd, float* knorm,
                                     float* dnorm, int B, int Hq, int Hkv, int d, int dd, int w,
                                     int r, int len, int n, int kv0, hipStream_t st) {
    if (!rope_vec_ok(d, r)) return hipErrorNotSupported;
    const int Tc = len + n - kv0, T_ = len + n, Td = T_ - w > 0 ? T_ - w : 0;
    const int lat0 = len - w > 0 ? len - w : 0;  // cached latents: positions < lat0
    const int nt = 32 * (d / 8);
    hipLaunchKernelGGL(rope_rows_vec_kernel<T>, dim3((n + 31) / 32, B * Hq), dim3(nt), 0, st, q, qr,
                       (float*)nullptr, tab, n, d, r, len);
    hipLaunchKernelGGL(rope_rows_vec_kernel<T>, dim3((Tc + 31) / 32, B * Hkv), dim3(nt), 0, st, ctx_k,
                       kr, (float*)nullptr, tab, Tc, d, r, kv0);
    const int nkb = (T_ + 31) / 32;
    hipLaunchKernelGGL(block_norm_kernel<T>, dim3(nkb - (kv0 >> 5), B * Hkv), dim3(256), 0, st,
                       (const T*)kr, Tc, kv0, Tc, d, knorm, nkb);
    if (Td > 0) {
        const size_t lds = sizeof(float) * (2 * (size_t)d * dd + 32 * (size_t)d + 32 * (size_t)dd);
        if (lds > 65536) return hipErrorNotSupported;
        const int ncache = lat0 < Td ? lat0 : Td;
        if (ncache > 0)
            hipLaunchKernelGGL(rope_lift_span_kernel<T>, dim3((ncache + 31) / 32, B * Hkv), dim3(256),
                               lds, st, (const T*)nullptr, (const T*)nullptr, 0, 0, k_lat, v_lat, cap,
                               wd, wu, kd, vd, Td, 0, ncache, tab, Hkv, d, dd, r);
        if (Td > lat0)
            hipLaunchKernelGGL(rope_lift_span_kernel<T>, dim3((Td - lat0 + 31) / 32, B * Hkv),
                               dim3(256), lds, st, ctx_k, ctx_v, Tc, lat0 - kv0, (const T*)nullptr,
                               (const T*)nullptr, 0, wd, wu, kd, vd, Td, lat0, Td - lat0, tab, Hkv,
                               d, dd, r);
        hipLaunchKernelGGL(block_norm_kernel<T>, dim3((Td + 31) / 32, B * Hkv), dim3(256), 0, st,
                           (const T*)kd, Td, 0, Td, d, dnorm, (Td + 31) / 32);
    }
    return hipGetLastError();
}

#define DAR_ROPE_INST(T)                                                                            \
    template hipError_t launch_rope_prepass<T>(const T*, const T*, const T*, const T*, const T*,   \
                                               const float*, T*, T*, T*, T*, float*, float*, int,  \
                                               int, int, int, int, int, int, int, int, hipStream_t); \
    template hipError_t launch_prefill_rope_valu<T>(const T*, const T*, const T*, const T*,        \
                                                    const T*, T*, float*, int, int, int, int, int, \
                                                    int, hipStream_t);                             \
    template hipError_t launch_rope_chunk_prepass<T>(const T*, const T*, const T*, const T*,       \
                                                     const T*, int, const T*, const T*,           \
                                                     const float*, T*, T*, T*, T*, float*, float*, \
                                                     int, int, int, int, int, int, int, int, int,  \
                                                     int, hipStream_t);
DAR_ROPE_INST(float)
DAR_ROPE_INST(bf16_t)
#undef DAR_ROPE_INST

}  // namespace dar

// ---------------------------------------------------------------- decode

namespace dar {

// Lanes that cover one row of `dim` elements, 8 elements a lane.
static __host__ __device__ inline int lanes_per_row_rope(int dim) {
    int lpt = 1;
    while (lpt * 8 < dim) lpt <<= 1;
    return lpt;
}

static constexpr int kRopeDecThreads = 256;
static constexpr int kRopeDecSlots = 8192;  // G * tokens-per-split scores in LDS

// Split-KV decode with the rotary embedding of Eq. 3 (generic kernel, every
// dtype and head size): one block per (batch, KV head, split) as the
// rotation-free generic decode, same splits and partial records
// {m, l, acc_lat[dd], acc_win[d]} (decode_combine_kernel finishes).
//
// The score of token j at position p against the query rotated at position
// len - 1, Qr . RoPE_p(x_j), is evaluated as (RoPE_p^T Qr) . x_j: the rotation
// moves to the query side per token, element e of the rotated-back query
// depending only on Qr[e], its pair partner and the angle of (p, e mod r/2),
// so each lane rotates its own 8-element segment without exchanging key
// elements. x_j is the ring key (window) or the lifted latent c^K_j W_up
// (distant: computed per token at full d, the rotation does not commute with
// W_up). Values are not rotated: the window accumulates v_j at d, the
// distant region sum p c^V at d_down, lifted once by the combine.
template <typename T, int G>
__global__ __launch_bounds__(kRopeDecThreads) void decode_rope_split_kernel(
    const T* __restrict__ q, const T* __restrict__ wd, const T* __restrict__ wu,
    const T* __restrict__ k_win, const T* __restrict__ v_win, const T* __restrict__ k_lat,
    const T* __restrict__ v_lat, const float* __restrict__ tab, float* __restrict__ part, int Hq,
    int Hkv, int d, int dd, int w, int cap, int len, int r, int chunk_lat, int chunk_win,
    int n_lat_split, int S, float qscale) {
    static_assert(4 * G * 256 <= kRopeDecSlots, "partial sums must fit in the score buffer");
    __shared__ float qsh[G][256];      // rotated query (scaled)
    __shared__ float ssh[kRopeDecSlots];
    __shared__ float mred[4][G];
    float (*red)[G][256] = reinterpret_cast<float (*)[G][256]>(ssh);

    const int s = wg_id_x();
    const int bg = wg_id_y();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int tid = lane_id_x();
    const int lane = tid & 63, wave = tid >> 6;
    const int n_lat = imax(0, len - w);
    const bool latent = s < n_lat_split;
    int t_begin, ntok;
    if (latent) {
        t_begin = s * chunk_lat;
        ntok = imin(chunk_lat, n_lat - t_begin);
    } else {
        t_begin = n_lat + (s - n_lat_split) * chunk_win;
        ntok = imin(chunk_win, len - t_begin);
    }
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;
    const int half = r / 2;

    // the query rotated at position len - 1, scaled by log2(e)/sqrt(d)
    const float* cq = tab + (size_t)(len - 1) * r;
    for (int idx = tid; idx < G * d; idx += kRopeDecThreads) {
        const int hh = idx / d, e = idx - (idx / d) * d;
        const T* qrow = q + ((size_t)b * Hq + (size_t)g * G + hh) * d;
        float y;
        if (e < half)
            y = __builtin_fmaf(elem<T>::load(qrow + e), cq[e], -(elem<T>::load(qrow + e + half) * cq[half + e]));
        else if (e < r)
            y = __builtin_fmaf(elem<T>::load(qrow + e), cq[e - half], elem<T>::load(qrow + e - half) * cq[e]);
        else
            y = elem<T>::load(qrow + e);
        qsh[hh][e] = y * qscale;
    }
    __syncthreads();

    const int lpt = lanes_per_row_rope(d);
    const int sub = tid & (lpt - 1);
    const int tpi = kRopeDecThreads / lpt;
    const int off = sub * 8;

    // pass 1: scores, at full d in both regions
    float mloc[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) mloc[hh] = -INFINITY;
    for (int t0 = 0; t0 < ntok; t0 += tpi) {
        const int t = t0 + tid / lpt;
        const int pos = t_begin + imin(t, ntok - 1);
        float x[8];
        if (latent) {
            const T* crow = k_lat + ((size_t)bg * cap + pos) * dd;
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = 0.f;
            for (int c = 0; c < dd; ++c) {
                const float cc = elem<T>::load(crow + c);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int e = imin(off + j, d - 1);
                    const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                        : elem<T>::load(wdg + (size_t)e * dd + c);
                    x[j] = __builtin_fmaf(cc, u, x[j]);
                }
            }
        } else {
            const T* krow = k_win + ((size_t)bg * w + pos % w) * d;
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = off + j < d ? elem<T>::load(krow + off + j) : 0.f;
        }
        const float* ca = tab + (size_t)pos * r;
        float sc[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int e = off + j;
                if (e >= d) break;
                float coef;  // element e of RoPE_pos^T Qr
                if (e < half) coef = __builtin_fmaf(qsh[hh][e], ca[e], qsh[hh][e + half] * ca[half + e]);
                else if (e < r) coef = __builtin_fmaf(qsh[hh][e], ca[e - half], -(qsh[hh][e - half] * ca[e]));
                else coef = qsh[hh][e];
                a = __builtin_fmaf(coef, x[j], a);
            }
            for (int o2 = 1; o2 < lpt; o2 <<= 1) a += __shfl_xor(a, o2, 64);
            sc[hh] = a;
        }
        if (t < ntok) {
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                mloc[hh] = fmaxf(mloc[hh], sc[hh]);
                if (sub == 0) ssh[hh * (kRopeDecSlots / G) + t] = sc[hh];
            }
        }
    }
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        const float mw = wave_max(mloc[hh]);
        if (lane == 0) mred[wave][hh] = mw;
    }
    __syncthreads();
    float mx[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
        mx[hh] = fmaxf(fmaxf(mred[0][hh], mred[1][hh]), fmaxf(mred[2][hh], mred[3][hh]));

    // pass 2: values (latent c^V in d_down space, ring values at d)
    const int dim = latent ? dd : d;
    const int lpv = lanes_per_row_rope(dim);
    const int subv = tid & (lpv - 1);
    const int tpv = kRopeDecThreads / lpv;
    const int offv = subv * 8;
    float acc[G][8];
    float lsum[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        lsum[hh] = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[hh][j] = 0.f;
    }
    for (int t0 = 0; t0 < ntok; t0 += tpv) {
        const int t = t0 + tid / lpv;
        if (t < ntok) {
            const int pos = t_begin + t;
            const T* vrow = latent ? v_lat + ((size_t)bg * cap + pos) * dd
                                   : v_win + ((size_t)bg * w + pos % w) * d;
            float x[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = offv + j < dim ? elem<T>::load(vrow + offv + j) : 0.f;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                const float p = exp2f(ssh[hh * (kRopeDecSlots / G) + t] - mx[hh]);
                if (subv == 0) lsum[hh] += p;
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[hh][j] = __builtin_fmaf(p, x[j], acc[hh][j]);
            }
        }
    }
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        lsum[hh] = wave_sum(lsum[hh]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float a = acc[hh][j];
            for (int o2 = lpv; o2 < 64; o2 <<= 1) a += __shfl_xor(a, o2, 64);
            acc[hh][j] = a;
        }
    }
    __syncthreads();  // scores and mred are reused below
    if (lane < lpv) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (offv + j < dim) red[wave][hh][offv + j] = acc[hh][j];
    }
    if (lane == 0) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) mred[wave][hh] = lsum[hh];
    }
    __syncthreads();
    const int stride = 2 + dd + d;
    const int lo = latent ? 2 : 2 + dd;
    for (int idx = tid; idx < G * stride; idx += kRopeDecThreads) {
        const int hh = idx / stride, f = idx - (idx / stride) * stride;
        float val = 0.f;
        if (f == 0) val = mx[hh];
        else if (f == 1) val = mred[0][hh] + mred[1][hh] + mred[2][hh] + mred[3][hh];
        else if (f >= lo && f < lo + dim)
            val = red[0][hh][f - lo] + red[1][hh][f - lo] + red[2][hh][f - lo] + red[3][hh][f - lo];
        const size_t bh = (size_t)b * Hq + (size_t)g * G + hh;
        part[(bh * S + s) * stride + f] = val;
    }
}

template <typename T, int G>
static hipError_t launch_decode_rope_g(const T* q, const T* wd, const T* wu, const T* k_win,
                                       const T* v_win, const T* k_lat, const T* v_lat,
                                       const float* tab, T* o, float* part, int B, int Hq, int Hkv,
                                       int d, int dd, int w, int cap, int len, int r,
                                       hipStream_t st) {
    DecodeSplits sp = decode_splits(len, w, d, dd, G);
    const int S = sp.n_lat_split + sp.n_win_split;
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    hipLaunchKernelGGL((decode_rope_split_kernel<T, G>), dim3(S, B * Hkv), dim3(kRopeDecThreads), 0,
                       st, q, wd, wu, k_win, v_win, k_lat, v_lat, tab, part, Hq, Hkv, d, dd, w, cap,
                       len, r, sp.chunk_lat, sp.chunk_win, sp.n_lat_split, S, qscale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_decode_combine<T>(part, wd, wu, o, B, Hq, Hkv, d, dd, S, st);
}

template <typename T>
hipError_t launch_decode_rope(const T* q, const T* wd, const T* wu, const T* k_win, const T* v_win,
                              const T* k_lat, const T* v_lat, const float* tab, int n_pos, T* o,
                              float* part, int B, int Hq, int Hkv, int d, int dd, int w, int cap,
                              int len, int r, hipStream_t st) {
    if (decode_mfma_rope_supported(d, dd, Hq / Hkv, r, sizeof(T) == 2)) {
        int P = 0;
        hipError_t e = launch_decode_mfma_rope((const bf16_t*)q, (const bf16_t*)wd, (const bf16_t*)wu,
                                               (const bf16_t*)k_win, (const bf16_t*)v_win,
                                               (const bf16_t*)k_lat, (const bf16_t*)v_lat, tab, n_pos,
                                               part, (bf16_t*)o, B, Hq, Hkv, dd, w, cap, len, r, P, st,
                                               d);
        if (e != hipSuccess || P == 1) return e;
        return launch_decode_combine<T>(part, wd, wu, o, B, Hq, Hkv, d, dd, P, st);
    }
    switch (Hq / Hkv) {
        case 1: return launch_decode_rope_g<T, 1>(q, wd, wu, k_win, v_win, k_lat, v_lat, tab, o, part, B, Hq, Hkv, d, dd, w, cap, len, r, st);
        case 2: return launch_decode_rope_g<T, 2>(q, wd, wu, k_win, v_win, k_lat, v_lat, tab, o, part, B, Hq, Hkv, d, dd, w, cap, len, r, st);
        case 4: return launch_decode_rope_g<T, 4>(q, wd, wu, k_win, v_win, k_lat, v_lat, tab, o, part, B, Hq, Hkv, d, dd, w, cap, len, r, st);
        case 8: return launch_decode_rope_g<T, 8>(q, wd, wu, k_win, v_win, k_lat, v_lat, tab, o, part, B, Hq, Hkv, d, dd, w, cap, len, r, st);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_decode_rope<float>(const float*, const float*, const float*, const float*,
                                              const float*, const float*, const float*, const float*,
                                              int, float*, float*, int, int, int, int, int, int, int,
                                              int, int, hipStream_t);
template hipError_t launch_decode_rope<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                               const bf16_t*, const bf16_t*, const bf16_t*,
                                               const bf16_t*, const float*, int, bf16_t*, float*, int,
                                               int, int, int, int, int, int, int, int, hipStream_t);

}  // namespace dar
