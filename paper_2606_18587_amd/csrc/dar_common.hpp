// Shared device helpers for the DAR kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dar {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

// Element traits: storage type <-> fp32.
template <typename T> struct elem;

template <> struct elem<float> {
    static __device__ __forceinline__ float load(const float* p) { return *p; }
    static __device__ __forceinline__ float to_f32(float x) { return x; }
    static __device__ __forceinline__ float from_f32(float x) { return x; }
};

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

template <> struct elem<bf16_t> {
    static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ float to_f32(bf16_t x) { return bf16_to_f32(x); }
    static __device__ __forceinline__ bf16_t from_f32(float x) { return f32_to_bf16(x); }
};

// Eq. 1 for one output column: c = sum_e x[e] * W_down[e][col], fp32 fused
// multiply-adds in increasing e. The vector-ALU kernels that produce a latent
// go through this function; on the matrix-core shapes (bf16, d 64/128,
// d_down 16/32) every latent comes from the MFMA projection instead (a fixed
// order too). Either way all latent producers of one shape share the same
// arithmetic, so prefill latents, bulk appends and single-token appends are
// bit-identical.
template <typename T>
__device__ __forceinline__ float project_col(const T* __restrict__ x, const T* __restrict__ wd,
                                             int d, int dd, int col) {
    float acc = 0.f;
    for (int e = 0; e < d; ++e)
        acc = __builtin_fmaf(elem<T>::load(x + e), elem<T>::load(wd + (size_t)e * dd + col), acc);
    return acc;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
    return x;
}

// Maximum over the 64 lanes with DPP lane moves (no LDS crossbar): quads,
// half rows, rows, then the two row broadcasts; lane 63 ends with the
// maximum, which is broadcast through a scalar register.
__device__ __forceinline__ float wave_max_dpp(float x) {
    auto step = [](float v, int ctrl, int row_mask) -> float {
        const int u = __float_as_int(v);
        int t;
        switch (ctrl) {  // the DPP control must be a constant
            case 0xB1: t = __builtin_amdgcn_update_dpp(u, u, 0xB1, 0xF, 0xF, false); break;
            case 0x4E: t = __builtin_amdgcn_update_dpp(u, u, 0x4E, 0xF, 0xF, false); break;
            case 0x141: t = __builtin_amdgcn_update_dpp(u, u, 0x141, 0xF, 0xF, false); break;
            case 0x140: t = __builtin_amdgcn_update_dpp(u, u, 0x140, 0xF, 0xF, false); break;
            case 0x142: t = __builtin_amdgcn_update_dpp(u, u, 0x142, 0xA, 0xF, false); break;
            default: t = __builtin_amdgcn_update_dpp(u, u, 0x143, 0xC, 0xF, false); break;
        }
        (void)row_mask;
        return fmaxf(v, __int_as_float(t));
    };
    x = step(x, 0xB1, 0xF);   // quad_perm [1,0,3,2]
    x = step(x, 0x4E, 0xF);   // quad_perm [2,3,0,1]
    x = step(x, 0x141, 0xF);  // row_half_mirror
    x = step(x, 0x140, 0xF);  // row_mirror
    x = step(x, 0x142, 0xA);  // row_bcast:15
    x = step(x, 0x143, 0xC);  // row_bcast:31
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// Storage position of latent column c (inside its group of 16) in the
// matrix-core prefill workspace: the two middle quads are swapped, so that
// the 8 contiguous bf16 a lane reads are the columns its query operand holds.
__host__ __device__ inline int latent_pos(int c) {
    const int q = (c >> 2) & 3;
    const int qq = (q == 1) ? 2 : (q == 2 ? 1 : q);
    return (c & ~15) | (qq << 2) | (c & 3);
}

// Workgroup and work-item indices read from the hardware registers. The
// blockIdx / threadIdx accessors go through device-library functions, which
// the compiler does not inline into code built with IEEE mode off
// (-mno-amdgpu-ieee): they become calls, and the workgroup index then lives
// in a vector register, so everything derived from it looks divergent.
__device__ __forceinline__ int wg_id_x() { return (int)__builtin_amdgcn_workgroup_id_x(); }
__device__ __forceinline__ int wg_id_y() { return (int)__builtin_amdgcn_workgroup_id_y(); }
__device__ __forceinline__ int wg_id_z() { return (int)__builtin_amdgcn_workgroup_id_z(); }
__device__ __forceinline__ int lane_id_x() { return (int)__builtin_amdgcn_workitem_id_x(); }

__device__ __forceinline__ int imin(int a, int b) { return a < b ? a : b; }
__device__ __forceinline__ int imax(int a, int b) { return a > b ? a : b; }

}  // namespace dar
