// Operand helpers for the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16),
// shared by the backward kernels.
//
// Operand layouts of the 32x32x16 bf16 instruction, lane l = 0..63:
//   A (32 x 16): lane l holds A[l % 32][8 (l / 32) + 0..7]
//   B (16 x 32): lane l holds B[8 (l / 32) + 0..7][l % 32]
//   C (32 x 32): register r of lane l holds C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32]
// So A is read as 16 contiguous bytes of a row-major [row][k] matrix, and B as
// 16 contiguous bytes of a row-major [col][k] matrix (B transposed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dar_common.hpp"

namespace dar {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

__device__ __forceinline__ bf16x8_t load_bf16x8(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}

__device__ __forceinline__ bf16x8_t zero_bf16x8() {
    return __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
}

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Eight consecutive accumulator registers x[o..o+7] as one bf16 operand.
__device__ __forceinline__ bf16x8_t pack8(const f32x16_t& x, int o, float f = 1.f) {
    return __builtin_bit_cast(bf16x8_t,
                              make_uint4(pack2(x[o] * f, x[o + 1] * f), pack2(x[o + 2] * f, x[o + 3] * f),
                                         pack2(x[o + 4] * f, x[o + 5] * f),
                                         pack2(x[o + 6] * f, x[o + 7] * f)));
}

// x[o..o+7] * f as a bf16 pair hi + lo (hi = bf16(v), lo = bf16(v - hi)):
// two products with hi and lo carry about 16 significant bits of v.
__device__ __forceinline__ void split8(const f32x16_t& x, int o, float f, bf16x8_t& hi,
                                       bf16x8_t& lo) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float a = x[o + 2 * k] * f, b = x[o + 2 * k + 1] * f;
        h[k] = pack2(a, b);
        const float ha = __uint_as_float(h[k] << 16), hb = __uint_as_float(h[k] & 0xffff0000u);
        l[k] = pack2(a - ha, b - hb);
    }
    hi = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
    lo = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}

__device__ __forceinline__ f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16_t splat16(float x) {
    f32x16_t r;
#pragma unroll
    for (int k = 0; k < 16; ++k) r[k] = x;
    return r;
}

// Workgroup -> (block, head) for a 1-D grid of nblk * BH workgroups, block 0
// first. Workgroups are dealt to the 8 XCDs round-robin; when BH % 8 == 0 all
// blocks of a head go to one XCD, so an XCD's L2 holds the operands of BH/8
// heads instead of all of them.
__device__ __forceinline__ void xcd_block_head(int L, int BH, int& blk, int& head) {
    if ((BH & 7) == 0) {
        const int xcd = L & 7, local = L >> 3, hpx = BH >> 3;
        blk = local / hpx;
        head = (local - blk * hpx) * 8 + xcd;
    } else {
        blk = L / BH;
        head = L - blk * BH;
    }
}

// Dot product of two 8-element bf16 operands, fp32 accumulation.
__device__ __forceinline__ float dot8(bf16x8_t a, bf16x8_t b, float acc) {
    const uint4 ua = __builtin_bit_cast(uint4, a), ub = __builtin_bit_cast(uint4, b);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.x), __builtin_bit_cast(bf16x2_t, ub.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.y), __builtin_bit_cast(bf16x2_t, ub.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.z), __builtin_bit_cast(bf16x2_t, ub.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.w), __builtin_bit_cast(bf16x2_t, ub.w), acc, false);
    return acc;
}

// Lanes l and l ^ 32 hold the same output column: combine them.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// With the A rows read in perm_row order, accumulator register r of a lane in
// half g holds output row acc_row(r, g): registers 0..7 are rows 8g..8g+7 and
// registers 8..15 rows 16+8g..16+8g+7, i.e. exactly the B operand layout of
// the next product over that index (two 16-wide k chunks), with no data
// movement.
__device__ __forceinline__ int acc_row(int r, int g) { return 16 * (r >> 3) + 8 * g + (r & 7); }

__device__ __forceinline__ int perm_row(int R) {
    const int a = R >> 3, gg = (R >> 2) & 1, b = R & 3;
    return 16 * (a >> 1) + 8 * gg + 4 * (a & 1) + b;
}

// A operand from a row-major LDS matrix M[k][col] read transposed: A rows are
// columns col0 + l % 32, k = k0 + 8 (l / 32) + 0..7 (two 64-bit transposing
// reads; ld and col0 multiples of 4 elements).
__device__ __forceinline__ bf16x8_t lds_tr_operand(const bf16_t* m, int ld, int k0, int col0,
                                                   int lane) {
    const int quad = lane >> 4, sl = lane & 15;
    const int kk = k0 + 8 * (quad >> 1) + (sl >> 2);
    const int col = col0 + 16 * (quad & 1) + 4 * (sl & 3);
    const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(m + kk * ld + col));
    const s16x4_t hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(m + (kk + 4) * ld + col));
    const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
    return __builtin_bit_cast(bf16x8_t, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
}

}  // namespace dar
