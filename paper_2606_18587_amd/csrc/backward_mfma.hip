// Matrix-core (MFMA) backward of the causal DAR prefill, bf16 storage, fp32
// accumulation, gfx950. The gradient formulas are those of the vector-ALU
// backward (backward.hip): one softmax over both regions (its log-sum-exp is
// the forward's), window pairs at full d, distant pairs in d_down space with
// W_up absorbed.
//
// Kernels, in launch order:
//  * bwd_prep_rows_kernel / bwd_prep_keys_kernel: q~ = q W_up^T (scaled by
//    log2(e)/sqrt(d)), dO~ = dO W_up^T, delta = dO . O and the log-sum-exp in
//    log2 units per query row; the latents c^K, c^V (Eq. 1) per key; all
//    operands bf16, each also stored in 32-token blocks transposed
//    ([T/32][d_down][32]) for the products that contract over tokens. Token
//    counts are padded to a multiple of 32 with zero rows.
//  * bwd_rows_dist_kernel: one wavefront per 32 query rows, distant keys only
//    (d_down wide), scores transposed (S^T = c^K q~^T, one query per lane
//    column, as in the forward): h^T += c^K^T dS^T and ol^T += c^V^T P^T.
//  * bwd_cols_dist_kernel: one wavefront per 32 keys, distant rows only, scores
//    in the other orientation (S = q~ c^K^T, one key per lane column) so that
//    P and dS are directly the B operands of gK^T += q~^T dS, gV^T += dO~^T P.
//  * bwd_rows_local_kernel: window keys at full d through LDS tiles,
//    dq^T += K^T dS^T (K^T read transposed from LDS); the epilogue adds the
//    lifted distant part (h W_up, h as a bf16 hi + lo pair) and the
//    workgroup's share of dW_up.
//  * bwd_cols_local_kernel: window rows, dV^T += dO^T P and dK^T += Q^T dS;
//    the epilogue adds gK W_down^T, gV W_down^T and the workgroup's share of
//    dW_down.
//  * bwd_wreduce_kernel (backward.hip): the shares summed in a fixed order.
// No kernel accumulates with atomics, so the result does not depend on
// timing. Masked pairs get a score of -inf (P = 0, dS = 0). Each row's
// exponentials use its log-sum-exp as the reference, fed as the accumulator
// input of the score product (distant) or through one FMA (window), and
// -delta is the accumulator input of dP, so dS = P * dP' needs one multiply.
#include "../../include/dar.h"
#include "dar_common.hpp"
#include "dar_kernels.hpp"
#include "mfma_common.hpp"

namespace dar {

namespace {

constexpr float kLog2eB = 1.4426950408889634f;

// 16 floats of a per-token array for the tokens acc_row(r, g) of a 32-token
// block: two runs of 8.
__device__ __forceinline__ f32x16_t load_row16(const float* p, int g, float sign) {
    const float4 a = *reinterpret_cast<const float4*>(p + 8 * g);
    const float4 b = *reinterpret_cast<const float4*>(p + 8 * g + 4);
    const float4 c = *reinterpret_cast<const float4*>(p + 16 + 8 * g);
    const float4 d = *reinterpret_cast<const float4*>(p + 16 + 8 * g + 4);
    f32x16_t r;
    r[0] = sign * a.x; r[1] = sign * a.y; r[2] = sign * a.z; r[3] = sign * a.w;
    r[4] = sign * b.x; r[5] = sign * b.y; r[6] = sign * b.z; r[7] = sign * b.w;
    r[8] = sign * c.x; r[9] = sign * c.y; r[10] = sign * c.z; r[11] = sign * c.w;
    r[12] = sign * d.x; r[13] = sign * d.y; r[14] = sign * d.z; r[15] = sign * d.w;
    return r;
}

// Store 4 consecutive fp32 accumulator registers as 4 bf16 (8 bytes).
__device__ __forceinline__ void store_bf16x4(bf16_t* p, float a, float b, float c, float d) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack2(a, b), pack2(c, d));
}

// A operand rows of a transposed latent block [32][32] (latent rows past
// d_down are zero): row R carries latent column perm_row(R), so the
// accumulator rows come out in B-operand order; tokens 16 half + 8 g + 0..7.
__device__ __forceinline__ bf16x8_t latT_operand(const bf16_t* blk, int qc, int hg, int half) {
    return load_bf16x8(blk + (size_t)perm_row(qc) * 32 + 16 * half + 8 * hg);
}

// Eight bf16 [hi, mid, lo, 0, 0, 0, 0, 0] of -x: hi + mid + lo carries about
// 24 significant bits of -x once summed in fp32.
__device__ __forceinline__ uint4 neg_split3(float x) {
    const float v = -x;
    const uint32_t h = pack2(v, 0.f) & 0xffffu;
    const float r1 = v - __uint_as_float(h << 16);
    const uint32_t m = pack2(r1, 0.f) & 0xffffu;
    const float r2 = r1 - __uint_as_float(m << 16);
    const uint32_t lo = pack2(r2, 0.f) & 0xffffu;
    return make_uint4(h | (m << 16), lo, 0u, 0u);
}

// B operand that sums the first three k slots of half `g1` (ones there, zeros
// elsewhere): with the row-constant A operand it adds -lse (g1 = 0) or
// -delta (g1 = 1) to every accumulator of the row.
__device__ __forceinline__ bf16x8_t ones3(int hg, int g1) {
    return hg == g1 ? __builtin_bit_cast(bf16x8_t, make_uint4(0x3f803f80u, 0x3f80u, 0u, 0u))
                    : zero_bf16x8();
}

// 8 fp32 values (16-byte aligned) times f, as a bf16 hi + lo pair.
__device__ __forceinline__ void split_load8(const float* p, float f, bf16x8_t& hi, bf16x8_t& lo) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    f32x16_t x;
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    split8(x, 0, f, hi, lo);
}

// 8 fp32 values (16-byte aligned) times f, as one bf16 operand.
__device__ __forceinline__ bf16x8_t pack_load8(const float* p, float f) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    return __builtin_bit_cast(bf16x8_t, make_uint4(pack2(a.x * f, a.y * f), pack2(a.z * f, a.w * f),
                                                   pack2(b.x * f, b.y * f), pack2(b.z * f, b.w * f)));
}

// Workgroup share of a weight gradient: every wavefront adds its C tiles
// (rows e = 32 t + accumulator row, column c = lane % 32 < DD) into pbuf in
// wavefront order, then the workgroup writes pbuf [D][DD] to `out`. Every
// wavefront of the workgroup must call this (it holds barriers).
template <int D, int DD, int NW>
__device__ __forceinline__ void wg_share(const f32x16_t (&acc)[D / 32], float* pbuf, int wave,
                                         int lane, int tid, float* __restrict__ out) {
    const int qc = lane & 31, hg = lane >> 5;
#pragma unroll
    for (int wv = 0; wv < NW; ++wv) {
        if (wave == wv && qc < DD) {
#pragma unroll
            for (int t = 0; t < D / 32; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int e = 32 * t + 8 * (r >> 2) + 4 * hg + (r & 3);
                    float* cell = pbuf + e * DD + qc;
                    *cell = (wv == 0) ? acc[t][r] : *cell + acc[t][r];
                }
        }
        __syncthreads();
    }
    for (int idx = tid; idx < D * DD; idx += NW * 64) out[idx] = pbuf[idx];
}

// Cooperative staging of a 64-row tile of two row-major [rows][D] bf16 arrays
// through registers into LDS (rows at or past `n` read as zero): fetch() for
// the next tile is issued before the current one is computed on, so its
// global latency hides behind that work.
template <int D, int NW>
struct TilePair {
    static constexpr int C8 = D / 8, PER = 64 * C8 / (NW * 64);  // 16-byte chunks per thread
    uint4 a[PER], b[PER];
    __device__ __forceinline__ void fetch(const bf16_t* ga, const bf16_t* gb, int t, int n,
                                          int tid) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int idx = tid + u * NW * 64;
            const int row = t + idx / C8, c8 = idx % C8;
            const size_t off = (size_t)imin(row, n - 1) * D + c8 * 8;  // clamped: no branch
            a[u] = *reinterpret_cast<const uint4*>(ga + off);
            b[u] = *reinterpret_cast<const uint4*>(gb + off);
            if (row >= n) {
                a[u] = make_uint4(0, 0, 0, 0);
                b[u] = make_uint4(0, 0, 0, 0);
            }
        }
    }
    __device__ __forceinline__ void store(bf16_t* la, bf16_t* lb, int ld, int tid) const {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int idx = tid + u * NW * 64;
            const int r = idx / C8, c8 = idx % C8;
            *reinterpret_cast<uint4*>(la + r * ld + c8 * 8) = a[u];
            *reinterpret_cast<uint4*>(lb + r * ld + c8 * 8) = b[u];
        }
    }
};

}  // namespace

// ---------------------------------------------------------------- preparation

// Per query row i (padded rows get zeros): q~s = (q W_up^T) log2(e)/sqrt(d)
// and dO~ = dO W_up^T in bf16, row-major and in transposed 32-row blocks, and
// -delta = -dO . O and -lse (the forward's, in log2 units), in fp32 and as
// bf16 hi + mid + lo row constants. One wavefront per 32 rows on the matrix
// cores: U W^T with U = W_up gives one latent row per lane column (the
// row-major store), Q U^T one token per lane column (the transposed store);
// latent rows past d_down come out zero from U's zero rows.
// Grid: (Tr / (32 NW), B * Hq).
template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_prep_rows_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ o, const bf16_t* __restrict__ dout,
    const float* __restrict__ lse, const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu,
    bf16_t* __restrict__ qts, bf16_t* __restrict__ qtT, bf16_t* __restrict__ dts,
    bf16_t* __restrict__ dtT, bf16_t* __restrict__ rc, float* __restrict__ nd,
    float* __restrict__ nl2, int Hq, int Hkv, int T, int Tr, float qscale) {
    constexpr int KS = D / 16, DS = DD / 16, LDU = D + 8;
    __shared__ __attribute__((aligned(16))) bf16_t U[32 * LDU];  // U[c][e] = W_up[c][e]
    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int bh = wg_id_y();
    const int g = (bh % Hq) / (Hq / Hkv);
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
    // (all of this thread's elements requested at once, indices clamped, no
    // load under a branch: one memory round trip before the barrier)
    constexpr int UPT = 32 * D / (NW * 64);
    bf16_t uv[UPT];
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
        const int idx = tid + j * NW * 64, c = imin(idx / D, DD - 1), e = idx % D;
        uv[j] = *(wug ? wug + (size_t)c * D + e : wdg + (size_t)e * DD + c);
    }
    // the rows and the row's lse are requested now too, so that the whole
    // kernel waits for one memory round trip (rows clamped into the array and
    // zeroed past T afterwards: no load under a branch)
    const int r0 = wg_id_x() * NW * 32 + wave * 32;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int rb = r0 + qc, ra = r0 + prow;  // B-layout row, A-layout row
    const int rbc = imin(rb, T - 1), rac = imin(ra, T - 1);
    const bf16_t* qh = q + (size_t)bh * T * D;
    const bf16_t* dh = dout + (size_t)bh * T * D;
    const bf16_t* oh = o + (size_t)bh * T * D;
    bf16x8_t qB[KS], dB[KS], oB[KS], qA[KS], dA[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int e = s * 16 + hg * 8;
        qB[s] = load_bf16x8(qh + (size_t)rbc * D + e);
        dB[s] = load_bf16x8(dh + (size_t)rbc * D + e);
        oB[s] = load_bf16x8(oh + (size_t)rbc * D + e);
        qA[s] = load_bf16x8(qh + (size_t)rac * D + e);
        dA[s] = load_bf16x8(dh + (size_t)rac * D + e);
    }
    const float lse_r = lse[(size_t)bh * T + rbc];
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
        const int idx = tid + j * NW * 64, c = idx / D, e = idx % D;
        U[c * LDU + e] = c < DD ? uv[j] : (bf16_t)0;
    }
    // the rows are consumed here, so they are loaded ahead of the barrier
    // rather than at their first use behind the early return
#pragma unroll
    for (int s = 0; s < KS; ++s)
        __asm__ volatile("" ::"v"(qB[s]), "v"(dB[s]), "v"(oB[s]), "v"(qA[s]), "v"(dA[s]));
    __asm__ volatile("" ::"v"(lse_r));
    __syncthreads();
    if (r0 >= Tr) return;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        if (rb >= T) { qB[s] = zero_bf16x8(); dB[s] = zero_bf16x8(); oB[s] = zero_bf16x8(); }
        if (ra >= T) { qA[s] = zero_bf16x8(); dA[s] = zero_bf16x8(); }
    }
    // latent rows of row rb: U Q^T, A rows = latent columns in perm_row order
    f32x16_t qt = splat16(0.f), dt = splat16(0.f), qn = splat16(0.f), dn = splat16(0.f);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const bf16x8_t ua = load_bf16x8(U + prow * LDU + s * 16 + hg * 8);
        const bf16x8_t ub = load_bf16x8(U + qc * LDU + s * 16 + hg * 8);
        qt = mfma(ua, qB[s], qt);
        dt = mfma(ua, dB[s], dt);
        qn = mfma(qA[s], ub, qn);
        dn = mfma(dA[s], ub, dn);
    }
    const size_t prw = (size_t)bh * Tr + rb;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        *reinterpret_cast<bf16x8_t*>(qts + prw * DD + s * 16 + hg * 8) = pack8(qt, 8 * s, qscale);
        *reinterpret_cast<bf16x8_t*>(dts + prw * DD + s * 16 + hg * 8) = pack8(dt, 8 * s);
    }
    // transposed block: lane column = latent c, registers = tokens 8 hg + r, 16 + 8 hg + r
    const size_t blk = (((size_t)bh * (Tr / 32) + r0 / 32) * 32 + qc) * 32;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
        *reinterpret_cast<bf16x8_t*>(qtT + blk + 16 * h2 + 8 * hg) = pack8(qn, 8 * h2, qscale);
        *reinterpret_cast<bf16x8_t*>(dtT + blk + 16 * h2 + 8 * hg) = pack8(dn, 8 * h2);
    }
    float dl = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) dl = dot8(dB[s], oB[s], dl);
    dl = pair_sum(dl);
    if (hg == 0) {
        const float L2 = rb < T ? lse_r * kLog2eB : 0.f;
        nd[prw] = -dl;
        nl2[prw] = -L2;
        *reinterpret_cast<uint4*>(rc + prw * 16) = neg_split3(L2);
        *reinterpret_cast<uint4*>(rc + prw * 16 + 8) = neg_split3(dl);
    }
}

// Per key token j (padded rows get zeros): c^K = k W_down, c^V = v W_down
// (Eq. 1) in bf16, row-major and in transposed 32-token blocks, computed as
// in bwd_prep_rows_kernel with U = W_down^T. Grid: (Tr / (32 NW), B * Hkv).
template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_prep_keys_kernel(
    const bf16_t* __restrict__ k, const bf16_t* __restrict__ v, const bf16_t* __restrict__ wd,
    bf16_t* __restrict__ ckb, bf16_t* __restrict__ ckT, bf16_t* __restrict__ cvb,
    bf16_t* __restrict__ cvT, int Hkv, int T, int Tr) {
    constexpr int KS = D / 16, DS = DD / 16, LDU = D + 8;
    __shared__ __attribute__((aligned(16))) bf16_t U[32 * LDU];  // U[c][e] = W_down[e][c]
    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int bg = wg_id_y();
    const bf16_t* wdg = wd + (size_t)(bg % Hkv) * D * DD;
    // (all of this thread's elements requested at once, indices clamped, no
    // load under a branch: one memory round trip before the barrier)
    constexpr int UPT = 32 * D / (NW * 64);
    bf16_t uv[UPT];
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
        const int idx = tid + j * NW * 64, c = imin(idx / D, DD - 1), e = idx % D;
        uv[j] = wdg[(size_t)e * DD + c];
    }
    // rows requested before the barrier, clamped and zeroed past T afterwards,
    // as in bwd_prep_rows_kernel
    const int r0 = wg_id_x() * NW * 32 + wave * 32;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int rb = r0 + qc, ra = r0 + prow;
    const int rbc = imin(rb, T - 1), rac = imin(ra, T - 1);
    const bf16_t* kh = k + (size_t)bg * T * D;
    const bf16_t* vh = v + (size_t)bg * T * D;
    bf16x8_t kB[KS], vB[KS], kA[KS], vA[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int e = s * 16 + hg * 8;
        kB[s] = load_bf16x8(kh + (size_t)rbc * D + e);
        vB[s] = load_bf16x8(vh + (size_t)rbc * D + e);
        kA[s] = load_bf16x8(kh + (size_t)rac * D + e);
        vA[s] = load_bf16x8(vh + (size_t)rac * D + e);
    }
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
        const int idx = tid + j * NW * 64, c = idx / D, e = idx % D;
        U[c * LDU + e] = c < DD ? uv[j] : (bf16_t)0;
    }
#pragma unroll
    for (int s = 0; s < KS; ++s)
        __asm__ volatile("" ::"v"(kB[s]), "v"(vB[s]), "v"(kA[s]), "v"(vA[s]));
    __syncthreads();
    if (r0 >= Tr) return;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        if (rb >= T) { kB[s] = zero_bf16x8(); vB[s] = zero_bf16x8(); }
        if (ra >= T) { kA[s] = zero_bf16x8(); vA[s] = zero_bf16x8(); }
    }
    f32x16_t kt = splat16(0.f), vt = splat16(0.f), kn = splat16(0.f), vn = splat16(0.f);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const bf16x8_t ua = load_bf16x8(U + prow * LDU + s * 16 + hg * 8);
        const bf16x8_t ub = load_bf16x8(U + qc * LDU + s * 16 + hg * 8);
        kt = mfma(ua, kB[s], kt);
        vt = mfma(ua, vB[s], vt);
        kn = mfma(kA[s], ub, kn);
        vn = mfma(vA[s], ub, vn);
    }
    const size_t prw = (size_t)bg * Tr + rb;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        *reinterpret_cast<bf16x8_t*>(ckb + prw * DD + s * 16 + hg * 8) = pack8(kt, 8 * s);
        *reinterpret_cast<bf16x8_t*>(cvb + prw * DD + s * 16 + hg * 8) = pack8(vt, 8 * s);
    }
    const size_t blk = (((size_t)bg * (Tr / 32) + r0 / 32) * 32 + qc) * 32;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
        *reinterpret_cast<bf16x8_t*>(ckT + blk + 16 * h2 + 8 * hg) = pack8(kn, 8 * h2);
        *reinterpret_cast<bf16x8_t*>(cvT + blk + 16 * h2 + 8 * hg) = pack8(vn, 8 * h2);
    }
}

// ---------------------------------------------------------------- distant tiles

// Cooperative copy of a 64-token operand tile through registers into LDS.
// The tile is up to five contiguous global segments of n_k 16-byte chunks
// (each a multiple of 64), laid out in LDS in the same order. Load u of
// wavefront `wave` moves the 64 chunks of group wave + NW u, so every load's
// segment is the same for the whole wavefront (no divergent address choice).
// seg_fetch() for the next tile is issued before the current one is computed
// on; the registers travel by value (a struct updated through a reference
// would be kept in scratch memory).
template <int NW, int NCH>
struct SegRegs {
    static_assert(NCH % 64 == 0, "tile segments are whole 64-chunk groups");
    static constexpr int NGRP = NCH / 64;
    static constexpr int PER = (NGRP + NW - 1) / NW;
    uint4 r[PER];
};

struct Segs {
    const uint4 *s0, *s1, *s2, *s3, *s4;
    int n0, n1, n2, n3;
};

template <int NW, int NCH>
__device__ __forceinline__ SegRegs<NW, NCH> seg_fetch(const Segs& g, int wave, int lane) {
    using R = SegRegs<NW, NCH>;
    R o;
#pragma unroll
    for (int u = 0; u < R::PER; ++u) {
        int grp = wave + NW * u;  // wave-uniform
        if (R::NGRP % NW != 0 && grp >= R::NGRP) grp = R::NGRP - 1;  // spare loads repeat a group
        const int c = grp * 64, b1 = g.n0, b2 = b1 + g.n1, b3 = b2 + g.n2, b4 = b3 + g.n3;
        const uint4* src = c < b1 ? g.s0 + c
                         : c < b2 ? g.s1 + (c - b1)
                         : c < b3 ? g.s2 + (c - b2)
                         : c < b4 ? g.s3 + (c - b3)
                                  : g.s4 + (c - b4);
        o.r[u] = src[lane];
    }
    return o;
}

// (lds points at the tile's first chunk, or at a later segment's)
template <int NW, int NCH>
__device__ __forceinline__ void seg_store(const SegRegs<NW, NCH> st, uint4* lds, int wave,
                                          int lane) {
    using R = SegRegs<NW, NCH>;
#pragma unroll
    for (int u = 0; u < R::PER; ++u) {
        const int grp = wave + NW * u;
        if (R::NGRP % NW == 0 || grp < R::NGRP) lds[grp * 64 + lane] = st.r[u];
    }
}

// ---------------------------------------------------------------- distant: h, ol

// One workgroup of NW wavefronts = 32 NW query rows of one (batch, query
// head); distant keys j <= i - w only. The d_down-wide key operands of each
// 64-key tile (c^K and c^V rows, their transposed blocks) are copied once into
// LDS for the workgroup, the next tile's loads in flight meanwhile. Tiles
// whose keys are distant for every row of the workgroup are computed without
// masks, both 32-key subtiles in one straight-line block so that the products
// of one overlap the exponentials of the other. Writes h = sum dS c^K and
// ol = sum P c^V (fp32) of every real row (zero without distant keys).
// Grid: ceil(T / (32 NW)) * B * Hq workgroups (xcd_block_head); row blocks
// with the most keys first.
template <int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_rows_dist_kernel(
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ ckT,
    const bf16_t* __restrict__ cvb, const bf16_t* __restrict__ cvT,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ dts,
    const float* __restrict__ nl2, const float* __restrict__ nd, float* __restrict__ hk,
    float* __restrict__ ol, int Hq, int Hkv, int T, int Tr, int w, int BH) {
    constexpr int DS = DD / 16, BM = NW * 32;
    constexpr int NK = 8 * DD, NT = 256;       // 16-byte chunks: 64 latent rows, 2 blocks
    constexpr int NCH = 2 * NK + 2 * NT;
    __shared__ __attribute__((aligned(16))) uint4 tile[NCH];
    const bf16_t* lck = reinterpret_cast<const bf16_t*>(tile);
    const bf16_t* lcv = lck + 64 * DD;
    const bf16_t* lkt = lcv + 64 * DD;
    const bf16_t* lvt = lkt + 2 * 1024;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nblk = (T + BM - 1) / BM;
    int rbi, bh;
    xcd_block_head(wg_id_x(), BH, rbi, bh);
    const int rb = nblk - 1 - rbi;  // row blocks with the most keys first
    const int b = bh / Hq, h = bh % Hq;
    const int bg = b * Hkv + h / (Hq / Hkv);
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc), lrow = perm_row(qc);
    const int i0 = rb * BM, r0 = i0 + wave * 32, i = r0 + qc;
    const bool live = r0 < T;
    const int i_hi = imin(r0 + 31, T - 1);
    const int ii = imin(i, T - 1);
    const int T32 = Tr / 32;
    const size_t prw = (size_t)bh * Tr + ii;

    bf16x8_t qtop[DS], dtop[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        qtop[s] = load_bf16x8(qts + prw * DD + s * 16 + hg * 8);
        dtop[s] = load_bf16x8(dts + prw * DD + s * 16 + hg * 8);
    }
    const f32x16_t negL = splat16(nl2[prw]), negd = splat16(nd[prw]);
    f32x16_t hT = splat16(0.f), olT = splat16(0.f);

    // one 32-key subtile at offset `sub` of the LDS tile (keys js..js+31)
    auto step = [&](int sub, int js, bool masked) {
        const bf16_t* ckr = lck + (sub * 32 + prow) * DD + hg * 8;
        const bf16_t* cvr = lcv + (sub * 32 + prow) * DD + hg * 8;
        f32x16_t x = mfma(load_bf16x8(ckr), qtop[0], negL);
        f32x16_t dp = mfma(load_bf16x8(cvr), dtop[0], negd);
        if (DS == 2) {
            x = mfma(load_bf16x8(ckr + 16), qtop[DS - 1], x);
            dp = mfma(load_bf16x8(cvr + 16), dtop[DS - 1], dp);
        }
        if (masked) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (js + acc_row(r, hg) > i - w) x[r] = -INFINITY;
        }
        f32x16_t p, ds;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            p[r] = __builtin_amdgcn_exp2f(x[r]);
            ds[r] = p[r] * dp[r];
        }
        const bf16_t* kt = lkt + sub * 1024 + lrow * 32 + hg * 8;
        const bf16_t* vt = lvt + sub * 1024 + lrow * 32 + hg * 8;
        hT = mfma(load_bf16x8(kt), pack8(ds, 0), hT);
        hT = mfma(load_bf16x8(kt + 16), pack8(ds, 8), hT);
        olT = mfma(load_bf16x8(vt), pack8(p, 0), olT);
        olT = mfma(load_bf16x8(vt + 16), pack8(p, 8), olT);
    };

    const int jd_wg = imin(i0 + BM - 1, T - 1) - w;  // last distant key of the workgroup
    const int jd_end = live ? i_hi - w : -1;         // ... of this wavefront
    if (jd_wg >= 0) {
        const uint4* g_ck = reinterpret_cast<const uint4*>(ckb + (size_t)bg * Tr * DD);
        const uint4* g_cv = reinterpret_cast<const uint4*>(cvb + (size_t)bg * Tr * DD);
        const uint4* g_kt = reinterpret_cast<const uint4*>(ckT + (size_t)bg * T32 * 1024);
        const uint4* g_vt = reinterpret_cast<const uint4*>(cvT + (size_t)bg * T32 * 1024);
        auto segs = [&](int t) {
            // rows t..t+63 (DD / 8 chunks each); transposed blocks t/32, t/32 + 1 (128 each)
            const size_t tb = (size_t)(t / 32) * 128;
            // four segments: the fifth is never read
            return Segs{g_ck + (size_t)t * DD / 8, g_cv + (size_t)t * DD / 8, g_kt + tb, g_vt + tb,
                        g_vt + tb, NK, NK, NT, NT};
        };
        SegRegs<NW, NCH> st = seg_fetch<NW, NCH>(segs(0), wave, lane);
        for (int t = 0; t <= jd_wg; t += 64) {
            __syncthreads();  // the previous tile is no longer read
            seg_store<NW, NCH>(st, tile, wave, lane);
            __syncthreads();
            if (t + 64 <= jd_wg) st = seg_fetch<NW, NCH>(segs(t + 64), wave, lane);
            const bool interior = t + 63 <= r0 - w;  // every key distant for every row
            if (live && interior) {
                step(0, t, false);
                step(1, t + 32, false);
            }
            if (live && !interior && t <= jd_end) step(0, t, t + 31 > r0 - w);
            if (live && !interior && t + 32 <= jd_end) step(1, t + 32, t + 63 > r0 - w);
        }
    }
    if (!live || i >= T) return;
    float* hr = hk + ((size_t)bh * T + i) * DD;
    float* orr = ol + ((size_t)bh * T + i) * DD;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const int c = 16 * s + 8 * hg;
        *reinterpret_cast<float4*>(hr + c) = make_float4(hT[8 * s], hT[8 * s + 1], hT[8 * s + 2], hT[8 * s + 3]);
        *reinterpret_cast<float4*>(hr + c + 4) = make_float4(hT[8 * s + 4], hT[8 * s + 5], hT[8 * s + 6], hT[8 * s + 7]);
        *reinterpret_cast<float4*>(orr + c) = make_float4(olT[8 * s], olT[8 * s + 1], olT[8 * s + 2], olT[8 * s + 3]);
        *reinterpret_cast<float4*>(orr + c + 4) = make_float4(olT[8 * s + 4], olT[8 * s + 5], olT[8 * s + 6], olT[8 * s + 7]);
    }
}

// ---------------------------------------------------------------- distant: gK, gV

// One workgroup of NW wavefronts = 32 NW keys of one (batch, KV head); the
// distant rows i >= j + w of every query head of the group. The row operands
// of each 64-row tile (q~ and dO~ rows, their transposed blocks, the row
// constants) are copied once into LDS for the workgroup, as in the query-side
// kernel. Each row's -lse and -delta enter through one more product each,
// the row-constant operand (hi + mid + lo) against ones3. Writes
// gK = sum dS q~ (q~ unscaled) and gV = sum P dO~ (fp32) of every real key.
// Grid: ceil(T / (32 NW)) * B * Hkv workgroups (xcd_block_head); key block 0
// (most rows) first.
template <int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_cols_dist_kernel(
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ cvb,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ qtT,
    const bf16_t* __restrict__ dts, const bf16_t* __restrict__ dtT,
    const bf16_t* __restrict__ rc, float* __restrict__ gk, float* __restrict__ gv, int Hq,
    int Hkv, int T, int Tr, int w, float gscale, int BKV) {
    constexpr int DS = DD / 16, BK = NW * 32;
    constexpr int NQ = 8 * DD, NT = 256, NC = 128;  // 16-byte chunks per 64-row tile
    constexpr int NCH = 2 * NQ + 2 * NT + NC;
    __shared__ __attribute__((aligned(16))) uint4 tile[NCH];
    const bf16_t* lq = reinterpret_cast<const bf16_t*>(tile);
    const bf16_t* ld = lq + 64 * DD;
    const bf16_t* lqt = ld + 64 * DD;
    const bf16_t* ldt = lqt + 2 * 1024;
    const bf16_t* lrc = ldt + 2 * 1024;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int cb, bg;
    xcd_block_head(wg_id_x(), BKV, cb, bg);
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int cwg = cb * BK;
    const int c0 = cwg + wave * 32, j = c0 + qc;
    const bool live = c0 < T;
    const int jj = imin(j, T - 1);
    const int T32 = Tr / 32;

    bf16x8_t ckop[DS], cvop[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        ckop[s] = load_bf16x8(ckb + ((size_t)bg * Tr + jj) * DD + s * 16 + hg * 8);
        cvop[s] = load_bf16x8(cvb + ((size_t)bg * Tr + jj) * DD + s * 16 + hg * 8);
    }
    const bf16x8_t b_lse = ones3(hg, 0), b_del = ones3(hg, 1);
    f32x16_t gkT = splat16(0.f), gvT = splat16(0.f);

    auto step = [&](int sub, int is, bool masked) {
        const bf16_t* qr = lq + (sub * 32 + prow) * DD + hg * 8;
        const bf16_t* dr = ld + (sub * 32 + prow) * DD + hg * 8;
        const bf16x8_t cst = load_bf16x8(lrc + (sub * 32 + prow) * 16 + hg * 8);
        f32x16_t x = mfma(cst, b_lse, splat16(0.f));
        f32x16_t dp = mfma(cst, b_del, splat16(0.f));
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            x = mfma(load_bf16x8(qr + s * 16), ckop[s], x);
            dp = mfma(load_bf16x8(dr + s * 16), cvop[s], dp);
        }
        if (masked) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int i = is + acc_row(r, hg);
                if (i - j < w || i >= T) x[r] = -INFINITY;
            }
        }
        f32x16_t p, ds;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            p[r] = __builtin_amdgcn_exp2f(x[r]);
            ds[r] = p[r] * dp[r];
        }
        const bf16_t* qt = lqt + sub * 1024 + prow * 32 + hg * 8;
        const bf16_t* dt = ldt + sub * 1024 + prow * 32 + hg * 8;
        gkT = mfma(load_bf16x8(qt), pack8(ds, 0), gkT);
        gkT = mfma(load_bf16x8(qt + 16), pack8(ds, 8), gkT);
        gvT = mfma(load_bf16x8(dt), pack8(p, 0), gvT);
        gvT = mfma(load_bf16x8(dt + 16), pack8(p, 8), gvT);
    };

    const int t0 = (cwg + w) & ~63;  // first row tile with a distant pair in the workgroup
    const int ntile = t0 < T ? (T - 1 - t0) / 64 + 1 : 0;
    const int ntot = G * ntile;
    // two copies per tile (the operand rows and blocks, then the row constants):
    // each keeps at most four loads per thread in registers
    constexpr int NA = NCH - NC;
    auto segs = [&](int n, bool consts) {
        const int hh = n / ntile, t = t0 + (n - hh * ntile) * 64;
        const size_t bh = (size_t)b * Hq + g * G + hh;
        const uint4* rcs = reinterpret_cast<const uint4*>(rc + (bh * Tr + t) * 16);
        if (consts) return Segs{rcs, rcs, rcs, rcs, rcs, NC, 0, 0, 0};
        return Segs{reinterpret_cast<const uint4*>(qts + (bh * Tr + t) * DD),
                    reinterpret_cast<const uint4*>(dts + (bh * Tr + t) * DD),
                    reinterpret_cast<const uint4*>(qtT + (bh * T32 + t / 32) * 1024),
                    reinterpret_cast<const uint4*>(dtT + (bh * T32 + t / 32) * 1024),
                    rcs, NQ, NQ, NT, NT};
    };
    if (ntot > 0) {  // workgroup-uniform
    SegRegs<NW, NA> sa = seg_fetch<NW, NA>(segs(0, false), wave, lane);
    SegRegs<NW, NC> sc = seg_fetch<NW, NC>(segs(0, true), wave, lane);
    for (int n = 0; n < ntot; ++n) {
        const int t = t0 + (n % ntile) * 64;
        __syncthreads();  // the previous tile is no longer read
        seg_store<NW, NA>(sa, tile, wave, lane);
        seg_store<NW, NC>(sc, tile + NA, wave, lane);
        __syncthreads();
        const int nn = imin(n + 1, ntot - 1);  // the last fetch repeats
        sa = seg_fetch<NW, NA>(segs(nn, false), wave, lane);
        sc = seg_fetch<NW, NC>(segs(nn, true), wave, lane);
        const bool interior = t >= c0 + 31 + w && t + 63 < T;  // every pair distant and real
        if (live && interior) {
            step(0, t, false);
            step(1, t + 32, false);
        }
        if (live && !interior && t + 31 >= c0 + w) step(0, t, true);
        if (live && !interior && t + 63 >= c0 + w && t + 32 < T) step(1, t + 32, true);
    }
    }
    if (!live || j >= T) return;
    float* gkr = gk + ((size_t)bg * T + j) * DD;
    float* gvr = gv + ((size_t)bg * T + j) * DD;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        const int c = 16 * s + 8 * hg;
        *reinterpret_cast<float4*>(gkr + c) =
            make_float4(gkT[8 * s] * gscale, gkT[8 * s + 1] * gscale, gkT[8 * s + 2] * gscale, gkT[8 * s + 3] * gscale);
        *reinterpret_cast<float4*>(gkr + c + 4) =
            make_float4(gkT[8 * s + 4] * gscale, gkT[8 * s + 5] * gscale, gkT[8 * s + 6] * gscale, gkT[8 * s + 7] * gscale);
        *reinterpret_cast<float4*>(gvr + c) = make_float4(gvT[8 * s], gvT[8 * s + 1], gvT[8 * s + 2], gvT[8 * s + 3]);
        *reinterpret_cast<float4*>(gvr + c + 4) = make_float4(gvT[8 * s + 4], gvT[8 * s + 5], gvT[8 * s + 6], gvT[8 * s + 7]);
    }
}

// ---------------------------------------------------------------- window: dq, dW_up

// One wavefront per 32 query rows, window keys i - w < j <= i through 64-key
// K/V tiles in LDS. Epilogue: dq = s (dq_win + h W_up) and the workgroup's
// share of dW_up^T = sum_i q_i^T (s h_i) + dO_i^T ol_i (chunk
// (b * G + h % G) * nblk + row block). Grid: ceil(T / (32 NW)) * B * Hq
// workgroups (xcd_block_head).
template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_rows_local_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dout, const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu,
    const float* __restrict__ hk, const float* __restrict__ ol, const float* __restrict__ nl2,
    const float* __restrict__ nd, bf16_t* __restrict__ dq, float* __restrict__ wpart, int Hq,
    int Hkv, int T, int Tr, int w, float qscale, float scale, int nchunk, int BH) {
    constexpr int KS = D / 16, NT = D / 32, DS = DD / 16, BN = 64, LDK = D + 8, LDH = 40;
    constexpr int BM = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_kv[2 * BN * LDK];  // K tile, V tile
    __shared__ __attribute__((aligned(16))) bf16_t lds_h[NW * 32 * LDH];
    __shared__ __attribute__((aligned(16))) float pbuf[D * DD];
    bf16_t* lds_k = lds_kv;
    bf16_t* lds_v = lds_kv + BN * LDK;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nblk = (T + BM - 1) / BM;
    int rbi, bh;
    xcd_block_head(wg_id_x(), BH, rbi, bh);
    const int rb = nblk - 1 - rbi;
    const int b = bh / Hq, h = bh % Hq;
    const int G = Hq / Hkv;
    const int g = h / G;
    const int bg = b * Hkv + g;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int i0 = rb * BM, r0 = i0 + wave * 32, i = r0 + qc;
    const bool live = r0 < T;
    const int i_hi = imin(r0 + 31, T - 1);
    const int iwg_hi = imin(i0 + BM - 1, T - 1);
    const int ii = imin(i, T - 1);

    const bf16_t* qrow = q + ((size_t)bh * T + ii) * D;
    const bf16_t* drow = dout + ((size_t)bh * T + ii) * D;
    bf16x8_t qop[KS], doop[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        qop[s] = load_bf16x8(qrow + s * 16 + hg * 8);
        doop[s] = load_bf16x8(drow + s * 16 + hg * 8);
    }
    const size_t prw = (size_t)bh * Tr + ii;
    const float nL = nl2[prw];
    const f32x16_t negd = splat16(nd[prw]);
    f32x16_t dqT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dqT[t] = splat16(0.f);

    const bf16_t* kg = k + (size_t)bg * T * D;
    const bf16_t* vg = v + (size_t)bg * T * D;
    if (w > 0) {
        const int t_first = imax(0, i0 - w + 1) & ~(BN - 1);
        TilePair<D, NW> tp;
        tp.fetch(kg, vg, t_first, T, tid);
        for (int t = t_first; t <= iwg_hi; t += BN) {
            __syncthreads();  // the previous tile is no longer read
            tp.store(lds_k, lds_v, LDK, tid);
            __syncthreads();
            if (t + BN <= iwg_hi) tp.fetch(kg, vg, t + BN, T, tid);
            if (!live) continue;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int js = t + sub * 32;
                if (js > i_hi || js + 31 <= r0 - w) continue;
                f32x16_t sc = splat16(0.f), dp = negd;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    sc = mfma(load_bf16x8(lds_k + (sub * 32 + prow) * LDK + s * 16 + hg * 8), qop[s], sc);
                    dp = mfma(load_bf16x8(lds_v + (sub * 32 + prow) * LDK + s * 16 + hg * 8), doop[s], dp);
                }
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, nL);
                if (!(js > i_hi - w && js + 31 <= r0)) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int j = js + acc_row(r, hg);
                        if (j <= i - w || j > i) x[r] = -INFINITY;
                    }
                }
                f32x16_t ds;
#pragma unroll
                for (int r = 0; r < 16; ++r) ds[r] = __builtin_amdgcn_exp2f(x[r]) * dp[r];
                const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    dqT[tt] = mfma(lds_tr_operand(lds_k, LDK, sub * 32, tt * 32, lane), s0, dqT[tt]);
                    dqT[tt] = mfma(lds_tr_operand(lds_k, LDK, sub * 32 + 16, tt * 32, lane), s1, dqT[tt]);
                }
            }
        }
    }
    __syncthreads();  // the K/V tiles are reused below

    // ---- dq = s (dq_win + h W_up), h from the distant kernel as hi + lo bf16
    const bool real = live && i < T;
    const float* hrow = hk + ((size_t)bh * T + ii) * DD;
    const float* orow = ol + ((size_t)bh * T + ii) * DD;
    const bool any_dist = live && i_hi - w >= 0;  // wave-uniform
    if (any_dist) {
        const bf16_t* wdg = wd + (size_t)g * D * DD;
        const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            bf16x8_t hhi, hlo;
            split_load8(hrow + s * 16 + hg * 8, 1.f, hhi, hlo);
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                // A[e][c] = W_up[c][e], rows e = 32 tt + qc, c = 16 s + 8 hg + 0..7
                const int e = tt * 32 + qc, cb = s * 16 + hg * 8;
                bf16x8_t a;
                if (wug) {
                    uint16_t a8[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) a8[u] = wug[(size_t)(cb + u) * D + e];
                    a = __builtin_bit_cast(bf16x8_t, a8);
                } else {
                    a = load_bf16x8(wdg + (size_t)e * DD + cb);
                }
                dqT[tt] = mfma(a, hhi, dqT[tt]);
                dqT[tt] = mfma(a, hlo, dqT[tt]);
            }
        }
    }
    if (real) {
        bf16_t* dqr = dq + ((size_t)bh * T + i) * D;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                store_bf16x4(dqr + tt * 32 + 8 * a + 4 * hg, dqT[tt][4 * a] * scale,
                             dqT[tt][4 * a + 1] * scale, dqT[tt][4 * a + 2] * scale,
                             dqT[tt][4 * a + 3] * scale);
    }

    // ---- share of dW_up^T [e][c] = sum_i q_i[e] s h_i[c] + dO_i[e] ol_i[c]
    f32x16_t pw[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pw[t] = splat16(0.f);
    if (any_dist) {
        bf16_t* xs = lds_kv + wave * 32 * LDK;  // this wavefront's 32 rows of q, then dO
        bf16_t* ys = lds_h + wave * 32 * LDH;   // its 32 rows of s h, then ol (bf16, zero padded)
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
            for (int s = 0; s < KS; ++s)
                *reinterpret_cast<bf16x8_t*>(xs + qc * LDK + s * 16 + hg * 8) = pass ? doop[s] : qop[s];
            const float* yr = pass ? orow : hrow;
            const float f = real ? (pass ? 1.f : scale) : 0.f;  // rows past T add nothing
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int c = s * 16 + hg * 8;
                *reinterpret_cast<bf16x8_t*>(ys + qc * LDH + c) =
                    (c < DD) ? pack_load8(yr + c, f) : zero_bf16x8();
            }
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const bf16x8_t bop = lds_tr_operand(ys, LDH, hf * 16, 0, lane);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    pw[tt] = mfma(lds_tr_operand(xs, LDK, hf * 16, tt * 32, lane), bop, pw[tt]);
            }
        }
    }
    const int chunk = (b * G + h % G) * nblk + rb;
    wg_share<D, DD, NW>(pw, pbuf, wave, lane, tid,
                        wpart + (((size_t)Hkv + g) * nchunk + chunk) * D * DD);
}

// ---------------------------------------------------------------- window: dk, dv, dW_down

// One wavefront per 32 keys, window rows j <= i < j + w of every query head
// of the group through 64-row Q / dO tiles in LDS. Epilogue: the distant part
// gK W_down^T, gV W_down^T (hi + lo bf16), and the workgroup's share of
// dW_down = sum_j k_j^T s gK_j + v_j^T gV_j (chunk b * nkb + key block).
// Grid: ceil(T / (32 NW)) * B * Hkv workgroups (xcd_block_head).
template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_cols_local_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dout, const bf16_t* __restrict__ wd,
    const float* __restrict__ gk, const float* __restrict__ gv, const float* __restrict__ nl2,
    const float* __restrict__ nd, bf16_t* __restrict__ dk, bf16_t* __restrict__ dv,
    float* __restrict__ wpart, int Hq, int Hkv, int T, int Tr, int w, float qscale, float scale,
    int nchunk, int BKV) {
    constexpr int KS = D / 16, NT = D / 32, DS = DD / 16, BN = 64, LDK = D + 8, LDH = 40;
    constexpr int BK = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_qd[2 * BN * LDK];  // Q tile, dO tile
    __shared__ __attribute__((aligned(16))) float lds_lse[BN];  // -lse (log2 units)
    __shared__ __attribute__((aligned(16))) float lds_del[BN];  // -delta
    __shared__ __attribute__((aligned(16))) bf16_t lds_g[NW * 32 * LDH];
    __shared__ __attribute__((aligned(16))) float pbuf[D * DD];
    bf16_t* lds_q = lds_qd;
    bf16_t* lds_do = lds_qd + BN * LDK;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int cb, bg;
    xcd_block_head(wg_id_x(), BKV, cb, bg);
    const int nkb = (T + BK - 1) / BK;
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int cwg_lo = cb * BK;
    const int c0 = cwg_lo + wave * 32, j = c0 + qc;
    const bool live = c0 < T;
    const int j_hi = imin(c0 + 31, T - 1);
    const int cwg_hi = imin(cwg_lo + BK - 1, T - 1);
    const int jj = imin(j, T - 1);

    bf16x8_t kop[KS], vop[KS];
    const bf16_t* krow = k + ((size_t)bg * T + jj) * D;
    const bf16_t* vrow = v + ((size_t)bg * T + jj) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        kop[s] = load_bf16x8(krow + s * 16 + hg * 8);
        vop[s] = load_bf16x8(vrow + s * 16 + hg * 8);
    }
    f32x16_t dkT[NT], dvT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { dkT[t] = splat16(0.f); dvT[t] = splat16(0.f); }
    const int loc_hi = w > 0 ? imin(T - 1, cwg_hi + w - 1) : -1;  // last row with a window pair

    // (head, 64-row tile) pairs in order, the next one fetched during the
    // current one's work
    const int ntile = loc_hi >= cwg_lo ? (loc_hi - cwg_lo) / BN + 1 : 0;
    TilePair<D, NW> tp;
    float sv = 0.f;  // -lse (threads 0..63) or -delta (64..127) of one tile row
    auto fetch = [&](int n) {
        const int hh = n / ntile, t = cwg_lo + (n - hh * ntile) * BN;
        const size_t bh = (size_t)b * Hq + g * G + hh;
        tp.fetch(q + bh * T * D, dout + bh * T * D, t, T, tid);
        if (tid < 2 * BN) {
            const int r = tid & (BN - 1);
            const float* src = (tid < BN ? nl2 : nd) + bh * Tr;
            sv = t + r < Tr ? src[imin(t + r, Tr - 1)] : 0.f;
        }
    };
    if (ntile > 0) fetch(0);
    for (int n = 0; n < G * ntile; ++n) {
        const int t = cwg_lo + (n % ntile) * BN;
        {
            __syncthreads();  // the previous tile is no longer read
            tp.store(lds_q, lds_do, LDK, tid);
            if (tid < BN) lds_lse[tid] = sv;
            else if (tid < 2 * BN) lds_del[tid - BN] = sv;
            __syncthreads();
            if (n + 1 < G * ntile) fetch(n + 1);
            if (!live) continue;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int is = t + sub * 32;
                if (is + 31 < c0 || is > j_hi + w - 1) continue;
                f32x16_t sc = splat16(0.f);
                f32x16_t dp = load_row16(lds_del + sub * 32, hg, 1.f);
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    sc = mfma(load_bf16x8(lds_q + (sub * 32 + prow) * LDK + s * 16 + hg * 8), kop[s], sc);
                    dp = mfma(load_bf16x8(lds_do + (sub * 32 + prow) * LDK + s * 16 + hg * 8), vop[s], dp);
                }
                const f32x16_t ln = load_row16(lds_lse + sub * 32, hg, 1.f);
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, ln[r]);
                if (!(is >= c0 + 31 && is + 31 - c0 < w && is + 31 < T)) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int i = is + acc_row(r, hg);
                        if (i < j || i - j >= w || i >= T) x[r] = -INFINITY;
                    }
                }
                f32x16_t p, ds;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    p[r] = __builtin_amdgcn_exp2f(x[r]);
                    ds[r] = p[r] * dp[r];
                }
                const bf16x8_t p0 = pack8(p, 0), p1 = pack8(p, 8);
                const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    dvT[tt] = mfma(lds_tr_operand(lds_do, LDK, sub * 32, tt * 32, lane), p0, dvT[tt]);
                    dvT[tt] = mfma(lds_tr_operand(lds_do, LDK, sub * 32 + 16, tt * 32, lane), p1, dvT[tt]);
                    dkT[tt] = mfma(lds_tr_operand(lds_q, LDK, sub * 32, tt * 32, lane), s0, dkT[tt]);
                    dkT[tt] = mfma(lds_tr_operand(lds_q, LDK, sub * 32 + 16, tt * 32, lane), s1, dkT[tt]);
                }
            }
        }
    }
    __syncthreads();  // the Q/dO tiles are reused below

    // ---- dk = s dk_win + (s gK) W_down^T, dv = dv_win + gV W_down^T
    const bool real = live && j < T;
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const float* gkr = gk + ((size_t)bg * T + jj) * DD;
    const float* gvr = gv + ((size_t)bg * T + jj) * DD;
    const bool any_dist = live && c0 + w < T;  // wave-uniform
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) dkT[tt][r] *= scale;
    if (any_dist) {
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            bf16x8_t khi, klo, vhi, vlo;
            split_load8(gkr + s * 16 + hg * 8, scale, khi, klo);
            split_load8(gvr + s * 16 + hg * 8, 1.f, vhi, vlo);
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                const bf16x8_t a = load_bf16x8(wdg + (size_t)(tt * 32 + qc) * DD + s * 16 + hg * 8);
                dkT[tt] = mfma(a, khi, dkT[tt]);
                dkT[tt] = mfma(a, klo, dkT[tt]);
                dvT[tt] = mfma(a, vhi, dvT[tt]);
                dvT[tt] = mfma(a, vlo, dvT[tt]);
            }
        }
    }
    if (real) {
        bf16_t* dkr = dk + ((size_t)bg * T + j) * D;
        bf16_t* dvr = dv + ((size_t)bg * T + j) * D;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                store_bf16x4(dkr + tt * 32 + 8 * a + 4 * hg, dkT[tt][4 * a], dkT[tt][4 * a + 1],
                             dkT[tt][4 * a + 2], dkT[tt][4 * a + 3]);
                store_bf16x4(dvr + tt * 32 + 8 * a + 4 * hg, dvT[tt][4 * a], dvT[tt][4 * a + 1],
                             dvT[tt][4 * a + 2], dvT[tt][4 * a + 3]);
            }
    }

    // ---- share of dW_down [e][c] = sum_j k_j[e] s gK_j[c] + v_j[e] gV_j[c]
    f32x16_t pw[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pw[t] = splat16(0.f);
    if (any_dist) {
        bf16_t* xs = lds_qd + wave * 32 * LDK;  // this wavefront's 32 keys, then values
        bf16_t* ys = lds_g + wave * 32 * LDH;   // s gK, then gV (bf16, zero padded)
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
            for (int s = 0; s < KS; ++s)
                *reinterpret_cast<bf16x8_t*>(xs + qc * LDK + s * 16 + hg * 8) = pass ? vop[s] : kop[s];
            const float* yr = pass ? gvr : gkr;
            const float f = real ? (pass ? 1.f : scale) : 0.f;  // keys past T add nothing
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int c = s * 16 + hg * 8;
                *reinterpret_cast<bf16x8_t*>(ys + qc * LDH + c) =
                    (c < DD) ? pack_load8(yr + c, f) : zero_bf16x8();
            }
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const bf16x8_t bop = lds_tr_operand(ys, LDH, hf * 16, 0, lane);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    pw[tt] = mfma(lds_tr_operand(xs, LDK, hf * 16, tt * 32, lane), bop, pw[tt]);
            }
        }
    }
    wg_share<D, DD, NW>(pw, pbuf, wave, lane, tid,
                        wpart + ((size_t)g * nchunk + b * nkb + cb) * D * DD);
}

// ---------------------------------------------------------------- host

bool bwd_mfma_supported(int d, int dd, bool bf16) {
    return bf16 && (d == 64 || d == 128) && (dd == 16 || dd == 32);
}

template <int D, int DD>
static hipError_t launch_bwd_mfma_t(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                    const bf16_t* o, const float* lse, const bf16_t* dout,
                                    const bf16_t* wd, const bf16_t* wu, bf16_t* dq, bf16_t* dk,
                                    bf16_t* dv, float* dwd, float* dwu, char* ws, const BwdWs& L,
                                    int B, int Hq, int Hkv, int T, int w, hipStream_t st) {
    constexpr int NW = 4;
    const int Tr = round_up(T, 64);
    const size_t nrow = (size_t)B * Hq * Tr * DD, ntok = (size_t)B * Hkv * Tr * DD;  // bf16
    float* nl2 = (float*)(ws + L.lse_off);
    float* nd = (float*)(ws + L.delta_off);
    bf16_t* rc = (bf16_t*)(ws + L.rc_off);
    bf16_t* qts = (bf16_t*)(ws + L.qt_off);
    bf16_t* qtT = qts + nrow;
    bf16_t* dts = (bf16_t*)(ws + L.dot_off);
    bf16_t* dtT = dts + nrow;
    bf16_t* ckb = (bf16_t*)(ws + L.ck_off);
    bf16_t* ckT = ckb + ntok;
    bf16_t* cvb = (bf16_t*)(ws + L.cv_off);
    bf16_t* cvT = cvb + ntok;
    float* hk = (float*)(ws + L.hk_off);
    float* ol = (float*)(ws + L.ol_off);
    float* gk = (float*)(ws + L.gk_off);
    float* gv = (float*)(ws + L.gv_off);
    float* part = (float*)(ws + L.wpart_off);
    const float scale = 1.f / sqrtf((float)D);
    const float qscale = scale * kLog2eB;
    const int nblk = (T + NW * 32 - 1) / (NW * 32);

    const int nprep = (Tr + NW * 32 - 1) / (NW * 32);
    hipLaunchKernelGGL((bwd_prep_rows_kernel<D, DD, NW>), dim3(nprep, B * Hq), dim3(NW * 64), 0,
                       st, q, o, dout, lse, wd, wu, qts, qtT, dts, dtT, rc, nd, nl2, Hq, Hkv, T, Tr,
                       qscale);
    hipLaunchKernelGGL((bwd_prep_keys_kernel<D, DD, NW>), dim3(nprep, B * Hkv), dim3(NW * 64), 0,
                       st, k, v, wd, ckb, ckT, cvb, cvT, Hkv, T, Tr);
    hipLaunchKernelGGL((bwd_rows_dist_kernel<DD, NW>), dim3(nblk * B * Hq), dim3(NW * 64), 0, st,
                       (const bf16_t*)ckb, (const bf16_t*)ckT, (const bf16_t*)cvb,
                       (const bf16_t*)cvT, (const bf16_t*)qts, (const bf16_t*)dts,
                       (const float*)nl2, (const float*)nd, hk, ol, Hq, Hkv, T, Tr, w, B * Hq);
    hipLaunchKernelGGL((bwd_cols_dist_kernel<DD, NW>), dim3(nblk * B * Hkv), dim3(NW * 64), 0, st,
                       (const bf16_t*)ckb, (const bf16_t*)cvb, (const bf16_t*)qts,
                       (const bf16_t*)qtT, (const bf16_t*)dts, (const bf16_t*)dtT,
                       (const bf16_t*)rc, gk, gv, Hq, Hkv, T, Tr, w, 1.f / qscale, B * Hkv);
    hipLaunchKernelGGL((bwd_rows_local_kernel<D, DD, NW>), dim3(nblk * B * Hq), dim3(NW * 64), 0,
                       st, q, k, v, dout, wd, wu, (const float*)hk, (const float*)ol,
                       (const float*)nl2, (const float*)nd, dq, part, Hq, Hkv, T, Tr, w,
                       qscale, scale, L.nchunk, B * Hq);
    hipLaunchKernelGGL((bwd_cols_local_kernel<D, DD, NW>), dim3(nblk * B * Hkv), dim3(NW * 64), 0,
                       st, q, k, v, dout, wd, (const float*)gk, (const float*)gv,
                       (const float*)nl2, (const float*)nd, dk, dv, part, Hq, Hkv, T, Tr, w,
                       qscale, scale, L.nchunk, B * Hkv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bwd_wreduce(part, dwd, dwu, Hkv, D, DD, L, st);
}

hipError_t launch_bwd_mfma(const bf16_t* q, const bf16_t* k, const bf16_t* v, const bf16_t* o,
                           const float* lse, const bf16_t* dout, const bf16_t* wd,
                           const bf16_t* wu, bf16_t* dq, bf16_t* dk, bf16_t* dv, float* dwd,
                           float* dwu, char* ws, const BwdWs& L, int B, int Hq, int Hkv, int T,
                           int d, int dd, int w, hipStream_t st) {
#define DAR_BWD_CASE(D_, DD_)                                                                   \
    if (d == D_ && dd == DD_)                                                                   \
        return launch_bwd_mfma_t<D_, DD_>(q, k, v, o, lse, dout, wd, wu, dq, dk, dv, dwd, dwu,  \
                                          ws, L, B, Hq, Hkv, T, w, st);
    DAR_BWD_CASE(64, 16)
    DAR_BWD_CASE(64, 32)
    DAR_BWD_CASE(128, 16)
    DAR_BWD_CASE(128, 32)
#undef DAR_BWD_CASE
    return hipErrorInvalidValue;
}


// ================================================================ rotary embedding
//
// Backward of dar_attn_prefill_rope (Eq. 3 with the rotation; Section 2.3
// trains through it). The forward attends at full d: rotated queries qr,
// rotated window keys kr with values v, lifted-then-rotated distant keys kd
// with lifted values vd (the rotary pre-pass writes them; kd, vd hold
// positions 0..Td-1, Td = T - w). The softmax is recomputed against the
// forward's log-sum-exp:
//   bwd_rope_rowprep_kernel  -lse (log2 units) and -delta = -dO . O per row
//   bwd_rope_rows_kernel     dqr = s sum_j dS_ij key_ij over both regions
//   bwd_rope_cols_kernel     per key, s sum_i dS_ij qr_i and sum_i P_ij dO_i over
//                            the rows that see it in the window (dkr, dvw) or
//                            at distance (dkd, dvd)
//   bwd_rope_post_rows_kernel  dq = R^T dqr
//   bwd_rope_post_keys_kernel  the rotation taken back (R^T) and the chain rule
//                            through the lift x' = (x W_down) W_up for keys and
//                            values, with the weight-gradient shares
//   bwd_wreduce_kernel       the shares summed in a fixed order
// with s = 1/sqrt(d). The rows and cols kernels are the window kernels'
// loops with the key range and mask of either region.

namespace {

// -lse (log2 units) and -delta per row, zero for the padding rows. One
// thread per row (16-byte loads along the row).
template <int D>
__global__ __launch_bounds__(256) void bwd_rope_rowprep_kernel(const bf16_t* __restrict__ o,
                                                               const bf16_t* __restrict__ dout,
                                                               const float* __restrict__ lse,
                                                               float* __restrict__ nl2,
                                                               float* __restrict__ nd, int T,
                                                               int Tr) {
    const int bh = wg_id_y();
    const int i = wg_id_x() * 256 + lane_id_x();
    if (i >= Tr) return;
    float acc = 0.f;
    if (i < T) {
        const size_t row = ((size_t)bh * T + i) * D;
#pragma unroll
        for (int e = 0; e < D; e += 8) {
            const uint4 a = *reinterpret_cast<const uint4*>(o + row + e);
            const uint4 b = *reinterpret_cast<const uint4*>(dout + row + e);
            const uint32_t ua[4] = {a.x, a.y, a.z, a.w}, ub[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc = __builtin_fmaf(__uint_as_float(ua[q] << 16), __uint_as_float(ub[q] << 16), acc);
                acc = __builtin_fmaf(__uint_as_float(ua[q] & 0xffff0000u), __uint_as_float(ub[q] & 0xffff0000u), acc);
            }
        }
    }
    nd[(size_t)bh * Tr + i] = i < T ? -acc : 0.f;
    nl2[(size_t)bh * Tr + i] = i < T ? -lse[(size_t)bh * T + i] * kLog2eB : 0.f;
}

// One wavefront per 32 query rows: dqr^T += K^T dS^T over the window keys
// (kr, v: i - w < j <= i) and the distant keys (kd, vd: j <= i - w), 64-key
// tiles staged through LDS for the workgroup. Writes s dqr (fp32) of every
// real row. Grid: ceil(T / (32 NW)) * B * Hq workgroups (xcd_block_head).
template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_rope_rows_kernel(
    const bf16_t* __restrict__ qr, const bf16_t* __restrict__ kr, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ kd, const bf16_t* __restrict__ vd, const bf16_t* __restrict__ dout,
    const float* __restrict__ nl2, const float* __restrict__ nd, float* __restrict__ dqr, int Hq,
    int Hkv, int T, int Tr, int w, float qscale, float scale, int BH) {
    constexpr int KS = D / 16, NT = D / 32, BN = 64, LDK = D + 8;
    constexpr int BM = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_kv[2 * BN * LDK];  // K tile, V tile
    bf16_t* lds_k = lds_kv;
    bf16_t* lds_v = lds_kv + BN * LDK;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nblk = (T + BM - 1) / BM;
    int rbi, bh;
    xcd_block_head(wg_id_x(), BH, rbi, bh);
    const int rb = nblk - 1 - rbi;
    const int b = bh / Hq, h = bh % Hq;
    const int G = Hq / Hkv;
    const int g = h / G;
    const int bg = b * Hkv + g;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int i0 = rb * BM, r0 = i0 + wave * 32, i = r0 + qc;
    const bool live = r0 < T;
    const int i_hi = imin(r0 + 31, T - 1);
    const int iwg_hi = imin(i0 + BM - 1, T - 1);
    const int ii = imin(i, T - 1);
    const int Td = imax(T - w, 0);

    const bf16_t* qrow = qr + ((size_t)bh * T + ii) * D;
    const bf16_t* drow = dout + ((size_t)bh * T + ii) * D;
    bf16x8_t qop[KS], doop[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        qop[s] = load_bf16x8(qrow + s * 16 + hg * 8);
        doop[s] = load_bf16x8(drow + s * 16 + hg * 8);
    }
    const size_t prw = (size_t)bh * Tr + ii;
    const float nL = nl2[prw];
    const f32x16_t negd = splat16(nd[prw]);
    f32x16_t dqT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dqT[t] = splat16(0.f);

    // keys [t_first, t_last] of one region (workgroup-uniform bounds: every
    // thread reaches the barriers)
    auto region = [&](const bf16_t* kg, const bf16_t* vg, int nkeys, int t_first, int t_last,
                      bool dist) {
        TilePair<D, NW> tp;
        tp.fetch(kg, vg, t_first, nkeys, tid);
        for (int t = t_first; t <= t_last; t += BN) {
            __syncthreads();  // the previous tile is no longer read
            tp.store(lds_k, lds_v, LDK, tid);
            __syncthreads();
            if (t + BN <= t_last) tp.fetch(kg, vg, t + BN, nkeys, tid);
            if (!live) continue;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int js = t + sub * 32;
                if (dist ? js > i_hi - w : (js > i_hi || js + 31 <= r0 - w)) continue;
                f32x16_t sc = splat16(0.f), dp = negd;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    sc = mfma(load_bf16x8(lds_k + (sub * 32 + prow) * LDK + s * 16 + hg * 8), qop[s], sc);
                    dp = mfma(load_bf16x8(lds_v + (sub * 32 + prow) * LDK + s * 16 + hg * 8), doop[s], dp);
                }
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, nL);
                const bool full = dist ? js + 31 <= r0 - w : (js > i_hi - w && js + 31 <= r0);
                if (!full) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int j = js + acc_row(r, hg);
                        if (dist ? j > i - w : (j <= i - w || j > i)) x[r] = -INFINITY;
                    }
                }
                f32x16_t ds;
#pragma unroll
                for (int r = 0; r < 16; ++r) ds[r] = __builtin_amdgcn_exp2f(x[r]) * dp[r];
                const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    dqT[tt] = mfma(lds_tr_operand(lds_k, LDK, sub * 32, tt * 32, lane), s0, dqT[tt]);
                    dqT[tt] = mfma(lds_tr_operand(lds_k, LDK, sub * 32 + 16, tt * 32, lane), s1, dqT[tt]);
                }
            }
        }
    };
    if (w > 0) region(kr + (size_t)bg * T * D, v + (size_t)bg * T * D, T, imax(0, i0 - w + 1) & ~(BN - 1),
                      iwg_hi, false);
    if (iwg_hi - w >= 0) region(kd + (size_t)bg * Td * D, vd + (size_t)bg * Td * D, Td, 0, iwg_hi - w, true);

    if (live && i < T) {
        float* out = dqr + ((size_t)bh * T + i) * D;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                *reinterpret_cast<float4*>(out + tt * 32 + 8 * a + 4 * hg) =
                    make_float4(dqT[tt][4 * a] * scale, dqT[tt][4 * a + 1] * scale,
                                dqT[tt][4 * a + 2] * scale, dqT[tt][4 * a + 3] * scale);
    }
}

// One wavefront per 32 keys of one region's key array (kx, vx: kr and v for
// the window, kd and vd at distance, nkeys rows a head), the rows of every
// query head of the group that see them there (window: j <= i < j + w; at
// distance: i >= j + w) through 64-row Q / dO tiles in LDS:
// dk^T += Q^T dS (times s), dv^T += dO^T P. Writes both (fp32) for every key.
// Grid: ceil(nkeys / (32 NW)) * B * Hkv workgroups (xcd_block_head).
template <int D, int NW, bool DIST>
__global__ __launch_bounds__(NW * 64) void bwd_rope_cols_kernel(
    const bf16_t* __restrict__ qr, const bf16_t* __restrict__ kx, const bf16_t* __restrict__ vx,
    const bf16_t* __restrict__ dout, const float* __restrict__ nl2, const float* __restrict__ nd,
    float* __restrict__ dk, float* __restrict__ dv, int Hq, int Hkv, int T, int Tr, int nkeys,
    int w, float qscale, float scale, int BKV) {
    constexpr int KS = D / 16, NT = D / 32, BN = 64, LDK = D + 8;
    constexpr int BK = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_qd[2 * BN * LDK];  // Q tile, dO tile
    __shared__ __attribute__((aligned(16))) float lds_lse[BN];  // -lse (log2 units)
    __shared__ __attribute__((aligned(16))) float lds_del[BN];  // -delta
    bf16_t* lds_q = lds_qd;
    bf16_t* lds_do = lds_qd + BN * LDK;

    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int cb, bg;
    xcd_block_head(wg_id_x(), BKV, cb, bg);
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int cwg_lo = cb * BK;
    const int c0 = cwg_lo + wave * 32, j = c0 + qc;
    const bool live = c0 < nkeys;
    const int j_hi = imin(c0 + 31, nkeys - 1);
    const int cwg_hi = imin(cwg_lo + BK - 1, nkeys - 1);
    const int jj = imin(j, nkeys - 1);

    bf16x8_t kop[KS], vop[KS];
    const bf16_t* krow = kx + ((size_t)bg * nkeys + jj) * D;
    const bf16_t* vrow = vx + ((size_t)bg * nkeys + jj) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        kop[s] = load_bf16x8(krow + s * 16 + hg * 8);
        vop[s] = load_bf16x8(vrow + s * 16 + hg * 8);
    }
    f32x16_t dkT[NT], dvT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { dkT[t] = splat16(0.f); dvT[t] = splat16(0.f); }
    // the workgroup's rows: window [cwg_lo, cwg_hi + w - 1], at distance [cwg_lo + w, T - 1]
    const int row_lo = DIST ? cwg_lo + w : cwg_lo;
    const int row_hi = DIST ? T - 1 : imin(T - 1, cwg_hi + w - 1);
    const int ntile = row_hi >= row_lo ? (row_hi - row_lo) / BN + 1 : 0;
    TilePair<D, NW> tp;
    float sv = 0.f;  // -lse (threads 0..63) or -delta (64..127) of one tile row
    auto fetch = [&](int n) {
        const int hh = n / ntile, t = row_lo + (n - hh * ntile) * BN;
        const size_t bh = (size_t)b * Hq + g * G + hh;
        tp.fetch(qr + bh * T * D, dout + bh * T * D, t, T, tid);
        if (tid < 2 * BN) {
            const int r = tid & (BN - 1);
            const float* src = (tid < BN ? nl2 : nd) + bh * Tr;
            sv = t + r < Tr ? src[imin(t + r, Tr - 1)] : 0.f;
        }
    };
    if (ntile > 0) fetch(0);
    for (int n = 0; n < G * ntile; ++n) {
        const int t = row_lo + (n % ntile) * BN;
        __syncthreads();  // the previous tile is no longer read
        tp.store(lds_q, lds_do, LDK, tid);
        if (tid < BN) lds_lse[tid] = sv;
        else if (tid < 2 * BN) lds_del[tid - BN] = sv;
        __syncthreads();
        if (n + 1 < G * ntile) fetch(n + 1);
        if (!live) continue;
#pragma unroll
        for (int sub = 0; sub < BN / 32; ++sub) {
            const int is = t + sub * 32;
            if (DIST ? is + 31 < c0 + w : (is + 31 < c0 || is > j_hi + w - 1)) continue;
            f32x16_t sc = splat16(0.f);
            f32x16_t dp = load_row16(lds_del + sub * 32, hg, 1.f);
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                sc = mfma(load_bf16x8(lds_q + (sub * 32 + prow) * LDK + s * 16 + hg * 8), kop[s], sc);
                dp = mfma(load_bf16x8(lds_do + (sub * 32 + prow) * LDK + s * 16 + hg * 8), vop[s], dp);
            }
            const f32x16_t ln = load_row16(lds_lse + sub * 32, hg, 1.f);
            f32x16_t x;
#pragma unroll
            for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, ln[r]);
            const bool full = DIST ? (is >= j_hi + w && is + 31 < T)
                                   : (is >= c0 + 31 && is + 31 - c0 < w && is + 31 < T);
            if (!full) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int i = is + acc_row(r, hg);
                    if (DIST ? (i - j < w || i >= T) : (i < j || i - j >= w || i >= T)) x[r] = -INFINITY;
                }
            }
            f32x16_t p, ds;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                p[r] = __builtin_amdgcn_exp2f(x[r]);
                ds[r] = p[r] * dp[r];
            }
            const bf16x8_t p0 = pack8(p, 0), p1 = pack8(p, 8);
            const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                dvT[tt] = mfma(lds_tr_operand(lds_do, LDK, sub * 32, tt * 32, lane), p0, dvT[tt]);
                dvT[tt] = mfma(lds_tr_operand(lds_do, LDK, sub * 32 + 16, tt * 32, lane), p1, dvT[tt]);
                dkT[tt] = mfma(lds_tr_operand(lds_q, LDK, sub * 32, tt * 32, lane), s0, dkT[tt]);
                dkT[tt] = mfma(lds_tr_operand(lds_q, LDK, sub * 32 + 16, tt * 32, lane), s1, dkT[tt]);
            }
        }
    }
    if (live && j < nkeys) {
        float* dkr = dk + ((size_t)bg * nkeys + j) * D;
        float* dvr = dv + ((size_t)bg * nkeys + j) * D;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                *reinterpret_cast<float4*>(dkr + tt * 32 + 8 * a + 4 * hg) =
                    make_float4(dkT[tt][4 * a] * scale, dkT[tt][4 * a + 1] * scale,
                                dkT[tt][4 * a + 2] * scale, dkT[tt][4 * a + 3] * scale);
                *reinterpret_cast<float4*>(dvr + tt * 32 + 8 * a + 4 * hg) =
                    make_float4(dvT[tt][4 * a], dvT[tt][4 * a + 1], dvT[tt][4 * a + 2], dvT[tt][4 * a + 3]);
            }
    }
}

// Element e of R_p^T x for a row x at position p: the rotation taken back,
// pairs (m, m + r/2) turned by -p base^(-2m/r) (tab [n_pos][r]: cos, then sin).
__device__ __forceinline__ float rot_back(const float* x, int e, int r, const float* tabp) {
    const int h = r >> 1;
    if (e >= r) return x[e];
    const int m = e < h ? e : e - h;
    const float c = tabp[m], s = tabp[h + m];
    return e < h ? __builtin_fmaf(x[e], c, x[e + h] * s) : __builtin_fmaf(x[e], c, -x[e - h] * s);
}

// dq = R^T dqr (bf16). One thread per element; grid (ceil(T D / 256), B Hq),
// so that the row and element come from shifts by the compile-time D rather
// than 64-bit divisions.
template <int D>
__global__ __launch_bounds__(256) void bwd_rope_post_rows_kernel(const float* __restrict__ dqr,
                                                                 const float* __restrict__ tab,
                                                                 bf16_t* __restrict__ dq, int T,
                                                                 int r, int pos0) {
    const int idx = wg_id_x() * 256 + lane_id_x();
    if (idx >= T * D) return;
    const int i = idx / D, e = idx % D;
    const size_t row = (size_t)wg_id_y() * T + i;
    dq[row * D + e] = f32_to_bf16(rot_back(dqr + row * D, e, r, tab + (size_t)(pos0 + i) * r));
}

// The chain rule per key, and the weight-gradient shares. A workgroup takes
// kRopeKeysPerWg keys of one (batch, KV head) in blocks of rope_post_block(D); per key j
// (u_j = R^T dkd_j and dvd_j zero at or past Td = T - w):
//   gK_j = u_j W_up^T,  gV_j = dvd_j W_up^T,  cK_j = k_j W_down,  cV_j = v_j W_down
//   dk_j = R^T dkr_j + gK_j W_down^T,  dv_j = dvw_j + gV_j W_down^T   (bf16)
// and over its keys, in key order, the shares [e][c]
//   dW_down += k_j[e] gK_j[c] + v_j[e] gV_j[c]
//   dW_up^T += u_j[e] cK_j[c] + dvd_j[e] cV_j[c]
// (chunk b * ceil(T / kRopeKeysPerWg) + workgroup). d_down <= D.
constexpr int kRopeKeysPerWg = 32;

// Keys per block of bwd_rope_post_keys_kernel (32 measured slower at d = 64:
// 310 against 256 us at the pythia70m shape), and its dynamic LDS in floats:
// a [KB][D + 1] block of four-float key entries (rows padded by one entry:
// the lanes reading one column of different rows hit different banks), four
// [KB][dd] latent blocks, the two weights interleaved and W_down transposed.
__host__ __device__ constexpr int rope_post_block(int) { return 16; }
static inline size_t rope_post_lds_bytes(int D, int dd) {
    const size_t kb = rope_post_block(D);
    return sizeof(float) * (4 * kb * (D + 1) + 4 * kb * dd + (size_t)3 * D * dd);
}

// NO bounds the weight columns a thread owns (cpt = ceil(d_down / (256 / D))),
// chosen at launch from d_down so that the share loop unrolls over registers
// that exist: sized for the largest d_down it would hold 16 (d = 64) or 64
// (d = 128) accumulator pairs and halve the occupancy.
template <int D, int NO>
__global__ __launch_bounds__(256) void bwd_rope_post_keys_kernel(
    const bf16_t* __restrict__ k, const bf16_t* __restrict__ v, const bf16_t* __restrict__ wd,
    const bf16_t* __restrict__ wu, const float* __restrict__ dkr, const float* __restrict__ dvw,
    const float* __restrict__ dkd, const float* __restrict__ dvd, const float* __restrict__ tab,
    bf16_t* __restrict__ dk, bf16_t* __restrict__ dv, float* __restrict__ wpart, int Hkv, int T,
    int dd, int w, int r, int pos0, int nchunk) {
    constexpr int KB = rope_post_block(D);
    constexpr int XJ = KB * D / 256, JS = 256 / D;  // keys of a thread in dk/dv, their stride
    extern __shared__ __align__(16) float sm[];
    constexpr int LD = D + 1;         // padded key row
    // the four key-side values of one (key, element) side by side, and the
    // two weights of one (e, c): one 16-byte and one 8-byte LDS read feed the
    // four products of an element
    float4* sx = reinterpret_cast<float4*>(sm);  // [KB][LD]  (u = R^T dkd, dvd, k, v)
    float* sg = sm + 4 * KB * LD;                // [4][KB][dd]  gK, gV, cK, cV
    float2* sw = reinterpret_cast<float2*>(sg + 4 * KB * dd);  // [D][dd]  (W_up[c][e], W_down[e][c])
    float* swt = sg + 4 * KB * dd + 2 * D * dd;  // [dd][D]  W_down[e][c] at [c][e]
    const int bg = wg_id_y(), b = bg / Hkv, g = bg % Hkv;
    const int tid = lane_id_x();
    const int Td = imax(T - w, 0);
    const int nkb = (T + kRopeKeysPerWg - 1) / kRopeKeysPerWg;
    const int j_lo = wg_id_x() * kRopeKeysPerWg;
    const int j_end = imin(j_lo + kRopeKeysPerWg, T);
    const bf16_t* wdg = wd + (size_t)g * D * dd;
    const bf16_t* wug = wu ? wu + (size_t)g * dd * D : nullptr;
    const int n_out = D * dd;
    // weight shares: TPE threads per element e, cpt columns each
    constexpr int TPE = 256 / D;
    const int we = tid / TPE, wq = tid % TPE;
    const int cpt = (dd + TPE - 1) / TPE;  // <= NO (checked at launch)
    for (int idx = tid; idx < n_out; idx += 256) {
        const int e = idx / dd, c = idx - (idx / dd) * dd;
        const float x = bf16_to_f32(wdg[idx]);
        swt[c * D + e] = x;
        sw[idx] = make_float2(wug ? bf16_to_f32(wug[(size_t)c * D + e]) : x, x);
    }
    float accd[NO], accu[NO];
#pragma unroll
    for (int x = 0; x < NO; ++x) accd[x] = accu[x] = 0.f;
    for (int j0 = j_lo; j0 < j_end; j0 += KB) {
        __syncthreads();  // the weights are staged; the previous block is no longer read
        // stage: u = R^T dkd, dvd, k, v of the block's keys (zero past the ends)
        for (int idx = tid; idx < KB * D; idx += 256) {
            const int jl = idx / D, e = idx - (idx / D) * D, j = j0 + jl;
            float uu = 0.f, vd = 0.f, kk = 0.f, vv = 0.f;
            if (j < j_end) {
                const size_t row = (size_t)bg * T + j;
                kk = bf16_to_f32(k[row * D + e]);
                vv = bf16_to_f32(v[row * D + e]);
                if (j < Td) {
                    const size_t drow = (size_t)bg * Td + j;
                    uu = rot_back(dkd + drow * D, e, r, tab + (size_t)(pos0 + j) * r);
                    vd = dvd[drow * D + e];
                }
            }
            sx[jl * LD + e] = make_float4(uu, vd, kk, vv);
        }
        __syncthreads();
        // gK, gV (through W_up) and cK, cV (through W_down), d_down wide: the
        // four products of one (key, column) together (independent chains)
        for (int idx = tid; idx < KB * dd; idx += 256) {
            const int jl = idx / dd, c = idx - (idx / dd) * dd;
            float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll 8
            for (int e = 0; e < D; ++e) {
                const float2 wt = sw[e * dd + c];  // (W_up, W_down)
                const float4 xv = sx[jl * LD + e];
                a0 = __builtin_fmaf(xv.x, wt.x, a0);
                a1 = __builtin_fmaf(xv.y, wt.x, a1);
                a2 = __builtin_fmaf(xv.z, wt.y, a2);
                a3 = __builtin_fmaf(xv.w, wt.y, a3);
            }
            sg[idx] = a0;
            sg[KB * dd + idx] = a1;
            sg[2 * KB * dd + idx] = a2;
            sg[3 * KB * dd + idx] = a3;
        }
        __syncthreads();
        // dk, dv of the block's keys: a thread keeps one element e of XJ keys,
        // so each weight it reads serves all of them
        {
            const int e = tid % D, jl0 = tid / D;
            float xk[XJ], xv[XJ];
#pragma unroll
            for (int x = 0; x < XJ; ++x) {
                const int j = imin(j0 + jl0 + JS * x, j_end - 1);
                const size_t row = (size_t)bg * T + j;
                xk[x] = rot_back(dkr + row * D, e, r, tab + (size_t)(pos0 + j) * r);
                xv[x] = dvw[row * D + e];
            }
            for (int c = 0; c < dd; ++c) {
                const float wdn = swt[c * D + e];
#pragma unroll
                for (int x = 0; x < XJ; ++x) {
                    xk[x] = __builtin_fmaf(sg[(jl0 + JS * x) * dd + c], wdn, xk[x]);
                    xv[x] = __builtin_fmaf(sg[(KB + jl0 + JS * x) * dd + c], wdn, xv[x]);
                }
            }
#pragma unroll
            for (int x = 0; x < XJ; ++x) {
                const int j = j0 + jl0 + JS * x;
                if (j < j_end) {
                    const size_t row = (size_t)bg * T + j;
                    dk[row * D + e] = f32_to_bf16(xk[x]);
                    dv[row * D + e] = f32_to_bf16(xv[x]);
                }
            }
        }
        // weight shares, key by key in order: a thread owns element e and the
        // columns [q cpt, q cpt + cpt) (independent chains; columns past
        // d_down are clamped and never stored)
#pragma unroll 1  // unrolled, its hoisted reads take the registers of a wave per SIMD
        for (int jl = 0; jl < KB; ++jl) {
            const float4 xv = sx[jl * LD + we];
            const float u_ = xv.x, d_ = xv.y, k_ = xv.z, v_ = xv.w;
            const float* g0 = sg + jl * dd;
            // a guard rather than a break: with a fixed trip count the loop
            // unrolls and accd / accu stay in statically named registers
#pragma unroll
            for (int y = 0; y < NO; ++y) {
                if (y < cpt) {  // uniform
                    const int c = imin(wq * cpt + y, dd - 1);
                    accd[y] = __builtin_fmaf(k_, g0[c], accd[y]);
                    accd[y] = __builtin_fmaf(v_, g0[KB * dd + c], accd[y]);
                    accu[y] = __builtin_fmaf(u_, g0[2 * KB * dd + c], accu[y]);
                    accu[y] = __builtin_fmaf(d_, g0[3 * KB * dd + c], accu[y]);
                }
            }
        }
    }
    const int chunk = b * nkb + wg_id_x();
    float* pd = wpart + ((size_t)g * nchunk + chunk) * n_out;
    float* pu = wpart + ((size_t)(Hkv + g) * nchunk + chunk) * n_out;
#pragma unroll
    for (int y = 0; y < NO; ++y) {
        const int c = wq * cpt + y;
        if (y < cpt && c < dd) {
            pd[we * dd + c] = accd[y];
            pu[we * dd + c] = accu[y];
        }
    }
}

}  // namespace

// (the post kernel's LDS, within the 160 KB of a compute unit: d_down <= 64 at d = 128)
bool bwd_rope_mfma_supported(int d, int dd, bool bf16) {
    return bf16 && (d == 64 || d == 128) && dd <= d && rope_post_lds_bytes(d, dd) <= 160 * 1024;
}

template <int D, int NO>
static hipError_t launch_rope_post_keys_t(const RopeBwdArgs& a, hipStream_t st) {
    const int nkb = (a.T + kRopeKeysPerWg - 1) / kRopeKeysPerWg;
    const size_t plds = rope_post_lds_bytes(D, a.dd);
    if (plds > 65536) {
        const hipError_t e = hipFuncSetAttribute((const void*)bwd_rope_post_keys_kernel<D, NO>,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)plds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((bwd_rope_post_keys_kernel<D, NO>), dim3(nkb, a.B * a.Hkv), dim3(256), plds, st,
                       a.k, a.v, a.wd, a.wu, (const float*)a.dkr, (const float*)a.dvw,
                       (const float*)a.dkd, (const float*)a.dvd, a.tab, a.dk, a.dv, a.wpart, a.Hkv,
                       a.T, a.dd, a.w, a.r, a.pos0, a.L.nchunk);
    return hipGetLastError();
}

// the smallest column bound that holds ceil(d_down / (256 / D)); d_down <= D
template <int D>
static hipError_t launch_rope_post_keys(const RopeBwdArgs& a, hipStream_t st) {
    const int cpt = (a.dd + 256 / D - 1) / (256 / D);
    if (cpt <= 4) return launch_rope_post_keys_t<D, 4>(a, st);
    if (cpt <= 8) return launch_rope_post_keys_t<D, 8>(a, st);
    if (cpt <= 16) return launch_rope_post_keys_t<D, 16>(a, st);
    if constexpr (D * D / 256 > 16) {
        if (cpt <= 32) return launch_rope_post_keys_t<D, 32>(a, st);
        if (cpt <= D * D / 256) return launch_rope_post_keys_t<D, D * D / 256>(a, st);
    }
    return hipErrorInvalidValue;
}

template <int D>
static hipError_t launch_bwd_rope_t(const RopeBwdArgs& a, hipStream_t st) {
    constexpr int NW = 4;
    const int B = a.B, Hq = a.Hq, Hkv = a.Hkv, T = a.T, w = a.w, dd = a.dd, r = a.r;
    const int Tr = round_up(T, 64);
    const int Td = T - w > 0 ? T - w : 0;
    const float scale = 1.f / sqrtf((float)D);
    const float qscale = scale * kLog2eB;
    const int BM = NW * 32;
    const int nblk = (T + BM - 1) / BM;
    hipLaunchKernelGGL(bwd_rope_rowprep_kernel<D>, dim3((Tr + 255) / 256, B * Hq), dim3(256), 0, st, a.o, a.dout,
                       a.lse, a.nl2, a.nd, T, Tr);
    hipLaunchKernelGGL((bwd_rope_rows_kernel<D, NW>), dim3(nblk * B * Hq), dim3(NW * 64), 0, st, a.qr,
                       a.kr, a.v, a.kd, a.vd, a.dout, (const float*)a.nl2, (const float*)a.nd, a.dqr, Hq,
                       Hkv, T, Tr, w, qscale, scale, B * Hq);
    hipLaunchKernelGGL((bwd_rope_cols_kernel<D, NW, false>), dim3(nblk * B * Hkv), dim3(NW * 64), 0, st,
                       a.qr, a.kr, a.v, a.dout, (const float*)a.nl2, (const float*)a.nd, a.dkr, a.dvw,
                       Hq, Hkv, T, Tr, T, w, qscale, scale, B * Hkv);
    if (Td > 0) {
        const int nkb = (Td + BM - 1) / BM;
        hipLaunchKernelGGL((bwd_rope_cols_kernel<D, NW, true>), dim3(nkb * B * Hkv), dim3(NW * 64), 0, st,
                           a.qr, a.kd, a.vd, a.dout, (const float*)a.nl2, (const float*)a.nd, a.dkd,
                           a.dvd, Hq, Hkv, T, Tr, Td, w, qscale, scale, B * Hkv);
    }
    hipLaunchKernelGGL(bwd_rope_post_rows_kernel<D>, dim3((T * D + 255) / 256, B * Hq), dim3(256), 0,
                       st, (const float*)a.dqr, a.tab, a.dq, T, r, a.pos0);
    const hipError_t e = launch_rope_post_keys<D>(a, st);
    if (e != hipSuccess) return e;
    return launch_bwd_wreduce(a.wpart, a.dwd, a.dwu, Hkv, D, dd, a.L, st);
}

hipError_t launch_bwd_rope_mfma(const RopeBwdArgs& a, int d, hipStream_t st) {
    if (d == 64) return launch_bwd_rope_t<64>(a, st);
    if (d == 128) return launch_bwd_rope_t<128>(a, st);
    return hipErrorInvalidValue;
}

}  // namespace dar
