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
    for (int idx = tid; idx < 32 * D; idx += NW * 64) {
        const int c = idx / D, e = idx % D;
        U[c * LDU + e] = c < DD ? (wug ? wug[(size_t)c * D + e] : wdg[(size_t)e * DD + c]) : (bf16_t)0;
    }
    __syncthreads();
    const int r0 = wg_id_x() * NW * 32 + wave * 32;
    if (r0 >= Tr) return;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int rb = r0 + qc, ra = r0 + prow;  // B-layout row, A-layout row
    const bf16_t* qh = q + (size_t)bh * T * D;
    const bf16_t* dh = dout + (size_t)bh * T * D;
    const bf16_t* oh = o + (size_t)bh * T * D;
    bf16x8_t qB[KS], dB[KS], oB[KS], qA[KS], dA[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int e = s * 16 + hg * 8;
        qB[s] = rb < T ? load_bf16x8(qh + (size_t)rb * D + e) : zero_bf16x8();
        dB[s] = rb < T ? load_bf16x8(dh + (size_t)rb * D + e) : zero_bf16x8();
        oB[s] = rb < T ? load_bf16x8(oh + (size_t)rb * D + e) : zero_bf16x8();
        qA[s] = ra < T ? load_bf16x8(qh + (size_t)ra * D + e) : zero_bf16x8();
        dA[s] = ra < T ? load_bf16x8(dh + (size_t)ra * D + e) : zero_bf16x8();
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
        const float L2 = rb < T ? lse[(size_t)bh * T + rb] * kLog2eB : 0.f;
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
    for (int idx = tid; idx < 32 * D; idx += NW * 64) {
        const int c = idx / D, e = idx % D;
        U[c * LDU + e] = c < DD ? wdg[(size_t)e * DD + c] : (bf16_t)0;
    }
    __syncthreads();
    const int r0 = wg_id_x() * NW * 32 + wave * 32;
    if (r0 >= Tr) return;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int rb = r0 + qc, ra = r0 + prow;
    const bf16_t* kh = k + (size_t)bg * T * D;
    const bf16_t* vh = v + (size_t)bg * T * D;
    bf16x8_t kB[KS], vB[KS], kA[KS], vA[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int e = s * 16 + hg * 8;
        kB[s] = rb < T ? load_bf16x8(kh + (size_t)rb * D + e) : zero_bf16x8();
        vB[s] = rb < T ? load_bf16x8(vh + (size_t)rb * D + e) : zero_bf16x8();
        kA[s] = ra < T ? load_bf16x8(kh + (size_t)ra * D + e) : zero_bf16x8();
        vA[s] = ra < T ? load_bf16x8(vh + (size_t)ra * D + e) : zero_bf16x8();
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

// ---------------------------------------------------------------- distant: h, ol

// One wavefront per 32 query rows of one (batch, query head), distant keys
// j <= i - w only. No LDS and no barriers: the d_down-wide operands are read
// straight from L2, one 32-key subtile ahead (two register sets used in
// turn). Writes h = sum dS c^K and ol = sum P c^V (fp32) of every real row
// (zero without distant keys). Grid: ceil(T / (32 NW)) * B * Hq workgroups,
// dealt XCD by XCD (xcd_block_head); row blocks with the most keys first.
template <int DD>
struct RowDistOps {
    bf16x8_t ck[DD / 16], cv[DD / 16], kt[2], vt[2];
};

template <int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_rows_dist_kernel(
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ ckT,
    const bf16_t* __restrict__ cvb, const bf16_t* __restrict__ cvT,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ dts,
    const float* __restrict__ nl2, const float* __restrict__ nd, float* __restrict__ hk,
    float* __restrict__ ol, int Hq, int Hkv, int T, int Tr, int w, int BH) {
    constexpr int DS = DD / 16, BM = NW * 32;
    const int lane = lane_id_x() & 63;
    const int wave = __builtin_amdgcn_readfirstlane(lane_id_x() >> 6);
    const int nblk = (T + BM - 1) / BM;
    int rbi, bh;
    xcd_block_head(wg_id_x(), BH, rbi, bh);
    const int rb = nblk - 1 - rbi;  // row blocks with the most keys first
    const int b = bh / Hq, h = bh % Hq;
    const int bg = b * Hkv + h / (Hq / Hkv);
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int r0 = rb * BM + wave * 32, i = r0 + qc;
    if (r0 >= T) return;  // no barriers in this kernel
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

    const int jd_end = i_hi - w;  // last distant key of any row here
    if (jd_end >= 0) {
        const bf16_t* ckg = ckb + (size_t)bg * Tr * DD + (size_t)prow * DD + hg * 8;
        const bf16_t* cvg = cvb + (size_t)bg * Tr * DD + (size_t)prow * DD + hg * 8;
        const bf16_t* ckTg = ckT + (size_t)bg * T32 * 32 * 32;
        const bf16_t* cvTg = cvT + (size_t)bg * T32 * 32 * 32;
        const int js_last = jd_end & ~31;
        auto load = [&](int js) {
            js = imin(js, js_last);  // loads past the last subtile repeat it
            RowDistOps<DD> o;
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                o.ck[s] = load_bf16x8(ckg + (size_t)js * DD + s * 16);
                o.cv[s] = load_bf16x8(cvg + (size_t)js * DD + s * 16);
            }
            const bf16_t* kb = ckTg + (size_t)(js >> 5) * 32 * 32;
            const bf16_t* vb = cvTg + (size_t)(js >> 5) * 32 * 32;
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                o.kt[hf] = latT_operand(kb, qc, hg, hf);
                o.vt[hf] = latT_operand(vb, qc, hg, hf);
            }
            return o;
        };
        auto step = [&](const RowDistOps<DD>& c, int js) {
            f32x16_t x = mfma(c.ck[0], qtop[0], negL);
            f32x16_t dp = mfma(c.cv[0], dtop[0], negd);
            if (DS == 2) {
                x = mfma(c.ck[DS - 1], qtop[DS - 1], x);
                dp = mfma(c.cv[DS - 1], dtop[DS - 1], dp);
            }
            if (js + 31 > r0 - w) {
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
            hT = mfma(c.kt[0], pack8(ds, 0), hT);
            hT = mfma(c.kt[1], pack8(ds, 8), hT);
            olT = mfma(c.vt[0], pack8(p, 0), olT);
            olT = mfma(c.vt[1], pack8(p, 8), olT);
        };
        RowDistOps<DD> bufa = load(0), bufb;
        for (int js = 0;; js += 64) {
            bufb = load(js + 32);
            step(bufa, js);
            if (js + 32 > jd_end) break;
            bufa = load(js + 64);
            step(bufb, js + 32);
            if (js + 64 > jd_end) break;
        }
    }
    if (i >= T) return;
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

// One wavefront per 32 keys of one (batch, KV head), the distant rows
// i >= j + w of every query head of the group. No LDS and no barriers; the
// row operands are read from L2 one 32-row subtile ahead (two register sets
// used in turn). Each row's -lse and -delta enter through one more product
// each, with the row-constant operand (hi + mid + lo) against ones3. Writes
// gK = sum dS q~ (q~ unscaled) and gV = sum P dO~ (fp32) of every real key.
// Grid: ceil(T / (32 NW)) * B * Hkv workgroups (xcd_block_head); key block 0
// (most rows) first.
template <int DD>
struct ColDistOps {
    bf16x8_t q[DD / 16], d[DD / 16], qt[2], dt[2], cst;
};

template <int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_cols_dist_kernel(
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ cvb,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ qtT,
    const bf16_t* __restrict__ dts, const bf16_t* __restrict__ dtT,
    const bf16_t* __restrict__ rc, float* __restrict__ gk, float* __restrict__ gv, int Hq,
    int Hkv, int T, int Tr, int w, float gscale, int BKV) {
    constexpr int DS = DD / 16, BK = NW * 32;
    const int lane = lane_id_x() & 63;
    const int wave = __builtin_amdgcn_readfirstlane(lane_id_x() >> 6);
    int cb, bg;
    xcd_block_head(wg_id_x(), BKV, cb, bg);  // key block 0 (most rows) first
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int c0 = cb * BK + wave * 32, j = c0 + qc;
    if (c0 >= T) return;  // no barriers in this kernel
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
    const int is0 = (c0 + w) & ~31;  // first row block with a distant pair
    const int is_last = (T - 1) & ~31;
    for (int hh = 0; hh < G && is0 < T; ++hh) {
        const int bh = b * Hq + g * G + hh;
        const bf16_t* qth = qts + (size_t)bh * Tr * DD + (size_t)prow * DD + hg * 8;
        const bf16_t* dth = dts + (size_t)bh * Tr * DD + (size_t)prow * DD + hg * 8;
        const bf16_t* rch = rc + (size_t)bh * Tr * 16 + (size_t)prow * 16 + hg * 8;
        const bf16_t* qtTh = qtT + (size_t)bh * T32 * 32 * 32;
        const bf16_t* dtTh = dtT + (size_t)bh * T32 * 32 * 32;
        auto load = [&](int is) {
            is = imin(is, is_last);  // loads past the last subtile repeat it
            ColDistOps<DD> o;
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                o.q[s] = load_bf16x8(qth + (size_t)is * DD + s * 16);
                o.d[s] = load_bf16x8(dth + (size_t)is * DD + s * 16);
            }
            o.cst = load_bf16x8(rch + (size_t)is * 16);
            const bf16_t* qb = qtTh + (size_t)(is >> 5) * 32 * 32;
            const bf16_t* db = dtTh + (size_t)(is >> 5) * 32 * 32;
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                o.qt[hf] = latT_operand(qb, qc, hg, hf);
                o.dt[hf] = latT_operand(db, qc, hg, hf);
            }
            return o;
        };
        auto step = [&](const ColDistOps<DD>& c, int is) {
            f32x16_t x = mfma(c.cst, b_lse, splat16(0.f));
            f32x16_t dp = mfma(c.cst, b_del, splat16(0.f));
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                x = mfma(c.q[s], ckop[s], x);
                dp = mfma(c.d[s], cvop[s], dp);
            }
            if (!(is >= c0 + 31 + w && is + 31 < T)) {
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
            gkT = mfma(c.qt[0], pack8(ds, 0), gkT);
            gkT = mfma(c.qt[1], pack8(ds, 8), gkT);
            gvT = mfma(c.dt[0], pack8(p, 0), gvT);
            gvT = mfma(c.dt[1], pack8(p, 8), gvT);
        };
        ColDistOps<DD> bufa = load(is0), bufb;
        for (int is = is0;; is += 64) {
            bufb = load(is + 32);
            step(bufa, is);
            if (is + 32 >= T) break;
            bufa = load(is + 64);
            step(bufb, is + 32);
            if (is + 64 >= T) break;
        }
    }
    if (j >= T) return;
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
    const int Tr = round_up(T, 32);
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

}  // namespace dar
