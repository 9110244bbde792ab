// Matrix-core (MFMA) backward of the causal DAR prefill, bf16 storage, fp32
// accumulation, gfx950. The gradient formulas are those of the vector-ALU
// backward (backward.hip): one softmax over both regions, window pairs at
// full d, distant pairs in d_down space with W_up absorbed.
//
// Kernels, in launch order:
//  * bwd_prep_rows_kernel / bwd_prep_keys_kernel: q~ = q W_up^T (scaled by
//    log2(e)/sqrt(d)), dO~ = dO W_up^T, delta = dO . O per query row, and the
//    latents c^K, c^V (Eq. 1) per key, all in bf16, each also stored in
//    32-token blocks transposed ([T/32][d_down][32]) for the operands that
//    contract over tokens. Token counts are padded to a multiple of 32 with
//    zero rows.
//  * bwd_rows_mfma_kernel: one wavefront per 32 query rows, scores
//    transposed (S^T = K Q^T, one query per lane column, as in the forward).
//    Pass 1 takes the row log-sum-exp; pass 2 recomputes P, forms
//    dP^T = V dO^T (or c^V dO~^T) and dS, and accumulates dq^T += K^T dS^T
//    (window keys, K^T read transposed from LDS) and h^T += c^K^T dS^T,
//    ol^T += c^V^T P^T (distant keys); the epilogue lifts h with W_up^T.
//  * bwd_cols_mfma_kernel: one wavefront per 32 keys, scores in the other
//    orientation (S = Q K^T, one key per lane column), so that P and dS are
//    directly the B operands of dV^T += dO^T P and dK^T += Q^T dS (window
//    rows, Q^T and dO^T read transposed from LDS) and of gK^T += q~^T dS,
//    gV^T += dO~^T P (distant rows); the epilogue lifts gK and gV with
//    W_down.
//  * the weight-gradient reduction of backward.hip, on the fp32 h, ol, gK, gV.
// Masked pairs get a score of -inf (P = 0, dS = 0). The reference of each
// row's exponentials is its log-sum-exp, fed as the accumulator input of the
// score product (distant) or through one FMA (window), and -delta is the
// accumulator input of dP, so dS = P * dP' needs one multiply.
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

// A operand rows of a transposed latent block [d_down][32]: row R carries
// latent column perm_row(R) (so the accumulator rows come out in B-operand
// order), tokens 16 * half + 8 g + 0..7; rows past d_down are zero.
template <int DD>
__device__ __forceinline__ bf16x8_t latT_operand(const bf16_t* blk, int qc, int hg, int half) {
    const int c = perm_row(qc);
    if (DD < 32 && c >= DD) return zero_bf16x8();
    return load_bf16x8(blk + (size_t)c * 32 + 16 * half + 8 * hg);
}

}  // namespace

// ---------------------------------------------------------------- preparation

// Per query row i (padded rows get zeros): q~s = (q W_up^T) log2(e)/sqrt(d),
// dO~ = dO W_up^T (bf16, row-major and in transposed 32-row blocks) and
// delta = dO . O (fp32). One thread per row. Grid: (ceil(Tr / 256), B * Hq).
template <int D, int DD>
__global__ __launch_bounds__(256) void bwd_prep_rows_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ o, const bf16_t* __restrict__ dout,
    const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu, bf16_t* __restrict__ qts,
    bf16_t* __restrict__ qtT, bf16_t* __restrict__ dts, bf16_t* __restrict__ dtT,
    float* __restrict__ delta, int Hq, int Hkv, int T, int Tr, float qscale) {
    __shared__ float U[DD * D];  // U[c][e] = W_up[c][e]
    const int bh = blockIdx.y;
    const int g = (bh % Hq) / (Hq / Hkv);
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
    for (int idx = threadIdx.x; idx < DD * D; idx += 256) {
        const int c = idx / D, e = idx % D;
        U[idx] = wug ? bf16_to_f32(wug[(size_t)c * D + e]) : bf16_to_f32(wdg[(size_t)e * DD + c]);
    }
    __syncthreads();
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= Tr) return;
    float aq[DD], ad[DD];
#pragma unroll
    for (int c = 0; c < DD; ++c) { aq[c] = 0.f; ad[c] = 0.f; }
    float dl = 0.f;
    if (i < T) {
        const size_t row = (size_t)bh * T + i;
#pragma unroll
        for (int e8 = 0; e8 < D; e8 += 8) {
            const uint4 uq = *reinterpret_cast<const uint4*>(q + row * D + e8);
            const uint4 ud = *reinterpret_cast<const uint4*>(dout + row * D + e8);
            const uint4 uo = *reinterpret_cast<const uint4*>(o + row * D + e8);
            const uint32_t wq[4] = {uq.x, uq.y, uq.z, uq.w};
            const uint32_t wdd[4] = {ud.x, ud.y, ud.z, ud.w};
            const uint32_t wo[4] = {uo.x, uo.y, uo.z, uo.w};
#pragma unroll
            for (int h2 = 0; h2 < 8; ++h2) {
                const int sh = (h2 & 1) ? 0 : 16;
                const float xq = __uint_as_float((wq[h2 >> 1] << sh) & 0xffff0000u);
                const float xd = __uint_as_float((wdd[h2 >> 1] << sh) & 0xffff0000u);
                const float xo = __uint_as_float((wo[h2 >> 1] << sh) & 0xffff0000u);
                dl = __builtin_fmaf(xd, xo, dl);
#pragma unroll
                for (int c = 0; c < DD; ++c) {
                    aq[c] = __builtin_fmaf(xq, U[c * D + e8 + h2], aq[c]);
                    ad[c] = __builtin_fmaf(xd, U[c * D + e8 + h2], ad[c]);
                }
            }
        }
    }
    const size_t prow = (size_t)bh * Tr + i;
    bf16_t* qr = qts + prow * DD;
    bf16_t* dr = dts + prow * DD;
#pragma unroll
    for (int c8 = 0; c8 < DD; c8 += 8) {
        *reinterpret_cast<uint4*>(qr + c8) =
            make_uint4(pack2(aq[c8] * qscale, aq[c8 + 1] * qscale), pack2(aq[c8 + 2] * qscale, aq[c8 + 3] * qscale),
                       pack2(aq[c8 + 4] * qscale, aq[c8 + 5] * qscale), pack2(aq[c8 + 6] * qscale, aq[c8 + 7] * qscale));
        *reinterpret_cast<uint4*>(dr + c8) =
            make_uint4(pack2(ad[c8], ad[c8 + 1]), pack2(ad[c8 + 2], ad[c8 + 3]),
                       pack2(ad[c8 + 4], ad[c8 + 5]), pack2(ad[c8 + 6], ad[c8 + 7]));
    }
    bf16_t* qb = qtT + ((size_t)bh * (Tr / 32) + i / 32) * DD * 32 + (i & 31);
    bf16_t* db = dtT + ((size_t)bh * (Tr / 32) + i / 32) * DD * 32 + (i & 31);
#pragma unroll
    for (int c = 0; c < DD; ++c) {
        qb[c * 32] = f32_to_bf16(aq[c] * qscale);
        db[c * 32] = f32_to_bf16(ad[c]);
    }
    delta[prow] = dl;
}

// Per key token j (padded rows get zeros): c^K = k W_down, c^V = v W_down
// (Eq. 1) in bf16, row-major and in transposed 32-token blocks. One thread per
// token. Grid: (ceil(Tr / 256), B * Hkv).
template <int D, int DD>
__global__ __launch_bounds__(256) void bwd_prep_keys_kernel(
    const bf16_t* __restrict__ k, const bf16_t* __restrict__ v, const bf16_t* __restrict__ wd,
    bf16_t* __restrict__ ckb, bf16_t* __restrict__ ckT, bf16_t* __restrict__ cvb,
    bf16_t* __restrict__ cvT, int Hkv, int T, int Tr) {
    __shared__ float W[D * DD];  // W[e][c] = W_down[e][c]
    const int bg = blockIdx.y;
    const int g = bg % Hkv;
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    for (int idx = threadIdx.x; idx < D * DD; idx += 256) W[idx] = bf16_to_f32(wdg[idx]);
    __syncthreads();
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (j >= Tr) return;
    float ak[DD], av[DD];
#pragma unroll
    for (int c = 0; c < DD; ++c) { ak[c] = 0.f; av[c] = 0.f; }
    if (j < T) {
        const size_t row = (size_t)bg * T + j;
#pragma unroll
        for (int e8 = 0; e8 < D; e8 += 8) {
            const uint4 uk = *reinterpret_cast<const uint4*>(k + row * D + e8);
            const uint4 uv = *reinterpret_cast<const uint4*>(v + row * D + e8);
            const uint32_t wk[4] = {uk.x, uk.y, uk.z, uk.w};
            const uint32_t wv[4] = {uv.x, uv.y, uv.z, uv.w};
#pragma unroll
            for (int h2 = 0; h2 < 8; ++h2) {
                const int sh = (h2 & 1) ? 0 : 16;
                const float xk = __uint_as_float((wk[h2 >> 1] << sh) & 0xffff0000u);
                const float xv = __uint_as_float((wv[h2 >> 1] << sh) & 0xffff0000u);
#pragma unroll
                for (int c = 0; c < DD; ++c) {
                    ak[c] = __builtin_fmaf(xk, W[(e8 + h2) * DD + c], ak[c]);
                    av[c] = __builtin_fmaf(xv, W[(e8 + h2) * DD + c], av[c]);
                }
            }
        }
    }
    const size_t prow = (size_t)bg * Tr + j;
#pragma unroll
    for (int c8 = 0; c8 < DD; c8 += 8) {
        *reinterpret_cast<uint4*>(ckb + prow * DD + c8) =
            make_uint4(pack2(ak[c8], ak[c8 + 1]), pack2(ak[c8 + 2], ak[c8 + 3]),
                       pack2(ak[c8 + 4], ak[c8 + 5]), pack2(ak[c8 + 6], ak[c8 + 7]));
        *reinterpret_cast<uint4*>(cvb + prow * DD + c8) =
            make_uint4(pack2(av[c8], av[c8 + 1]), pack2(av[c8 + 2], av[c8 + 3]),
                       pack2(av[c8 + 4], av[c8 + 5]), pack2(av[c8 + 6], av[c8 + 7]));
    }
    bf16_t* kb = ckT + ((size_t)bg * (Tr / 32) + j / 32) * DD * 32 + (j & 31);
    bf16_t* vb = cvT + ((size_t)bg * (Tr / 32) + j / 32) * DD * 32 + (j & 31);
#pragma unroll
    for (int c = 0; c < DD; ++c) {
        kb[c * 32] = f32_to_bf16(ak[c]);
        vb[c * 32] = f32_to_bf16(av[c]);
    }
}

// ---------------------------------------------------------------- rows: dq, h, ol

template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_rows_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dout, const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu,
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ ckT,
    const bf16_t* __restrict__ cvb, const bf16_t* __restrict__ cvT,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ dts,
    const float* __restrict__ delta, float* __restrict__ lse, float* __restrict__ hk,
    float* __restrict__ ol, bf16_t* __restrict__ dq, int Hq, int Hkv, int T, int Tr, int w,
    float qscale, float scale) {
    constexpr int KS = D / 16, NT = D / 32, DS = DD / 16, BN = 64, LDK = D + 8, LDU = DD + 8;
    constexpr int BM = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_k[BN * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t lds_v[BN * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t ut[D * LDU];  // ut[e][c] = W_up[c][e]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nblk = (T + BM - 1) / BM;
    const int rb = nblk - 1 - (int)blockIdx.x;  // longest row blocks first
    const int bh = blockIdx.y;
    const int b = bh / Hq, h = bh % Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int i0 = rb * BM, r0 = i0 + wave * 32, i = r0 + qc;
    const bool live = r0 < T;                // this wavefront has real rows
    const int i_hi = imin(r0 + 31, T - 1);   // its last real row
    const int iwg_hi = imin(i0 + BM - 1, T - 1);
    const int ii = imin(i, T - 1);
    const int T32 = Tr / 32;

    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
    for (int idx = tid; idx < D * DD; idx += NW * 64) {
        const int e = idx / DD, c = idx % DD;
        ut[e * LDU + c] = wug ? wug[(size_t)c * D + e] : wdg[(size_t)e * DD + c];
    }

    // B operands of the query row: S^T = K Q^T, dP^T = V dO^T and the distant
    // forms with q~s, dO~.
    const bf16_t* qrow = q + ((size_t)bh * T + ii) * D;
    const bf16_t* drow = dout + ((size_t)bh * T + ii) * D;
    bf16x8_t qop[KS], doop[KS], qtop[DS], dtop[DS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        qop[s] = load_bf16x8(qrow + s * 16 + hg * 8);
        doop[s] = load_bf16x8(drow + s * 16 + hg * 8);
    }
    const size_t prw = (size_t)bh * Tr + ii;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        qtop[s] = load_bf16x8(qts + prw * DD + s * 16 + hg * 8);
        dtop[s] = load_bf16x8(dts + prw * DD + s * 16 + hg * 8);
    }
    const float dl = delta[prw];
    __syncthreads();

    const int jd_end = live ? i_hi - w : -1;  // last distant key of any row here
    const bool wg_local = w > 0 && i0 < T;
    const int jlo = imax(0, i0 - w + 1);
    const bf16_t* ckg = ckb + (size_t)bg * Tr * DD;
    const bf16_t* cvg = cvb + (size_t)bg * Tr * DD;
    const bf16_t* ckTg = ckT + (size_t)bg * T32 * DD * 32;
    const bf16_t* cvTg = cvT + (size_t)bg * T32 * DD * 32;
    const bf16_t* kg = k + (size_t)bg * T * D;
    const bf16_t* vg = v + (size_t)bg * T * D;

    auto load_tile = [&](int t, bool with_v) {
        constexpr int C8 = D / 8;
        for (int idx = tid; idx < BN * C8; idx += NW * 64) {
            const int r = idx / C8, c8 = idx % C8;
            const int key = t + r;
            uint4 uk = make_uint4(0, 0, 0, 0), uv = make_uint4(0, 0, 0, 0);
            if (key < T) {
                uk = *reinterpret_cast<const uint4*>(kg + (size_t)key * D + c8 * 8);
                if (with_v) uv = *reinterpret_cast<const uint4*>(vg + (size_t)key * D + c8 * 8);
            }
            *reinterpret_cast<uint4*>(lds_k + r * LDK + c8 * 8) = uk;
            if (with_v) *reinterpret_cast<uint4*>(lds_v + r * LDK + c8 * 8) = uv;
        }
    };

    // ---- pass 1: log-sum-exp of the row (log2 domain)
    float m = -INFINITY, l = 0.f;
    auto stats = [&](const f32x16_t& x) {
        float mx = x[0];
#pragma unroll
        for (int r = 1; r < 16; ++r) mx = fmaxf(mx, x[r]);
        mx = pair_max(mx);
        if (mx > m) {
            l *= exp2f(m - mx);
            m = mx;
        }
        if (m != -INFINITY) {
            float s = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) s += __builtin_amdgcn_exp2f(x[r] - m);
            l += s;
        }
    };
    for (int js = 0; js <= jd_end; js += 32) {
        const bf16_t* cr = ckg + (size_t)(js + prow) * DD + hg * 8;
        f32x16_t x = mfma(load_bf16x8(cr), qtop[0], splat16(0.f));
        if (DS == 2) x = mfma(load_bf16x8(cr + 16), qtop[DS - 1], x);
        if (js + 31 > r0 - w) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (js + acc_row(r, hg) > i - w) x[r] = -INFINITY;
        }
        stats(x);
    }
    if (wg_local) {
        for (int t = jlo & ~(BN - 1); t <= iwg_hi; t += BN) {
            __syncthreads();
            load_tile(t, false);
            __syncthreads();
            if (!live) continue;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int js = t + sub * 32;
                if (js > i_hi || js + 31 <= r0 - w) continue;
                f32x16_t sc = splat16(0.f);
#pragma unroll
                for (int s = 0; s < KS; ++s)
                    sc = mfma(load_bf16x8(lds_k + (sub * 32 + prow) * LDK + s * 16 + hg * 8), qop[s], sc);
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = sc[r] * qscale;
                if (!(js > i_hi - w && js + 31 <= r0)) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int j = js + acc_row(r, hg);
                        if (j <= i - w || j > i) x[r] = -INFINITY;
                    }
                }
                stats(x);
            }
        }
    }
    l = pair_sum(l);
    const float L = (m == -INFINITY) ? 0.f : m + log2f(l);
    if (live && i < Tr && hg == 0) lse[(size_t)bh * Tr + i] = L;  // padded rows: finite

    // ---- pass 2: gradients
    f32x16_t dqT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dqT[t] = splat16(0.f);
    f32x16_t hT = splat16(0.f), olT = splat16(0.f);
    const f32x16_t negL = splat16(-L), negd = splat16(-dl);

    for (int js = 0; js <= jd_end; js += 32) {
        const bf16_t* cr = ckg + (size_t)(js + prow) * DD + hg * 8;
        const bf16_t* vr = cvg + (size_t)(js + prow) * DD + hg * 8;
        f32x16_t x = mfma(load_bf16x8(cr), qtop[0], negL);
        f32x16_t dp = mfma(load_bf16x8(vr), dtop[0], negd);
        if (DS == 2) {
            x = mfma(load_bf16x8(cr + 16), qtop[DS - 1], x);
            dp = mfma(load_bf16x8(vr + 16), dtop[DS - 1], dp);
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
        const bf16x8_t p0 = pack8(p, 0), p1 = pack8(p, 8);
        const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
        const bf16_t* kblk = ckTg + (size_t)(js >> 5) * DD * 32;
        const bf16_t* vblk = cvTg + (size_t)(js >> 5) * DD * 32;
        hT = mfma(latT_operand<DD>(kblk, qc, hg, 0), s0, hT);
        hT = mfma(latT_operand<DD>(kblk, qc, hg, 1), s1, hT);
        olT = mfma(latT_operand<DD>(vblk, qc, hg, 0), p0, olT);
        olT = mfma(latT_operand<DD>(vblk, qc, hg, 1), p1, olT);
    }
    if (wg_local) {
        for (int t = jlo & ~(BN - 1); t <= iwg_hi; t += BN) {
            __syncthreads();
            load_tile(t, true);
            __syncthreads();
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
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, -L);
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
    // ---- epilogue: dq = s (dq_win + h W_up); h and ol (fp32) for dW_up.
    // The matrix-core lift runs for the whole wavefront (wave-uniform
    // condition); only the stores are per row.
    if (!live) return;
    if (jd_end >= 0) {
        bf16x8_t hhi[DS], hlo[DS];  // h as hi + lo bf16: the lift keeps ~16 bits of h
#pragma unroll
        for (int s = 0; s < DS; ++s) split8(hT, 8 * s, 1.f, hhi[s], hlo[s]);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                const bf16x8_t a = load_bf16x8(ut + (tt * 32 + qc) * LDU + s * 16 + hg * 8);
                dqT[tt] = mfma(a, hhi[s], dqT[tt]);
                dqT[tt] = mfma(a, hlo[s], dqT[tt]);
            }
    }
    if (i >= T) return;
    bf16_t* dqr = dq + ((size_t)bh * T + i) * D;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int a = 0; a < 4; ++a)
            store_bf16x4(dqr + tt * 32 + 8 * a + 4 * hg, dqT[tt][4 * a] * scale,
                         dqT[tt][4 * a + 1] * scale, dqT[tt][4 * a + 2] * scale,
                         dqT[tt][4 * a + 3] * scale);
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

// ---------------------------------------------------------------- columns: dk, dv, gK, gV

template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_cols_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dout, const bf16_t* __restrict__ wd,
    const bf16_t* __restrict__ ckb, const bf16_t* __restrict__ cvb,
    const bf16_t* __restrict__ qts, const bf16_t* __restrict__ qtT,
    const bf16_t* __restrict__ dts, const bf16_t* __restrict__ dtT,
    const float* __restrict__ lse, const float* __restrict__ delta, float* __restrict__ gk,
    float* __restrict__ gv, bf16_t* __restrict__ dk, bf16_t* __restrict__ dv, int Hq, int Hkv,
    int T, int Tr, int w, float qscale, float scale) {
    constexpr int KS = D / 16, NT = D / 32, DS = DD / 16, BN = 64, LDK = D + 8;
    constexpr int BK = NW * 32;
    __shared__ __attribute__((aligned(16))) bf16_t lds_q[BN * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t lds_do[BN * LDK];
    __shared__ __attribute__((aligned(16))) float lds_lse[BN];
    __shared__ __attribute__((aligned(16))) float lds_del[BN];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cb = blockIdx.x;  // key block 0 (most rows) first
    const int bg = blockIdx.y;
    const int b = bg / Hkv, g = bg % Hkv;
    const int G = Hq / Hkv;
    const int qc = lane & 31, hg = lane >> 5, prow = perm_row(qc);
    const int cwg_lo = cb * BK;
    const int c0 = cwg_lo + wave * 32, j = c0 + qc;
    const bool live = c0 < T;
    const int j_hi = imin(c0 + 31, T - 1);
    const int cwg_hi = imin(cwg_lo + BK - 1, T - 1);
    const int jj = imin(j, T - 1);
    const int T32 = Tr / 32;

    // B operands of the key column: S = Q K^T, dP = dO V^T and the distant
    // forms with c^K, c^V.
    bf16x8_t kop[KS], vop[KS], ckop[DS], cvop[DS];
    const bf16_t* krow = k + ((size_t)bg * T + jj) * D;
    const bf16_t* vrow = v + ((size_t)bg * T + jj) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        kop[s] = load_bf16x8(krow + s * 16 + hg * 8);
        vop[s] = load_bf16x8(vrow + s * 16 + hg * 8);
    }
#pragma unroll
    for (int s = 0; s < DS; ++s) {
        ckop[s] = load_bf16x8(ckb + ((size_t)bg * Tr + jj) * DD + s * 16 + hg * 8);
        cvop[s] = load_bf16x8(cvb + ((size_t)bg * Tr + jj) * DD + s * 16 + hg * 8);
    }

    f32x16_t dkT[NT], dvT[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { dkT[t] = splat16(0.f); dvT[t] = splat16(0.f); }
    f32x16_t gkT = splat16(0.f), gvT = splat16(0.f);
    const int loc_hi = w > 0 ? imin(T - 1, cwg_hi + w - 1) : -1;  // last row with a window pair

    for (int hh = 0; hh < G; ++hh) {
        const int bh = b * Hq + g * G + hh;
        const bf16_t* qh = q + (size_t)bh * T * D;
        const bf16_t* dh = dout + (size_t)bh * T * D;
        const float* lh = lse + (size_t)bh * Tr;
        const float* delh = delta + (size_t)bh * Tr;

        // window rows: 64-row Q / dO tiles staged in LDS for the workgroup
        for (int t = cwg_lo; t <= loc_hi; t += BN) {
            __syncthreads();
            {
                constexpr int C8 = D / 8;
                for (int idx = tid; idx < BN * C8; idx += NW * 64) {
                    const int r = idx / C8, c8 = idx % C8;
                    const int row = t + r;
                    uint4 uq = make_uint4(0, 0, 0, 0), ud = make_uint4(0, 0, 0, 0);
                    if (row < T) {
                        uq = *reinterpret_cast<const uint4*>(qh + (size_t)row * D + c8 * 8);
                        ud = *reinterpret_cast<const uint4*>(dh + (size_t)row * D + c8 * 8);
                    }
                    *reinterpret_cast<uint4*>(lds_q + r * LDK + c8 * 8) = uq;
                    *reinterpret_cast<uint4*>(lds_do + r * LDK + c8 * 8) = ud;
                }
                for (int r = tid; r < BN; r += NW * 64) {
                    const bool in = t + r < Tr;
                    lds_lse[r] = in ? lh[t + r] : 0.f;
                    lds_del[r] = in ? delh[t + r] : 0.f;
                }
            }
            __syncthreads();
            if (!live) continue;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int is = t + sub * 32;
                if (is + 31 < c0 || is > j_hi + w - 1) continue;
                f32x16_t sc = splat16(0.f);
                f32x16_t dp = load_row16(lds_del + sub * 32, hg, -1.f);
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    sc = mfma(load_bf16x8(lds_q + (sub * 32 + prow) * LDK + s * 16 + hg * 8), kop[s], sc);
                    dp = mfma(load_bf16x8(lds_do + (sub * 32 + prow) * LDK + s * 16 + hg * 8), vop[s], dp);
                }
                const f32x16_t ln = load_row16(lds_lse + sub * 32, hg, 1.f);
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, -ln[r]);
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

        // distant rows i >= j + w, straight from L2 for each wavefront
        if (live) {
            const bf16_t* qth = qts + (size_t)bh * Tr * DD;
            const bf16_t* dth = dts + (size_t)bh * Tr * DD;
            const bf16_t* qtTh = qtT + (size_t)bh * T32 * DD * 32;
            const bf16_t* dtTh = dtT + (size_t)bh * T32 * DD * 32;
            for (int is = (c0 + w) & ~31; is < T; is += 32) {
                const bf16_t* ar = qth + (size_t)(is + prow) * DD + hg * 8;
                const bf16_t* dr = dth + (size_t)(is + prow) * DD + hg * 8;
                f32x16_t x = mfma(load_bf16x8(ar), ckop[0], load_row16(lh + is, hg, -1.f));
                f32x16_t dp = mfma(load_bf16x8(dr), cvop[0], load_row16(delh + is, hg, -1.f));
                if (DS == 2) {
                    x = mfma(load_bf16x8(ar + 16), ckop[DS - 1], x);
                    dp = mfma(load_bf16x8(dr + 16), cvop[DS - 1], dp);
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
                const bf16x8_t p0 = pack8(p, 0), p1 = pack8(p, 8);
                const bf16x8_t s0 = pack8(ds, 0), s1 = pack8(ds, 8);
                const bf16_t* qblk = qtTh + (size_t)(is >> 5) * DD * 32;
                const bf16_t* dblk = dtTh + (size_t)(is >> 5) * DD * 32;
                gkT = mfma(latT_operand<DD>(qblk, qc, hg, 0), s0, gkT);
                gkT = mfma(latT_operand<DD>(qblk, qc, hg, 1), s1, gkT);
                gvT = mfma(latT_operand<DD>(dblk, qc, hg, 0), p0, gvT);
                gvT = mfma(latT_operand<DD>(dblk, qc, hg, 1), p1, gvT);
            }
        }
    }
    // ---- epilogue: dk = s dk_win + (s gK) W_down^T, dv = dv_win + gV W_down^T,
    // with gK = sum dS q~ (q~ unscaled: the operand above carried qscale).
    // The matrix-core lift runs for the whole wavefront (wave-uniform
    // condition; keys without distant rows have gK = gV = 0).
    if (!live) return;
    const float gscale = 1.f / qscale;
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    if (c0 + w < T) {
        // gK and gV as hi + lo bf16 pairs: the lift keeps ~16 bits of them
        bf16x8_t gkh[DS], gkl[DS], gvh[DS], gvl[DS];
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            split8(gkT, 8 * s, gscale * scale, gkh[s], gkl[s]);
            split8(gvT, 8 * s, 1.f, gvh[s], gvl[s]);
        }
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) dkT[tt][r] *= scale;
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                const bf16x8_t a = load_bf16x8(wdg + (size_t)(tt * 32 + qc) * DD + s * 16 + hg * 8);
                dkT[tt] = mfma(a, gkh[s], dkT[tt]);
                dkT[tt] = mfma(a, gkl[s], dkT[tt]);
                dvT[tt] = mfma(a, gvh[s], dvT[tt]);
                dvT[tt] = mfma(a, gvl[s], dvT[tt]);
            }
        }
    } else {
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int r = 0; r < 16; ++r) dkT[tt][r] *= scale;
    }
    if (j >= T) return;
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

// ---------------------------------------------------------------- host

bool bwd_mfma_supported(int d, int dd, bool bf16) {
    return bf16 && (d == 64 || d == 128) && (dd == 16 || dd == 32);
}

template <int D, int DD>
static hipError_t launch_bwd_mfma_t(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                    const bf16_t* o, const bf16_t* dout, const bf16_t* wd,
                                    const bf16_t* wu, bf16_t* dq, bf16_t* dk, bf16_t* dv,
                                    float* dwd, float* dwu, char* ws, const BwdWs& L, int B,
                                    int Hq, int Hkv, int T, int w, hipStream_t st) {
    constexpr int NW = 4;
    const int Tr = round_up(T, 32);
    const size_t nrow = (size_t)B * Hq * Tr * DD, ntok = (size_t)B * Hkv * Tr * DD;
    float* lse = (float*)(ws + L.lse_off);
    float* delta = (float*)(ws + L.delta_off);
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

    hipLaunchKernelGGL((bwd_prep_rows_kernel<D, DD>), dim3((Tr + 255) / 256, B * Hq), dim3(256), 0,
                       st, q, o, dout, wd, wu, qts, qtT, dts, dtT, delta, Hq, Hkv, T, Tr, qscale);
    hipLaunchKernelGGL((bwd_prep_keys_kernel<D, DD>), dim3((Tr + 255) / 256, B * Hkv), dim3(256),
                       0, st, k, v, wd, ckb, ckT, cvb, cvT, Hkv, T, Tr);
    const int nblk = (T + NW * 32 - 1) / (NW * 32);
    hipLaunchKernelGGL((bwd_rows_mfma_kernel<D, DD, NW>), dim3(nblk, B * Hq), dim3(NW * 64), 0, st,
                       q, k, v, dout, wd, wu, (const bf16_t*)ckb, (const bf16_t*)ckT,
                       (const bf16_t*)cvb, (const bf16_t*)cvT, (const bf16_t*)qts,
                       (const bf16_t*)dts, (const float*)delta, lse, hk, ol, dq, Hq, Hkv, T, Tr, w,
                       qscale, scale);
    hipLaunchKernelGGL((bwd_cols_mfma_kernel<D, DD, NW>), dim3(nblk, B * Hkv), dim3(NW * 64), 0,
                       st, q, k, v, dout, wd, (const bf16_t*)ckb, (const bf16_t*)cvb,
                       (const bf16_t*)qts, (const bf16_t*)qtT, (const bf16_t*)dts,
                       (const bf16_t*)dtT, (const float*)lse, (const float*)delta, gk, gv, dk, dv,
                       Hq, Hkv, T, Tr, w, qscale, scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bwd_weights<bf16_t>(q, k, v, dout, gk, gv, hk, ol, part, dwd, dwu, B, Hq, Hkv, T,
                                      D, DD, L, st);
}

hipError_t launch_bwd_mfma(const bf16_t* q, const bf16_t* k, const bf16_t* v, const bf16_t* o,
                           const bf16_t* dout, const bf16_t* wd, const bf16_t* wu, bf16_t* dq,
                           bf16_t* dk, bf16_t* dv, float* dwd, float* dwu, char* ws,
                           const BwdWs& L, int B, int Hq, int Hkv, int T, int d, int dd, int w,
                           hipStream_t st) {
#define DAR_BWD_CASE(D_, DD_)                                                                   \
    if (d == D_ && dd == DD_)                                                                   \
        return launch_bwd_mfma_t<D_, DD_>(q, k, v, o, dout, wd, wu, dq, dk, dv, dwd, dwu, ws, L, \
                                          B, Hq, Hkv, T, w, st);
    DAR_BWD_CASE(64, 16)
    DAR_BWD_CASE(64, 32)
    DAR_BWD_CASE(128, 16)
    DAR_BWD_CASE(128, 32)
#undef DAR_BWD_CASE
    return hipErrorInvalidValue;
}

}  // namespace dar
