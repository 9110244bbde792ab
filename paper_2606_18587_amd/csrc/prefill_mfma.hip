// Matrix-core (MFMA) causal DAR prefill, bf16 storage, fp32 accumulation,
// gfx950 (v_mfma_f32_32x32x16_bf16).
//
// Work unit: one workgroup = NW wavefronts = NW*32 query rows of one
// (batch, query head); one wavefront = 32 query rows, and lane l owns query
// row r0 + l%32 (lanes l and l^32 share a row and split its keys).
//
// Scores are computed transposed, S^T = K Q^T, so each lane holds 16 scores of
// its own query per 32-key subtile. The key rows of the A operand are read in
// a permuted order so that, in the accumulator layout, a lane's 16 scores are
// keys 8g..8g+7 and 16+8g..16+8g+7 (g = l/32): converted to bf16 they are the
// P^T operand of O^T += V^T P^T without any data movement. V^T is read from a
// row-major LDS tile with ds_read_b64_tr_b16.
//
// Two regions under one online softmax (Eq. 4):
//  * distant keys j <= i - w (Eq. 3, lifted branch): scores q~ . c^K_j with
//    q~ = q W_up^T (W_up absorbed into the query, Limitations section) and
//    c^K the window-exit latents of the pre-pass; values accumulate in d_down
//    space, O_lat^T += c^V^T P^T, and are lifted once in the epilogue,
//    O^T += W_up^T O_lat^T. These latent streams are small and are read per
//    wavefront straight from L2, without LDS or barriers.
//  * local keys i - w < j <= i (Eq. 3, full branch): q . k_j and P V at full
//    d, K/V tiles of 64 keys staged through LDS for the whole workgroup.
// Both regions use scale 1/sqrt(d); log2(e) is folded in so that p = exp2(x).
//
// Softmax bookkeeping (the distant region is bound by the exponential rate,
// so per-score work is kept to exp2, a max and a bf16 pack):
//  * the running reference m (per row) is subtracted inside the MFMA: the
//    accumulator input is a register block holding -m, so S' = S - m arrives
//    ready for exp2 (distant region); in the local region one FMA applies the
//    scale and subtracts m;
//  * m is only moved when a subtile's maximum exceeds it by more than kTau
//    (then the accumulators are rescaled), so p <= 2^kTau;
//  * with d_down = 16 the padding row 16 of the O_lat^T tile is fed ones, so
//    the MFMA also produces the distant row sums.
#include "../../include/dar.h"
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

static constexpr float kTau = 8.0f;

__device__ __forceinline__ bf16x8_t load_bf16x8(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}

__device__ __forceinline__ bf16x8_t zero_bf16x8() { return __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0)); }

__device__ __forceinline__ bf16x8_t ones_bf16x8() {
    return __builtin_bit_cast(bf16x8_t, make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u));
}

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ bf16x8_t pack8(float a0, float a1, float a2, float a3, float a4, float a5,
                                          float a6, float a7) {
    return __builtin_bit_cast(bf16x8_t, make_uint4(pack2(a0, a1), pack2(a2, a3), pack2(a4, a5), pack2(a6, a7)));
}

// value of lane l ^ 32
__device__ __forceinline__ float swap32(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    // lanes 0-31 receive the upper half in r[1], lanes 32-63 the lower half in r[0]
    return (threadIdx.x & 32) ? __uint_as_float(r[0]) : __uint_as_float(r[1]);
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

// Key offset (inside a 32-key subtile) held by accumulator register r of a
// lane in half g of the wavefront, given the permuted A-operand rows below.
__device__ __forceinline__ int acc_key(int r, int g) { return 16 * (r >> 3) + 8 * g + (r & 7); }

// Key loaded as A-operand row R (R = lane % 32) so that acc_key holds.
__device__ __forceinline__ int perm_row(int R) {
    const int a = R >> 3, gg = (R >> 2) & 1, b = R & 3;
    return 16 * (a >> 1) + 8 * gg + 4 * (a & 1) + b;
}

struct SoftmaxState {
    float m;    // reference (scaled log2 units); -inf until the row has seen a key
    float cm;   // -m, or 0 while m is -inf
    float l;    // partial row sum of this lane (bf16-rounded p)
};

// One 32-key subtile of the online softmax on x[16] (already relative to the
// reference). Returns P^T as two bf16x8 operands; rescales ow/ol if needed.
template <int NT, bool SUM_VALU>
__device__ __forceinline__ void softmax_step(f32x16_t& x, SoftmaxState& st, f32x16_t (&ow)[NT],
                                             f32x16_t& ol, bf16x8_t& p0, bf16x8_t& p1) {
    float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), x[2]), fmaxf(x[3], x[4]));
    mx = fmaxf(fmaxf(mx, x[5]), fmaxf(x[6], x[7]));
    mx = fmaxf(fmaxf(mx, x[8]), fmaxf(x[9], x[10]));
    mx = fmaxf(fmaxf(mx, x[11]), fmaxf(x[12], x[13]));
    mx = fmaxf(fmaxf(mx, x[14]), x[15]);
    mx = fmaxf(mx, swap32(mx));
    const bool fresh = st.m == -INFINITY;
    const bool need = fresh ? (mx > -INFINITY) : (mx > kTau);
    if (__builtin_amdgcn_ballot_w64(need)) {
        const float delta = need ? mx : 0.f;
        const float fac = need ? (fresh ? 0.f : exp2f(-delta)) : 1.f;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) ow[t][r] *= fac;
#pragma unroll
        for (int r = 0; r < 16; ++r) ol[r] *= fac;
        st.l *= fac;
        if (need) st.m = fresh ? mx : st.m + delta;
        st.cm = (st.m == -INFINITY) ? 0.f : -st.m;
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] -= delta;
    }
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(x[r]);
    p0 = pack8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
    p1 = pack8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    if (SUM_VALU) {
        const bf16x2_t one2 = {(__bf16)1.0f, (__bf16)1.0f};
        const uint4 u0 = __builtin_bit_cast(uint4, p0), u1 = __builtin_bit_cast(uint4, p1);
        float s = st.l;
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.w), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.w), one2, s, false);
        st.l = s;
    }
}

template <int D, int DD, int NW>
__global__ __launch_bounds__(NW * 64) void prefill_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu, const bf16_t* __restrict__ cK,
    const bf16_t* __restrict__ cVt, bf16_t* __restrict__ o, int Hq, int Hkv, int T, int w, int Tp,
    int nblk, int BH, float c_scale) {
    constexpr int BM = NW * 32;
    constexpr int KS = D / 16;   // 16-wide k slabs of q . k
    constexpr int DS = DD / 16;  // 16-wide k slabs of q~ . c^K
    constexpr int NT = D / 32;   // 32-row tiles of O_win^T
    constexpr int BN = 64;       // keys per LDS tile (local region)
    constexpr int LDK = D + 8;   // padded LDS row (bf16 elements)
    constexpr int CH = BN * D / 8 / (NW * 64);  // 16-byte chunks per thread per tile
    static_assert(CH >= 1 && BN * D / 8 == CH * NW * 64, "tile load split");
    extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
    bf16_t* lds_k = smem;                    // [2][BN][LDK]
    bf16_t* lds_v = smem + 2 * BN * LDK;     // [2][BN][LDK]

    const int idx = blockIdx.x;
    const int rb = nblk - 1 - idx / BH;  // longest row blocks first
    const int bh = idx - (idx / BH) * BH;
    const int b = bh / Hq, h = bh - (bh / Hq) * Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    const int i0 = rb * BM;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int qc = lane & 31, hg = lane >> 5;
    const int r0 = i0 + wave * 32;
    const int i = r0 + qc;
    const int i_hi = imin(r0 + 31, T - 1);  // last real row of this wavefront (< r0 if none)

    // ---- query operand (B of S^T = K Q^T): q[i][s*16 + hg*8 + 0..7]
    bf16x8_t qop[KS];
    {
        const bf16_t* qrow = q + ((size_t)bh * T + imin(i, T - 1)) * D;
#pragma unroll
        for (int s = 0; s < KS; ++s) qop[s] = (i < T) ? load_bf16x8(qrow + s * 16 + hg * 8) : zero_bf16x8();
    }

    SoftmaxState st{-INFINITY, 0.f, 0.f};
    f32x16_t ow[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) ow[t] = splat16(0.f);
    f32x16_t ol = splat16(0.f);

    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;

    // ---------------------------------------------------------------- distant region
    const int jd_end = (r0 < T) ? i_hi - w : -1;  // last distant key of any row here
    if (jd_end >= 0) {
        // q~^T = W_up q^T (scaled): A rows = latent column c, k = e.
        f32x16_t qt = splat16(0.f);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            bf16x8_t a = zero_bf16x8();
            if (qc < DD) {
                if (wug) {
                    a = load_bf16x8(wug + (size_t)qc * D + s * 16 + hg * 8);
                } else {
                    uint16_t t8[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) t8[j] = wdg[(size_t)(s * 16 + hg * 8 + j) * DD + qc];
                    a = __builtin_bit_cast(bf16x8_t, t8);
                }
            }
            qt = mfma(a, qop[s], qt);
        }
        // accumulator register 8*s + j holds latent column 16*s + (j<4 ? 4hg+j : 8+4hg+j-4)
        bf16x8_t qtop[DS];
#pragma unroll
        for (int s = 0; s < DS; ++s)
            qtop[s] = pack8(qt[8 * s + 0] * c_scale, qt[8 * s + 1] * c_scale, qt[8 * s + 2] * c_scale,
                            qt[8 * s + 3] * c_scale, qt[8 * s + 4] * c_scale, qt[8 * s + 5] * c_scale,
                            qt[8 * s + 6] * c_scale, qt[8 * s + 7] * c_scale);

        const bf16_t* ckb = cK + (size_t)bg * Tp * DD;
        const bf16_t* cvb = cVt + (size_t)bg * Tp * DD;
        const int prow = perm_row(qc);
        auto load_k = [&](int js, bf16x8_t (&ak)[DS]) {
#pragma unroll
            for (int s = 0; s < DS; ++s) ak[s] = load_bf16x8(ckb + (size_t)(js + prow) * DD + s * 16 + hg * 8);
        };
        auto load_v = [&](int js, bf16x8_t& a0, bf16x8_t& a1) {
            if (qc < DD) {
                const bf16_t* base = cvb + ((size_t)(js >> 6) * DD + qc) * 64 + (js & 63) + hg * 8;
                a0 = load_bf16x8(base);
                a1 = load_bf16x8(base + 16);
            } else if (DD == 16 && qc == 16) {
                a0 = ones_bf16x8();
                a1 = ones_bf16x8();
            } else {
                a0 = zero_bf16x8();
                a1 = zero_bf16x8();
            }
        };
        bf16x8_t ak[DS], av0, av1;
        load_k(0, ak);
        load_v(0, av0, av1);
        for (int js = 0; js <= jd_end; js += 32) {
            bf16x8_t akn[DS], avn0, avn1;
            const bool more = js + 32 <= jd_end;
            if (more) {
                load_k(js + 32, akn);
                load_v(js + 32, avn0, avn1);
            }
            f32x16_t x = splat16(st.cm);
#pragma unroll
            for (int s = 0; s < DS; ++s) x = mfma(ak[s], qtop[s], x);
            if (js + 31 > r0 - w) {  // staircase subtile: keep j <= i - w
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (js + acc_key(r, hg) > i - w) x[r] = -INFINITY;
            }
            bf16x8_t p0, p1;
            softmax_step<NT, DD != 16>(x, st, ow, ol, p0, p1);
            ol = mfma(av0, p0, ol);
            ol = mfma(av1, p1, ol);
            if (more) {
#pragma unroll
                for (int s = 0; s < DS; ++s) ak[s] = akn[s];
                av0 = avn0;
                av1 = avn1;
            }
        }
    }

    // ---------------------------------------------------------------- local region
    const int iwg_hi = imin(i0 + BM - 1, T - 1);
    const int jb_lo = imax(0, i0 - w + 1);
    if (w > 0 && jb_lo <= iwg_hi) {
        const int t_first = jb_lo & ~(BN - 1);
        const int ntile = (iwg_hi - t_first) / BN + 1;
        const bf16_t* kb = k + (size_t)bg * T * D;
        const bf16_t* vb = v + (size_t)bg * T * D;
        uint4 pk[CH], pv[CH];
        auto gload = [&](int t0) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int chunk = tid + c * NW * 64;
                const int row = chunk / (D / 8), col = (chunk % (D / 8)) * 8;
                const int key = t0 + row;
                if (key < T) {
                    pk[c] = *reinterpret_cast<const uint4*>(kb + (size_t)key * D + col);
                    pv[c] = *reinterpret_cast<const uint4*>(vb + (size_t)key * D + col);
                } else {
                    pk[c] = make_uint4(0, 0, 0, 0);
                    pv[c] = make_uint4(0, 0, 0, 0);
                }
            }
        };
        auto lstore = [&](int buf) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int chunk = tid + c * NW * 64;
                const int row = chunk / (D / 8), col = (chunk % (D / 8)) * 8;
                *reinterpret_cast<uint4*>(lds_k + (size_t)buf * BN * LDK + row * LDK + col) = pk[c];
                *reinterpret_cast<uint4*>(lds_v + (size_t)buf * BN * LDK + row * LDK + col) = pv[c];
            }
        };
        gload(t_first);
        lstore(0);
        __syncthreads();
        const int prow = perm_row(qc);
        const int quad = lane >> 4, sl = lane & 15;
        for (int n = 0; n < ntile; ++n) {
            const int t0 = t_first + n * BN;
            const int buf = n & 1;
            if (n + 1 < ntile) gload(t0 + BN);
            const bf16_t* lk = lds_k + (size_t)buf * BN * LDK;
            const bf16_t* lv = lds_v + (size_t)buf * BN * LDK;
#pragma unroll
            for (int sub = 0; sub < BN / 32; ++sub) {
                const int js = t0 + sub * 32;
                if (r0 < T && js <= i_hi && js + 31 > r0 - w) {
                    f32x16_t s = splat16(0.f);
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
                        s = mfma(load_bf16x8(lk + (sub * 32 + prow) * LDK + ks * 16 + hg * 8), qop[ks], s);
                    f32x16_t x;
#pragma unroll
                    for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(s[r], c_scale, st.cm);
                    if (!(js > i_hi - w && js + 31 <= r0)) {  // edge subtile: keep i - w < j <= i
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const int j = js + acc_key(r, hg);
                            if (j <= i - w || j > i) x[r] = -INFINITY;
                        }
                    }
                    bf16x8_t p0, p1;
                    softmax_step<NT, true>(x, st, ow, ol, p0, p1);
                    // O_win^T += V^T P^T; V^T operand via transposing LDS reads
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
#pragma unroll
                        for (int half = 0; half < 2; ++half) {
                            const int key = sub * 32 + half * 16 + 8 * (quad >> 1) + (sl >> 2);
                            const int col = t * 32 + 16 * (quad & 1) + 4 * (sl & 3);
                            const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                (lds_s16x4_t*)(lv + key * LDK + col));
                            const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                (lds_s16x4_t*)(lv + (key + 4) * LDK + col));
                            const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                            const bf16x8_t a = __builtin_bit_cast(bf16x8_t, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
                            ow[t] = mfma(a, half ? p1 : p0, ow[t]);
                        }
                    }
                }
            }
            if (n + 1 < ntile) lstore(buf ^ 1);
            __syncthreads();
        }
    }

    if (r0 >= T) return;

    // ---------------------------------------------------------------- epilogue
    float lt = st.l;
    if (DD == 16) lt += ol[8];  // ones row (row 16, held by lanes of half 0)
    lt += swap32(lt);

    if (jd_end >= 0) {
        // O^T += W_up^T O_lat^T, O_lat split into bf16 hi + lo parts
#pragma unroll
        for (int s = 0; s < DS; ++s) {
            float hi_f[8], lo_f[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float x = ol[8 * s + j];
                const uint32_t hb = pack2(x, 0.f) & 0xffffu;
                const float hv = __uint_as_float(hb << 16);
                hi_f[j] = hv;
                lo_f[j] = x - hv;
            }
            const bf16x8_t bhi = pack8(hi_f[0], hi_f[1], hi_f[2], hi_f[3], hi_f[4], hi_f[5], hi_f[6], hi_f[7]);
            const bf16x8_t blo = pack8(lo_f[0], lo_f[1], lo_f[2], lo_f[3], lo_f[4], lo_f[5], lo_f[6], lo_f[7]);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int e = t * 32 + qc;
                uint16_t a8[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int c = s * 16 + ((j < 4) ? 4 * hg + j : 8 + 4 * hg + (j - 4));
                    a8[j] = wug ? wug[(size_t)c * D + e] : wdg[(size_t)e * DD + c];
                }
                const bf16x8_t a = __builtin_bit_cast(bf16x8_t, a8);
                ow[t] = mfma(a, bhi, ow[t]);
                ow[t] = mfma(a, blo, ow[t]);
            }
        }
    }

    if (i < T) {
        const float inv = 1.f / lt;
        bf16_t* orow = o + ((size_t)bh * T + i) * D;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int e = t * 32 + grp * 8 + hg * 4;
                uint2 u;
                u.x = pack2(ow[t][grp * 4 + 0] * inv, ow[t][grp * 4 + 1] * inv);
                u.y = pack2(ow[t][grp * 4 + 2] * inv, ow[t][grp * 4 + 3] * inv);
                *reinterpret_cast<uint2*>(orow + e) = u;
            }
    }
}

bool prefill_mfma_supported(const dar_shape* s) {
    if (s->dtype != DAR_BF16) return false;
    if (s->d != 64 && s->d != 128) return false;
    if (s->d_down != 16 && s->d_down != 32) return false;
    return true;
}

template <int D, int DD>
static hipError_t launch_dd(int B, int Hq, int Hkv, int T, int w, const void* q, const void* k,
                            const void* v, const void* wd, const void* wu, void* o,
                            const void* cK, const void* cVt, hipStream_t st) {
    constexpr int NW = 4;
    constexpr int BM = NW * 32;
    const int nblk = (T + BM - 1) / BM;
    const int BH = B * Hq;
    const int Tp = (T - w > 0) ? round_up(T - w, 64) : 0;
    const float c_scale = 1.4426950408889634f / sqrtf((float)D);
    const size_t lds = sizeof(bf16_t) * 4 * 64 * (D + 8);
    auto kern = prefill_mfma_kernel<D, DD, NW>;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(nblk * BH), dim3(NW * 64), lds, st, (const bf16_t*)q,
                       (const bf16_t*)k, (const bf16_t*)v, (const bf16_t*)wd, (const bf16_t*)wu,
                       (const bf16_t*)cK, (const bf16_t*)cVt, (bf16_t*)o, Hq, Hkv, T, w, Tp, nblk,
                       BH, c_scale);
    return hipGetLastError();
}

hipError_t launch_prefill_mfma(const dar_shape* s, int T, const void* q, const void* k,
                               const void* v, const void* wd, const void* wu, void* o,
                               const void* cK, const void* cVt, hipStream_t st) {
    const int B = s->B, Hq = s->Hq, Hkv = s->Hkv, w = s->w;
    if (s->d == 64 && s->d_down == 16) return launch_dd<64, 16>(B, Hq, Hkv, T, w, q, k, v, wd, wu, o, cK, cVt, st);
    if (s->d == 64 && s->d_down == 32) return launch_dd<64, 32>(B, Hq, Hkv, T, w, q, k, v, wd, wu, o, cK, cVt, st);
    if (s->d == 128 && s->d_down == 16) return launch_dd<128, 16>(B, Hq, Hkv, T, w, q, k, v, wd, wu, o, cK, cVt, st);
    if (s->d == 128 && s->d_down == 32) return launch_dd<128, 32>(B, Hq, Hkv, T, w, q, k, v, wd, wu, o, cK, cVt, st);
    return hipErrorNotSupported;
}

}  // namespace dar
