// Split-KV DAR decode on the matrix cores (bf16; d in {64, 128}, d_down in
// {16, 32}, up to 8 query heads per KV head).
//
// One workgroup = 4 wavefronts = one split of one (batch, KV head); each
// wavefront walks its own run of 32-token subtiles of one region:
//   latent region (tokens [0, len - w)): S = C^K Q~^T with q~ = q W_up^T
//     (W_up absorbed, Limitations section), values in d_down space;
//   window region (the ring, tokens [len - w, len)): S = K Q^T, full d.
// As in the prefill kernel, scores are computed transposed so that a lane
// owns one query head (lane l: head l%32, tokens split between l and l^32),
// the key rows are read in a permuted order that makes the score registers
// the P^T operand of O^T += V^T P^T, and V^T comes from an LDS copy of the
// subtile through ds_read_b64_tr_b16. The query heads of a KV head are the
// MFMA columns, so every cache byte is read once per step for all of them.
// The softmax keeps a running reference per head that moves only when a
// subtile maximum exceeds it by kTau. With d_down = 16 the V^T operand rows
// 16..31 carry a constant [1, 0, 0, 0] chunk, so O^T row 16 is the row sum.
//
// Per split the four wavefronts merge through LDS and write one partial
// {m, l, acc} per query head; decode_combine_kernel merges the splits, lifts
// the latent part with W_up and normalises (Eq. 4, one softmax).
#include "../../include/dar.h"
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

namespace {

typedef __bf16 dbf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 dbf16x2 __attribute__((ext_vector_type(2)));
typedef float df32x16 __attribute__((ext_vector_type(16)));
typedef float df32x2 __attribute__((ext_vector_type(2)));
typedef short ds16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) ds16x4 lds_ds16x4;

constexpr float kTau = 8.0f;
constexpr int kWaves = 4;

__device__ __forceinline__ dbf16x8 ld8(const bf16_t* p) {
    return __builtin_bit_cast(dbf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ dbf16x8 zero8() { return __builtin_bit_cast(dbf16x8, make_uint4(0, 0, 0, 0)); }
__device__ __forceinline__ uint32_t pk2(float a, float b) {
    df32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, dbf16x2));
}
__device__ __forceinline__ dbf16x8 pk8(const float* p) {
    return __builtin_bit_cast(dbf16x8, make_uint4(pk2(p[0], p[1]), pk2(p[2], p[3]), pk2(p[4], p[5]), pk2(p[6], p[7])));
}
__device__ __forceinline__ df32x16 mma(dbf16x8 a, dbf16x8 b, df32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ df32x16 fill16(float x) {
    df32x16 r;
#pragma unroll
    for (int i = 0; i < 16; ++i) r[i] = x;
    return r;
}
__device__ __forceinline__ float pmax(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float psum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// token (inside a 32-token subtile) of accumulator register r in half g
__device__ __forceinline__ int dkey(int r, int g) { return 16 * (r >> 3) + 8 * g + (r & 7); }
// token read as A-operand row R so that dkey holds
__device__ __forceinline__ int dperm(int R) {
    const int a = R >> 3, gg = (R >> 2) & 1, b = R & 3;
    return 16 * (a >> 1) + 8 * gg + 4 * (a & 1) + b;
}

struct DecState {
    float m, cm, thr, l;
};

// Online softmax over one subtile's 16 scores per lane (already relative to
// the reference). Rescales acc on a reference move; packs P^T; adds the
// bf16-rounded p to l when SUMV.
template <int NT, bool SUMV>
__device__ __forceinline__ void dstep(df32x16& x, DecState& st, df32x16 (&acc)[NT], dbf16x8& p0, dbf16x8& p1) {
    float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), x[2]), fmaxf(x[3], x[4]));
    mx = fmaxf(fmaxf(mx, x[5]), fmaxf(x[6], x[7]));
    mx = fmaxf(fmaxf(mx, x[8]), fmaxf(x[9], x[10]));
    mx = fmaxf(fmaxf(mx, x[11]), fmaxf(x[12], x[13]));
    mx = fmaxf(fmaxf(mx, x[14]), x[15]);
    mx = pmax(mx);
    const bool need = mx > st.thr;
    if (__builtin_amdgcn_ballot_w64(need)) {
        const bool fresh = st.m == -INFINITY;
        const float delta = need ? mx : 0.f;
        const float fac = need ? (fresh ? 0.f : exp2f(-delta)) : 1.f;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[t][r] *= fac;
        st.l *= fac;
        if (need) st.m = fresh ? mx : st.m + delta;
        st.cm = (st.m == -INFINITY) ? 0.f : -st.m;
        st.thr = (st.m == -INFINITY) ? -INFINITY : kTau;
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] -= delta;
    }
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(x[r]);
    p0 = pk8(p);
    p1 = pk8(p + 8);
    if (SUMV) {
        const dbf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
        const uint4 u0 = __builtin_bit_cast(uint4, p0), u1 = __builtin_bit_cast(uint4, p1);
        float s = st.l;
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u0.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u0.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u0.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u0.w), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u1.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u1.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u1.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dbf16x2, u1.w), one2, s, false);
        st.l = s;
    }
}

}  // namespace

// Tokens per wavefront in each region (multiples of 32).
constexpr int kDecWaveLat = 512;
constexpr int kDecWaveWin = 128;
constexpr int kDecMaxGroup = 8;  // query heads per KV head on this path

template <int D, int DD>
__global__ __launch_bounds__(256) void decode_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu,
    const bf16_t* __restrict__ k_win, const bf16_t* __restrict__ v_win,
    const bf16_t* __restrict__ k_lat, const bf16_t* __restrict__ v_lat, float* __restrict__ part,
    int Hq, int Hkv, int w, int cap, int len, int n_lat_split, int S, float qscale) {
    constexpr int KS = D / 16, DS = DD / 16, NT = D / 32;
    constexpr int LDW = D + 8;                      // padded ring row in LDS (bf16)
    constexpr int VBUF = 32 * LDW;                  // per-wave V staging (bf16 elements)
    __shared__ __attribute__((aligned(16))) bf16_t vbuf[kWaves][VBUF + 8];
    __shared__ float red_m[kWaves][kDecMaxGroup], red_l[kWaves][kDecMaxGroup];
    __shared__ float red_o[kWaves][kDecMaxGroup][D + 1];

    const int s = blockIdx.x;
    const int bg = blockIdx.y;
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int G = Hq / Hkv;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int col = lane & 31, hg = lane >> 5;
    const int n_lat = imax(0, len - w);
    const bool latent = s < n_lat_split;
    int t_begin, t_end;  // this wavefront's token range (positions)
    if (latent) {
        t_begin = imin(n_lat, s * kWaves * kDecWaveLat + wave * kDecWaveLat);
        t_end = imin(n_lat, t_begin + kDecWaveLat);
    } else {
        const int s2 = s - n_lat_split;
        t_begin = imin(len, n_lat + s2 * kWaves * kDecWaveWin + wave * kDecWaveWin);
        t_end = imin(len, t_begin + kDecWaveWin);
    }
    bf16_t* vb = vbuf[wave];
    // constant chunk [1, 0, 0, 0] for the rows of the latent V^T operand past d_down
    if (lane == 0) {
        vb[VBUF + 0] = 0x3f80;
        vb[VBUF + 1] = 0;
        vb[VBUF + 2] = 0;
        vb[VBUF + 3] = 0;
    }

    // query heads of this KV head as MFMA columns: qop = q^T slabs (unscaled)
    const bool hval = col < G;
    const bf16_t* qrow = q + ((size_t)b * Hq + (size_t)g * G + (hval ? col : 0)) * D;
    dbf16x8 qop[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) qop[k] = hval ? ld8(qrow + k * 16 + hg * 8) : zero8();

    DecState st{-INFINITY, 0.f, -INFINITY, 0.f};
    df32x16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = fill16(0.f);
    const int quad = lane >> 4, sl = lane & 15;
    const int prow = dperm(col);

    if (t_begin < t_end && latent) {
        // ---- q~^T = W_up q^T, scaled; rearranged from the accumulator layout
        // (lane half g holds columns 4g..4g+3, 8+4g..8+4g+3 of each 16) to the
        // B-operand layout (half g holds 8g..8g+7) with one swap across halves.
        const bf16_t* wdg = wd + (size_t)g * D * DD;
        const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
        df32x16 qt = fill16(0.f);
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            dbf16x8 a = zero8();
            if (col < DD) {
                if (wug) {
                    a = ld8(wug + (size_t)col * D + k * 16 + hg * 8);
                } else {
                    uint16_t t8[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) t8[j] = wdg[(size_t)(k * 16 + hg * 8 + j) * DD + col];
                    a = __builtin_bit_cast(dbf16x8, t8);
                }
            }
            qt = mma(a, qop[k], qt);
        }
        dbf16x8 qtop[DS];
#pragma unroll
        for (int k = 0; k < DS; ++k) {
            float v8[8];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(qt[8 * k + j]),
                                                          __float_as_uint(qt[8 * k + 4 + j]), false, false);
                v8[j] = __uint_as_float(r[0]) * qscale;
                v8[4 + j] = __uint_as_float(r[1]) * qscale;
            }
            qtop[k] = pk8(v8);
        }

        const bf16_t* kl = k_lat + (size_t)bg * cap * DD;
        const bf16_t* vl = v_lat + (size_t)bg * cap * DD;
        const int last = t_end - 1;
        // V subtile copy: lane l moves 16 bytes (DS chunks of 64 lanes)
        auto load = [&](int t0, dbf16x8 (&ak)[DS], uint4 (&vv)[DS]) {
            const int kr = imin(t0 + prow, last);
#pragma unroll
            for (int k = 0; k < DS; ++k) ak[k] = ld8(kl + (size_t)kr * DD + k * 16 + hg * 8);
#pragma unroll
            for (int k = 0; k < DS; ++k) {
                const int chunk = lane + 64 * k;            // 16-byte chunk of the 32 x DD tile
                const int tr = imin(t0 + chunk / (DD / 8), last);
                vv[k] = *reinterpret_cast<const uint4*>(vl + (size_t)tr * DD + (chunk % (DD / 8)) * 8);
            }
        };
        auto body = [&](int t0, const dbf16x8 (&ak)[DS], const uint4 (&vv)[DS]) {
#pragma unroll
            for (int k = 0; k < DS; ++k) *reinterpret_cast<uint4*>(vb + (lane + 64 * k) * 8) = vv[k];
            df32x16 x = mma(ak[0], qtop[0], fill16(st.cm));
#pragma unroll
            for (int k = 1; k < DS; ++k) x = mma(ak[k], qtop[k], x);
            if (t0 + 31 > last) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (t0 + dkey(r, hg) > last) x[r] = -INFINITY;
            }
            dbf16x8 p0, p1;
            dstep<NT, DD != 16>(x, st, acc, p0, p1);
            // V^T operand: rows c = lane%32 of the DD-wide tile
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int key = half * 16 + 8 * (quad >> 1) + (sl >> 2);
                const int c = 16 * (quad & 1) + 4 * (sl & 3);
                const bf16_t* plo;
                const bf16_t* phi;
                if (DD == 16 && (quad & 1)) {
                    plo = vb + VBUF;
                    phi = vb + VBUF;
                } else {
                    plo = vb + key * DD + c;
                    phi = vb + (key + 4) * DD + c;
                }
                const ds16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)plo);
                const ds16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)phi);
                const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                const dbf16x8 a = __builtin_bit_cast(dbf16x8, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
                acc[0] = mma(a, half ? p1 : p0, acc[0]);
            }
        };
        dbf16x8 akA[DS], akB[DS];
        uint4 vA[DS], vB[DS];
        load(t_begin, akA, vA);
        load(t_begin + 32, akB, vB);
        int t0 = t_begin;
        for (; t0 + 32 < t_end; t0 += 64) {
            body(t0, akA, vA);
            load(t0 + 64, akA, vA);
            body(t0 + 32, akB, vB);
            load(t0 + 96, akB, vB);
        }
        if (t0 < t_end) body(t0, akA, vA);
        if (DD == 16) st.l = acc[0][8];  // ones row: full row sum on both halves
        else st.l = psum(st.l);
    } else if (t_begin < t_end) {
        // ---- window region: full-d keys and values from the ring
        const bf16_t* kw = k_win + (size_t)bg * w * D;
        const bf16_t* vw = v_win + (size_t)bg * w * D;
        const int last = t_end - 1;
        constexpr int CPT = 32 * D / 8 / 64;  // 16-byte chunks per lane per subtile
        auto load = [&](int t0, dbf16x8 (&ak)[KS], uint4 (&vv)[CPT]) {
            const int kr = imin(t0 + prow, last) % w;
#pragma unroll
            for (int k = 0; k < KS; ++k) ak[k] = ld8(kw + (size_t)kr * D + k * 16 + hg * 8);
#pragma unroll
            for (int k = 0; k < CPT; ++k) {
                const int chunk = lane + 64 * k;
                const int tr = imin(t0 + chunk / (D / 8), last) % w;
                vv[k] = *reinterpret_cast<const uint4*>(vw + (size_t)tr * D + (chunk % (D / 8)) * 8);
            }
        };
        auto body = [&](int t0, const dbf16x8 (&ak)[KS], const uint4 (&vv)[CPT]) {
#pragma unroll
            for (int k = 0; k < CPT; ++k) {
                const int chunk = lane + 64 * k;
                *reinterpret_cast<uint4*>(vb + (chunk / (D / 8)) * LDW + (chunk % (D / 8)) * 8) = vv[k];
            }
            df32x16 sc = fill16(0.f);
#pragma unroll
            for (int k = 0; k < KS; ++k) sc = mma(ak[k], qop[k], sc);
            df32x16 x;
#pragma unroll
            for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], qscale, st.cm);
            if (t0 + 31 > last) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (t0 + dkey(r, hg) > last) x[r] = -INFINITY;
            }
            dbf16x8 p0, p1;
            dstep<NT, true>(x, st, acc, p0, p1);
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int key = half * 16 + 8 * (quad >> 1) + (sl >> 2);
                    const int c = t * 32 + 16 * (quad & 1) + 4 * (sl & 3);
                    const ds16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)(vb + key * LDW + c));
                    const ds16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)(vb + (key + 4) * LDW + c));
                    const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                    const dbf16x8 a = __builtin_bit_cast(dbf16x8, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
                    acc[t] = mma(a, half ? p1 : p0, acc[t]);
                }
        };
        dbf16x8 akA[KS];
        uint4 vA[CPT];
        for (int t0 = t_begin; t0 < t_end; t0 += 32) {
            load(t0, akA, vA);
            body(t0, akA, vA);
        }
        st.l = psum(st.l);
    }

    // ---- merge the wavefronts of this split and write the partials
    const int dim = latent ? DD : D;
    if (col < G && hg == 0) {
        red_m[wave][col] = st.m;
        red_l[wave][col] = st.l;
    }
    if (col < G) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = t * 32 + 8 * (r >> 2) + 4 * hg + (r & 3);
                if (row < dim) red_o[wave][col][row] = acc[t][r];
            }
    }
    __syncthreads();
    const int stride = 2 + D;
    for (int idx = tid; idx < G * (dim + 2); idx += 256) {
        const int h = idx / (dim + 2), f = idx - (idx / (dim + 2)) * (dim + 2);
        float M = -INFINITY;
#pragma unroll
        for (int v = 0; v < kWaves; ++v) M = fmaxf(M, red_m[v][h]);
        float val = 0.f;
        if (f == 0) {
            val = M;
        } else {
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                const float mv = red_m[v][h];
                if (mv != -INFINITY) {
                    const float wgt = exp2f(mv - M);
                    val += wgt * (f == 1 ? red_l[v][h] : red_o[v][h][f - 2]);
                }
            }
        }
        const size_t bh = (size_t)b * Hq + (size_t)g * G + h;
        part[(bh * S + s) * stride + f] = val;
    }
}

bool decode_mfma_supported(int d, int dd, int G, bool bf16) {
    return bf16 && (d == 64 || d == 128) && (dd == 16 || dd == 32) && G >= 1 && G <= kDecMaxGroup;
}

void decode_mfma_splits(int len, int w, int& n_lat_split, int& n_win_split) {
    const int n_lat = len - w > 0 ? len - w : 0;
    const int n_win = len - n_lat;
    n_lat_split = (n_lat + kWaves * kDecWaveLat - 1) / (kWaves * kDecWaveLat);
    n_win_split = (n_win + kWaves * kDecWaveWin - 1) / (kWaves * kDecWaveWin);
}

hipError_t launch_decode_mfma(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                              const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_lat,
                              const bf16_t* v_lat, float* part, int B, int Hq, int Hkv, int d,
                              int dd, int w, int cap, int len, int& n_lat_split, int& S,
                              hipStream_t st) {
    int n_win_split;
    decode_mfma_splits(len, w, n_lat_split, n_win_split);
    S = n_lat_split + n_win_split;
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    dim3 grid(S, B * Hkv);
#define DAR_DEC_LAUNCH(D_, DD_)                                                                   \
    hipLaunchKernelGGL((decode_mfma_kernel<D_, DD_>), grid, dim3(256), 0, st, q, wd, wu, k_win,   \
                       v_win, k_lat, v_lat, part, Hq, Hkv, w, cap, len, n_lat_split, S, qscale)
    if (d == 64 && dd == 16) DAR_DEC_LAUNCH(64, 16);
    else if (d == 64 && dd == 32) DAR_DEC_LAUNCH(64, 32);
    else if (d == 128 && dd == 16) DAR_DEC_LAUNCH(128, 16);
    else DAR_DEC_LAUNCH(128, 32);
#undef DAR_DEC_LAUNCH
    return hipGetLastError();
}

}  // namespace dar
