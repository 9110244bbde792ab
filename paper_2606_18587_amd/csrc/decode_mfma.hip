// Split-KV DAR decode on the matrix cores (bf16; d in {64, 128}, d_down in
// {16, 32}, up to 8 query heads per KV head).
//
// Work split: each (batch, KV head) gets P workgroups of NW wavefronts, P
// chosen so that the whole grid is about one round of resident workgroups
// (no tail). The P*NW wavefronts are dealt to the two regions in proportion
// to the cache bytes each region holds, and each wavefront walks one
// contiguous run of 32-token subtiles of one region:
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
// The wavefronts of a workgroup merge through LDS. With one workgroup per
// (batch, KV head) it lifts the latent part with W_up, normalises (Eq. 4, one
// softmax) and writes the output itself; otherwise it writes one partial
// {m, l, acc_lat[d_down], acc_win[d]} per query head and
// decode_combine_kernel finishes.
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
// fp16 pairs and operands: the rotated distant keys and the query they meet
// (the rotation runs on packed fp16 pairs; fp16 keeps more mantissa than the
// bf16 operands elsewhere)
typedef _Float16 dh2 __attribute__((ext_vector_type(2)));
typedef _Float16 dh16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ dh2 h2(float a, float b) {
    return __builtin_bit_cast(dh2, __builtin_amdgcn_cvt_pkrtz(a, b));
}
__device__ __forceinline__ dh16x8 h8(dh2 a, dh2 b, dh2 c, dh2 d) {
    return __builtin_bit_cast(dh16x8, make_uint4(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b),
                                                 __builtin_bit_cast(uint32_t, c), __builtin_bit_cast(uint32_t, d)));
}
__device__ __forceinline__ df32x16 mmah(dh16x8 a, dh16x8 b, df32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
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

// RoPE (rotate-half, rotary dimension R) of a row held as KS slabs of 8
// elements in the operand layout (lane half hg holds elements 16k + 8hg + j),
// at the position whose table row is cs (cos of the R/2 angles, then sin).
// With R a multiple of 32 the partner of element e (e + R/2) is in this
// lane (slab k + R/32); with R = 16 it is in the other half (one swap).
template <int KS, int R>
__device__ __forceinline__ void rotate_slabs(float (&x)[KS][8], const float* cs, int hg) {
    if constexpr (R % 32 == 0) {
#pragma unroll
        for (int k = 0; k < R / 32; ++k) {
            const int m0 = 16 * k + 8 * hg;
            const float4 c0 = *reinterpret_cast<const float4*>(cs + m0);
            const float4 c1 = *reinterpret_cast<const float4*>(cs + m0 + 4);
            const float4 s0 = *reinterpret_cast<const float4*>(cs + R / 2 + m0);
            const float4 s1 = *reinterpret_cast<const float4*>(cs + R / 2 + m0 + 4);
            const float c8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
            const float s8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float a = x[k][j], b = x[k + R / 32][j];
                x[k][j] = __builtin_fmaf(a, c8[j], -(b * s8[j]));
                x[k + R / 32][j] = __builtin_fmaf(b, c8[j], a * s8[j]);
            }
        }
    } else {
        static_assert(R == 16, "rotary dimension 16 or a multiple of 32");
        // slab 0: half 0 holds elements 0..7 (first of their pairs), half 1
        // elements 8..15 (the partners); both use angles m = j
        const float4 c0 = *reinterpret_cast<const float4*>(cs);
        const float4 c1 = *reinterpret_cast<const float4*>(cs + 4);
        const float4 s0 = *reinterpret_cast<const float4*>(cs + 8);
        const float4 s1 = *reinterpret_cast<const float4*>(cs + 12);
        const float c8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        const float s8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float own = x[0][j];
            auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(own), __float_as_uint(own), false, false);
            // the partner's value: lanes of half 0 find it in r[1], half 1 in r[0]
            const float other = __uint_as_float(hg == 0 ? r[1] : r[0]);
            x[0][j] = hg == 0 ? __builtin_fmaf(own, c8[j], -(other * s8[j]))
                              : __builtin_fmaf(own, c8[j], other * s8[j]);
        }
    }
}

// The reference m is kept exactly representable in bf16 (rounded up when it
// moves), so that the latent scores can subtract it inside the MFMA: a rank-1
// product of a constant operand (1 in contraction slot 0 of every key row)
// and negm (-m of each head in slot 0) yields -m in every accumulator.
struct DecState {
    float m, cm, thr, l;
    dbf16x8 negm;  // B operand: -m at contraction slot 0 (lanes of half 0), zeros elsewhere
};

// 16-byte non-temporal load (a cache byte read once per step)
typedef unsigned int du32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ du32x4 ld_stream(const bf16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const du32x4*>(p));
}

// Marks a rarely taken, wave-uniform branch: the compiler may not execute its
// body unconditionally (if-converted, every subtile would pay for it).
__device__ __forceinline__ void keep_branch() { __asm__ volatile(""); }

// A pointer every lane of the wavefront holds, moved to scalar registers.
__device__ __forceinline__ const bf16_t* uniform_ptr(const bf16_t* p) {
    const uint64_t u = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return (const bf16_t*)(((uint64_t)hi << 32) | lo);
}

// bf16 value >= x (x finite): round the fp32 bit pattern up to 16 bits
__device__ __forceinline__ float bf16_ceil(float x) {
    uint32_t u = __float_as_uint(x);
    const uint32_t low = u & 0xffffu;
    u &= 0xffff0000u;
    if (low != 0) u += (x > 0.f) ? 0x10000u : 0u;  // away from zero for positives, truncation for negatives
    return __uint_as_float(u);
}

// Online softmax over one subtile's 16 scores per lane (already relative to
// the reference). Rescales acc on a reference move; packs P^T; adds the
// bf16-rounded p to l when SUMV.
// B operand with -m (= cm, bf16-exact) at contraction slot 0: lane half 0,
// element 0 of the 8-element run
__device__ __forceinline__ dbf16x8 negm_operand(float cm, int hg) {
    const uint32_t b = __float_as_uint(cm) >> 16;  // exact: cm is a bf16 value
    return __builtin_bit_cast(dbf16x8, make_uint4(hg == 0 ? b : 0u, 0u, 0u, 0u));
}

template <int NT, bool SUMV>
__device__ __forceinline__ void dstep(df32x16& x, DecState& st, df32x16 (&acc)[NT], dbf16x8& p0, dbf16x8& p1,
                                      int hg, df32x16* xnext = nullptr) {
    float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), x[2]), fmaxf(x[3], x[4]));
    mx = fmaxf(fmaxf(mx, x[5]), fmaxf(x[6], x[7]));
    mx = fmaxf(fmaxf(mx, x[8]), fmaxf(x[9], x[10]));
    mx = fmaxf(fmaxf(mx, x[11]), fmaxf(x[12], x[13]));
    mx = fmaxf(fmaxf(mx, x[14]), x[15]);
    mx = pmax(mx);
    const bool need = mx > st.thr;
    if (__builtin_amdgcn_ballot_w64(need)) {
        keep_branch();
        // new reference: the subtile maximum, rounded up to a bf16 value
        const bool fresh = st.m == -INFINITY;
        const float mnew = need ? bf16_ceil(fresh ? mx : st.m + mx) : st.m;
        const float delta = need ? (fresh ? mnew : mnew - st.m) : 0.f;  // x is relative to the old reference (0 if none)
        const float fac = need ? (fresh ? 0.f : exp2f(-delta)) : 1.f;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[t][r] *= fac;
        st.l *= fac;
        st.m = mnew;
        st.cm = (st.m == -INFINITY) ? 0.f : -st.m;
        st.thr = (st.m == -INFINITY) ? -INFINITY : kTau;
        st.negm = negm_operand(st.cm, hg);
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] -= delta;
        if (xnext) {  // scores already computed against the old reference
#pragma unroll
            for (int r = 0; r < 16; ++r) (*xnext)[r] -= delta;
        }
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

constexpr int kDecMaxGroup = 8;   // query heads per KV head on this path
// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data
// format; with stride 0, accesses at or past num_records return zero).
constexpr int kBufWord3 = 0x00020000;
// Cache policy of the cache streams: non-temporal (every cache byte is read
// once per step; measured 12% faster than the default policy at 32K tokens).
constexpr int kStream = 2;
constexpr int kDecMinSub = 4;     // fewest subtiles a wavefront is given, when possible

// Subtile run of wavefront `idx` (of nwave per (batch, KV head)). Waves
// [0, nwl) share the latent subtiles, waves [nwl, nwave) the ring subtiles;
// nwl is proportional to the latent region's share of the cache bytes.
struct WaveRun {
    int latent;        // 1: latent region, 0: window region
    int t_begin, t_end;  // token positions [t_begin, t_end)
};

// Subtile run of wavefront idx (of nwave) over latent subtiles [ls0, ls1)
// and ring subtiles [ws0, ws1) of a cache of len tokens.
__host__ __device__ inline WaveRun decode_wave_run_range(int len, int w, int D, int DD, int ls0,
                                                         int ls1, int ws0, int ws1, int nwave,
                                                         int idx) {
    const int n_lat = len - w > 0 ? len - w : 0;
    const int n_win = len - n_lat;
    const long long nls = ls1 - ls0, nws = ws1 - ws0;
    int nwr = 0;  // wavefronts on the ring
    if (nws > 0) {
        if (nls == 0) {
            nwr = nwave;
        } else {
            const long long cw = nws * D, cl = nls * DD;
            nwr = (int)((2 * nwave * cw + cl + cw) / (2 * (cl + cw)));  // rounded share
            nwr = nwr < 1 ? 1 : (nwr > nwave - 1 ? nwave - 1 : nwr);
        }
    }
    const int nwl = nwave - nwr;
    WaveRun r;
    if (idx < nwl) {
        const long long s0 = ls0 + nls * idx / nwl, s1 = ls0 + nls * (idx + 1) / nwl;
        r.latent = 1;
        r.t_begin = (int)(32 * s0);
        r.t_end = (int)(32 * s1 < n_lat ? 32 * s1 : n_lat);
    } else {
        const int j = idx - nwl;
        const long long s0 = ws0 + nws * j / nwr, s1 = ws0 + nws * (j + 1) / nwr;
        r.latent = 0;
        r.t_begin = n_lat + (int)(32 * s0);
        r.t_end = n_lat + (int)(32 * s1 < n_win ? 32 * s1 : n_win);
    }
    return r;
}

__host__ __device__ inline WaveRun decode_wave_run(int len, int w, int D, int DD, int nwave, int idx) {
    const int n_lat = len - w > 0 ? len - w : 0;
    return decode_wave_run_range(len, w, D, DD, 0, (n_lat + 31) / 32, 0, (len - n_lat + 31) / 32,
                                 nwave, idx);
}

// NW = 8 wavefronts per workgroup: one workgroup per compute unit, 2 waves
// per SIMD, so that each wavefront can keep many subtiles in flight.
template <int D>
struct DecWaves {
    static constexpr int value = 8;
};
// Latent subtiles in flight per wavefront (register budget of 2 waves/SIMD).
template <int D, int DD, int R = 0>
struct DecStages {
    static constexpr int value = R > 0 ? (DD <= 16 ? 6 : 4)
                                       : (D <= 64 ? (DD <= 16 ? 12 : 7) : (DD <= 16 ? 10 : 5));
};

// Jobs of a paged batch. The work of a (sequence, KV head) pair is counted
// in units of one latent subtile's bytes (a ring subtile is D / DD units). A
// pair of U units is cut into n = ceil(U / cu) parts of cu units (the last one
// the remainder), cu = max(ceil(4 total / (3 kPagedGroups)), kPagedMinPart,
// ceil(U(cap) / kPagedMaxParts)): a third more than one compute unit's share
// of the batch (measured on a ragged batch: 1, 1.25, 4/3, 1.5 and 2 shares
// gave 80, 70, 69, 74 and 80 us). One workgroup per part; the full parts of
// all pairs come first in
// the grid, then the remainders from the largest down (longest processing
// time first), so that the last workgroups to start are the shortest. A pair
// of one part is finished by its workgroup; the others' parts leave partial
// records (slot = part index, count n in pg.counts) for the combine kernel.
constexpr int kPagedGroups = 256;   // compute units
constexpr long kPagedMinPart = 32;  // units
constexpr int kPagedMaxParts = 16;  // parts of one pair, at most
constexpr int kPagedRankMax = 512;  // sequences ranked by remainder (more: in batch order)
__host__ __device__ inline long paged_units(int len, int w, int cap, int D, int DD) {
    len = len < 0 ? 0 : (len > cap ? cap : len);  // empty or overflowed: no work
    const int n_lat = len - w > 0 ? len - w : 0;
    return (long)((n_lat + 31) / 32) + (long)((len - n_lat + 31) / 32) * (D / DD);
}
// the part size for a batch of `total` units
__host__ __device__ inline long paged_part(long total, int cap, int w, int D, int DD) {
    long cu = (total * 4 + kPagedGroups * 3 - 1) / (kPagedGroups * 3);
    const long cmin = (paged_units(cap, w, cap, D, DD) + kPagedMaxParts - 1) / kPagedMaxParts;
    cu = cu > cmin ? cu : cmin;
    return cu > kPagedMinPart ? cu : kPagedMinPart;
}


// R > 0: the rotary embedding of Eq. 3 with rotary dimension R (rotate-half
// pairs; d 64 or 128, R <= 64). The query is rotated at position len - 1, each ring key at
// its position as it is loaded. A distant key has to be lifted to full d
// before its rotation: per 32-token subtile the latent keys are lifted on
// the matrix cores, K'^T = W_up^T C^T (the latent rows as loaded are the B
// operand), and each lane rotates its token's elements in registers. Token
// p = t0 + delta of a subtile starting at t0 takes cos/sin(p f) from the
// angle-addition formula, with the subtile's table row (t0) read per subtile
// and the lane's offset row (delta) held in registers for the whole run.
// The rotated K' is the A operand of the scores as it stands (its element
// order is matched by a permuted query operand). Values are not rotated:
// the distant ones stay in d_down space and are lifted once, as without
// rotation. tab: [n_pos][R] (cos of the R/2 angles, then their sin).
// PAGED: the latents come from the pages of a paged cache and the cache
// length of each sequence from pg.lens; each 32-token subtile lies inside one
// page (ps is a multiple of 32), whose descriptor is built per subtile. The
// grid is one workgroup per job (part of a pair; see kPagedGroups).
// SHARED: one latent array for keys and values (v_lat == k_lat): each
// latent subtile is loaded once, in the key operand's layout; the scores use
// it as loaded, and the same registers, stored at their token rows, are the
// LDS tile the value operand is read from.
// The kernel's arguments, as one piece of work reads them.
struct DecArgs {
    const bf16_t *q, *wd, *wu, *k_win, *v_win, *k_lat, *v_lat;
    float* part;
    bf16_t* o;
    const float* tab;
    const bf16_t* wv;
    const int* block_table;
    PagedArgs pg;
    int Hq, Hkv, w, cap, P, n_pos;
    float qscale;
};
static_assert(sizeof(DecArgs) % 4 == 0, "copied as 32-bit words");

// A wave-uniform load through the scalar cache (the data is not written
// while the kernel runs): a vector load here would be waited for behind the
// cache stream's loads in flight, which retire in order.
__device__ __forceinline__ int scalar_load(const int* p) {
    return *(const __attribute__((address_space(4))) int*)p;
}


template <int D, int DD, int NW, int R = 0, bool PAGED = false, bool SHARED = false>
__global__ __launch_bounds__(NW * 64) void decode_mfma_kernel(
    const bf16_t* __restrict__ q_, const bf16_t* __restrict__ wd_, const bf16_t* __restrict__ wu_,
    const bf16_t* __restrict__ k_win_, const bf16_t* __restrict__ v_win_,
    const bf16_t* __restrict__ k_lat_, const bf16_t* __restrict__ v_lat_, float* __restrict__ part_,
    bf16_t* __restrict__ o_, int Hq_, int Hkv_, int w_, int cap_, int len_arg, int P_, float qscale_,
    const float* __restrict__ tab_, int n_pos_, const bf16_t* __restrict__ wv_, PagedArgs pg_,
    const int* __restrict__ block_table_) {
    static_assert(R == 0 || ((D == 64 || D == 128) && R % 16 == 0 && R <= 64),
                  "rotary: d 64 or 128, R a multiple of 16 up to 64");
    constexpr int KS = D / 16, DS = DD / 16, NT = D / 32;
    // With rotation only elements [0, R) of a lifted distant key turn, R <= 64:
    // the first 64 elements are lifted and rotated per subtile (NL tiles of
    // 32, KL query slabs against them); with D = 128 elements [64, 128) are
    // not rotated, so their part of the score stays absorbed in the query,
    // (q_hi W_up,hi^T) . c, one more MFMA on the latent rows as loaded.
    constexpr int NL = R > 0 ? 2 : NT, KL = R > 0 ? 4 : KS;
    constexpr int QK0 = R > 0 ? (D > 64 ? 4 : KS) : 0;  // first query slab absorbed
    constexpr int LDW = D + 8;                      // padded ring row in LDS (bf16)
    constexpr int VBUF = 32 * LDW;                  // per-wave V staging (bf16 elements)
    constexpr int stride = 2 + DD + D;              // partial record {m, l, acc_lat, acc_win}
    __shared__ __attribute__((aligned(16))) bf16_t vbuf[NW][VBUF + 8];
    __shared__ float red_m[NW][kDecMaxGroup], red_l[NW][kDecMaxGroup];
    __shared__ float red_o[NW][kDecMaxGroup][D + 1];
    __shared__ int red_lat[NW];
    __shared__ float wsh[DD][D];                    // W_up (fp32), used when P == 1
    __shared__ float mrg[kDecMaxGroup][stride];     // merged record, used when P == 1
    const DecArgs args_in{q_, wd_, wu_, k_win_, v_win_, k_lat_, v_lat_, part_, o_, tab_, wv_,
                          block_table_, pg_, Hq_, Hkv_, w_, cap_, P_, n_pos_, qscale_};

    // One piece of work: latent subtiles [ls0, ls1) and ring subtiles
    // [ws0, ws1) of (sequence b, KV head g), whose cache holds len tokens,
    // shared by nwave wavefronts of which this one is number widx. fuse: the
    // workgroup has the whole pair and writes the output; else it writes
    // partial record srec of each head.
    auto piece = [&](const int b, const int g, const int len, const bool fuse, const int srec,
                     const int ls0, const int ls1, const int ws0, const int ws1, const int nwave,
                     const int widx) {
    const DecArgs A = args_in;
    const bf16_t* __restrict__ const q = A.q;
    const bf16_t* __restrict__ const wd = A.wd;
    const bf16_t* __restrict__ const wu = A.wu;
    const bf16_t* __restrict__ const k_win = A.k_win;
    const bf16_t* __restrict__ const v_win = A.v_win;
    const bf16_t* __restrict__ const k_lat = A.k_lat;
    const bf16_t* __restrict__ const v_lat = A.v_lat;
    float* __restrict__ const part = A.part;
    bf16_t* __restrict__ const o = A.o;
    const float* __restrict__ const tab = A.tab;
    const bf16_t* __restrict__ const wv = A.wv;
    const int* __restrict__ const block_table = A.block_table;
    const PagedArgs pg = A.pg;
    const int Hq = A.Hq, Hkv = A.Hkv, w = A.w, cap = A.cap, P = A.P, n_pos = A.n_pos;
    const float qscale = A.qscale;
    const int G = Hq / Hkv;
    // (the thread's indices are computed here, not captured: captured, they
    // cost the loops below registers)
    const int tid = lane_id_x();
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int col = lane & 31, hg = lane >> 5;
    const int bg = b * Hkv + g;
    if (fuse) {
        const bf16_t* wdg = wd + (size_t)g * D * DD;
        const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
        // the lift's matrix: W_up, or (shared latent) the value matrix
        const bf16_t* wlift = wv ? wv + (size_t)g * DD * D : wug;
        // (all of this thread's elements requested at once, no load under a
        // branch: the cache stream below is not held up by them)
        constexpr int UPT = (DD * D + NW * 64 - 1) / (NW * 64);
        bf16_t uv[UPT];
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int idx = imin(tid + j * NW * 64, DD * D - 1);
            const int c = idx / D, e = idx - (idx / D) * D;
            uv[j] = *(wlift ? wlift + (size_t)c * D + e : wdg + (size_t)e * DD + c);
        }
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int idx = tid + j * NW * 64;
            if (idx < DD * D) wsh[idx / D][idx - (idx / D) * D] = bf16_to_f32(uv[j]);
        }
    }
    // (computed after the W_up loads are issued: earlier costs registers)
    const WaveRun run = decode_wave_run_range(len, w, D, DD, ls0, ls1, ws0, ws1, nwave, widx);
    const bool latent = run.latent != 0;
    const int t_begin = run.t_begin, t_end = run.t_end;  // this wavefront's tokens
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
    // with rotation: the query rotated at len - 1 (fp32 until packed); qopr is
    // its scaled operand in the element order of the lifted keys' registers
    dh16x8 qopr[R > 0 ? KL : 1];
    if constexpr (R == 0) {
#pragma unroll
        for (int k = 0; k < KS; ++k) qop[k] = hval ? ld8(qrow + k * 16 + hg * 8) : zero8();
    } else {
        float qf[KS][8];
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            const uint4 u = hval ? *reinterpret_cast<const uint4*>(qrow + k * 16 + hg * 8) : make_uint4(0, 0, 0, 0);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                qf[k][2 * j] = __uint_as_float(w4[j] << 16);
                qf[k][2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
            }
        }
        rotate_slabs<KS, R>(qf, tab + (size_t)(len - 1) * R, hg);
#pragma unroll
        for (int k = 0; k < KS; ++k) qop[k] = pk8(qf[k]);
#pragma unroll
        for (int k = 0; k < KL; ++k) {
            // element order 16k + (j < 4 ? 4hg + j : 8 + 4hg + j - 4): swap
            // the middle quads across the lane halves
            float v8[8];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(qf[k][j]), __float_as_uint(qf[k][4 + j]), false, false);
                v8[j] = __uint_as_float(r[0]) * qscale;
                v8[4 + j] = __uint_as_float(r[1]) * qscale;
            }
            qopr[k] = h8(h2(v8[0], v8[1]), h2(v8[2], v8[3]), h2(v8[4], v8[5]), h2(v8[6], v8[7]));
        }
    }

    DecState st{-INFINITY, 0.f, -INFINITY, 0.f, zero8()};
    const int quad = lane >> 4, sl = lane & 15;
    const int prow = dperm(col);

    if (t_begin < t_end && latent) {
        df32x16 acc[1] = {fill16(0.f)};  // O_lat^T (rows < d_down; row 16 = row sum when d_down = 16)
        // Latent rows through buffer loads whose size ends at the run's last
        // token: rows at or past t_end read as zeros, so the prefetches past
        // the run need no clamping and stay inside this head's latents.
        const bf16_t* kl = k_lat + (size_t)bg * cap * DD;
        const bf16_t* vl = v_lat + (size_t)bg * cap * DD;
        const int last = t_end - 1;
        // the descriptors are wave-uniform: keep them in scalar registers
        const int nbytes = __builtin_amdgcn_readfirstlane(t_end * DD * 2);
        const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(kl), (short)0, nbytes, kBufWord3);
        const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(vl), (short)0, nbytes, kBufWord3);
        const int koff = (t_begin + prow) * DD * 2 + hg * 16;  // A-operand row of subtile 0
        const int voff = t_begin * DD * 2 + lane * 16;         // 16-byte chunk of subtile 0
        constexpr int kSubBytes = 32 * DD * 2;
        // A operand of the rank-1 reference product: 1 at contraction slot 0
        const dbf16x8 ones_a = __builtin_bit_cast(dbf16x8, make_uint4(hg == 0 ? 0x3f80u : 0u, 0u, 0u, 0u));
        // paged: this sequence's row of the block table (the index of a
        // subtile's block is wave-uniform: a scalar load, kept apart from the
        // vector loads in flight)
        const int* btb = PAGED ? block_table + (size_t)b * pg.maxb : nullptr;
        auto load = [&](int t0, dbf16x8 (&ak)[DS], uint4 (&vv)[DS]) {
            if constexpr (PAGED) {
                // this subtile's page: rows past the run (or of an unmapped
                // page) are outside the descriptor's size and read as zeros
                const int blk = imin(t0 >> pg.ps_shift, pg.maxb - 1);
                const int page = scalar_load(btb + blk);
                const int pstart = blk * pg.ps;
                const bool ok = t0 < t_end && page >= 0 && page < pg.n_pages;
                const int nrow = ok ? imin(pg.ps, t_end - pstart) : 0;
                const size_t poff = ((size_t)(ok ? page : 0) * Hkv + g) * pg.ps * DD;
                const int nb = __builtin_amdgcn_readfirstlane(nrow * DD * 2);
                const __amdgpu_buffer_rsrc_t rkp = __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(k_lat + poff), (short)0, nb, kBufWord3);
                const __amdgpu_buffer_rsrc_t rvp = __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(v_lat + poff), (short)0, nb, kBufWord3);
                const int r0 = t0 - pstart;
#pragma unroll
                for (int k = 0; k < DS; ++k)
                    ak[k] = __builtin_bit_cast(dbf16x8, __builtin_amdgcn_raw_buffer_load_b128(rkp, (r0 + prow) * DD * 2 + hg * 16 + k * 32, 0, kStream));
#pragma unroll
                for (int k = 0; k < DS; ++k)
                    vv[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rvp, r0 * DD * 2 + lane * 16 + k * 1024, 0, kStream));
            } else {
                const int o = (t0 - t_begin) * DD * 2;
#pragma unroll
                for (int k = 0; k < DS; ++k)
                    ak[k] = __builtin_bit_cast(dbf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, koff + o + k * 32, 0, kStream));
                if constexpr (!SHARED) {
#pragma unroll
                    for (int k = 0; k < DS; ++k)
                        vv[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, voff + o + k * 1024, 0, kStream));
                }
            }
        };
        static_assert(kSubBytes == 1024 * DS, "one V chunk of 16 bytes per lane per 16 latent columns");
        // NST subtiles in flight per wavefront (the stream is latency bound:
        // the depth, not the arithmetic, sets its rate), issued before the
        // query absorption below so that its latency overlaps theirs
        constexpr int NST = DecStages<D, DD, R>::value;
        dbf16x8 aks[NST][DS];
        uint4 vs[NST][DS];
#pragma unroll
        for (int j = 0; j < NST; ++j) load(t_begin + 32 * j, aks[j], vs[j]);

        // ---- q~^T = W_up q^T, scaled; rearranged from the accumulator layout
        // (lane half g holds columns 4g..4g+3, 8+4g..8+4g+3 of each 16) to the
        // B-operand layout (half g holds 8g..8g+7) with one swap across halves.
        // (With rotation only slabs QK0.. not touched by it: the keys are lifted
        // instead for the rotated ones.)
        const bf16_t* wdg = wd + (size_t)g * D * DD;
        const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
        df32x16 qt = fill16(0.f);
#pragma unroll
        for (int k = QK0; k < KS; ++k) {
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

        // rotation: W_up^T rows (A operand of the lift; contraction slot
        // 8 hg + j = latent column 16 s2 + 8 hg + j) and the lane's offset
        // angles (token prow of the subtile) for its rotated pairs
        constexpr int NP = R / 4;  // rotated pairs per lane
        dbf16x8 aU[R > 0 ? NL : 1][R > 0 ? DS : 1];
        dh2 co[NP > 1 ? NP / 2 : 1], so[NP > 1 ? NP / 2 : 1];  // fp16 pairs of elements i, i + 1
        if constexpr (R > 0) {
#pragma unroll
            for (int t = 0; t < NL; ++t)
#pragma unroll
                for (int s2 = 0; s2 < DS; ++s2) {
                    uint16_t e8[8];
                    const int e = 32 * t + col;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int c = 16 * s2 + 8 * hg + j;
                        e8[j] = wug ? wug[(size_t)c * D + e] : wdg[(size_t)e * DD + c];
                    }
                    aU[t][s2] = __builtin_bit_cast(dbf16x8, e8);
                }
            // (an offset row past the table belongs to a token past the run: masked)
            const float* orow = tab + (size_t)imin(prow, n_pos - 1) * R;
#pragma unroll
            for (int f = 0; f < R / 16; ++f) {
                const float4 c4 = *reinterpret_cast<const float4*>(orow + 8 * f + 4 * hg);
                const float4 s4 = *reinterpret_cast<const float4*>(orow + R / 2 + 8 * f + 4 * hg);
                co[2 * f] = h2(c4.x, c4.y); co[2 * f + 1] = h2(c4.z, c4.w);
                so[2 * f] = h2(s4.x, s4.y); so[2 * f + 1] = h2(s4.z, s4.w);
            }
        }

        // Software pipelined: the scores of subtile n+1 are on the matrix
        // cores while the exponentials of subtile n run.
        auto scores = [&](int t0, const dbf16x8 (&ak)[DS]) {
            df32x16 x;
            if constexpr (R == 0) {
                x = mma(ak[0], qtop[0], mma(ones_a, st.negm, fill16(0.f)));
#pragma unroll
                for (int k = 1; k < DS; ++k) x = mma(ak[k], qtop[k], x);
            } else {
                // K'^T tiles: lane = token prow, register 4 mm + i of tile t =
                // element 32 t + 8 mm + 4 hg + i
                df32x16 kx[NL];
#pragma unroll
                for (int t = 0; t < NL; ++t) {
                    kx[t] = mma(aU[t][0], ak[0], fill16(0.f));
#pragma unroll
                    for (int s2 = 1; s2 < DS; ++s2) kx[t] = mma(aU[t][s2], ak[s2], kx[t]);
                }
                // the lifted keys as fp16 pairs (registers 2 p, 2 p + 1 of a tile)
                dh2 kh[NL][8];
#pragma unroll
                for (int t = 0; t < NL; ++t)
#pragma unroll
                    for (int p2 = 0; p2 < 8; ++p2) kh[t][p2] = h2(kx[t][2 * p2], kx[t][2 * p2 + 1]);
                // the subtile's base angles (row t0; t0 <= last < n_pos)
                const float* brow = tab + (size_t)t0 * R;
#pragma unroll
                for (int f = 0; f < R / 16; ++f) {
                    const float4 c4 = *reinterpret_cast<const float4*>(brow + 8 * f + 4 * hg);
                    const float4 s4 = *reinterpret_cast<const float4*>(brow + R / 2 + 8 * f + 4 * hg);
                    const dh2 cb[2] = {h2(c4.x, c4.y), h2(c4.z, c4.w)}, sb[2] = {h2(s4.x, s4.y), h2(s4.z, s4.w)};
                    constexpr int q8 = R / 16;  // partner: 8 q8 elements on
#pragma unroll
                    for (int i2 = 0; i2 < 2; ++i2) {  // elements 2 i2, 2 i2 + 1 of the group
                        const dh2 c = cb[i2] * co[2 * f + i2] - sb[i2] * so[2 * f + i2];
                        const dh2 sn = sb[i2] * co[2 * f + i2] + cb[i2] * so[2 * f + i2];
                        const int F2 = f + q8;
                        const dh2 av = kh[f / 4][2 * (f % 4) + i2], bv = kh[F2 / 4][2 * (F2 % 4) + i2];
                        kh[f / 4][2 * (f % 4) + i2] = av * c - bv * sn;
                        kh[F2 / 4][2 * (F2 % 4) + i2] = bv * c + av * sn;
                    }
                }
                x = mma(ones_a, st.negm, fill16(0.f));
#pragma unroll
                for (int k = 0; k < KL; ++k) {
                    const int t = k / 2, p0 = 4 * (k % 2);
                    x = mmah(h8(kh[t][p0], kh[t][p0 + 1], kh[t][p0 + 2], kh[t][p0 + 3]), qopr[k], x);
                }
                if constexpr (D > 64) {  // the unrotated half, absorbed
#pragma unroll
                    for (int k = 0; k < DS; ++k) x = mma(ak[k], qtop[k], x);
                }
            }
            if (t0 + 31 > last) {
                keep_branch();
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (t0 + dkey(r, hg) > last) x[r] = -INFINITY;
            }
            return x;
        };
        auto finish = [&](int t0, df32x16& x, const dbf16x8 (&ak)[DS], const uint4 (&vv)[DS],
                          df32x16* xnext) {
            const bf16_t* vbs = vb;
            if constexpr (SHARED) {
                // the key operand as loaded holds token prow's latent row:
                // stored at that row it is the value tile
#pragma unroll
                for (int k = 0; k < DS; ++k)
                    *reinterpret_cast<dbf16x8*>(vb + prow * DD + k * 16 + hg * 8) = ak[k];
            } else {
#pragma unroll
                for (int k = 0; k < DS; ++k) *reinterpret_cast<uint4*>(vb + (lane + 64 * k) * 8) = vv[k];
            }
            dbf16x8 p0, p1;
            dstep<1, DD != 16>(x, st, acc, p0, p1, hg, xnext);
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
                    plo = vbs + key * DD + c;
                    phi = vbs + (key + 4) * DD + c;
                }
                const ds16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)plo);
                const ds16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ds16x4*)phi);
                const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
                const dbf16x8 a = __builtin_bit_cast(dbf16x8, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
                acc[0] = mma(a, half ? p1 : p0, acc[0]);
            }
        };
        int t0 = t_begin;
        df32x16 x = scores(t_begin, aks[0]);
        for (; t0 + 32 * (NST - 1) < t_end; t0 += 32 * NST) {
#pragma unroll
            for (int j = 0; j < NST; ++j) {
                const int tj = t0 + 32 * j;
                df32x16 xn = scores(tj + 32, aks[(j + 1) % NST]);
                finish(tj, x, aks[j], vs[j], &xn);
                load(tj + 32 * NST, aks[j], vs[j]);
                x = xn;
            }
        }
#pragma unroll
        for (int j = 0; j < NST - 1; ++j) {
            const int tj = t0 + 32 * j;
            if (tj < t_end) {
                if (tj + 32 < t_end) {
                    df32x16 xn = scores(tj + 32, aks[j + 1]);
                    finish(tj, x, aks[j], vs[j], &xn);
                    x = xn;
                } else {
                    finish(tj, x, aks[j], vs[j], nullptr);
                }
            }
        }
        if (DD == 16) st.l = acc[0][8];  // ones row: full row sum on both halves
        else st.l = psum(st.l);
        if (col < G) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = 8 * (r >> 2) + 4 * hg + (r & 3);
                if (row < DD) red_o[wave][col][row] = acc[0][r];
            }
        }
    } else if (t_begin < t_end) {
        df32x16 acc[NT];  // O_win^T
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = fill16(0.f);
        // ---- window region: full-d keys and values from the ring
        const bf16_t* kw = k_win + (size_t)bg * w * D;
        const bf16_t* vw = v_win + (size_t)bg * w * D;
        const int last = t_end - 1;
        constexpr int CPT = 32 * D / 8 / 64;  // 16-byte chunks per lane per subtile
        auto load = [&](int t0, dbf16x8 (&ak)[KS], uint4 (&vv)[CPT]) {
            const int kpos = imin(t0 + prow, last);
            const int kr = kpos % w;
#pragma unroll
            for (int k = 0; k < KS; ++k) ak[k] = __builtin_bit_cast(dbf16x8, ld_stream(kw + (size_t)kr * D + k * 16 + hg * 8));
            if constexpr (R > 0) {  // the key rotated at its position
                float kf[KS][8];
#pragma unroll
                for (int k = 0; k < KS; ++k) {
                    const uint4 u = __builtin_bit_cast(uint4, ak[k]);
                    const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        kf[k][2 * j] = __uint_as_float(w4[j] << 16);
                        kf[k][2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
                    }
                }
                rotate_slabs<KS, R>(kf, tab + (size_t)kpos * R, hg);
#pragma unroll
                for (int k = 0; k < KS; ++k) ak[k] = pk8(kf[k]);
            }
#pragma unroll
            for (int k = 0; k < CPT; ++k) {
                const int chunk = lane + 64 * k;
                const int tr = imin(t0 + chunk / (D / 8), last) % w;
                vv[k] = __builtin_bit_cast(uint4, ld_stream(vw + (size_t)tr * D + (chunk % (D / 8)) * 8));
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
                keep_branch();
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (t0 + dkey(r, hg) > last) x[r] = -INFINITY;
            }
            dbf16x8 p0, p1;
            dstep<NT, true>(x, st, acc, p0, p1, hg);
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
        // NSW subtiles in flight (positions past the run are clamped to its
        // last token, so the prefetches need no branch)
        constexpr int NSW = D > 64 ? 1 : (R > 0 ? 2 : 3);
        dbf16x8 akw[NSW][KS];
        uint4 vw4[NSW][CPT];
#pragma unroll
        for (int j = 0; j < NSW; ++j) load(t_begin + 32 * j, akw[j], vw4[j]);
        int t0 = t_begin;
        for (; t0 + 32 * (NSW - 1) < t_end; t0 += 32 * NSW) {
#pragma unroll
            for (int j = 0; j < NSW; ++j) {
                body(t0 + 32 * j, akw[j], vw4[j]);
                load(t0 + 32 * (j + NSW), akw[j], vw4[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < NSW - 1; ++j)
            if (t0 + 32 * j < t_end) body(t0 + 32 * j, akw[j], vw4[j]);
        st.l = psum(st.l);
        if (col < G) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) red_o[wave][col][t * 32 + 8 * (r >> 2) + 4 * hg + (r & 3)] = acc[t][r];
        }
    }

    // ---- merge the wavefronts of this workgroup and write the partials
    // {m, l, acc_lat[DD], acc_win[D]}; each wavefront contributes to the part
    // of its region (an empty run has m = -inf and contributes nothing)
    if (col < G && hg == 0) {
        red_m[wave][col] = st.m;
        red_l[wave][col] = st.l;
    }
    if (lane == 0) red_lat[wave] = latent ? 1 : 0;
    __syncthreads();
    for (int idx = tid; idx < G * stride; idx += NW * 64) {
        const int h = idx / stride, f = idx - (idx / stride) * stride;
        float M = -INFINITY;
#pragma unroll
        for (int v = 0; v < NW; ++v) M = fmaxf(M, red_m[v][h]);
        float val = 0.f;
        if (f == 0) {
            val = M;
        } else {
            const int want_lat = f < 2 + DD ? 1 : 0;
            const int row = f < 2 + DD ? f - 2 : f - 2 - DD;
#pragma unroll
            for (int v = 0; v < NW; ++v) {
                const float mv = red_m[v][h];
                if (mv != -INFINITY && (f == 1 || red_lat[v] == want_lat)) {
                    const float wgt = exp2f(mv - M);
                    val += wgt * (f == 1 ? red_l[v][h] : red_o[v][h][row]);
                }
            }
        }
        if (fuse) {
            mrg[h][f] = val;
        } else {
            const size_t bh = (size_t)b * Hq + (size_t)g * G + h;
            part[(bh * P + srec) * stride + f] = val;
        }
    }
    if (!fuse) return;
    // o = (acc_win + acc_lat W_up) / l (Eq. 2 lift applied once, Eq. 4 normalisation)
    __syncthreads();
    for (int idx = tid; idx < G * D; idx += NW * 64) {
        const int h = idx / D, e = idx - (idx / D) * D;
        float acc = mrg[h][2 + DD + e];
#pragma unroll
        for (int c = 0; c < DD; ++c) acc = __builtin_fmaf(mrg[h][2 + c], wsh[c][e], acc);
        o[((size_t)b * Hq + (size_t)g * G + h) * D + e] = f32_to_bf16(acc / mrg[h][1]);
    }
    };  // piece

    const int tid = lane_id_x();
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    if constexpr (!PAGED) {
        // P workgroups per (sequence, KV head): this one is part s
        const int s = wg_id_x(), bg = wg_id_y();
        const int b = bg / Hkv_, g = bg - (bg / Hkv_) * Hkv_;
        const int n_lat = imax(len_arg - w_, 0);
        piece(b, g, len_arg, P_ == 1, s, 0, (n_lat + 31) / 32, 0, (len_arg - n_lat + 31) / 32, P_ * NW,
              s * NW + wave);
    } else {
        // ---- this workgroup's job (every workgroup derives the same plan
        // from the lengths). Block-wide sums and exclusive prefixes:
        __shared__ long red[NW];
        __shared__ int job[3];  // sequence, KV head, part
        auto block_scan = [&](long v, long& excl, long& tot) {
            long inc = v;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const long t = __shfl_up(inc, off, 64);
                if (lane >= off) inc += t;
            }
            if (lane == 63) red[wave] = inc;
            __syncthreads();
            long before = 0;
            tot = 0;
#pragma unroll
            for (int v2 = 0; v2 < NW; ++v2) {
                const long t = red[v2];
                tot += t;
                if (v2 < wave) before += t;
            }
            excl = before + inc - v;
            __syncthreads();  // red is reused
        };
        const int B = pg_.nseq;
        const int per = (B + NW * 64 - 1) / (NW * 64);
        const int b0 = tid * per;  // this thread's sequences: [b0, b0 + per)
        // units of this thread's sequences (the first kKeep kept in registers)
        constexpr int kKeep = 2;
        long uk[kKeep];
        auto units_of = [&](int i) -> long {
            if (i < kKeep) {
                long u = 0;
#pragma unroll
                for (int t = 0; t < kKeep; ++t) u = t == i ? uk[t] : u;
                return u;
            }
            return b0 + i < B ? paged_units(pg_.lens[b0 + i], w_, cap_, D, DD) : 0;
        };
#pragma unroll
        for (int t = 0; t < kKeep; ++t)
            uk[t] = t < per && b0 + t < B ? paged_units(pg_.lens[b0 + t], w_, cap_, D, DD) : 0;
        long myU = 0, myLive = 0;
        for (int i = 0; i < per; ++i) {
            const long u = units_of(i);
            myU += u;
            myLive += u > 0;
        }
        long ex, totU, totLive;
        block_scan(myU, ex, totU);
        block_scan(myLive, ex, totLive);
        const long liveBefore = ex;
        const long cu = paged_part(totU * Hkv_, cap_, w_, D, DD);
        auto nparts = [&](long u) { return (u + cu - 1) / cu; };
        long myFull = 0;  // full parts (all but the last) of this thread's pairs
        for (int i = 0; i < per; ++i) {
            const long u = units_of(i);
            if (u > 0) myFull += (nparts(u) - 1) * Hkv_;
        }
        long fullBefore, F;
        block_scan(myFull, fullBefore, F);
        const long i0 = wg_id_x();
        if (i0 >= F + totLive * Hkv_) return;  // no job (uniform)
        if (i0 < F) {
            // a full part: the thread whose pairs hold full part i0
            long pos = fullBefore;
            for (int i = 0; i < per; ++i) {
                const long u = units_of(i);
                const long nf = u > 0 ? nparts(u) - 1 : 0;  // full parts per pair
                if (nf > 0 && pos <= i0 && i0 < pos + nf * Hkv_) {
                    job[0] = b0 + i;
                    job[1] = (int)((i0 - pos) / nf);
                    job[2] = (int)((i0 - pos) % nf);
                }
                pos += nf * Hkv_;
            }
        } else {
            // a last part: the sequence of rank (i0 - F) / Hkv among the live
            // ones, ranked by remainder (largest first, then batch order)
            const long j = i0 - F, target = j / Hkv_;
            __shared__ int rem[kPagedRankMax];
            if (B <= kPagedRankMax) {
                // (per == 1 here)
                long u = 0, r = -1;
                if (tid < B) {
                    u = uk[0];
                    r = u > 0 ? u - (nparts(u) - 1) * cu : -1;
                    rem[tid] = (int)r;
                }
                __syncthreads();
                if (tid < B && r >= 0) {
                    int rank = 0;
                    for (int b2 = 0; b2 < B; ++b2) {
                        const int r2 = rem[b2];
                        rank += (r2 > r || (r2 == r && b2 < tid)) ? 1 : 0;
                    }
                    if (rank == target) {
                        job[0] = tid;
                        job[1] = (int)(j % Hkv_);
                        job[2] = (int)(nparts(u) - 1);
                    }
                }
            } else {
                long pos = liveBefore;
                for (int i = 0; i < per; ++i) {
                    const long u = units_of(i);
                    if (u > 0) {
                        if (pos == target) {
                            job[0] = b0 + i;
                            job[1] = (int)(j % Hkv_);
                            job[2] = (int)(nparts(u) - 1);
                        }
                        ++pos;
                    }
                }
            }
        }
        __syncthreads();
        const int b = __builtin_amdgcn_readfirstlane(job[0]);
        const int g = __builtin_amdgcn_readfirstlane(job[1]);
        const int p = __builtin_amdgcn_readfirstlane(job[2]);
        const int len = imin(imax(scalar_load(pg_.lens + b), 0), cap_);
        const long U = paged_units(len, w_, cap_, D, DD);
        const int n = (int)nparts(U);
        const long u0 = p * cu, u1 = u0 + cu < U ? u0 + cu : U;  // this part's units
        constexpr int RU = D / DD;
        const int n_lat = imax(len - w_, 0);
        const int nls = (n_lat + 31) / 32, nws = (len - n_lat + 31) / 32;
        const int ls0 = (int)(u0 < nls ? u0 : nls), ls1 = (int)(u1 < nls ? u1 : nls);
        const int ws0 = imin((int)(u0 > nls ? (u0 - nls + RU - 1) / RU : 0), nws);
        const int ws1 = imin((int)(u1 > nls ? (u1 - nls + RU - 1) / RU : 0), nws);
        if (p == 0 && tid == 0) pg_.counts[b * Hkv_ + g] = n;
        piece(b, g, len, n == 1, p, ls0, ls1, ws0, ws1, NW, wave);
    }
}

bool decode_mfma_supported(int d, int dd, int G, bool bf16) {
    return bf16 && (d == 64 || d == 128) && (dd == 16 || dd == 32) && G >= 1 && G <= kDecMaxGroup;
}

int decode_mfma_parts(int B, int Hkv, int len, int w, int d) {
    // about one round of resident workgroups on the 256 compute units of a
    // gfx950 part, one workgroup per unit. Fixed, so that the workspace size
    // is a pure function of the shape.
    const int nw = d <= 64 ? DecWaves<64>::value : DecWaves<128>::value;
    const long long pairs = (long long)B * Hkv;
    long long P = (256 + pairs - 1) / pairs;
    const int n_lat = len - w > 0 ? len - w : 0;
    const long long nsub = (n_lat + 31) / 32 + (len - n_lat + 31) / 32;
    const long long by_work = nsub / (nw * kDecMinSub);
    if (P > by_work) P = by_work;
    if (P < 1) P = 1;
    if (P > 1024) P = 1024;
    return (int)P;
}

hipError_t launch_decode_mfma(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                              const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_lat,
                              const bf16_t* v_lat, float* part, bf16_t* o, int B, int Hq, int Hkv,
                              int d, int dd, int w, int cap, int len, int& P, hipStream_t st,
                              const bf16_t* wv) {
    P = decode_mfma_parts(B, Hkv, len, w, d);
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    dim3 grid(P, B * Hkv);
    if (k_lat == v_lat) {  // one shared latent array: each subtile loaded once
#define DAR_DEC_SHARED(D_, DD_)                                                                     \
    hipLaunchKernelGGL((decode_mfma_kernel<D_, DD_, DecWaves<D_>::value, 0, false, true>), grid,    \
                       dim3(64 * DecWaves<D_>::value), 0, st, q, wd, wu, k_win, v_win, k_lat, v_lat, \
                       part, o, Hq, Hkv, w, cap, len, P, qscale, (const float*)nullptr, 0, wv, PagedArgs{}, \
                       (const int*)nullptr)
        if (d == 64 && dd == 16) DAR_DEC_SHARED(64, 16);
        else if (d == 64 && dd == 32) DAR_DEC_SHARED(64, 32);
        else if (d == 128 && dd == 16) DAR_DEC_SHARED(128, 16);
        else DAR_DEC_SHARED(128, 32);
#undef DAR_DEC_SHARED
        return hipGetLastError();
    }
#define DAR_DEC_LAUNCH(D_, DD_)                                                                     \
    hipLaunchKernelGGL((decode_mfma_kernel<D_, DD_, DecWaves<D_>::value>), grid,                    \
                       dim3(64 * DecWaves<D_>::value), 0, st, q, wd, wu, k_win, v_win, k_lat, v_lat, \
                       part, o, Hq, Hkv, w, cap, len, P, qscale, (const float*)nullptr, 0, wv, PagedArgs{}, \
                       (const int*)nullptr)
    if (d == 64 && dd == 16) DAR_DEC_LAUNCH(64, 16);
    else if (d == 64 && dd == 32) DAR_DEC_LAUNCH(64, 32);
    else if (d == 128 && dd == 16) DAR_DEC_LAUNCH(128, 16);
    else DAR_DEC_LAUNCH(128, 32);
#undef DAR_DEC_LAUNCH
    return hipGetLastError();
}

bool decode_mfma_rope_supported(int d, int dd, int G, int r, bool bf16) {
    return bf16 && (d == 64 || d == 128) && (dd == 16 || dd == 32) && G >= 1 && G <= kDecMaxGroup &&
           (r == 16 || r == 32 || r == 64);
}

hipError_t launch_decode_mfma_rope(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                                   const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_lat,
                                   const bf16_t* v_lat, const float* tab, int n_pos, float* part,
                                   bf16_t* o, int B, int Hq, int Hkv, int dd, int w, int cap,
                                   int len, int r, int& P, hipStream_t st, int d) {
    P = decode_mfma_parts(B, Hkv, len, w, d);
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    dim3 grid(P, B * Hkv);
#define DAR_DEC_ROPE(D_, DD_, R_)                                                                    \
    hipLaunchKernelGGL((decode_mfma_kernel<D_, DD_, DecWaves<D_>::value, R_>), grid,                 \
                       dim3(64 * DecWaves<D_>::value), 0, st, q, wd, wu, k_win, v_win, k_lat, v_lat, \
                       part, o, Hq, Hkv, w, cap, len, P, qscale, tab, n_pos, (const bf16_t*)nullptr, PagedArgs{}, \
                       (const int*)nullptr)
#define DAR_DEC_ROPE_D(D_)                                    \
    if (dd == 16) {                                           \
        if (r == 16) DAR_DEC_ROPE(D_, 16, 16);                \
        else if (r == 32) DAR_DEC_ROPE(D_, 16, 32);           \
        else DAR_DEC_ROPE(D_, 16, 64);                        \
    } else {                                                  \
        if (r == 16) DAR_DEC_ROPE(D_, 32, 16);                \
        else if (r == 32) DAR_DEC_ROPE(D_, 32, 32);           \
        else DAR_DEC_ROPE(D_, 32, 64);                        \
    }
    if (d == 64) {
        DAR_DEC_ROPE_D(64)
    } else {
        DAR_DEC_ROPE_D(128)
    }
#undef DAR_DEC_ROPE_D
#undef DAR_DEC_ROPE
    return hipGetLastError();
}

int decode_paged_slots(int Hkv, int cap, int w, int d, int dd) {
    // cu >= ceil(U(cap) / kPagedMaxParts): a pair has at most that many parts
    (void)Hkv; (void)cap; (void)w; (void)d; (void)dd;
    return kPagedMaxParts;
}

hipError_t launch_decode_mfma_paged(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                                    const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_pool,
                                    const bf16_t* v_pool, const PagedArgs& pg_in, float* part,
                                    bf16_t* o, int B, int Hq, int Hkv, int d, int dd, int w, int& P,
                                    int*& counts, hipStream_t st, const float* tab, int n_pos, int r) {
    const int cap = pg_in.maxb * pg_in.ps;
    P = decode_paged_slots(Hkv, cap, w, d, dd);
    counts = reinterpret_cast<int*>(part + (size_t)B * Hq * P * (2 + dd + d));
    PagedArgs pg = pg_in;
    pg.nseq = B;
    pg.counts = counts;
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    // jobs: at most kPagedGroups full parts (cu >= total / kPagedGroups) and
    // one last part per pair
    dim3 grid(kPagedGroups + B * Hkv);
#define DAR_DEC_PAGED(D_, DD_, R_)                                                                   \
    hipLaunchKernelGGL((decode_mfma_kernel<D_, DD_, DecWaves<D_>::value, R_, true>), grid,           \
                       dim3(64 * DecWaves<D_>::value), 0, st, q, wd, wu, k_win, v_win, k_pool, v_pool, \
                       part, o, Hq, Hkv, w, cap, 0, P, qscale, tab, n_pos,                            \
                       (const bf16_t*)nullptr, pg, pg.bt)
#define DAR_DEC_PAGED_R(D_, DD_)                          \
    if (r == 0) DAR_DEC_PAGED(D_, DD_, 0);                \
    else if (r == 16) DAR_DEC_PAGED(D_, DD_, 16);         \
    else if (r == 32) DAR_DEC_PAGED(D_, DD_, 32);         \
    else DAR_DEC_PAGED(D_, DD_, 64);
    if (d == 64 && dd == 16) { DAR_DEC_PAGED_R(64, 16) }
    else if (d == 64 && dd == 32) { DAR_DEC_PAGED_R(64, 32) }
    else if (d == 128 && dd == 16) { DAR_DEC_PAGED_R(128, 16) }
    else { DAR_DEC_PAGED_R(128, 32) }
#undef DAR_DEC_PAGED_R
#undef DAR_DEC_PAGED
    return hipGetLastError();
}

}  // namespace dar
