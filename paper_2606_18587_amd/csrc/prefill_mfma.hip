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

// Combine lane l with lane l ^ 32. After the swap one result holds the lane's
// own value and the other its partner's, in an order that depends on the
// half, so max and sum can use both without a select.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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

// p = exp2(x) for the 16 scores, packed to bf16 as the two P^T operands; with
// SUM_VALU the bf16-rounded p are also added to the row sum l.
template <bool SUM_VALU>
__device__ __forceinline__ void exp_pack(const f32x16_t& x, float& l, bf16x8_t& p0, bf16x8_t& p1) {
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(x[r]);
    p0 = pack8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
    p1 = pack8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    if (SUM_VALU) {
        const bf16x2_t one2 = {(__bf16)1.0f, (__bf16)1.0f};
        const uint4 u0 = __builtin_bit_cast(uint4, p0), u1 = __builtin_bit_cast(uint4, p1);
        float s = l;
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0.w), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.x), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.y), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.z), one2, s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1.w), one2, s, false);
        l = s;
    }
}

struct SoftmaxState {
    float m;       // reference (scaled log2 units); -inf until the row has seen a key
    float cm;      // -m, or 0 while m is -inf
    float thr;     // a subtile maximum above thr moves m: -inf until m is set, then kTau
    float l;       // partial row sum of this lane (bf16-rounded p)
    f32x16_t cmv;  // cm in every register: the accumulator input of distant S^T
};

// One 32-key subtile of the online softmax on x[16] (already relative to the
// reference). Returns P^T as two bf16x8 operands; rescales ow/ol if needed.
// OL: the latent accumulator ol is still separate (distant region); after
// it has been lifted into ow (window region) only ow is rescaled. OW: ow
// holds something to rescale (in the distant region, which runs before any
// window key, it is still zero).
template <int NT, bool SUM_VALU, bool OL = true, bool OW = true>
__device__ __forceinline__ void softmax_step(f32x16_t& x, SoftmaxState& st, f32x16_t (&ow)[NT],
                                             f32x16_t& ol, bf16x8_t& p0, bf16x8_t& p1,
                                             f32x16_t* xnext = nullptr) {
    float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), x[2]), fmaxf(x[3], x[4]));
    mx = fmaxf(fmaxf(mx, x[5]), fmaxf(x[6], x[7]));
    mx = fmaxf(fmaxf(mx, x[8]), fmaxf(x[9], x[10]));
    mx = fmaxf(fmaxf(mx, x[11]), fmaxf(x[12], x[13]));
    mx = fmaxf(fmaxf(mx, x[14]), x[15]);
    mx = pair_max(mx);
    const bool need = mx > st.thr;
    if (__builtin_amdgcn_ballot_w64(need)) {
        __asm__ volatile("");  // a real branch: never if-converted into every subtile
        const bool fresh = st.m == -INFINITY;
        const float delta = need ? mx : 0.f;
        const float fac = need ? (fresh ? 0.f : exp2f(-delta)) : 1.f;
        if (OW) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) ow[t][r] *= fac;
        }
        if (OL) {
#pragma unroll
            for (int r = 0; r < 16; ++r) ol[r] *= fac;
        }
        st.l *= fac;
        if (need) st.m = fresh ? mx : st.m + delta;
        st.cm = (st.m == -INFINITY) ? 0.f : -st.m;
        st.thr = (st.m == -INFINITY) ? -INFINITY : kTau;
        st.cmv = splat16(st.cm);
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] -= delta;
        if (xnext) {  // scores already computed against the old reference
#pragma unroll
            for (int r = 0; r < 16; ++r) (*xnext)[r] -= delta;
        }
    }
    exp_pack<SUM_VALU>(x, st.l, p0, p1);
}

// dot product of two 8-element bf16 operands (fp32 accumulation)
__device__ __forceinline__ float dot8(bf16x8_t a, bf16x8_t b, float acc) {
    const uint4 ua = __builtin_bit_cast(uint4, a), ub = __builtin_bit_cast(uint4, b);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.x), __builtin_bit_cast(bf16x2_t, ub.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.y), __builtin_bit_cast(bf16x2_t, ub.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.z), __builtin_bit_cast(bf16x2_t, ub.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, ua.w), __builtin_bit_cast(bf16x2_t, ub.w), acc, false);
    return acc;
}

// Everything a wavefront needs to walk one row block. Row indices are
// positions (r0, i, i_hi < T); key/value row t of k and v holds position
// kv0 + t (t < Tkv).
struct RowCtx {
    int T, w, Tp, r0, i, i_hi, qc, hg, prow, bg, tid, kv0, Tkv;
    int Td;  // with rotary embedding: rows of the lifted keys and values (T - w)
    float c_scale;
};

// The key range one call of the window-tile loop covers. LOCAL: the window,
// i - w < j <= i, from the token's own keys and values. DIST (rotary
// embedding only): the distant keys j <= i - w at full d, from the lifted
// and rotated keys and the lifted values (rows 0..Td-1).
template <bool DIST>
struct Region {
    static __device__ __forceinline__ int first_tile(int i0, int w, int bn) {
        return DIST ? 0 : (imax(0, i0 - w + 1) & ~(bn - 1));
    }
    static __device__ __forceinline__ int last_key(int iwg_hi, int w) { return DIST ? iwg_hi - w : iwg_hi; }
    // source row of key t (clamped: rows past the range are masked)
    static __device__ __forceinline__ int row(const RowCtx& c, int t) {
        return DIST ? imin(t, c.Td - 1) : imax(imin(t, c.T - 1) - c.kv0, 0);
    }
    static __device__ __forceinline__ size_t rows(const RowCtx& c) { return DIST ? c.Td : c.Tkv; }
    // some row of this wavefront has a key of the region in [js, js + 31]
    static __device__ __forceinline__ bool active(const RowCtx& c, int js) {
        return DIST ? (c.r0 < c.T && js <= c.i_hi - c.w)
                    : (c.r0 < c.T && js <= c.i_hi && js + 31 > c.r0 - c.w);
    }
    // every key of [js, js + 31] is in the region for every row
    static __device__ __forceinline__ bool full(const RowCtx& c, int js) {
        return DIST ? (js + 31 <= c.r0 - c.w) : (js > c.i_hi - c.w && js + 31 <= c.r0);
    }
    static __device__ __forceinline__ bool masked(const RowCtx& c, int j) {
        return DIST ? (j > c.i - c.w) : (j <= c.i - c.w || j > c.i);
    }
};

// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data
// format; with stride 0, lanes whose offset is past num_records read zero).
static constexpr int kBufWord3 = 0x00020000;

// A pointer every lane of the wavefront holds, moved to scalar registers.
__device__ __forceinline__ const bf16_t* uniform_ptr(const bf16_t* p) {
    const uint64_t u = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return (const bf16_t*)(((uint64_t)hi << 32) | lo);
}

// Kernel modes: the whole-sequence prefill; the rotary embedding (full-d
// distant keys from the pre-pass); a chunk whose distant latents are read in
// place from a dense or a paged cache (LatCache).
enum { kModePlain = 0, kModeRope = 1, kModeDense = 2, kModePaged = 3 };

// A load of a wavefront-uniform int through the scalar data cache.
__device__ __forceinline__ int sload(const int* p) {
    return *(const __attribute__((address_space(4))) int*)p;
}

// Buffer descriptor over the latent rows of positions [t0, t0 + 32) of one
// (batch, KV head) in a cache array (t0 a multiple of 32; a page holds at
// least 32 tokens, so the rows are contiguous): rows at or past Td (not
// latent yet), and all rows of an unmapped page, read as zeros.
template <int DD, bool PAGED>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t lat_rsrc(const LatCache& lc, const bf16_t* arr,
                                                           int b, int g, int bg, int Hkv, int t0,
                                                           int Td) {
    int rows = imax(imin(Td - t0, 32), 0);
    size_t row0;
    if constexpr (PAGED) {
        const int page = sload(lc.bt + (size_t)b * lc.maxb + imin(t0 >> lc.ps_shift, lc.maxb - 1));
        const bool ok = page >= 0 && page < lc.n_pages;
        if (!ok) rows = 0;
        row0 = ((((size_t)(ok ? page : 0)) * Hkv + g) << lc.ps_shift) + (t0 & ((1 << lc.ps_shift) - 1));
    } else {
        row0 = (size_t)bg * lc.cap + t0;
    }
    // (size and base moved to scalar registers: a descriptor in vector
    // registers would make every load a loop over its distinct values)
    return __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(arr + row0 * DD), (short)0,
                                             __builtin_amdgcn_readfirstlane(rows * DD * 2), kBufWord3);
}

// The latent key row of position t (nullptr when its page is not mapped).
template <int DD, bool PAGED>
__device__ __forceinline__ const bf16_t* lat_row(const LatCache& lc, int b, int g, int bg, int Hkv, int t) {
    if constexpr (PAGED) {
        const int page = lc.bt[(size_t)b * lc.maxb + (t >> lc.ps_shift)];
        if (page < 0 || page >= lc.n_pages) return nullptr;
        return lc.k + (((((size_t)page) * Hkv + g) << lc.ps_shift) + (t & ((1 << lc.ps_shift) - 1))) * DD;
    } else {
        return lc.k + ((size_t)bg * lc.cap + t) * DD;
    }
}

// Distant region: subtiles of 32 keys [0, js_last] against the latents of
// the pre-pass, software pipelined: the scores of subtile n+1 are on the
// matrix cores while the exponentials of subtile n run, so neither unit
// waits for the other. Latent keys are loaded three subtiles ahead, values
// three ahead of their use, through buffer loads whose subtile offset is a
// scalar (no per-subtile address arithmetic); lanes of the V^T operand past
// the stored rows read zeros (out-of-range offset), and with d_down = 16 the
// stored ones row makes O_lat^T row 16 the row sum.
// FIXED: the reference is final, every score is <= 0 relative to it: no
// maximum, no rescaling. Otherwise the online maximum is tracked.
template <int D, int DD, bool FIXED>
__device__ __forceinline__ void distant_region(const RowCtx& c, const bf16_t* __restrict__ cK,
                                               const bf16_t* __restrict__ cVt,
                                               const bf16x8_t (&qtop)[DD / 16], int js_last,
                                               SoftmaxState& st, f32x16_t (&ow)[D / 32],
                                               f32x16_t& ol) {
    constexpr int DS = DD / 16, NT = D / 32;
    constexpr int RB = DD == 16 ? 17 : DD;  // stored rows per 32-token block of c^V^T
    const int n_sub = (js_last >> 5) + 1;
    const int max_sub = (c.Tp >> 5) - 1;    // last subtile with storage
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        (void*)uniform_ptr(cK + (size_t)c.bg * c.Tp * DD), (short)0, c.Tp * DD * 2, kBufWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        (void*)uniform_ptr(cVt + (size_t)c.bg * (c.Tp / 32) * RB * 32), (short)0, (c.Tp / 32) * RB * 64,
        kBufWord3);
    const int koff = (c.prow * DD + c.hg * 8) * 2;
    const int voff = c.qc < RB ? (c.qc * 32 + c.hg * 8) * 2 : 0x40000000;  // past the end: zeros
    struct KT {
        bf16x8_t k[DS];
    };
    struct VT {
        bf16x8_t v[2];
    };
    auto loadK = [&](int sub) {
        const int so = __builtin_amdgcn_readfirstlane(imin(sub, max_sub) * 32 * DD * 2);
        KT r;
#pragma unroll
        for (int s = 0; s < DS; ++s)
            r.k[s] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rk, koff + s * 32, so, 0));
        return r;
    };
    auto loadV = [&](int sub) {
        const int so = __builtin_amdgcn_readfirstlane(imin(sub, max_sub) * RB * 64);
        VT r;
        r.v[0] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rv, voff, so, 0));
        r.v[1] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rv, voff + 32, so, 0));
        return r;
    };
    auto scores = [&](int sub, const KT& kt) {
        f32x16_t x = mfma(kt.k[0], qtop[0], st.cmv);
#pragma unroll
        for (int s = 1; s < DS; ++s) x = mfma(kt.k[s], qtop[s], x);
        return x;
    };
    // staircase subtile: keep j <= i - w
    auto mask = [&](f32x16_t& x, int sub) {
        const int js = sub * 32;
        if (js + 31 > c.r0 - c.w) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (js + acc_key(r, c.hg) > c.i - c.w) x[r] = -INFINITY;
        }
    };
    auto finish = [&](f32x16_t& x, const VT& vt, f32x16_t* xnext) {
        bf16x8_t p0, p1;
        if (FIXED) exp_pack<DD != 16>(x, st.l, p0, p1);
        else softmax_step<NT, DD != 16, true, false>(x, st, ow, ol, p0, p1, xnext);
        ol = mfma(vt.v[0], p0, ol);
        ol = mfma(vt.v[1], p1, ol);
    };
    // Subtiles [0, n_full) need no mask for any row of the wavefront; the
    // pipelined loop finishes only those, so it carries no lane-dependent
    // mask state (at the register limit such state was spilled, and its
    // reload before the loop made every iteration wait for nearly all of
    // the loads in flight). At most two staircase subtiles remain.
    const int n_full = imin(n_sub, imax(0, (c.r0 - c.w + 1) >> 5));
    KT ka = loadK(0), kb = loadK(1), kc = loadK(2);
    VT va = loadV(0), vb = loadV(1), vc = loadV(2);
    f32x16_t x = scores(0, ka);
    ka = loadK(3);
    int n = 0;
    // (scheduling fences keep each load where it is written: left free, the
    // scheduler sank all of an iteration's loads to its end, right before
    // the next iteration waits for them)
    for (; n + 2 < n_full; n += 3) {
        // x = scores of n; kb, kc, ka hold keys n+1..n+3; va, vb, vc values n..n+2
        f32x16_t xn = scores(n + 1, kb);
        kb = loadK(n + 4);
        __builtin_amdgcn_sched_barrier(0);
        finish(x, va, &xn);
        va = loadV(n + 3);
        __builtin_amdgcn_sched_barrier(0);
        x = xn;
        xn = scores(n + 2, kc);
        kc = loadK(n + 5);
        __builtin_amdgcn_sched_barrier(0);
        finish(x, vb, &xn);
        vb = loadV(n + 4);
        __builtin_amdgcn_sched_barrier(0);
        x = xn;
        xn = scores(n + 3, ka);
        ka = loadK(n + 6);
        __builtin_amdgcn_sched_barrier(0);
        finish(x, vc, &xn);
        vc = loadV(n + 5);
        __builtin_amdgcn_sched_barrier(0);
        x = xn;
    }
    // the rest, at most four subtiles, one at a time (keys n..n+3 and values
    // n..n+2 are in flight; x holds the scores of n)
    if (n < n_sub) {
        mask(x, n);
        finish(x, va, nullptr);
    }
    if (n + 1 < n_sub) {
        f32x16_t y = scores(n + 1, kb);
        mask(y, n + 1);
        finish(y, vb, nullptr);
    }
    if (n + 2 < n_sub) {
        f32x16_t y = scores(n + 2, kc);
        mask(y, n + 2);
        finish(y, vc, nullptr);
    }
    if (n + 3 < n_sub) {
        const VT vd = loadV(n + 3);
        f32x16_t y = scores(n + 3, ka);
        mask(y, n + 3);
        finish(y, vd, nullptr);
    }
}

// Distant region of a chunk, latents read in place from the cache: the
// schedule of distant_region (scores of subtile n+1 on the matrix cores while
// the exponentials of subtile n run; keys and values three subtiles ahead).
// The key latents are in natural column order, so qtop must be too. The
// value latents are token-major in the cache: each wavefront stores its
// subtile into its own LDS block (vst, 32 rows of DD) and reads the V^T
// operand from it with transposing reads; with d_down = 16 the operand rows
// 16..31 come from two constant chunks stored after the block, [1, 0, 0, 0]
// for the lanes that supply row 16 and zeros for the others, so O_lat^T row
// 16 is the row sum and rows 17..31 are zero, as with the pre-pass layout.
template <int D, int DD, bool FIXED, bool PAGED>
__device__ __forceinline__ void distant_region_cache(const RowCtx& c, const LatCache& lc, int b,
                                                     int g, int Hkv, bf16_t* vst,
                                                     const bf16x8_t (&qtop)[DD / 16], int js_last,
                                                     SoftmaxState& st, f32x16_t (&ow)[D / 32],
                                                     f32x16_t& ol) {
    constexpr int DS = DD / 16, NT = D / 32;
    const int n_sub = (js_last >> 5) + 1;
    const int lane = c.tid & 63;
    const int quad = lane >> 4, sl = lane & 15;
    const int koff = (c.prow * DD + c.hg * 8) * 2;
    const int voff = lane * 16;
    if (DD == 16 && lane < 8) vst[32 * DD + lane] = lane == 0 ? (bf16_t)0x3f80 : (bf16_t)0;
    struct KT {
        bf16x8_t k[DS];
    };
    struct VT {
        uint4 v[DS];  // bytes 16 lane + 1024 k of the subtile
    };
    auto loadK = [&](int sub) {
        const __amdgpu_buffer_rsrc_t rk = lat_rsrc<DD, PAGED>(lc, lc.k, b, g, c.bg, Hkv, sub * 32, c.Td);
        KT r;
#pragma unroll
        for (int s = 0; s < DS; ++s)
            r.k[s] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rk, koff + s * 32, 0, 0));
        return r;
    };
    auto loadV = [&](int sub) {
        const __amdgpu_buffer_rsrc_t rv = lat_rsrc<DD, PAGED>(lc, lc.v, b, g, c.bg, Hkv, sub * 32, c.Td);
        VT r;
#pragma unroll
        for (int k = 0; k < DS; ++k)
            r.v[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, voff + k * 1024, 0, 0));
        return r;
    };
    auto scores = [&](int sub, const KT& kt) {
        f32x16_t x = mfma(kt.k[0], qtop[0], st.cmv);
#pragma unroll
        for (int s = 1; s < DS; ++s) x = mfma(kt.k[s], qtop[s], x);
        const int js = sub * 32;
        if (js + 31 > c.r0 - c.w) {  // staircase subtile: keep j <= i - w
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (js + acc_key(r, c.hg) > c.i - c.w) x[r] = -INFINITY;
        }
        return x;
    };
    auto finish = [&](f32x16_t& x, const VT& vt, f32x16_t* xnext) {
        // the wavefront's own LDS block: its stores complete before its reads
#pragma unroll
        for (int k = 0; k < DS; ++k) *reinterpret_cast<uint4*>(vst + (lane + 64 * k) * 8) = vt.v[k];
        bf16x8_t p0, p1;
        if (FIXED) exp_pack<DD != 16>(x, st.l, p0, p1);
        else softmax_step<NT, DD != 16, true, false>(x, st, ow, ol, p0, p1, xnext);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int key = half * 16 + 8 * (quad >> 1) + (sl >> 2);
            const int cc = 16 * (quad & 1) + 4 * (sl & 3);
            // (a lane reads 4 columns of one row of a 4 x 16 block that the
            // transposing read hands out column by column: the lanes with
            // sl % 4 == 0 supply operand rows 16..19, of which only row 16 is
            // ones)
            const bool pad = DD == 16 && (quad & 1);
            const bf16_t* cst = vst + 32 * DD + ((sl & 3) ? 4 : 0);
            const bf16_t* plo = pad ? cst : vst + key * DD + cc;
            const bf16_t* phi = pad ? cst : vst + (key + 4) * DD + cc;
            const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)plo);
            const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)phi);
            const uint2 ulo = __builtin_bit_cast(uint2, lo), uhi = __builtin_bit_cast(uint2, hi);
            const bf16x8_t a = __builtin_bit_cast(bf16x8_t, make_uint4(ulo.x, ulo.y, uhi.x, uhi.y));
            ol = mfma(a, half ? p1 : p0, ol);
        }
    };
    KT ka = loadK(0), kb = loadK(1), kc = loadK(2);
    VT va = loadV(0), vb = loadV(1), vc = loadV(2);
    f32x16_t x = scores(0, ka);
    ka = loadK(3);
    int n = 0;
    for (; n + 2 < n_sub; n += 3) {
        f32x16_t xn = scores(n + 1, kb);
        kb = loadK(n + 4);
        finish(x, va, &xn);
        va = loadV(n + 3);
        x = xn;
        xn = scores(n + 2, kc);
        kc = loadK(n + 5);
        finish(x, vb, &xn);
        vb = loadV(n + 4);
        x = xn;
        xn = scores(n + 3, ka);
        ka = loadK(n + 6);
        finish(x, vc, &xn);
        vc = loadV(n + 5);
        x = xn;
    }
    if (n + 1 < n_sub) {
        f32x16_t xn = scores(n + 1, kb);
        finish(x, va, &xn);
        finish(xn, vb, nullptr);
    } else if (n < n_sub) {
        finish(x, va, nullptr);
    }
}

// Local region at d = 128 (where a register set for the next tile does not
// fit): 64-key K/V tiles loaded straight from global memory into LDS
// (global_load_lds, no registers), the next tile's loads in flight while
// the current one is computed on. One wavefront instruction fills 1 KB of
// LDS, lane l at byte 16 l: the padded tile (rows of d + 8 elements, 17
// chunks of 16 bytes) is 17 such instructions per array, and a lane whose
// chunk is a row's pad loads a chunk of that row again (never read). The
// query operand is the unscaled bf16 query (scaling it in bf16 would add a
// rounding proportional to the score); one FMA per score applies
// log2(e)/sqrt(d) and the reference.
template <int D, int DD, int NW, bool FIXED, bool DIST = false>
__device__ __forceinline__ void local_region_1deep(const RowCtx& c, const bf16_t* __restrict__ k,
                                             const bf16_t* __restrict__ v, bf16_t* lds_k,
                                             bf16_t* lds_v, const bf16x8_t (&qop)[D / 16],
                                             int i0, int iwg_hi, SoftmaxState& st,
                                             f32x16_t (&ow)[D / 32], f32x16_t& ol) {
    constexpr int KS = D / 16, NT = D / 32, BN = 64, LDK = D + 8;
    constexpr int RC = LDK / 8;                 // 16-byte chunks per padded row
    constexpr int NI = BN * RC / 64;            // 1 KB instructions per array and tile
    static_assert(LDK % 8 == 0 && BN * RC % 64 == 0, "whole chunks, whole instructions");
    using R = Region<DIST>;
    const int w = c.w;
    const int t_first = R::first_tile(i0, w, BN);
    const int ntile = (R::last_key(iwg_hi, w) - t_first) / BN + 1;
    const bf16_t* kb = k + (size_t)c.bg * R::rows(c) * D;
    const bf16_t* vb = v + (size_t)c.bg * R::rows(c) * D;
    const int lane = c.tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(c.tid >> 6);
    // stage the tile of keys t0..t0+63 into buffer `buf`: instructions m =
    // wave, wave + NW, ... (keys past the range repeat its last key and keys
    // below kv0 read row 0: their scores are masked)
    // (the lane index is made opaque here so that no address is hoisted out
    // of the tile loop: held across it, the addresses were spilled, and each
    // reload waited for every load in flight)
    // (its wave-uniform inputs are read into scalar registers there too)
    auto issue = [&](int buf, int t0) {
        typedef __attribute__((address_space(3))) void lds_void_t;
        int ln = lane;
        __asm__ volatile("" : "+v"(ln));
        const bf16_t* kbu = uniform_ptr(kb);
        const bf16_t* vbu = uniform_ptr(vb);
        const int last = __builtin_amdgcn_readfirstlane(DIST ? c.Td - 1 : c.T - 1);
        const int base = __builtin_amdgcn_readfirstlane(DIST ? 0 : c.kv0);
#pragma unroll
        for (int j = 0; j < (NI + NW - 1) / NW; ++j) {
            const int m = wave + NW * j;  // wave-uniform
            if (NI % NW != 0 && m >= NI) break;
            const int qc = m * 64 + ln;  // chunk of the padded tile
            const int r = qc / RC, cp = qc - (qc / RC) * RC;
            const int col = (cp < D / 8 ? cp : 0) * 8;  // the pad chunk loads column 0 again
            const int key = imax(imin(t0 + r, last) - base, 0);  // R::row
            __builtin_amdgcn_global_load_lds((const void*)(kbu + (size_t)key * D + col),
                                             (lds_void_t*)(lds_k + (size_t)buf * BN * LDK + m * 512), 16, 0, 0);
            __builtin_amdgcn_global_load_lds((const void*)(vbu + (size_t)key * D + col),
                                             (lds_void_t*)(lds_v + (size_t)buf * BN * LDK + m * 512), 16, 0, 0);
        }
    };
    // this wavefront's loads into LDS are complete (then a barrier for the
    // workgroup)
    auto drain = [] { __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
    issue(0, t_first);
    drain();
    __syncthreads();
    const int quad = lane >> 4, sl = lane & 15;
    for (int n = 0; n < ntile; ++n) {
        const int t0 = t_first + n * BN;
        const int buf = n & 1;
        // (the other buffer was last read before the barrier that ended the
        // previous tile)
        if (n + 1 < ntile) issue(buf ^ 1, t0 + BN);
        const bf16_t* lk = lds_k + (size_t)buf * BN * LDK;
        const bf16_t* lv = lds_v + (size_t)buf * BN * LDK;
#pragma unroll
        for (int sub = 0; sub < BN / 32; ++sub) {
            const int js = t0 + sub * 32;
            if (R::active(c, js)) {
                f32x16_t sc = mfma(load_bf16x8(lk + (sub * 32 + c.prow) * LDK + c.hg * 8), qop[0], splat16(0.f));
#pragma unroll
                for (int ks = 1; ks < KS; ++ks)
                    sc = mfma(load_bf16x8(lk + (sub * 32 + c.prow) * LDK + ks * 16 + c.hg * 8), qop[ks], sc);
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], c.c_scale, st.cm);
                if (!R::full(c, js)) {  // edge subtile: mask the keys outside the region
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (R::masked(c, js + acc_key(r, c.hg))) x[r] = -INFINITY;
                }
                bf16x8_t p0, p1;
                if (FIXED) exp_pack<true>(x, st.l, p0, p1);
                else softmax_step<NT, true, false>(x, st, ow, ol, p0, p1);
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
        drain();
        __syncthreads();
    }
}

// Local region: 64-key K/V tiles staged through LDS for the workgroup. The
// query operand is the unscaled bf16 query (scaling it in bf16 would add a
// rounding proportional to the score); one FMA per score applies
// log2(e)/sqrt(d) and the reference.
template <int D, int DD, int NW, bool FIXED, bool DIST = false>
__device__ __forceinline__ void local_region(const RowCtx& c, const bf16_t* __restrict__ k,
                                             const bf16_t* __restrict__ v, bf16_t* lds_k,
                                             bf16_t* lds_v, const bf16x8_t (&qop)[D / 16],
                                             int i0, int iwg_hi, SoftmaxState& st,
                                             f32x16_t (&ow)[D / 32], f32x16_t& ol) {
    constexpr int KS = D / 16, NT = D / 32, BN = 64, LDK = D + 8;
    constexpr int CH = BN * D / 8 / (NW * 64);
    using R = Region<DIST>;
    const int w = c.w;
    const int t_first = R::first_tile(i0, w, BN);
    const int ntile = (R::last_key(iwg_hi, w) - t_first) / BN + 1;
    const bf16_t* kb = k + (size_t)c.bg * R::rows(c) * D;
    const bf16_t* vb = v + (size_t)c.bg * R::rows(c) * D;
    // d = 64: two register sets; the loads of tile n+2 are issued when tile n
    // starts and reach LDS when tile n+1 ends, so two tiles of work cover
    // their latency.
    // (tiles travel by value: no array of them ever has its address taken,
    // so they stay in registers whatever the compiler does with the loop)
    struct Tile {
        uint4 k[CH], v[CH];
    };
    auto gload = [&](int t0) {
        Tile r;
#pragma unroll
        for (int q = 0; q < CH; ++q) {
            const int chunk = c.tid + q * NW * 64;
            const int row = chunk / (D / 8), col = (chunk % (D / 8)) * 8;
            // keys past the range repeat its last key: their scores are
            // masked and their weights are zero; keys below kv0 (the first
            // rows a tile start rounded down may cover) are never local and
            // read row 0
            const int key = R::row(c, t0 + row);
            r.k[q] = *reinterpret_cast<const uint4*>(kb + (size_t)key * D + col);
            r.v[q] = *reinterpret_cast<const uint4*>(vb + (size_t)key * D + col);
        }
        return r;
    };
    auto lstore = [&](int buf, const Tile& tl) {
#pragma unroll
        for (int q = 0; q < CH; ++q) {
            const int chunk = c.tid + q * NW * 64;
            const int row = chunk / (D / 8), col = (chunk % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(lds_k + (size_t)buf * BN * LDK + row * LDK + col) = tl.k[q];
            *reinterpret_cast<uint4*>(lds_v + (size_t)buf * BN * LDK + row * LDK + col) = tl.v[q];
        }
    };
    const int lane = c.tid & 63;
    const int quad = lane >> 4, sl = lane & 15;
    auto compute = [&](int buf, int t0) {
        const bf16_t* lk = lds_k + (size_t)buf * BN * LDK;
        const bf16_t* lv = lds_v + (size_t)buf * BN * LDK;
#pragma unroll
        for (int sub = 0; sub < BN / 32; ++sub) {
            const int js = t0 + sub * 32;
            if (R::active(c, js)) {
                f32x16_t sc = mfma(load_bf16x8(lk + (sub * 32 + c.prow) * LDK + c.hg * 8), qop[0], splat16(0.f));
#pragma unroll
                for (int ks = 1; ks < KS; ++ks)
                    sc = mfma(load_bf16x8(lk + (sub * 32 + c.prow) * LDK + ks * 16 + c.hg * 8), qop[ks], sc);
                f32x16_t x;
#pragma unroll
                for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(sc[r], c.c_scale, st.cm);
                if (!R::full(c, js)) {  // edge subtile: mask the keys outside the region
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (R::masked(c, js + acc_key(r, c.hg))) x[r] = -INFINITY;
                }
                bf16x8_t p0, p1;
                if (FIXED) exp_pack<true>(x, st.l, p0, p1);
                else softmax_step<NT, true, false>(x, st, ow, ol, p0, p1);
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
    };
    // The loads are unconditional (tiles past the last one read clamped keys
    // and are never used): a load under a branch would make every later wait
    // drain all loads in flight.
    Tile ta = gload(t_first);
    Tile tb = gload(t_first + BN);
    lstore(0, ta);
    __syncthreads();
    for (int n = 0; n < ntile; n += 2) {
        const int t0 = t_first + n * BN;
        // tile n is in LDS buffer 0, tile n+1 in tb
        ta = gload(t0 + 2 * BN);
        compute(0, t0);
        lstore(1, tb);
        __syncthreads();
        if (n + 1 >= ntile) break;
        // tile n+1 is in LDS buffer 1, tile n+2 in ta
        tb = gload(t0 + 3 * BN);
        compute(1, t0 + BN);
        lstore(0, ta);
        __syncthreads();
    }
}

// kModeRope: rotary embedding inside Eq. 3. q, k are the rotated queries and
// keys, cK / cVt the lifted-and-rotated distant keys and the lifted values
// ([B*Hkv][T - w][D] each), cnorm their 32-row block norms (Tp / 32 per
// head); the distant region then runs the full-d tile loop (no absorbed
// query, no lift in the epilogue), and W_down / W_up are not read.
// kModeDense / kModePaged: a chunk (rows q0.., k / v the context rows) whose
// distant latents are read in place from lc (cK / cVt unused); the norm
// arrays have lc.ncb / lc.nkb blocks a head; paged: each sequence's q0 and
// row count come from lc, and Tkv is the context rows' stride.
template <int D, int DD, int NW, int MODE>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void prefill_mfma_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wu, const bf16_t* __restrict__ cK,
    const bf16_t* __restrict__ cVt, const float* __restrict__ cnorm,
    const float* __restrict__ knorm, const bf16_t* __restrict__ consts, bf16_t* __restrict__ o,
    float* __restrict__ lse, int Hq, int Hkv, int T, int w, int Tp, int nblk, int BH,
    float c_scale, int q0, int n_rows, int kv0, int Tkv, const bf16_t* __restrict__ wv,
    const int* __restrict__ seq_lens, LatCache lc) {
    constexpr bool ROPE = MODE == kModeRope;
    constexpr bool CACHE = MODE == kModeDense || MODE == kModePaged;
    constexpr bool PAGED = MODE == kModePaged;
    constexpr int BM = NW * 32;
    constexpr int KS = D / 16;   // 16-wide k slabs of q . k
    constexpr int DS = DD / 16;  // 16-wide k slabs of q~ . c^K
    constexpr int NT = D / 32;   // 32-row tiles of O_win^T
    constexpr int BN = 64;       // keys per LDS tile (local region)
    constexpr int LDK = D + 8;   // padded LDS row (bf16 elements)
    constexpr int LDU = D + 8;   // padded row of wU (bf16 elements)
    static_assert(NW * (32 * DD + 8) <= BN * LDK, "value blocks of the cache mode fit one tile buffer");
    extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
    bf16_t* lds_k = smem;                    // [2][BN][LDK]
    bf16_t* lds_v = smem + 2 * BN * LDK;     // [2][BN][LDK]
    bf16_t* wU = smem + 4 * BN * LDK;        // [DD][LDU]: U[c][e] = W_up[c][e]
    // the value lift's matrix: W_up itself, or (shared latent) a second one
    // [Hkv][DD][D] staged after it
    bf16_t* wV = wv ? wU + DD * LDU : wU;

    // Each workgroup takes row blocks p and nblk-1-p of one (batch, head): a
    // short and a long causal row block, so every workgroup has the same work.
    // Workgroups are dealt to the 8 XCDs round-robin; when BH % 8 == 0 all
    // workgroups of a head are placed on one XCD so its L2 holds only the
    // K/V/latents of BH/8 heads.
    int pair, bh;
    const int G = Hq / Hkv;
    const int BG = BH / G;  // (batch, KV head) groups
    if ((BG & 7) == 0) {
        // the G query heads of a KV head share its XCD (and its L2)
        const int xcd = wg_id_x() & 7, local = wg_id_x() >> 3;
        const int hpx = BH >> 3;  // query heads per XCD
        pair = local / hpx;
        const int rem = local - pair * hpx;
        bh = ((rem / G) * 8 + xcd) * G + rem % G;
    } else {
        pair = wg_id_x() / BH;
        bh = wg_id_x() - pair * BH;
    }
    const int b = bh / Hq, h = bh - (bh / Hq) * Hq;
    const int g = h / (Hq / Hkv);
    const int bg = b * Hkv + g;
    const int tid = lane_id_x();
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // A paged chunk: this sequence's first row position and row count; one
    // the chunk does not fit gets NaN rows and nothing is read for it.
    int T_ = T, kv0_ = kv0;
    if constexpr (PAGED) {
        const int len_b = sload(lc.lens + b);
        const int nb = lc.n_new ? imin(imax(sload(lc.n_new + b), 0), n_rows) : n_rows;
        if (nb > 0 && (len_b < 0 || len_b + nb > lc.cap)) {
            for (int part = 0; part < 2; ++part) {
                const int rb = part == 0 ? nblk - 1 - pair : pair;
                if (part == 1 && rb >= nblk - 1 - pair) break;
                for (int idx = tid; idx < BM * D; idx += NW * 64) {
                    const int r = rb * BM + idx / D;
                    if (r < nb) {
                        o[((size_t)bh * n_rows + r) * D + idx % D] = (bf16_t)0x7fc0;
                        if (lse && idx % D == 0) lse[(size_t)bh * n_rows + r] = __builtin_nanf("");
                    }
                }
            }
            return;
        }
        q0 = imax(len_b, 0);
        T_ = q0 + nb;
        kv0_ = imax(q0 - w, 0);
    }
    // this sequence's length (a ragged batch; T, the padded length, stays the
    // layout of every array)
    const int Tb = seq_lens ? imin(imax(seq_lens[b], 0), T) : T_;
    const bf16_t* wdg = wd + (size_t)g * D * DD;
    const bf16_t* wug = wu ? wu + (size_t)g * DD * D : nullptr;
    const int nkb = CACHE ? lc.nkb : (T + 31) >> 5;  // 32-key blocks of a head with a key norm
    const int ncb = CACHE ? lc.ncb : Tp / 32;        // 32-key blocks of a head with a latent norm

    // U = W_up (W_down^T when tied), once per workgroup: its rows are the A
    // operand of q~ = q W_up^T, its columns that of the lift
    // O^T += W_up^T O_lat^T.
    // (all of this thread's elements requested at once, no load under a
    // branch: one memory round trip before the barrier)
    constexpr int UPT = DD * D / (NW * 64);
    static_assert(DD * D % (NW * 64) == 0, "whole W_up elements per thread");
    bf16_t uv[UPT];
    if constexpr (!ROPE) {
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int idx = tid + j * NW * 64, cc = idx / D, e = idx - (idx / D) * D;
            uv[j] = *(wug ? wug + (size_t)cc * D + e : wdg + (size_t)e * DD + cc);
        }
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int idx = tid + j * NW * 64, cc = idx / D, e = idx - (idx / D) * D;
            wU[cc * LDU + e] = uv[j];
        }
        if (wv) {
            const bf16_t* wvg = wv + (size_t)g * DD * D;
#pragma unroll
            for (int j = 0; j < UPT; ++j) {
                const int idx = tid + j * NW * 64;
                uv[j] = wvg[idx];
            }
#pragma unroll
            for (int j = 0; j < UPT; ++j) {
                const int idx = tid + j * NW * 64, cc = idx / D, e = idx - (idx / D) * D;
                wV[cc * LDU + e] = uv[j];
            }
        }
    }
    __syncthreads();

#pragma nounroll
    for (int part = 0; part < 2; ++part) {
        // Lane-dependent addresses are recomputed for each row block from an
        // opaque copy of the lane id: hoisted out of this loop they would hold
        // (and spill) dozens of registers across both blocks.
        int lane = tid & 63;
        __asm__ volatile("" : "+v"(lane));
        const int rb = part == 0 ? nblk - 1 - pair : pair;
        if (part == 1 && rb >= nblk - 1 - pair) break;  // odd block count: middle block once
        if (q0 + rb * BM >= Tb) continue;  // past this sequence's end (workgroup-uniform)
        RowCtx c;
        c.T = Tb;
        c.w = w;
        c.Tp = Tp;
        c.qc = lane & 31;
        c.hg = lane >> 5;
        c.prow = perm_row(c.qc);
        c.bg = bg;
        c.tid = tid;
        c.c_scale = c_scale;
        c.kv0 = kv0_;
        c.Tkv = Tkv;
        c.Td = imax(T_ - w, 0);
        const int i0 = q0 + rb * BM;  // position of the block's first row
        c.r0 = i0 + wave * 32;
        c.i = c.r0 + c.qc;
        c.i_hi = imin(c.r0 + 31, Tb - 1);  // last real row of this wavefront (< r0 if none)
        const int qc = c.qc, hg = c.hg, i = c.i;

        const int jd_end = (c.r0 < Tb) ? c.i_hi - w : -1;  // last distant key of any row here
        const int js_last = jd_end & ~31;
        const int iwg_hi = imin(i0 + BM - 1, Tb - 1);
        const bool has_local = w > 0 && imax(0, i0 - w + 1) <= iwg_hi;
        const int ii = imin(i, Tb - 1);

        // Every global load of the setup is issued here, before any of its
        // results is used: the query row and the first norm maxima of both
        // regions.
        const bf16_t* qrow = q + ((size_t)bh * n_rows + (ii - q0)) * D;
        bf16x8_t qop[KS];  // B operand of S^T = K Q^T: q[i][s*16 + hg*8 + 0..7]
#pragma unroll
        for (int s = 0; s < KS; ++s) qop[s] = load_bf16x8(qrow + s * 16 + hg * 8);
        const int nsb = jd_end >= 0 ? (js_last >> 5) + 1 : 0;  // latent blocks with a norm
        const int kb_lo = imax(0, c.r0 - w + 1) >> 5, kb_hi = imax(0, c.i_hi) >> 5;
        float cmax = lane < nsb ? cnorm[(size_t)bg * ncb + lane] : 0.f;
        float kmax = (has_local && kb_lo + lane <= kb_hi) ? knorm[(size_t)bg * nkb + kb_lo + lane] : 0.f;
        if (i >= Tb) {
#pragma unroll
            for (int s = 0; s < KS; ++s) qop[s] = zero_bf16x8();
        }
        float qs2 = dot8(qop[0], qop[0], 0.f);
#pragma unroll
        for (int s = 1; s < KS; ++s) qs2 = dot8(qop[s], qop[s], qs2);
        qs2 = pair_sum(qs2);

        SoftmaxState st;
        st.m = -INFINITY;
        st.cm = 0.f;
        st.thr = -INFINITY;
        st.l = 0.f;
        st.cmv = splat16(0.f);
        f32x16_t ow[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) ow[t] = splat16(0.f);
        f32x16_t ol = splat16(0.f);

        // ---- absorbed query q~ = q W_up^T (scaled): A rows = latent column c, k = e
        bf16x8_t qtop[DS];
        float bound = -INFINITY;
        if (ROPE && jd_end >= 0) {
            // full-d distant keys: |q . k| <= |q| |k|
            for (int sb = lane + 64; sb < nsb; sb += 64) cmax = fmaxf(cmax, cnorm[(size_t)bg * ncb + sb]);
            cmax = wave_max(cmax);
            bound = c_scale * sqrtf(qs2) * cmax;
        } else if (jd_end >= 0) {
            f32x16_t qt = splat16(0.f);
            // A row qc is latent column qa: qc itself (the pre-pass stores its
            // key latents in that permuted order), or, for latents read in
            // natural column order from a cache, qc with bits 2 and 3 swapped
            const int qa = CACHE ? (qc & ~12) | ((qc & 4) << 1) | ((qc & 8) >> 1) : qc;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const bf16x8_t a = qc < DD ? load_bf16x8(wU + qa * LDU + s * 16 + hg * 8) : zero_bf16x8();
                qt = mfma(a, qop[s], qt);
            }
            // accumulator register 8*s + j holds latent column qa(16*s + (j<4 ? 4hg+j : 8+4hg+j-4)):
            // natural order 16*s + 8hg + j when the bits were swapped
            float qn2 = 0.f;
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                qtop[s] = pack8(qt[8 * s + 0] * c_scale, qt[8 * s + 1] * c_scale, qt[8 * s + 2] * c_scale,
                                qt[8 * s + 3] * c_scale, qt[8 * s + 4] * c_scale, qt[8 * s + 5] * c_scale,
                                qt[8 * s + 6] * c_scale, qt[8 * s + 7] * c_scale);
                qn2 = dot8(qtop[s], qtop[s], qn2);
            }
            qn2 = pair_sum(qn2);
            // |q~ . c| <= |q~| |c| on the bf16 values the MFMA multiplies (Cauchy-Schwarz)
            for (int sb = lane + 64; sb < nsb; sb += 64) cmax = fmaxf(cmax, cnorm[(size_t)bg * ncb + sb]);
            cmax = wave_max(cmax);
            bound = sqrtf(qn2) * cmax;
        }
        if (has_local) {
            for (int kb = kb_lo + lane + 64; kb <= kb_hi; kb += 64) kmax = fmaxf(kmax, knorm[(size_t)bg * nkb + kb]);
            kmax = wave_max(kmax);
            bound = fmaxf(bound, c_scale * sqrtf(qs2) * kmax);
        }
        // Fixed reference: the bound (inflated for fp32 rounding) bounds |s|
        // for every real score s of the row (Cauchy-Schwarz), so when it is at
        // most 50 every weight 2^(s - bound) is at least 2^-100. A row with a
        // larger bound needs a witness: a real score of that row (its own key
        // or latent) within 100 of the bound, so that its largest weight
        // cannot underflow. Only a wavefront with such a row loads it.
        bound = bound * 1.001f + 1e-6f;
        bool fixed = c.r0 < Tb;
        if (fixed && __builtin_amdgcn_ballot_w64(i < Tb && bound > 50.f)) {
            bf16x8_t wit[KS];  // own key (w >= 1) or own latent key (w = 0)
            if (w >= 1) {
                const bf16_t* krow = k + ((size_t)bg * Tkv + (ii - kv0_)) * D;
#pragma unroll
                for (int s = 0; s < KS; ++s) wit[s] = load_bf16x8(krow + s * 16 + hg * 8);
            } else if (ROPE) {
                const bf16_t* crow = cK + ((size_t)bg * c.Td + ii) * D;  // lifted, rotated own key
#pragma unroll
                for (int s = 0; s < KS; ++s) wit[s] = load_bf16x8(crow + s * 16 + hg * 8);
            } else if (CACHE) {
                const bf16_t* crow = lat_row<DD, PAGED>(lc, b, g, bg, Hkv, ii);  // own latent key
#pragma unroll
                for (int s = 0; s < KS; ++s)
                    wit[s] = s < DS && crow ? load_bf16x8(crow + s * 16 + hg * 8) : zero_bf16x8();
            } else {
                const bf16_t* crow = cK + ((size_t)bg * Tp + ii) * DD;
#pragma unroll
                for (int s = 0; s < KS; ++s) wit[s] = s < DS ? load_bf16x8(crow + s * 16 + hg * 8) : zero_bf16x8();
            }
            float witness = 0.f;
            if (w >= 1 || ROPE) {
#pragma unroll
                for (int s = 0; s < KS; ++s) witness = dot8(qop[s], wit[s], witness);
                witness *= c_scale;
            } else {
#pragma unroll
                for (int s = 0; s < DS; ++s) witness = dot8(qtop[s], wit[s], witness);
            }
            witness = pair_sum(witness);
            fixed = !__builtin_amdgcn_ballot_w64(i < Tb && bound - witness > 100.f);
        }
        if (fixed) {
            st.m = bound;
            st.cm = -bound;
            st.thr = kTau;
            st.cmv = splat16(-bound);
        }

        // ------------------------------------------------------------ distant region
        if constexpr (ROPE) {
            // full d, tiles staged for the workgroup (a barrier per tile: the
            // condition is the workgroup's)
            if (iwg_hi - w >= 0) {
                if constexpr (D > 64) {
                    if (fixed) local_region_1deep<D, DD, NW, true, true>(c, cK, cVt, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                    else local_region_1deep<D, DD, NW, false, true>(c, cK, cVt, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                } else {
                    if (fixed) local_region<D, DD, NW, true, true>(c, cK, cVt, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                    else local_region<D, DD, NW, false, true>(c, cK, cVt, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                }
            }
        } else if (jd_end >= 0) {
            if constexpr (CACHE) {
                // the wavefront's value block: in the second local-region value
                // buffer, which the local region first writes after a barrier
                // that every wavefront reaches only after its distant region
                bf16_t* vst = lds_v + BN * LDK + wave * (32 * DD + 8);
                if (fixed) distant_region_cache<D, DD, true, PAGED>(c, lc, b, g, Hkv, vst, qtop, js_last, st, ow, ol);
                else distant_region_cache<D, DD, false, PAGED>(c, lc, b, g, Hkv, vst, qtop, js_last, st, ow, ol);
            } else {
                if (fixed) distant_region<D, DD, true>(c, cK, cVt, qtop, js_last, st, ow, ol);
                else distant_region<D, DD, false>(c, cK, cVt, qtop, js_last, st, ow, ol);
            }
        }
        // The latent part is complete: lift it now (Eq. 2 by linearity), so the
        // window region below carries ow only.
        if (DD == 16 && !ROPE) st.l += ol[8];  // ones row (row 16, held by lanes of half 0)
        if (jd_end >= 0 && !ROPE) {
            // O^T += W_up^T O_lat^T, O_lat split into bf16 hi + lo parts
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                float hi_f[8], lo_f[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float x = ol[8 * s + j];
                    const float hv = __uint_as_float((pack2(x, 0.f) & 0xffffu) << 16);
                    hi_f[j] = hv;
                    lo_f[j] = x - hv;
                }
                const bf16x8_t bhi = pack8(hi_f[0], hi_f[1], hi_f[2], hi_f[3], hi_f[4], hi_f[5], hi_f[6], hi_f[7]);
                const bf16x8_t blo = pack8(lo_f[0], lo_f[1], lo_f[2], lo_f[3], lo_f[4], lo_f[5], lo_f[6], lo_f[7]);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    // A row e = t*32 + qc, k = latent columns s*16 + {4hg..4hg+3, 8+4hg..8+4hg+3}
                    const bf16_t* ur = wV + (s * 16 + 4 * hg) * LDU + t * 32 + qc;
                    uint16_t a8[8];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        a8[j] = ur[j * LDU];
                        a8[4 + j] = ur[(8 + j) * LDU];
                    }
                    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, a8);
                    ow[t] = mfma(a, bhi, ow[t]);
                    ow[t] = mfma(a, blo, ow[t]);
                }
            }
        }


        // ------------------------------------------------------------ local region
        if (has_local) {
            if constexpr (D > 64) {
                if (fixed) local_region_1deep<D, DD, NW, true>(c, k, v, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                else local_region_1deep<D, DD, NW, false>(c, k, v, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
            } else {
                if (fixed) local_region<D, DD, NW, true>(c, k, v, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
                else local_region<D, DD, NW, false>(c, k, v, lds_k, lds_v, qop, i0, iwg_hi, st, ow, ol);
            }
        }

        if (c.r0 >= Tb) continue;

        // ------------------------------------------------------------ epilogue
        const float lt = pair_sum(st.l);

        if (i < Tb) {
            // log of the row's softmax denominator (natural log), for a backward pass
            if (lse && hg == 0) lse[(size_t)bh * n_rows + (i - q0)] = (st.m + log2f(lt)) * 0.6931471805599453f;
            const float inv = 1.f / lt;
            bf16_t* orow = o + ((size_t)bh * n_rows + (i - q0)) * D;
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
}

bool prefill_mfma_supported(const dar_shape* s) {
    if (s->dtype != DAR_BF16) return false;
    if (s->d != 64 && s->d != 128) return false;
    if (s->d_down != 16 && s->d_down != 32) return false;
    return true;
}

template <int D, int DD, int MODE = kModePlain>
static hipError_t launch_dd(int B, int Hq, int Hkv, const PrefillGeo& geo, int w, const void* q, const void* k,
                            const void* v, const void* wd, const void* wu, void* o, float* lse,
                            const void* cK, const void* cVt, const float* cnorm,
                            const float* knorm, const void* consts, hipStream_t st,
                            const void* wv = nullptr, const LatCache& lc = LatCache{}) {
    constexpr bool ROPE = MODE == kModeRope;
    constexpr int NW = 4;
    constexpr int BM = NW * 32;
    const int T = geo.total();
    const int nblk = (geo.n_rows + BM - 1) / BM;
    const int npair = (nblk + 1) / 2;
    const int BH = B * Hq;
    const int Tp = ROPE ? round_up(T - w > 0 ? T - w : 0, 32) : prefill_tp(T, w);
    const float c_scale = 1.4426950408889634f / sqrtf((float)D);
    const size_t lds = sizeof(bf16_t) * (4 * 64 * (D + 8) + (wv ? 2 : 1) * DD * (D + 8));
    auto kern = prefill_mfma_kernel<D, DD, NW, MODE>;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(npair * BH), dim3(NW * 64), lds, st, (const bf16_t*)q,
                       (const bf16_t*)k, (const bf16_t*)v, (const bf16_t*)wd, (const bf16_t*)wu,
                       (const bf16_t*)cK, (const bf16_t*)cVt, cnorm, knorm, (const bf16_t*)consts,
                       (bf16_t*)o, lse, Hq, Hkv, T, w, Tp, nblk, BH, c_scale, geo.q0,
                       geo.n_rows, geo.kv0, geo.Tkv, (const bf16_t*)wv, geo.seq_lens, lc);
    return hipGetLastError();
}

hipError_t launch_prefill_mfma(const dar_shape* s, const PrefillGeo& geo, const void* q, const void* k,
                               const void* v, const void* wd, const void* wu, void* o, float* lse,
                               const void* cK, const void* cVt, const float* cnorm,
                               const float* knorm, const void* consts, hipStream_t st,
                               const void* wv) {
    const int B = s->B, Hq = s->Hq, Hkv = s->Hkv, w = s->w;
    if (s->d == 64 && s->d_down == 16) return launch_dd<64, 16>(B, Hq, Hkv, geo, w, q, k, v, wd, wu, o, lse, cK, cVt, cnorm, knorm, consts, st, wv);
    if (s->d == 64 && s->d_down == 32) return launch_dd<64, 32>(B, Hq, Hkv, geo, w, q, k, v, wd, wu, o, lse, cK, cVt, cnorm, knorm, consts, st, wv);
    if (s->d == 128 && s->d_down == 16) return launch_dd<128, 16>(B, Hq, Hkv, geo, w, q, k, v, wd, wu, o, lse, cK, cVt, cnorm, knorm, consts, st, wv);
    if (s->d == 128 && s->d_down == 32) return launch_dd<128, 32>(B, Hq, Hkv, geo, w, q, k, v, wd, wu, o, lse, cK, cVt, cnorm, knorm, consts, st, wv);
    return hipErrorNotSupported;
}

hipError_t launch_prefill_mfma_cache(const dar_shape* s, const PrefillGeo& geo, const LatCache& lc,
                                     const void* q, const void* ctx_k, const void* ctx_v,
                                     const void* wd, const void* wu, void* o, float* lse,
                                     const float* cnorm, const float* knorm, hipStream_t st) {
    const int B = s->B, Hq = s->Hq, Hkv = s->Hkv, w = s->w;
#define DAR_CACHE_LAUNCH(D_, DD_)                                                                     \
    if (s->d == D_ && s->d_down == DD_) {                                                            \
        if (lc.bt)                                                                                   \
            return launch_dd<D_, DD_, kModePaged>(B, Hq, Hkv, geo, w, q, ctx_k, ctx_v, wd, wu, o, lse, \
                                                  nullptr, nullptr, cnorm, knorm, nullptr, st,       \
                                                  nullptr, lc);                                      \
        return launch_dd<D_, DD_, kModeDense>(B, Hq, Hkv, geo, w, q, ctx_k, ctx_v, wd, wu, o, lse,     \
                                              nullptr, nullptr, cnorm, knorm, nullptr, st, nullptr, \
                                              lc);                                                   \
    }
    DAR_CACHE_LAUNCH(64, 16)
    DAR_CACHE_LAUNCH(64, 32)
    DAR_CACHE_LAUNCH(128, 16)
    DAR_CACHE_LAUNCH(128, 32)
#undef DAR_CACHE_LAUNCH
    return hipErrorNotSupported;
}

}  // namespace dar

namespace dar {

// Rotary embedding inside Eq. 3 (bf16, d in {64, 128}, any d_down: the
// lift happened in the pre-pass): qr, kr the rotated queries and keys, v the
// values, kd / vd the lifted-and-rotated distant keys and lifted values
// [B*Hkv][T - w][d], knorm / dnorm the 32-row block norms of kr and kd.
bool prefill_mfma_rope_supported(const dar_shape* s) {
    return s->dtype == DAR_BF16 && (s->d == 64 || s->d == 128);
}

hipError_t launch_prefill_mfma_rope_geo(const dar_shape* s, const PrefillGeo& geo, const void* qr,
                                        const void* kr, const void* v, const void* kd,
                                        const void* vd, void* o, float* lse, const float* knorm,
                                        const float* dnorm, hipStream_t st) {
    if (s->d == 64)
        return launch_dd<64, 16, kModeRope>(s->B, s->Hq, s->Hkv, geo, s->w, qr, kr, v, nullptr, nullptr, o,
                                       lse, kd, vd, dnorm, knorm, nullptr, st);
    return launch_dd<128, 16, kModeRope>(s->B, s->Hq, s->Hkv, geo, s->w, qr, kr, v, nullptr, nullptr, o, lse,
                                    kd, vd, dnorm, knorm, nullptr, st);
}

hipError_t launch_prefill_mfma_rope(const dar_shape* s, int T, const void* qr, const void* kr,
                                    const void* v, const void* kd, const void* vd, void* o,
                                    float* lse, const float* knorm, const float* dnorm,
                                    hipStream_t st) {
    const PrefillGeo geo = whole_sequence(T);
    if (s->d == 64)
        return launch_dd<64, 16, kModeRope>(s->B, s->Hq, s->Hkv, geo, s->w, qr, kr, v, nullptr, nullptr, o,
                                       lse, kd, vd, dnorm, knorm, nullptr, st);
    return launch_dd<128, 16, kModeRope>(s->B, s->Hq, s->Hkv, geo, s->w, qr, kr, v, nullptr, nullptr, o, lse,
                                    kd, vd, dnorm, knorm, nullptr, st);
}

}  // namespace dar
