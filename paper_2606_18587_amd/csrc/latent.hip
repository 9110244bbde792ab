// Window-exit down-projection (Eq. 1, applied per KV head to keys and values).
//
//  * prefill pre-pass: latents of every token that is distant for some query
//    of the sequence (tokens [0, T - w)), into the prefill workspace;
//  * cache append: each token that leaves the window is projected into its
//    latent slot, the newest tokens go to the ring.
//
// Both accumulate c[col] = sum_e x[e] * W_down[e][col] in fp32 in a fixed
// order: on the vector ALUs with fused multiply-adds in increasing e
// (dar::project_col), on the matrix cores (bf16, d 64/128, d_down 16/32) with
// the MFMA sequence of project_mfma. Each shape takes the same one of the two
// in the pre-pass and in every append kernel, so they produce identical bits
// for identical inputs, however tokens are batched.
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

// One block = 64 tokens of one (batch, KV head). Lane = token; the 4 waves
// share the 2*dd output columns (K and V) in chunks of 8.
//   cK:  [B*Hkv][Tp][dd]               token-major (columns in latent_pos order
//                                       when perm is set)
//   cVt: [B*Hkv][Tp/32][dd][32]        32-token blocks, transposed inside
// Rows [Tl, Tp) are written as zeros.
template <typename T>
__global__ __launch_bounds__(256) void prefill_latent_kernel(
    const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ wd,
    T* __restrict__ cK, T* __restrict__ cVt, int Hkv, int d, int dd, int Tl, int Tp, int perm,
    int kv0, int Tkv, int lat0, const T* __restrict__ k_lat, const T* __restrict__ v_lat,
    int cap) {
    extern __shared__ float xs[];  // [2][64][d+1]
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    const int t0 = wg_id_x() * 64;
    const int ld = d + 1;
    const T* wdg = wd + (size_t)g * d * dd;
    // rows of the positions whose latent is projected here (k/v row = position - kv0)
    for (int which = 0; which < 2; ++which) {
        const T* x = (which ? v : k) + (size_t)bg * Tkv * d;
        float* dst = xs + which * 64 * ld;
        for (int idx = lane_id_x(); idx < 64 * d; idx += 256) {
            const int t = idx / d, e = idx - (idx / d) * d;
            const int p = t0 + t;
            dst[t * ld + e] = (p < Tl && p >= lat0 && p >= kv0 && p - kv0 < Tkv)
                                  ? elem<T>::load(x + (size_t)(p - kv0) * d + e) : 0.f;
        }
    }
    __syncthreads();
    const int lane = lane_id_x() & 63;
    const int wave = __builtin_amdgcn_readfirstlane(lane_id_x() >> 6);
    const int t = t0 + lane;
    const int nchunk = (dd + 7) / 8;
    for (int ch = wave; ch < 2 * nchunk; ch += 4) {
        const int which = ch / nchunk;
        const int c0 = (ch - which * nchunk) * 8;
        const float* xr = xs + which * 64 * ld + lane * ld;
        float acc[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = 0.f;
        for (int e = 0; e < d; ++e) {
            const float xv = xr[e];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (c0 + j < dd)
                    acc[j] = __builtin_fmaf(xv, elem<T>::load(wdg + (size_t)e * dd + c0 + j), acc[j]);
        }
        if (t < Tp) {
            // positions below lat0: the cache's latent, copied
            const bool fromc = t < lat0;
            const T* cached = (which ? v_lat : k_lat) + ((size_t)bg * cap + imin(t, imax(lat0 - 1, 0))) * dd;
            if (which == 0) {
                T* out = cK + ((size_t)bg * Tp + t) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd)
                        out[perm ? latent_pos(c0 + j) : c0 + j] =
                            fromc ? cached[c0 + j] : elem<T>::from_f32(acc[j]);
            } else {
                T* out = cVt + ((size_t)bg * Tp + (size_t)(t >> 5) * 32) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd)
                        out[(size_t)(c0 + j) * 32 + (t & 31)] =
                            fromc ? cached[c0 + j] : elem<T>::from_f32(acc[j]);
            }
        }
    }
}

// Cache append. One block = up to 64 new tokens of one (batch, KV head).
// New token t (position p = len + t) makes token e = p - w leave the window:
// its latent is projected from the ring (e < len) or from the new tokens
// (e >= len). Token t itself is written to ring slot p % w if it is still in
// the window after the whole append (t >= n - w).
// mode 0: project and write the ring (safe when n <= w: the slot a block
//         reads is only rewritten by the same block, after its barrier);
// mode 1: project only; mode 2: ring only (mode 1 then mode 2 when n > w).
template <typename T>
__global__ __launch_bounds__(256) void append_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, const T* __restrict__ wd,
    T* k_win, T* v_win, T* __restrict__ k_lat, T* __restrict__ v_lat, int Hkv, int d, int dd,
    int w, int cap, int len, int n, int mode) {
    extern __shared__ float xs[];  // [2][64][d+1]
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    const int t0 = wg_id_x() * 64;
    const int ld = d + 1;
    const size_t new_base = (size_t)bg * n * d;
    const size_t win_base = (size_t)bg * w * d;
    if (mode != 2) {
        for (int which = 0; which < 2; ++which) {
            const T* src_new = (which ? v_new : k_new) + new_base;
            const T* src_win = (which ? v_win : k_win) + win_base;
            float* dst = xs + which * 64 * ld;
            for (int idx = lane_id_x(); idx < 64 * d; idx += 256) {
                const int tl = idx / d, e = idx - (idx / d) * d;
                const int tt = t0 + tl;
                const int ex = len + tt - w;  // position leaving the window
                float val = 0.f;
                if (tt < n && ex >= 0) {
                    const T* row = (ex < len) ? src_win + (size_t)(ex % w) * d
                                              : src_new + (size_t)(ex - len) * d;
                    val = elem<T>::load(row + e);
                }
                dst[tl * ld + e] = val;
            }
        }
    }
    __syncthreads();  // every ring read of this block is done before any ring write
    if (mode != 2) {
        const int lane = lane_id_x() & 63;
        const int wave = __builtin_amdgcn_readfirstlane(lane_id_x() >> 6);
        const int tt = t0 + lane;
        const int ex = len + tt - w;
        const int nchunk = (dd + 7) / 8;
        const T* wdg = wd + (size_t)g * d * dd;
        for (int ch = wave; ch < 2 * nchunk; ch += 4) {
            const int which = ch / nchunk;
            const int c0 = (ch - which * nchunk) * 8;
            const float* xr = xs + which * 64 * ld + lane * ld;
            float acc[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j] = 0.f;
            for (int e = 0; e < d; ++e) {
                const float xv = xr[e];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd)
                        acc[j] = __builtin_fmaf(xv, elem<T>::load(wdg + (size_t)e * dd + c0 + j), acc[j]);
            }
            if (tt < n && ex >= 0) {
                T* out = (which ? v_lat : k_lat) + ((size_t)bg * cap + ex) * dd;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (c0 + j < dd) out[c0 + j] = elem<T>::from_f32(acc[j]);
            }
        }
    }
    if (mode != 1 && w > 0) {
        for (int which = 0; which < 2; ++which) {
            const T* src = (which ? v_new : k_new) + new_base;
            T* ring = (which ? v_win : k_win) + win_base;
            for (int idx = lane_id_x(); idx < 64 * d; idx += 256) {
                const int tl = idx / d, e = idx - (idx / d) * d;
                const int tt = t0 + tl;
                if (tt < n && tt >= n - w)
                    ring[(size_t)((len + tt) % w) * d + e] = src[(size_t)tt * d + e];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Matrix-core projection for bf16 (d % 16 == 0, d_down <= 32). Per group of 32
// tokens, latent^T = W_down^T x^T with v_mfma_f32_32x32x16_bf16: A = W_down^T
// (row = latent column c, k = e), B = x^T (column = token, k = e, a 16-byte
// load from the token's row). The accumulator of lane l holds token l%32 and
// latent columns c = 8*(r/4) + 4*(l/32) + r%4 for register r. A token's
// latent depends only on its own row and W_down, and every bf16 path (prefill
// pre-pass, bulk and single-token append) runs this same instruction
// sequence, so their latents are bit-identical.
typedef __bf16 lbf16x8 __attribute__((ext_vector_type(8)));
typedef float lf32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ lbf16x8 lload8(const bf16_t* p) {
    return __builtin_bit_cast(lbf16x8, *reinterpret_cast<const uint4*>(p));
}

// Two fp32 values rounded to bf16 (nearest even, one v_cvt_pk_bf16_f32) and
// packed, a in the low half. Equal to f32_to_bf16 on every non-NaN input.
__device__ __forceinline__ uint32_t rne_pack2(float a, float b) {
    typedef float lf32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 lbf16x2 __attribute__((ext_vector_type(2)));
    const lf32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, lbf16x2));
}

template <int D>
__device__ __forceinline__ void load_wd_operand(const bf16_t* __restrict__ wdg, int dd, int lane,
                                                lbf16x8 (&wa)[D / 16]) {
    const int c = lane & 31, hg = lane >> 5;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
        uint16_t t8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) t8[j] = (c < dd) ? wdg[(size_t)(s * 16 + hg * 8 + j) * dd + c] : 0;
        wa[s] = __builtin_bit_cast(lbf16x8, t8);
    }
}

template <int D>
__device__ __forceinline__ lf32x16 project_mfma(const lbf16x8 (&wa)[D / 16], const lbf16x8 (&x)[D / 16]) {
    lf32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[s], x[s], acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ int acc_col(int r, int hg) { return 8 * (r >> 2) + 4 * hg + (r & 3); }

// Prefill pre-pass. Block (x, y) serves positions [128x, 128x + 128) of
// (batch, KV head) y; wavefront w takes positions [32w, 32w + 32) of them.
// Writes the latents of positions [0, T - w), and per 32-position block the
// largest L2 norm of the stored c^K rows and of the key rows that k holds
// (positions [kv0, T)); the matrix-core prefill bounds its scores with them.
// k and v row t holds position kv0 + t; positions below lat0 take their
// latents from the cache arrays k_lat / v_lat (row stride cap) instead of a
// projection (chunked prefill: the tokens that left the window earlier).
//
// Latency layout: W_down is requested first and brought into LDS (stored
// transposed as the A operand rows); the key and value rows are in flight
// meanwhile; the transposed value latents go out through LDS as 16-byte
// stores.
template <int D>
__global__ __launch_bounds__(256) void prefill_latent_mfma_kernel(
    const bf16_t* __restrict__ k, const bf16_t* __restrict__ v, const bf16_t* __restrict__ wd,
    bf16_t* __restrict__ cK, bf16_t* __restrict__ cVt, float* __restrict__ cnorm,
    float* __restrict__ knorm, bf16_t* __restrict__ consts, int Hkv, int T_, int dd, int Tl,
    int Tp, int kv0, int Tkv, int lat0, const bf16_t* __restrict__ k_lat,
    const bf16_t* __restrict__ v_lat, int cap, const int* __restrict__ seq_lens) {
    constexpr int KS = D / 16;
    constexpr int LDW = D + 8;   // W^T row in LDS (bf16 elements)
    constexpr int LDT = 32 + 8;  // transposed value-latent row in LDS
    __shared__ __attribute__((aligned(16))) bf16_t wsh[32 * LDW];
    __shared__ __attribute__((aligned(16))) bf16_t vtr[4][32 * LDT];
    if (wg_id_x() == 0 && wg_id_y() == 0 && lane_id_x() < 16)
        consts[lane_id_x()] = lane_id_x() < 8 ? (bf16_t)0x3f80 : (bf16_t)0;
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    // a ragged batch: this sequence's length Tv (positions at or past it are
    // padding: no norm, zero latents), its latent count Tlv
    const int Tv = seq_lens ? imin(imax(seq_lens[bg / Hkv], 0), T_) : T_;
    const int Tlv = Tl - (T_ - Tv);
    const int tid = lane_id_x();
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tl = lane & 31, hg = lane >> 5;
    const int Tk = (T_ + 31) & ~31;
    const bf16_t* kbase = k + (size_t)bg * Tkv * D;
    const bf16_t* vbase = v + (size_t)bg * Tkv * D;

    // key and value rows of a wavefront's 32 positions (row indices clamped;
    // rows of positions k does not hold are zeroed before use)
    struct Rows {
        lbf16x8 k[KS], v[KS];
    };
    auto load = [&](int chunk) {
        Rows r;
        const int t = chunk * 128 + wave * 32 + tl;
        const int row = imax(imin(t - kv0, Tkv - 1), 0);
        const bf16_t* kr = kbase + (size_t)row * D;
        const bf16_t* vr = vbase + (size_t)row * D;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            r.k[s] = lload8(kr + s * 16 + hg * 8);
            r.v[s] = lload8(vr + s * 16 + hg * 8);
        }
        return r;
    };

    // W_down^T into LDS: row c (latent column, zero for c >= dd), k = e.
    // This thread's elements are requested together, before any key or value
    // row (loads return in order, so the LDS stores wait for W only and the
    // rows stay in flight through the barrier). Column indices are clamped so
    // that no load sits under a branch.
    // A workgroup whose 128 positions all take their latents from the cache
    // and lie below the first key row (chunked prefill: no key norm either)
    // projects nothing: it only copies the cached latents into this kernel's
    // layouts with their norms (workgroup-uniform, so the barrier below is
    // skipped by every thread of it or by none).
    const int chunk = wg_id_x();
    const bool cached = chunk * 128 + 127 < imin(lat0, kv0);
    const lbf16x8 zero8 = __builtin_bit_cast(lbf16x8, make_uint4(0, 0, 0, 0));
    constexpr int WPT = D * 32 / 256;  // W elements per thread
    const bf16_t* wdg = wd + (size_t)g * D * dd;
    Rows cur;
    lbf16x8 wa[KS];
    if (!cached) {
        bf16_t wv[WPT];
#pragma unroll
        for (int j = 0; j < WPT; ++j) {
            const int idx = tid + 256 * j, e = idx >> 5, c = idx & 31;
            wv[j] = wdg[(size_t)e * dd + imin(c, dd - 1)];
        }
        cur = load(chunk);
#pragma unroll
        for (int j = 0; j < WPT; ++j) {
            const int idx = tid + 256 * j, e = idx >> 5, c = idx & 31;
            wsh[c * LDW + e] = c < dd ? wv[j] : (bf16_t)0;
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < KS; ++s) wa[s] = *reinterpret_cast<const lbf16x8*>(wsh + tl * LDW + s * 16 + hg * 8);
    } else {
#pragma unroll
        for (int s = 0; s < KS; ++s) cur.k[s] = cur.v[s] = wa[s] = zero8;
    }

    {
        const int ts = chunk * 128 + wave * 32;  // first token of this wavefront
        const int t = ts + tl;
        if (ts < T_) {
            float n2 = 0.f;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const uint4 u = __builtin_bit_cast(uint4, t < Tv && t >= kv0 ? cur.k[s] : zero8);
                const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float lo = __uint_as_float(w4[j] << 16), hi = __uint_as_float(w4[j] & 0xffff0000u);
                    n2 = __builtin_fmaf(lo, lo, n2);
                    n2 = __builtin_fmaf(hi, hi, n2);
                }
            }
            n2 += __shfl_xor(n2, 32, 64);
            const float nmax = wave_max_dpp(n2);
            if (lane == 0) knorm[(size_t)bg * (Tk / 32) + (ts >> 5)] = sqrtf(nmax);
        }
        if (ts < Tp) {
            lbf16x8 xk[KS], xv[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                xk[s] = t < Tlv ? cur.k[s] : zero8;
                xv[s] = t < Tlv ? cur.v[s] : zero8;
            }
            // Latents read from the cache for positions below lat0: per lane
            // the columns 8q + 4hg + 0..3 of its token, i.e. the register
            // pairs (4q, 4q + 1) and (4q + 2, 4q + 3) of the projection.
            const bool fromc = t < lat0;
            uint2 ck[4], cv[4];
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) ck[q4] = cv[q4] = make_uint2(0, 0);
            if (ts < lat0) {  // wave-uniform
                const size_t rowc = ((size_t)bg * cap + imin(t, lat0 - 1)) * dd;
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4)
                    if (8 * q4 < dd) {
                        ck[q4] = *reinterpret_cast<const uint2*>(k_lat + rowc + 8 * q4 + 4 * hg);
                        cv[q4] = *reinterpret_cast<const uint2*>(v_lat + rowc + 8 * q4 + 4 * hg);
                    }
            }
            auto cpair = [&](const uint2 (&c)[4], int m) { return (m & 1) ? c[m >> 1].y : c[m >> 1].x; };
            const lf32x16 zacc = {};
            // key latents: token-major, columns in latent_pos order, plus the norm
            {
                const lf32x16 acc = cached ? zacc : project_mfma<D>(wa, xk);
                // squared norm of the stored (bf16-rounded) row; columns past
                // d_down are zero (W^T rows past d_down are zero)
                float n2 = 0.f;
                uint32_t pk[8];  // the row's bf16 values, pairs of registers
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    const uint32_t u = fromc ? cpair(ck, r >> 1) : rne_pack2(acc[r], acc[r + 1]);
                    pk[r >> 1] = u;
                    const float c0 = __uint_as_float(u << 16), c1 = __uint_as_float(u & 0xffff0000u);
                    n2 = __builtin_fmaf(c0, c0, n2);
                    n2 = __builtin_fmaf(c1, c1, n2);
                }
                n2 += __shfl_xor(n2, 32, 64);
                const float nmax = wave_max_dpp(n2);
                if (lane == 0) cnorm[(size_t)bg * (Tp / 32) + (ts >> 5)] = sqrtf(nmax);
                bf16_t* out = cK + ((size_t)bg * Tp + t) * dd;
                // latent_pos order: positions 16s + 8hg + j hold registers 8s + j
#pragma unroll
                for (int s = 0; s < 2; ++s)
                    if (16 * s < dd)
                        *reinterpret_cast<uint4*>(out + 16 * s + 8 * hg) =
                            make_uint4(pk[4 * s], pk[4 * s + 1], pk[4 * s + 2], pk[4 * s + 3]);
            }
            // value latents, transposed per 32-token block: [c][token], via LDS
            {
                const lf32x16 acc = cached ? zacc : project_mfma<D>(wa, xv);
                bf16_t* tb = vtr[wave];
                // all 32 rows of the block (rows past d_down are zero and not read)
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    const uint32_t u = fromc ? cpair(cv, r >> 1) : rne_pack2(acc[r], acc[r + 1]);
                    tb[acc_col(r, hg) * LDT + tl] = (bf16_t)(u & 0xffffu);
                    tb[acc_col(r + 1, hg) * LDT + tl] = (bf16_t)(u >> 16);
                }
                // same wavefront: its LDS writes complete before its reads
                const int rb = cvt_rows(dd);  // block rows: dd, plus a ones row when dd == 16
                bf16_t* out = cVt + ((size_t)bg * (Tp / 32) + (size_t)(ts >> 5)) * rb * 32;
                for (int q = lane; q < dd * 4; q += 64) {
                    const int c = q >> 2, t0 = (q & 3) * 8;
                    *reinterpret_cast<uint4*>(out + q * 8) = *reinterpret_cast<const uint4*>(tb + c * LDT + t0);
                }
                if (rb > dd && lane < 4)
                    *reinterpret_cast<uint4*>(out + dd * 32 + lane * 8) =
                        make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
            }
        }
    }
}

// Cache append for bf16 with the matrix-core projection. One wavefront per 32
// new tokens of one (batch, KV head); modes as in append_kernel. The lane that
// reads elements [16s + 8hg, +8) of the token leaving ring slot p % w is the
// lane that writes the same elements of the new token into that slot, after
// its read, so mode 0 needs no barrier.
template <int D>
__global__ __launch_bounds__(64) void append_mfma_kernel(
    const bf16_t* __restrict__ k_new, const bf16_t* __restrict__ v_new, const bf16_t* __restrict__ wd,
    bf16_t* k_win, bf16_t* v_win, bf16_t* __restrict__ k_lat, bf16_t* __restrict__ v_lat, int Hkv,
    int dd, int w, int cap, int len, int n, int mode) {
    constexpr int KS = D / 16;
    const int bg = wg_id_y();
    const int g = bg % Hkv;
    const int lane = lane_id_x();
    const int tl = lane & 31, hg = lane >> 5;
    const int tt = wg_id_x() * 32 + tl;      // new token index
    const int ex = len + tt - w;              // position leaving the window
    const bool valid = tt < n;
    const bool project = mode != 2 && valid && ex >= 0;
    const bool to_ring = mode != 1 && valid && w > 0 && tt >= n - w;
    lbf16x8 wa[KS];
    if (mode != 2) load_wd_operand<D>(wd + (size_t)g * D * dd, dd, lane, wa);
    for (int which = 0; which < 2; ++which) {
        const bf16_t* src_new = (which ? v_new : k_new) + (size_t)bg * n * D;
        bf16_t* ring = (which ? v_win : k_win) + (size_t)bg * w * D;
        if (mode != 2) {
            const bf16_t* row = src_new;
            if (project) row = (ex < len) ? ring + (size_t)(ex % w) * D : src_new + (size_t)(ex - len) * D;
            lbf16x8 x[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                x[s] = lload8(row + s * 16 + hg * 8);
                if (!project) x[s] = __builtin_bit_cast(lbf16x8, make_uint4(0, 0, 0, 0));
            }
            const lf32x16 acc = project_mfma<D>(wa, x);
            if (project) {
                bf16_t* out = (which ? v_lat : k_lat) + ((size_t)bg * cap + ex) * dd;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int c = acc_col(r, hg);
                    if (c < dd) out[c] = f32_to_bf16(acc[r]);
                }
            }
        }
        if (to_ring) {
            const bf16_t* src = src_new + (size_t)tt * D;
            bf16_t* dst = ring + (size_t)((len + tt) % w) * D;
#pragma unroll
            for (int s = 0; s < KS; ++s)
                *reinterpret_cast<uint4*>(dst + s * 16 + hg * 8) = *reinterpret_cast<const uint4*>(src + s * 16 + hg * 8);
        }
    }
}

// The matrix-core projection is used exactly on the shapes the matrix-core
// prefill takes (bf16, d 64/128, d_down 16/32), by the pre-pass and by every
// append kernel alike: one projection per shape, so the latents a chunked
// prefill attends with are the bits the cache keeps.
static bool mfma_projection(int d, int dd) { return (d == 64 || d == 128) && (dd == 16 || dd == 32); }

template <typename T>
static hipError_t launch_prefill_latent_valu(const T* k, const T* v, const T* wd, T* cK, T* cVt,
                                             int B, int Hkv, const PrefillGeo& geo, int d, int dd,
                                             int w, bool perm, hipStream_t st) {
    const int T_ = geo.total();
    const int Tl = T_ - w;
    if (Tl <= 0) return hipSuccess;
    const int Tp = prefill_tp(T_, w);
    dim3 grid((Tp + 63) / 64, B * Hkv);
    const size_t lds = sizeof(float) * 2 * 64 * (d + 1);
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)prefill_latent_kernel<T>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(prefill_latent_kernel<T>, grid, dim3(256), lds, st, k, v, wd, cK, cVt, Hkv,
                       d, dd, Tl, Tp, perm ? 1 : 0, geo.kv0, geo.Tkv, geo.lat0,
                       (const T*)geo.k_lat, (const T*)geo.v_lat, geo.cap);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_append_valu(const T* k_new, const T* v_new, const T* wd, T* k_win,
                                     T* v_win, T* k_lat, T* v_lat, int B, int Hkv, int d, int dd,
                                     int w, int cap, int len, int n, hipStream_t st) {
    dim3 grid((n + 63) / 64, B * Hkv);
    const size_t lds = sizeof(float) * 2 * 64 * (d + 1);
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)append_kernel<T>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    if (n <= w || w == 0) {
        hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), lds, st, k_new, v_new, wd, k_win,
                           v_win, k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), lds, st, k_new, v_new, wd, k_win, v_win,
                       k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(append_kernel<T>, grid, dim3(256), 0, st, k_new, v_new, wd, k_win, v_win,
                       k_lat, v_lat, Hkv, d, dd, w, cap, len, n, 2);
    return hipGetLastError();
}

// perm is set exactly when the matrix-core prefill consumes the workspace: it
// then needs the norms and constant rows even when no token is distant.
template <>
hipError_t launch_prefill_latent<bf16_t>(const bf16_t* k, const bf16_t* v, const bf16_t* wd,
                                         bf16_t* cK, bf16_t* cVt, float* cnorm, float* knorm,
                                         bf16_t* consts, int B, int Hkv, const PrefillGeo& geo,
                                         int d, int dd, int w, bool perm, hipStream_t st) {
    const int T_ = geo.total();
    const int Tl = T_ - w;
    const int Tp = prefill_tp(T_, w);
    if (!perm || !mfma_projection(d, dd)) {
        if (Tl <= 0) return hipSuccess;
        return launch_prefill_latent_valu<bf16_t>(k, v, wd, cK, cVt, B, Hkv, geo, d, dd, w, perm, st);
    }
    const int Tk = (T_ + 31) & ~31;
    const int ntok = Tp > Tk ? Tp : Tk;
    dim3 grid((ntok + 127) / 128, B * Hkv);
    auto kern = d == 64 ? prefill_latent_mfma_kernel<64> : prefill_latent_mfma_kernel<128>;
    hipLaunchKernelGGL(kern, grid, dim3(256), 0, st, k, v, wd, cK, cVt, cnorm, knorm, consts, Hkv,
                       T_, dd, Tl, Tp, geo.kv0, geo.Tkv, geo.lat0, (const bf16_t*)geo.k_lat,
                       (const bf16_t*)geo.v_lat, geo.cap, geo.seq_lens);
    return hipGetLastError();
}

template <>
hipError_t launch_append<bf16_t>(const bf16_t* k_new, const bf16_t* v_new, const bf16_t* wd,
                                 bf16_t* k_win, bf16_t* v_win, bf16_t* k_lat, bf16_t* v_lat, int B,
                                 int Hkv, int d, int dd, int w, int cap, int len, int n,
                                 hipStream_t st) {
    if (!mfma_projection(d, dd))
        return launch_append_valu<bf16_t>(k_new, v_new, wd, k_win, v_win, k_lat, v_lat, B, Hkv, d, dd, w, cap, len, n, st);
    dim3 grid((n + 31) / 32, B * Hkv);
    auto kern = (d == 64) ? append_mfma_kernel<64> : append_mfma_kernel<128>;
    if (n <= w || w == 0) {
        hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_lat, v_lat, Hkv, dd, w, cap, len, n, 0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_lat, v_lat, Hkv, dd, w, cap, len, n, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_lat, v_lat, Hkv, dd, w, cap, len, n, 2);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_prefill_latent(const T* k, const T* v, const T* wd, T* cK, T* cVt,
                                 float* cnorm, float* knorm, T* consts, int B, int Hkv,
                                 const PrefillGeo& geo, int d, int dd, int w, bool perm,
                                 hipStream_t st) {
    (void)cnorm;   // only the matrix-core prefill reads the norms
    (void)knorm;
    (void)consts;  // and the constant rows
    if (geo.total() - w <= 0) return hipSuccess;
    return launch_prefill_latent_valu<T>(k, v, wd, cK, cVt, B, Hkv, geo, d, dd, w, perm, st);
}

// One thread per 4-byte word of a context row; positions below len come from
// the ring (slot p % w), the others from the new tokens.
template <typename T>
__global__ __launch_bounds__(256) void chunk_gather_kernel(
    const T* __restrict__ k_win, const T* __restrict__ v_win, const T* __restrict__ k_new,
    const T* __restrict__ v_new, T* __restrict__ ctx_k, T* __restrict__ ctx_v, int d, int w,
    int len, int n, int kv0, int Tc) {
    const int bg = wg_id_y();
    const int words = d * (int)sizeof(T) / 4;  // d * esize is a multiple of 4
    const long long idx = (long long)wg_id_x() * 256 + lane_id_x();
    if (idx >= (long long)Tc * words) return;
    const int r = (int)(idx / words), wd4 = (int)(idx - (long long)r * words);
    const int p = kv0 + r;
    const size_t src_row = p < len ? (size_t)bg * w + p % w : (size_t)bg * n + (p - len);
    const uint32_t* sk = reinterpret_cast<const uint32_t*>(p < len ? k_win : k_new) + src_row * words;
    const uint32_t* sv = reinterpret_cast<const uint32_t*>(p < len ? v_win : v_new) + src_row * words;
    const size_t dst = ((size_t)bg * Tc + r) * words + wd4;
    reinterpret_cast<uint32_t*>(ctx_k)[dst] = sk[wd4];
    reinterpret_cast<uint32_t*>(ctx_v)[dst] = sv[wd4];
}

template <typename T>
hipError_t launch_chunk_gather(const T* k_win, const T* v_win, const T* k_new, const T* v_new,
                               T* ctx_k, T* ctx_v, int B, int Hkv, int d, int w, int len, int n,
                               int kv0, hipStream_t st) {
    const int Tc = len + n - kv0;
    const long long words = (long long)Tc * d * (long long)sizeof(T) / 4;
    dim3 grid((unsigned)((words + 255) / 256), B * Hkv);
    hipLaunchKernelGGL(chunk_gather_kernel<T>, grid, dim3(256), 0, st, k_win, v_win, k_new, v_new,
                       ctx_k, ctx_v, d, w, len, n, kv0, Tc);
    return hipGetLastError();
}

template hipError_t launch_chunk_gather<float>(const float*, const float*, const float*,
                                               const float*, float*, float*, int, int, int, int,
                                               int, int, int, hipStream_t);
template hipError_t launch_chunk_gather<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                                const bf16_t*, bf16_t*, bf16_t*, int, int, int,
                                                int, int, int, int, hipStream_t);

template <typename T>
hipError_t launch_append(const T* k_new, const T* v_new, const T* wd, T* k_win, T* v_win,
                         T* k_lat, T* v_lat, int B, int Hkv, int d, int dd, int w, int cap, int len,
                         int n, hipStream_t st) {
    return launch_append_valu<T>(k_new, v_new, wd, k_win, v_win, k_lat, v_lat, B, Hkv, d, dd, w, cap, len, n, st);
}

template hipError_t launch_prefill_latent<float>(const float*, const float*, const float*, float*,
                                                 float*, float*, float*, float*, int, int,
                                                 const PrefillGeo&, int, int, int, bool,
                                                 hipStream_t);
template hipError_t launch_append<float>(const float*, const float*, const float*, float*, float*,
                                         float*, float*, int, int, int, int, int, int, int, int,
                                         hipStream_t);

}  // namespace dar

namespace dar {

// Append with a single shared latent per token (its latent is given, one
// per token and KV head): grid (ceil(n / 64), B*Hkv), 256 threads; a block
// copies the latents of 64 consecutive tokens (positions len + t) into their
// slots (one contiguous run in both arrays), and the rows of those among the
// newest min(n, w) tokens into ring slots (len + t) % w. Plain copies, so the
// cache holds the given bits.
template <typename T>
__global__ __launch_bounds__(256) void append_shared_kernel(const T* __restrict__ k_new,
                                                            const T* __restrict__ v_new,
                                                            const T* __restrict__ c_new,
                                                            T* __restrict__ k_win, T* __restrict__ v_win,
                                                            T* __restrict__ lat, int d, int dd, int w,
                                                            int cap, int len, int n) {
    const int t0 = wg_id_x() * 64, bg = wg_id_y();
    const int tid = lane_id_x();
    const int nt = imin(64, n - t0);
    const T* cs = c_new + ((size_t)bg * n + t0) * dd;
    T* cd = lat + ((size_t)bg * cap + len + t0) * dd;
    for (int i = tid; i < nt * dd; i += 256) cd[i] = cs[i];
    if (w > 0) {
        const int first = imax(t0, n - imin(n, w));  // first token of this block bound for the ring
        for (int i = tid; i < (t0 + nt - first) * d; i += 256) {
            const int t = first + i / d, e = i - (i / d) * d;
            const size_t src = ((size_t)bg * n + t) * d + e;
            const size_t dst = ((size_t)bg * w + (len + t) % w) * d + e;
            k_win[dst] = k_new[src];
            v_win[dst] = v_new[src];
        }
    }
}

template <typename T>
hipError_t launch_append_shared(const T* k_new, const T* v_new, const T* c_new, T* k_win, T* v_win,
                                T* lat, int B, int Hkv, int d, int dd, int w, int cap, int len,
                                int n, hipStream_t st) {
    hipLaunchKernelGGL(append_shared_kernel<T>, dim3((n + 63) / 64, B * Hkv), dim3(256), 0, st, k_new,
                       v_new, c_new, k_win, v_win, lat, d, dd, w, cap, len, n);
    return hipGetLastError();
}

template hipError_t launch_append_shared<float>(const float*, const float*, const float*, float*,
                                                float*, float*, int, int, int, int, int, int, int,
                                                int, hipStream_t);
template hipError_t launch_append_shared<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                                 bf16_t*, bf16_t*, bf16_t*, int, int, int, int, int,
                                                 int, int, int, hipStream_t);

}  // namespace dar

namespace dar {

// Paged append, one token per sequence (grid B*Hkv, one wavefront each): the
// new token of sequence b sits at position len = lens[b]; the token leaving
// the window, ex = len - w (the new token itself when w = 0), is projected
// into its page slot with the same instruction sequence as the dense append
// (matrix cores: token in column 0), then the new token goes to ring slot
// len % w (after the read of the same slot). A sequence at capacity, or whose
// page is not mapped, stores nothing.
template <int D>
__global__ __launch_bounds__(64) void append_paged_mfma_kernel(
    const bf16_t* __restrict__ k_new, const bf16_t* __restrict__ v_new, const bf16_t* __restrict__ wd,
    bf16_t* k_win, bf16_t* v_win, bf16_t* __restrict__ k_pool, bf16_t* __restrict__ v_pool,
    PagedArgs pg, int Hkv, int dd, int w) {
    constexpr int KS = D / 16;
    const int bg = wg_id_x();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int lane = lane_id_x();
    const int tl = lane & 31, hg = lane >> 5;
    const int len = pg.lens[b];
    if (len < 0 || len >= pg.maxb * pg.ps) return;  // overflowed, or at capacity: nothing stored
    const int ex = len - w;
    int page = -1;
    if (ex >= 0) page = pg.bt[(size_t)b * pg.maxb + ex / pg.ps];
    const bool project = ex >= 0 && page >= 0 && page < pg.n_pages;
    lbf16x8 wa[KS];
    load_wd_operand<D>(wd + (size_t)g * D * dd, dd, lane, wa);
    for (int which = 0; which < 2; ++which) {
        const bf16_t* src_new = (which ? v_new : k_new) + (size_t)bg * D;
        bf16_t* ring = (which ? v_win : k_win) + (size_t)bg * w * D;
        const bf16_t* row = w > 0 ? ring + (size_t)(imax(ex, 0) % w) * D : src_new;
        lbf16x8 x[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s)
            x[s] = (project && tl == 0) ? lload8(row + s * 16 + hg * 8)
                                        : __builtin_bit_cast(lbf16x8, make_uint4(0, 0, 0, 0));
        const lf32x16 acc = project_mfma<D>(wa, x);
        if (project && tl == 0) {
            bf16_t* out = (which ? v_pool : k_pool) + (((size_t)page * Hkv + g) * pg.ps + ex % pg.ps) * dd;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int c = acc_col(r, hg);
                if (c < dd) out[c] = f32_to_bf16(acc[r]);
            }
        }
        if (w > 0 && tl == 0) {
            bf16_t* dst = ring + (size_t)(len % w) * D;
#pragma unroll
            for (int s = 0; s < KS; ++s)
                *reinterpret_cast<uint4*>(dst + s * 16 + hg * 8) = *reinterpret_cast<const uint4*>(src_new + s * 16 + hg * 8);
        }
    }
}

// The same for every dtype and head size, on the vector ALUs (project_col:
// the dense append's arithmetic). One workgroup of 64 per (batch, KV head).
template <typename T>
__global__ __launch_bounds__(64) void append_paged_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, const T* __restrict__ wd, T* k_win,
    T* v_win, T* __restrict__ k_pool, T* __restrict__ v_pool, PagedArgs pg, int Hkv, int d, int dd,
    int w) {
    const int bg = wg_id_x();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int lane = lane_id_x();
    const int len = pg.lens[b];
    if (len < 0 || len >= pg.maxb * pg.ps) return;  // overflowed, or at capacity: nothing stored
    const int ex = len - w;
    int page = -1;
    if (ex >= 0) page = pg.bt[(size_t)b * pg.maxb + ex / pg.ps];
    const bool project = ex >= 0 && page >= 0 && page < pg.n_pages;
    const T* wdg = wd + (size_t)g * d * dd;
    for (int which = 0; which < 2; ++which) {
        const T* src_new = (which ? v_new : k_new) + (size_t)bg * d;
        T* ring = (which ? v_win : k_win) + (size_t)bg * w * d;
        const T* row = w > 0 ? ring + (size_t)(imax(ex, 0) % w) * d : src_new;
        if (project) {
            T* out = (which ? v_pool : k_pool) + (((size_t)page * Hkv + g) * pg.ps + ex % pg.ps) * dd;
            for (int c = lane; c < dd; c += 64) out[c] = elem<T>::from_f32(project_col<T>(row, wdg, d, dd, c));
        }
        __syncthreads();  // every read of the ring slot before it is overwritten
        if (w > 0)
            for (int e = lane; e < d; e += 64) ring[(size_t)(len % w) * d + e] = src_new[e];
    }
}

// A sequence whose token could not be stored (at capacity) is marked as
// overflowed: its length becomes -1 - len (the held length stays readable),
// later appends leave it alone and the decode writes NaN for it.
__global__ __launch_bounds__(64) void lens_advance_kernel(int* __restrict__ lens, int B, int cap) {
    const int b = wg_id_x() * 64 + lane_id_x();
    if (b < B) {
        const int len = lens[b];
        if (len >= 0 && len < cap) lens[b] = len + 1;
        else if (len >= cap) lens[b] = -1 - len;
    }
}

template <typename T>
hipError_t launch_append_paged(const T* k_new, const T* v_new, const T* wd, T* k_win, T* v_win,
                               T* k_pool, T* v_pool, const PagedArgs& pg, int* lens, int B, int Hkv,
                               int d, int dd, int w, hipStream_t st) {
    if (sizeof(T) == 2 && mfma_projection(d, dd)) {
        auto kern = d == 64 ? append_paged_mfma_kernel<64> : append_paged_mfma_kernel<128>;
        hipLaunchKernelGGL(kern, dim3(B * Hkv), dim3(64), 0, st, (const bf16_t*)k_new,
                           (const bf16_t*)v_new, (const bf16_t*)wd, (bf16_t*)k_win, (bf16_t*)v_win,
                           (bf16_t*)k_pool, (bf16_t*)v_pool, pg, Hkv, dd, w);
    } else {
        hipLaunchKernelGGL(append_paged_kernel<T>, dim3(B * Hkv), dim3(64), 0, st, k_new, v_new, wd,
                           k_win, v_win, k_pool, v_pool, pg, Hkv, d, dd, w);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // after every workgroup above has read lens (stream order)
    hipLaunchKernelGGL(lens_advance_kernel, dim3((B + 63) / 64), dim3(64), 0, st, lens, B,
                       pg.maxb * pg.ps);
    return hipGetLastError();
}

template hipError_t launch_append_paged<float>(const float*, const float*, const float*, float*,
                                               float*, float*, float*, const PagedArgs&, int*, int,
                                               int, int, int, int, hipStream_t);
template hipError_t launch_append_paged<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                                bf16_t*, bf16_t*, bf16_t*, bf16_t*, const PagedArgs&,
                                                int*, int, int, int, int, int, hipStream_t);

}  // namespace dar

namespace dar {

// ---------------------------------------------------------------------------
// Chunked prefill reading the cached latents in place. The chunk's own window
// exits are appended first (so every distant latent of its rows is in the
// cache), the context rows (window tokens of the ring, then the new ones) are
// gathered before that append overwrites the ring, and the norms below give
// the attention kernel its score bounds.

// Sum of squares of m bf16 values (m a multiple of 8, 16-byte aligned).
__device__ __forceinline__ float sq_sum_bf16(const bf16_t* p, int m) {
    float s = 0.f;
    for (int j = 0; j < m; j += 8) {
        const uint4 u = *reinterpret_cast<const uint4*>(p + j);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float lo = __uint_as_float(w4[q] << 16), hi = __uint_as_float(w4[q] & 0xffff0000u);
            s = __builtin_fmaf(lo, lo, s);
            s = __builtin_fmaf(hi, hi, s);
        }
    }
    return s;
}

// A sequence's geometry for this chunk: false when it takes no part (no new
// tokens) or the chunk does not fit (overflowed before, or past capacity).
__device__ __forceinline__ bool chunk_seq(const LatCache& lc, int b, int len, int n, int& L, int& nb) {
    L = len;
    nb = n;
    if (!lc.lens) return true;
    L = lc.lens[b];
    nb = lc.n_new ? imin(imax(lc.n_new[b], 0), n) : n;
    return nb > 0 && L >= 0 && L + nb <= lc.cap;
}

// Each wavefront takes kNormBlocks 32-position blocks of one (batch, KV head)
// (all its latent loads issued before the first reduction); lanes l and
// l + 32 take the two halves of the row of position 32 blk + l % 32.
constexpr int kNormBlocks = 8;

template <int DD>
__global__ __launch_bounds__(256) void chunk_norms_kernel(LatCache lc, const bf16_t* __restrict__ ctx_k,
                                                          int kst, float* __restrict__ cnorm,
                                                          float* __restrict__ knorm, int Hkv, int d,
                                                          int w, int len, int n, int nblk) {
    const int bg = wg_id_y();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int tid = lane_id_x(), lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int blk0 = (wg_id_x() * 4 + wave) * kNormBlocks;
    if (blk0 >= nblk) return;
    int L, nb;
    if (!chunk_seq(lc, b, len, n, L, nb)) return;
    const int T = L + nb, Td = imax(T - w, 0), kv0 = imax(L - w, 0);
    const int tl = lane & 31, hg = lane >> 5;
    constexpr int NL = DD / 16;  // 16-byte loads per half row
    // latent keys: every row of the wavefront's blocks requested at once
    // (unconditional loads from a clamped address, zeroed after: a load
    // under a branch would wait for all loads before it)
    uint4 u[kNormBlocks][NL];
    bool ok[kNormBlocks];
#pragma unroll
    for (int j = 0; j < kNormBlocks; ++j) {
        const int p = (blk0 + j) * 32 + tl;
        ok[j] = p < Td;
        size_t row = 0;
        if (lc.bt) {
            const int page = ok[j] ? lc.bt[(size_t)b * lc.maxb + (p >> lc.ps_shift)] : -1;
            ok[j] = ok[j] && page >= 0 && page < lc.n_pages;
            if (ok[j]) row = ((((size_t)page) * Hkv + g) << lc.ps_shift) + (p & ((1 << lc.ps_shift) - 1));
        } else if (ok[j]) {
            row = (size_t)bg * lc.cap + p;
        }
        const bf16_t* src = lc.k + row * DD + hg * (DD / 2);
#pragma unroll
        for (int h = 0; h < NL; ++h) u[j][h] = *reinterpret_cast<const uint4*>(src + 8 * h);
    }
#pragma unroll
    for (int j = 0; j < kNormBlocks; ++j) {
        const int blk = blk0 + j;
        if (blk < nblk && blk * 32 < Td) {  // wavefront-uniform
            float n2 = 0.f;
#pragma unroll
            for (int h = 0; h < NL; ++h) {
                const uint4 uu = ok[j] ? u[j][h] : make_uint4(0, 0, 0, 0);
                const uint32_t w4[4] = {uu.x, uu.y, uu.z, uu.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float lo = __uint_as_float(w4[q] << 16), hi = __uint_as_float(w4[q] & 0xffff0000u);
                    n2 = __builtin_fmaf(lo, lo, n2);
                    n2 = __builtin_fmaf(hi, hi, n2);
                }
            }
            n2 += __shfl_xor(n2, 32, 64);
            const float m = wave_max_dpp(n2);
            if (lane == 0) cnorm[(size_t)bg * lc.ncb + blk] = sqrtf(m);
        }
    }
    // context keys (the window and the chunk: a few blocks of each head)
    for (int j = 0; j < kNormBlocks; ++j) {
        const int blk = blk0 + j;
        if (blk < nblk && blk * 32 < T && blk * 32 + 31 >= kv0) {  // wavefront-uniform
            const int p = blk * 32 + tl;
            float n2 = 0.f;
            if (p < T && p >= kv0)
                n2 = sq_sum_bf16(ctx_k + ((size_t)bg * kst + (p - kv0)) * d + hg * (d / 2), d / 2);
            n2 += __shfl_xor(n2, 32, 64);
            const float m = wave_max_dpp(n2);
            if (lane == 0) knorm[(size_t)bg * lc.nkb + blk] = sqrtf(m);
        }
    }
}

hipError_t launch_chunk_norms(const LatCache& lc, const bf16_t* ctx_k, int kst, float* cnorm,
                              float* knorm, int B, int Hkv, int d, int dd, int w, int len, int n,
                              int nblk, hipStream_t st) {
    if (nblk <= 0) return hipSuccess;
    const int per_wg = 4 * kNormBlocks;
    auto kern = dd == 16 ? chunk_norms_kernel<16> : chunk_norms_kernel<32>;
    hipLaunchKernelGGL(kern, dim3((nblk + per_wg - 1) / per_wg, B * Hkv), dim3(256), 0, st, lc, ctx_k, kst,
                       cnorm, knorm, Hkv, d, w, len, n, nblk);
    return hipGetLastError();
}

// Paged chunk context rows, one thread per 4-byte word: row r of sequence b's
// block holds position kv0 + r (kv0 = max(0, lens[b] - w)), from ring slot
// (kv0 + r) % w below lens[b], else the new token kv0 + r - lens[b].
__global__ __launch_bounds__(256) void chunk_gather_paged_kernel(
    const bf16_t* __restrict__ k_win, const bf16_t* __restrict__ v_win, const bf16_t* __restrict__ k_new,
    const bf16_t* __restrict__ v_new, bf16_t* __restrict__ ctx_k, bf16_t* __restrict__ ctx_v, LatCache lc,
    int Hkv, int d, int w, int n) {
    const int bg = wg_id_y(), b = bg / Hkv;
    int L, nb;
    if (!chunk_seq(lc, b, 0, n, L, nb)) return;
    const int kv0 = imax(L - w, 0);
    const int Tc = L + nb - kv0;
    const int words = d / 2;
    const int idx = wg_id_x() * 256 + lane_id_x();
    if (idx >= Tc * words) return;
    const int r = idx / words, wd4 = idx - (idx / words) * words;
    const int p = kv0 + r;
    const size_t src_row = p < L ? (size_t)bg * w + p % w : (size_t)bg * n + (p - L);
    const uint32_t* sk = reinterpret_cast<const uint32_t*>(p < L ? k_win : k_new) + src_row * words;
    const uint32_t* sv = reinterpret_cast<const uint32_t*>(p < L ? v_win : v_new) + src_row * words;
    const size_t dst = ((size_t)bg * (w + n) + r) * words + wd4;
    reinterpret_cast<uint32_t*>(ctx_k)[dst] = sk[wd4];
    reinterpret_cast<uint32_t*>(ctx_v)[dst] = sv[wd4];
}

hipError_t launch_chunk_gather_paged(const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_new,
                                     const bf16_t* v_new, bf16_t* ctx_k, bf16_t* ctx_v,
                                     const LatCache& lc, int B, int Hkv, int d, int w, int n,
                                     hipStream_t st) {
    const long long words = (long long)(w + n) * (d / 2);
    hipLaunchKernelGGL(chunk_gather_paged_kernel, dim3((unsigned)((words + 255) / 256), B * Hkv), dim3(256), 0,
                       st, k_win, v_win, k_new, v_new, ctx_k, ctx_v, lc, Hkv, d, w, n);
    return hipGetLastError();
}

// Paged chunk append (matrix-core projection): one wavefront per 32 new
// tokens of one (sequence, KV head), the modes of append_mfma_kernel (0:
// project and ring, safe when n <= w: the lane that reads a ring slot is the
// one that rewrites it; 1: project only; 2: ring only). The window exit of
// new token tt is position lens[b] + tt - w, written to its page slot.
template <int D>
__global__ __launch_bounds__(64) void append_chunk_paged_mfma_kernel(
    const bf16_t* __restrict__ k_new, const bf16_t* __restrict__ v_new, const bf16_t* __restrict__ wd,
    bf16_t* k_win, bf16_t* v_win, bf16_t* __restrict__ k_pool, bf16_t* __restrict__ v_pool, LatCache lc,
    int Hkv, int dd, int w, int n, int mode) {
    constexpr int KS = D / 16;
    const int bg = wg_id_y();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    int L, nb;
    if (!chunk_seq(lc, b, 0, n, L, nb)) return;
    const int lane = lane_id_x();
    const int tl = lane & 31, hg = lane >> 5;
    const int tt = wg_id_x() * 32 + tl;  // new token index
    const int ex = L + tt - w;           // position leaving the window
    const bool valid = tt < nb;
    int page = -1;
    if (mode != 2 && valid && ex >= 0) page = lc.bt[(size_t)b * lc.maxb + (ex >> lc.ps_shift)];
    const bool project = mode != 2 && valid && ex >= 0 && page >= 0 && page < lc.n_pages;
    const bool to_ring = mode != 1 && valid && w > 0 && tt >= nb - w;
    lbf16x8 wa[KS];
    if (mode != 2) load_wd_operand<D>(wd + (size_t)g * D * dd, dd, lane, wa);
    for (int which = 0; which < 2; ++which) {
        const bf16_t* src_new = (which ? v_new : k_new) + (size_t)bg * n * D;
        bf16_t* ring = (which ? v_win : k_win) + (size_t)bg * w * D;
        if (mode != 2) {
            const bf16_t* row = src_new;
            if (project) row = (ex < L) ? ring + (size_t)(ex % w) * D : src_new + (size_t)(ex - L) * D;
            lbf16x8 x[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                x[s] = lload8(row + s * 16 + hg * 8);
                if (!project) x[s] = __builtin_bit_cast(lbf16x8, make_uint4(0, 0, 0, 0));
            }
            const lf32x16 acc = project_mfma<D>(wa, x);
            if (project) {
                bf16_t* out = (which ? v_pool : k_pool) +
                              (((((size_t)page) * Hkv + g) << lc.ps_shift) + (ex & ((1 << lc.ps_shift) - 1))) * dd;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int c = acc_col(r, hg);
                    if (c < dd) out[c] = f32_to_bf16(acc[r]);
                }
            }
        }
        if (to_ring) {
            const bf16_t* src = src_new + (size_t)tt * D;
            bf16_t* dst = ring + (size_t)((L + tt) % w) * D;
#pragma unroll
            for (int s = 0; s < KS; ++s)
                *reinterpret_cast<uint4*>(dst + s * 16 + hg * 8) = *reinterpret_cast<const uint4*>(src + s * 16 + hg * 8);
        }
    }
}

hipError_t launch_append_chunk_paged(const bf16_t* k_new, const bf16_t* v_new, const bf16_t* wd,
                                     bf16_t* k_win, bf16_t* v_win, bf16_t* k_pool, bf16_t* v_pool,
                                     const LatCache& lc, int B, int Hkv, int d, int dd, int w, int n,
                                     hipStream_t st) {
    if (!mfma_projection(d, dd)) return hipErrorNotSupported;
    dim3 grid((n + 31) / 32, B * Hkv);
    auto kern = (d == 64) ? append_chunk_paged_mfma_kernel<64> : append_chunk_paged_mfma_kernel<128>;
    if (n <= w || w == 0) {
        hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_pool, v_pool, lc, Hkv,
                           dd, w, n, 0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_pool, v_pool, lc, Hkv, dd,
                       w, n, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, dim3(64), 0, st, k_new, v_new, wd, k_win, v_win, k_pool, v_pool, lc, Hkv, dd,
                       w, n, 2);
    return hipGetLastError();
}

__global__ __launch_bounds__(64) void lens_advance_n_kernel(int* __restrict__ lens,
                                                            const int* __restrict__ n_new, int B,
                                                            int cap, int n) {
    const int b = wg_id_x() * 64 + lane_id_x();
    if (b >= B) return;
    const int nb = n_new ? imin(imax(n_new[b], 0), n) : n;
    if (nb == 0) return;
    const int L = lens[b];
    if (L >= 0 && L + nb <= cap) lens[b] = L + nb;
    else if (L >= 0) lens[b] = -1 - L;
}

hipError_t launch_lens_advance(int* lens, const int* n_new, int B, int cap, int n, hipStream_t st) {
    hipLaunchKernelGGL(lens_advance_n_kernel, dim3((B + 63) / 64), dim3(64), 0, st, lens, n_new, B, cap, n);
    return hipGetLastError();
}

}  // namespace dar
