// Split-KV DAR decode over the split cache (Limitations section: the last w
// tokens at full d in a ring, every older token as its d_down latent).
//
// Stage 1 (decode_split_kernel): one block per (batch, KV head, split). A
// split is a run of consecutive tokens of one region: latent tokens
// [0, len - w) are read from k_lat/v_lat and scored with q~ = q W_up^T
// (W_up absorbed into the query); window tokens [len - w, len) are read from
// the ring and scored with q. All G = Hq/Hkv query heads of the KV head are
// handled by the block, so every cache byte is read once per step. Two
// passes over the split: keys (scores kept in LDS, exact per-head max), then
// values with p = exp2(s - max). Output per (head, split): {m, l, acc} with
// acc in d_down space for latent splits and in d space for window splits.
//
// Stage 2 (decode_combine_kernel): one wavefront per (batch, query head)
// merges the partial records under one max (Eq. 4 is a single softmax over
// both regions) and lifts the latent part once, o = (o_win + o_lat W_up) / l.
#include "dar_common.hpp"
#include "dar_kernels.hpp"

namespace dar {

static constexpr int kDecThreads = 256;
static constexpr int kDecScoreSlots = 8192;  // G * tokens-per-split scores in LDS

// Each lane owns an 8-element segment of a row; lanes_per_token lanes cover
// one row. Loads are 16-byte vectors when the segment is whole.
template <typename T>
__device__ __forceinline__ void load_seg(const T* __restrict__ row, int off, int dim, bool vec,
                                         float (&x)[8]);

template <>
__device__ __forceinline__ void load_seg<bf16_t>(const bf16_t* __restrict__ row, int off, int dim,
                                                 bool vec, float (&x)[8]) {
    if (vec) {
        const uint4 u = *reinterpret_cast<const uint4*>(row + off);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            x[2 * j] = __uint_as_float(w4[j] << 16);
            x[2 * j + 1] = __uint_as_float(w4[j] & 0xffff0000u);
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = (off + j < dim) ? bf16_to_f32(row[off + j]) : 0.f;
    }
}

template <>
__device__ __forceinline__ void load_seg<float>(const float* __restrict__ row, int off, int dim,
                                                bool vec, float (&x)[8]) {
    if (vec) {
        const float4 a = *reinterpret_cast<const float4*>(row + off);
        const float4 b = *reinterpret_cast<const float4*>(row + off + 4);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = (off + j < dim) ? row[off + j] : 0.f;
    }
}

static __host__ __device__ inline int lanes_per_row(int dim) {
    int lpt = 1;
    while (lpt * 8 < dim) lpt <<= 1;
    return lpt;
}

template <typename T, int G>
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(
    const T* __restrict__ q, const T* __restrict__ wd, const T* __restrict__ wu,
    const T* __restrict__ k_win, const T* __restrict__ v_win, const T* __restrict__ k_lat,
    const T* __restrict__ v_lat, float* __restrict__ part, int Hq, int Hkv, int d, int dd, int w,
    int cap, int len, int chunk_lat, int chunk_win, int n_lat_split, int S, float qscale) {
    static_assert(4 * G * 256 <= kDecScoreSlots, "partial sums must fit in the score buffer");
    __shared__ float qsh[G][256];
    __shared__ float ssh[kDecScoreSlots];
    __shared__ float mred[4][G];
    // after pass 2 the score buffer holds the cross-wave partial sums
    float (*red)[G][256] = reinterpret_cast<float (*)[G][256]>(ssh);

    const int s = wg_id_x();
    const int bg = wg_id_y();
    const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
    const int tid = lane_id_x();
    const int lane = tid & 63, wave = tid >> 6;
    const int n_lat = imax(0, len - w);
    const bool latent = s < n_lat_split;
    const int dim = latent ? dd : d;
    int t_begin, ntok;
    if (latent) {
        t_begin = s * chunk_lat;
        ntok = imin(chunk_lat, n_lat - t_begin);
    } else {
        t_begin = n_lat + (s - n_lat_split) * chunk_win;
        ntok = imin(chunk_win, len - t_begin);
    }
    const T* wdg = wd + (size_t)g * d * dd;
    const T* wug = wu ? wu + (size_t)g * dd * d : nullptr;

    // query (window region) or absorbed query q W_up^T (latent region),
    // scaled by log2(e)/sqrt(d)
    for (int idx = tid; idx < G * dim; idx += kDecThreads) {
        const int hh = idx / dim, c = idx - (idx / dim) * dim;
        const T* qrow = q + ((size_t)b * Hq + (size_t)g * G + hh) * d;
        float acc;
        if (latent) {
            acc = 0.f;
            for (int e = 0; e < d; ++e) {
                const float u = wug ? elem<T>::load(wug + (size_t)c * d + e)
                                    : elem<T>::load(wdg + (size_t)e * dd + c);
                acc = __builtin_fmaf(elem<T>::load(qrow + e), u, acc);
            }
        } else {
            acc = elem<T>::load(qrow + c);
        }
        qsh[hh][c] = acc * qscale;
    }
    __syncthreads();

    const int lpt = lanes_per_row(dim);
    const int sub = tid & (lpt - 1);
    const int tpi = kDecThreads / lpt;  // tokens per block iteration
    const int off = sub * 8;
    const bool vec = (dim % 8) == 0 && off < dim;
    float qreg[G][8];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int j = 0; j < 8; ++j) qreg[hh][j] = (off + j < dim) ? qsh[hh][off + j] : 0.f;

    const T* kbase = latent ? k_lat + (size_t)bg * cap * dd : k_win + (size_t)bg * w * d;
    const T* vbase = latent ? v_lat + (size_t)bg * cap * dd : v_win + (size_t)bg * w * d;
    auto row_of = [&](const T* base, int t) -> const T* {
        const int pos = t_begin + t;
        return latent ? base + (size_t)pos * dd : base + (size_t)(pos % w) * d;
    };

    // pass 1: scores
    float mloc[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) mloc[hh] = -INFINITY;
    for (int t0 = 0; t0 < ntok; t0 += tpi) {
        const int t = t0 + tid / lpt;
        float x[8];
        if (t < ntok) load_seg<T>(row_of(kbase, t), off, dim, vec, x);
        else {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = 0.f;
        }
        float sc[G];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) a = __builtin_fmaf(qreg[hh][j], x[j], a);
            for (int o2 = 1; o2 < lpt; o2 <<= 1) a += __shfl_xor(a, o2, 64);
            sc[hh] = a;
        }
        if (t < ntok) {
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                mloc[hh] = fmaxf(mloc[hh], sc[hh]);
                if (sub == 0) ssh[hh * (kDecScoreSlots / G) + t] = sc[hh];
            }
        }
    }
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        const float mw = wave_max(mloc[hh]);
        if (lane == 0) mred[wave][hh] = mw;
    }
    __syncthreads();
    float mx[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
        mx[hh] = fmaxf(fmaxf(mred[0][hh], mred[1][hh]), fmaxf(mred[2][hh], mred[3][hh]));

    // pass 2: values
    float acc[G][8];
    float lsum[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        lsum[hh] = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[hh][j] = 0.f;
    }
    for (int t0 = 0; t0 < ntok; t0 += tpi) {
        const int t = t0 + tid / lpt;
        if (t < ntok) {
            float x[8];
            load_seg<T>(row_of(vbase, t), off, dim, vec, x);
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                const float p = exp2f(ssh[hh * (kDecScoreSlots / G) + t] - mx[hh]);
                if (sub == 0) lsum[hh] += p;
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[hh][j] = __builtin_fmaf(p, x[j], acc[hh][j]);
            }
        }
    }
    // reduce over the lanes that share a segment (same sub), then over waves
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        lsum[hh] = wave_sum(lsum[hh]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float a = acc[hh][j];
            for (int o2 = lpt; o2 < 64; o2 <<= 1) a += __shfl_xor(a, o2, 64);
            acc[hh][j] = a;
        }
    }
    __syncthreads();  // scores and mred are reused below
    if (lane < lpt) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (off + j < dim) red[wave][hh][off + j] = acc[hh][j];
    }
    if (lane == 0) {
#pragma unroll
        for (int hh = 0; hh < G; ++hh) mred[wave][hh] = lsum[hh];
    }
    __syncthreads();
    // partial record {m, l, acc_lat[dd], acc_win[d]}: this split fills the
    // part of its region and zeroes the other
    const int stride = 2 + dd + d;
    const int lo = latent ? 2 : 2 + dd;
    for (int idx = tid; idx < G * stride; idx += kDecThreads) {
        const int hh = idx / stride, f = idx - (idx / stride) * stride;
        float val = 0.f;
        if (f == 0) val = mx[hh];
        else if (f == 1) val = mred[0][hh] + mred[1][hh] + mred[2][hh] + mred[3][hh];
        else if (f >= lo && f < lo + dim)
            val = red[0][hh][f - lo] + red[1][hh][f - lo] + red[2][hh][f - lo] + red[3][hh][f - lo];
        const size_t bh = (size_t)b * Hq + (size_t)g * G + hh;
        part[(bh * S + s) * stride + f] = val;
    }
}

// One wavefront per (batch, query head) merges its S partial records
// {m, l, acc_lat[dd], acc_win[d]} under one maximum (Eq. 4 is a single
// softmax over both regions), lifts the latent part once and normalises:
// o = (acc_win + acc_lat W_up) / l. Every global load of a phase is
// independent of the others, so each phase costs one memory round trip: the
// W_up column of the lane is fetched first, split weights are broadcast from
// the lane that owns the split, and partial rows are read eight at a time.
// NR: output columns per lane (lane + 64 r, r < NR; d <= 64 NR).
template <typename T, int NR>
__global__ __launch_bounds__(64) void decode_combine_kernel(
    const float* __restrict__ part, const T* __restrict__ wd, const T* __restrict__ wu,
    T* __restrict__ o, int Hq, int Hkv, int d, int dd, int S_all, const T* __restrict__ wv,
    const int* __restrict__ lens, const int* __restrict__ counts) {
    constexpr int kLiftCols = 32;  // W_up rows held in registers (d_down <= 32)
    const int bh = wg_id_x();
    const int h = bh % Hq;
    const int g = h / (Hq / Hkv);
    // records per head: S_all, or (a paged batch) the records the decode
    // kernel wrote for this (sequence, KV head)
    const int S = lens ? imin(S_all, counts[(bh / Hq) * Hkv + g]) : S_all;
    if (lens && lens[bh / Hq] < 1) {
        // an empty or overflowed sequence (paged batch): no query position, NaN
        for (int e = lane_id_x(); e < d; e += 64) {
            if (sizeof(T) == 2) reinterpret_cast<uint16_t*>(o)[(size_t)bh * d + e] = 0x7fc0;
            else reinterpret_cast<uint32_t*>(o)[(size_t)bh * d + e] = 0x7fc00000u;
        }
        return;
    }
    if (lens && S <= 1) return;
    const int lane = lane_id_x();
    const int stride = 2 + dd + d;
    const float* pp = part + (size_t)bh * S_all * stride;
    const T* wdg = wd + (size_t)g * d * dd;
    // the lift's matrix: W_up (W_down^T when tied), or (shared latent) the
    // value matrix
    const T* wug = wv ? wv + (size_t)g * dd * d : (wu ? wu + (size_t)g * dd * d : nullptr);
    const bool lift_regs = dd <= kLiftCols;

    // the lane's W_up columns: every load issued before any is used, none
    // under a branch (clamped addresses; the values past d_down are zeroed)
    const int wstep = wug ? d : 1;  // distance between consecutive latent columns c
    const int cmax = imin(dd, kLiftCols) - 1;
    float wcol[NR][kLiftCols];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int e = imin(lane + 64 * r, d - 1);
        const T* wp = wug ? wug + e : wdg + (size_t)e * dd;
#pragma unroll
        for (int c = 0; c < kLiftCols; ++c) wcol[r][c] = elem<T>::load(wp + (size_t)imin(c, cmax) * wstep);
    }
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int c = 0; c < kLiftCols; ++c)
            if (c >= dd) wcol[r][c] = 0.f;

    // (d_down <= d <= 64 NR: the lane's columns are lane + 64 r, r < NR.)
    // The first kFirst records' rows and the first 64 records' {m, l},
    // requested together (clamped addresses, no load under a branch), so that
    // a merge of few records costs one memory round trip after W_up.
    constexpr int kFirst = 8;
    const int n0 = imin(S, kFirst);
    float al0[kFirst][NR], aw0[kFirst][NR];
#pragma unroll
    for (int j = 0; j < kFirst; ++j) {
        const float* row = pp + (size_t)imin(j, n0 - 1) * stride + 2;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int e = lane + 64 * r;
            al0[j][r] = row[imin(e, dd - 1)];
            aw0[j][r] = row[dd + imin(e, d - 1)];
        }
    }
    const int s_ml = imin(lane, S - 1);
    const float m_l = pp[(size_t)s_ml * stride], l_l = pp[(size_t)s_ml * stride + 1];

    // split weights: w_s = 2^(m_s - M), L = sum_s w_s l_s
    float M = lane < S ? m_l : -INFINITY;
    for (int s = lane + 64; s < S; s += 64) M = fmaxf(M, pp[(size_t)s * stride]);
    M = wave_max(M);
    float L = lane < S && m_l != -INFINITY ? exp2f(m_l - M) * l_l : 0.f;
    for (int s = lane + 64; s < S; s += 64) {
        const float ms = pp[(size_t)s * stride];
        if (ms != -INFINITY) L += exp2f(ms - M) * pp[(size_t)s * stride + 1];
    }
    L = wave_sum(L);
    const float inv = 1.f / L;

    // lane owns latent columns lane + 64 r (< dd) and window columns lane + 64 r (< d)
    float lat[4] = {0.f, 0.f, 0.f, 0.f};
    float win[4] = {0.f, 0.f, 0.f, 0.f};
    {
        const float w0 = lane < S && m_l != -INFINITY ? exp2f(m_l - M) : 0.f;
#pragma unroll
        for (int j = 0; j < kFirst; ++j) {
            const float ws = j < n0 ? __shfl(w0, j, 64) : 0.f;
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const int e = lane + 64 * r;
                lat[r] = __builtin_fmaf(ws, e < dd ? al0[j][r] : 0.f, lat[r]);
                win[r] = __builtin_fmaf(ws, e < d ? aw0[j][r] : 0.f, win[r]);
            }
        }
    }
    // the records past the first kFirst
    for (int s0 = 0; s0 < S; s0 += 64) {
        float wl = 0.f;  // weight of split s0 + lane, broadcast below
        if (s0 + lane < S) {
            const float ms = pp[(size_t)(s0 + lane) * stride];
            wl = ms == -INFINITY ? 0.f : exp2f(ms - M);
        }
        const int ns = imin(64, S - s0);
        for (int j0 = s0 == 0 ? kFirst : 0; j0 < ns; j0 += 8) {
            float al[8][4], aw[8][4];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float* row = pp + (size_t)(s0 + imin(j0 + j, ns - 1)) * stride + 2;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int e = lane + 64 * r;
                    al[j][r] = e < dd ? row[e] : 0.f;
                    aw[j][r] = e < d ? row[dd + e] : 0.f;
                }
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float ws = (j0 + j < ns) ? __shfl(wl, j0 + j, 64) : 0.f;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    lat[r] = __builtin_fmaf(ws, al[j][r], lat[r]);
                    win[r] = __builtin_fmaf(ws, aw[j][r], win[r]);
                }
            }
        }
    }
    if (lift_regs) {
        float acc[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) acc[r] = win[r];
        // (columns past d_down add zero: their W_up values are zeroed)
#pragma unroll
        for (int c = 0; c < kLiftCols; ++c) {
            const float lc = __shfl(lat[0], c, 64);
#pragma unroll
            for (int r = 0; r < NR; ++r) acc[r] = __builtin_fmaf(lc, wcol[r][c], acc[r]);
        }
#pragma unroll
        for (int r = 0; r < NR; ++r)
            if (lane + 64 * r < d) o[(size_t)bh * d + lane + 64 * r] = elem<T>::from_f32(acc[r] * inv);
        return;
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int e = lane + 64 * r;
        float acc = win[r];
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2)
#pragma unroll 8
            for (int c2 = 0; c2 < 64 && 64 * r2 + c2 < dd; ++c2) {
                const int c = 64 * r2 + c2;
                const float lc = __shfl(lat[r2], c2, 64);
                const float u = wug ? elem<T>::load(wug + (size_t)c * d + (e < d ? e : 0))
                                    : elem<T>::load(wdg + (size_t)(e < d ? e : 0) * dd + c);
                acc = __builtin_fmaf(lc, u, acc);
            }
        if (e < d) o[(size_t)bh * d + e] = elem<T>::from_f32(acc * inv);
    }
}

template <typename T>
hipError_t launch_decode_combine(const float* part, const T* wd, const T* wu, T* o, int B, int Hq,
                                 int Hkv, int d, int dd, int S, hipStream_t st, const T* wv,
                                 const int* lens, const int* counts) {
#define DAR_COMBINE(NR_)                                                                          \
    hipLaunchKernelGGL((decode_combine_kernel<T, NR_>), dim3(B * Hq), dim3(64), 0, st, part, wd, wu, \
                       o, Hq, Hkv, d, dd, S, wv, lens, counts)
    if (d <= 64) DAR_COMBINE(1);
    else if (d <= 128) DAR_COMBINE(2);
    else DAR_COMBINE(4);
#undef DAR_COMBINE
    return hipGetLastError();
}
template hipError_t launch_decode_combine<float>(const float*, const float*, const float*, float*,
                                                 int, int, int, int, int, int, hipStream_t,
                                                 const float*, const int*, const int*);
template hipError_t launch_decode_combine<bf16_t>(const float*, const bf16_t*, const bf16_t*,
                                                  bf16_t*, int, int, int, int, int, int,
                                                  hipStream_t, const bf16_t*, const int*,
                                                  const int*);

static int group_chunk(int G) { return kDecScoreSlots / G; }

DecodeSplits decode_splits(int len, int w, int d, int dd, int G) {
    DecodeSplits sp;
    const int n_lat = len - w > 0 ? len - w : 0;
    const int n_win = len - n_lat;
    const int cmax = group_chunk(G);
    // about 64 KB of keys+values per split in each region
    int cl = 65536 / (4 * (dd > 0 ? dd : 1));
    int cw = 65536 / (4 * d);
    cl = cl < 64 ? 64 : (cl > cmax ? cmax : cl);
    cw = cw < 64 ? 64 : (cw > cmax ? cmax : cw);
    sp.chunk_lat = cl;
    sp.chunk_win = cw;
    sp.n_lat_split = (n_lat + cl - 1) / cl;
    sp.n_win_split = (n_win + cw - 1) / cw;
    return sp;
}

int decode_max_partials(int B, int Hkv, int cap, int w, int d, int dd, int G) {
    // both counts grow with the cache length: bound them at len = cap
    DecodeSplits a = decode_splits(cap, w, d, dd, G);
    DecodeSplits b = decode_splits(cap, 0, d, dd, G);
    int m = a.n_lat_split + a.n_win_split;
    m = m > b.n_lat_split + b.n_win_split ? m : b.n_lat_split + b.n_win_split;
    int p = decode_mfma_parts(B, Hkv, cap, w, d);
    if (dd == 16 || dd == 32) {  // a paged decode of this shape
        const int ps = decode_paged_slots(Hkv, cap, w, d, dd);
        p = p > ps ? p : ps;
    }
    return m > p ? m : p;
}

int decode_partials_at(int B, int Hkv, int len, int w, int d, int dd, int G, bool bf16) {
    // the same choice of path and split count as launch_decode below
    if (decode_mfma_supported(d, dd, G, bf16)) {
        const int P = decode_mfma_parts(B, Hkv, len, w, d);
        return P > 1 ? P : 0;
    }
    const DecodeSplits sp = decode_splits(len, w, d, dd, G);
    return sp.n_lat_split + sp.n_win_split;
}

template <typename T, int G>
static hipError_t launch_decode_g(const T* q, const T* wd, const T* wu, const T* k_win,
                                  const T* v_win, const T* k_lat, const T* v_lat, T* o,
                                  float* part, int B, int Hq, int Hkv, int d, int dd, int w,
                                  int cap, int len, hipStream_t st, const T* wv) {
    DecodeSplits sp = decode_splits(len, w, d, dd, G);
    const int S = sp.n_lat_split + sp.n_win_split;
    const float qscale = 1.4426950408889634f / sqrtf((float)d);
    hipLaunchKernelGGL((decode_split_kernel<T, G>), dim3(S, B * Hkv), dim3(kDecThreads), 0, st, q,
                       wd, wu, k_win, v_win, k_lat, v_lat, part, Hq, Hkv, d, dd, w, cap, len,
                       sp.chunk_lat, sp.chunk_win, sp.n_lat_split, S, qscale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_decode_combine<T>(part, wd, wu, o, B, Hq, Hkv, d, dd, S, st, wv, nullptr, 0);
}

template <typename T>
hipError_t launch_decode(const T* q, const T* wd, const T* wu, const T* k_win, const T* v_win,
                         const T* k_lat, const T* v_lat, T* o, float* part, int B, int Hq, int Hkv,
                         int d, int dd, int w, int cap, int len, hipStream_t st, const T* wv) {
    if (decode_mfma_supported(d, dd, Hq / Hkv, sizeof(T) == 2)) {
        int P = 0;
        hipError_t e = launch_decode_mfma((const bf16_t*)q, (const bf16_t*)wd, (const bf16_t*)wu,
                                          (const bf16_t*)k_win, (const bf16_t*)v_win,
                                          (const bf16_t*)k_lat, (const bf16_t*)v_lat, part,
                                          (bf16_t*)o, B, Hq, Hkv, d, dd, w, cap, len, P, st,
                                          (const bf16_t*)wv);
        if (e != hipSuccess || P == 1) return e;
        return launch_decode_combine<T>(part, wd, wu, o, B, Hq, Hkv, d, dd, P, st, wv, nullptr, 0);
    }
    switch (Hq / Hkv) {
        case 1: return launch_decode_g<T, 1>(q, wd, wu, k_win, v_win, k_lat, v_lat, o, part, B, Hq, Hkv, d, dd, w, cap, len, st, wv);
        case 2: return launch_decode_g<T, 2>(q, wd, wu, k_win, v_win, k_lat, v_lat, o, part, B, Hq, Hkv, d, dd, w, cap, len, st, wv);
        case 4: return launch_decode_g<T, 4>(q, wd, wu, k_win, v_win, k_lat, v_lat, o, part, B, Hq, Hkv, d, dd, w, cap, len, st, wv);
        case 8: return launch_decode_g<T, 8>(q, wd, wu, k_win, v_win, k_lat, v_lat, o, part, B, Hq, Hkv, d, dd, w, cap, len, st, wv);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_decode<float>(const float*, const float*, const float*, const float*,
                                         const float*, const float*, const float*, float*, float*,
                                         int, int, int, int, int, int, int, int, hipStream_t,
                                         const float*);
template hipError_t launch_decode<bf16_t>(const bf16_t*, const bf16_t*, const bf16_t*,
                                          const bf16_t*, const bf16_t*, const bf16_t*,
                                          const bf16_t*, bf16_t*, float*, int, int, int, int, int,
                                          int, int, int, hipStream_t, const bf16_t*);

}  // namespace dar
