// C ABI of libdar: argument validation, workspace sizing, cache bookkeeping
// and kernel dispatch. Nothing is enqueued unless every check passes.
#include "../../include/dar.h"
#include "dar_kernels.hpp"

#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <mutex>

namespace dar {

PrefillWs prefill_ws_layout(int B, int Hkv, int T, int dd, int w, size_t esize) {
    PrefillWs ws{0, 0, 0, 0, 0, 0};
    const size_t Tp = (size_t)prefill_tp(T, w);
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    // c^K: Tp rows of dd; c^V^T: Tp/32 blocks of up to dd + 1 rows of 32
    const size_t kbytes = al((size_t)B * Hkv * Tp * dd * esize);
    const size_t vbytes = al((size_t)B * Hkv * Tp * (dd + 1) * esize);
    ws.ck_off = 0;
    ws.cv_off = kbytes;
    ws.norm_off = kbytes + vbytes;
    ws.knorm_off = ws.norm_off + al((size_t)B * Hkv * (Tp / 32) * sizeof(float));
    ws.const_off = ws.knorm_off + al((size_t)B * Hkv * ((T + 31) / 32) * sizeof(float));
    ws.bytes = ws.const_off + 256;
    return ws;
}

// Both fast paths (matrix-core prefill) and the generic kernels live in this
// library; the generic path handles everything the fast one does not.
bool prefill_mfma_supported(const dar_shape* s);
hipError_t launch_prefill_mfma(const dar_shape* s, const PrefillGeo& geo, const void* q, const void* k,
                               const void* v, const void* wd, const void* wu, void* o, float* lse,
                               const void* cK, const void* cVt, const float* cnorm,
                               const float* knorm, const void* consts, hipStream_t st,
                               const void* wv = nullptr);
bool prefill_mfma_rope_supported(const dar_shape* s);
// The attention kernel on a chunk (rows q0.., geo as for launch_prefill_mfma
// with k / v the context rows) with the distant latents read from lc; for a
// paged lc the per-sequence geometry comes from lc.lens / lc.n_new and geo.Tkv
// is the context rows' stride (w + n).
hipError_t launch_prefill_mfma_cache(const dar_shape* s, const PrefillGeo& geo, const LatCache& lc,
                                     const void* q, const void* ctx_k, const void* ctx_v,
                                     const void* wd, const void* wu, void* o, float* lse,
                                     const float* cnorm, const float* knorm, hipStream_t st);
// The matrix-core rotary attention over a chunk geometry (see PrefillGeo):
// qr the rotated chunk queries, kr / v the rotated keys and the values of the
// context rows (from geo.kv0), kd / vd the distant rows (positions 0..).
hipError_t launch_prefill_mfma_rope_geo(const dar_shape* s, const PrefillGeo& geo, const void* qr,
                                        const void* kr, const void* v, const void* kd,
                                        const void* vd, void* o, float* lse, const float* knorm,
                                        const float* dnorm, hipStream_t st);
hipError_t launch_prefill_mfma_rope(const dar_shape* s, int T, const void* qr, const void* kr,
                                    const void* v, const void* kd, const void* vd, void* o,
                                    float* lse, const float* knorm, const float* dnorm,
                                    hipStream_t st);

// Prefill workspace with rotary embedding: rotated queries and keys, the
// lifted-and-rotated distant keys and lifted values of positions < T - w,
// and the 32-row block norms of the two key arrays; 256-byte aligned parts.
struct RopeWs {
    size_t qr_off, kr_off, kd_off, vd_off, knorm_off, dnorm_off, bytes;
};

RopeWs rope_ws_layout(const dar_shape* s, int T) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t es = s->dtype == DAR_BF16 ? 2 : 4;
    const size_t Td = T > s->w ? (size_t)(T - s->w) : 0;
    RopeWs L{};
    L.qr_off = 0;
    L.kr_off = L.qr_off + al((size_t)s->B * s->Hq * T * s->d * es);
    L.kd_off = L.kr_off + al((size_t)s->B * s->Hkv * T * s->d * es);
    L.vd_off = L.kd_off + al((size_t)s->B * s->Hkv * Td * s->d * es);
    L.knorm_off = L.vd_off + al((size_t)s->B * s->Hkv * Td * s->d * es);
    L.dnorm_off = L.knorm_off + al((size_t)s->B * s->Hkv * ((T + 31) / 32) * sizeof(float));
    L.bytes = L.dnorm_off + al((size_t)s->B * s->Hkv * ((Td + 31) / 32) * sizeof(float)) + 256;
    return L;
}

}  // namespace dar

using namespace dar;

namespace {

bool log_enabled() {
    static int on = -1;
    if (on < 0) {
        const char* e = getenv("DAR_LOG");
        on = (e && e[0] == '1') ? 1 : 0;
    }
    return on == 1;
}

// An environment switch ("1" = on), read at each call. DAR_BWD_VALU=1 sends
// the backward to the vector-ALU kernels for every shape (used to test them
// on shapes the matrix-core kernels also cover).
bool env_flag(const char* name) {
    const char* e = getenv(name);
    return e && e[0] == '1';
}

size_t esize_of(dar_dtype t) { return t == DAR_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// A device tensor argument: non-NULL and 16-byte aligned.
bool dev_ok(const void* p) { return p != nullptr && aligned16(p); }

dar_status check_shape(const dar_shape* s) {
    if (!s) return DAR_E_ARG;
    if (s->B < 1 || s->Hq < 1 || s->Hkv < 1 || s->d < 1 || s->d_down < 1 || s->w < 0)
        return DAR_E_ARG;
    if (s->Hq % s->Hkv != 0) return DAR_E_ARG;
    if (s->d_down > s->d) return DAR_E_ARG;
    if (s->dtype != DAR_F32 && s->dtype != DAR_BF16) return DAR_E_ARG;
    if (s->d > 256) return DAR_E_UNSUPPORTED;
    if ((long long)s->B * s->Hq > 65535) return DAR_E_UNSUPPORTED;
    return DAR_OK;
}

bool group_supported(const dar_shape* s) {
    const int G = s->Hq / s->Hkv;
    return G == 1 || G == 2 || G == 4 || G == 8;
}

void clear_hip_error() { (void)hipGetLastError(); }

// Pre-pass and attention kernels of one prefill (whole sequence or chunk):
// k and v hold the positions geo describes, ws the prefill workspace laid out
// as L for geo.total() positions.
hipError_t run_prefill(const dar_shape* s, const PrefillGeo& geo, const void* q, const void* k,
                       const void* v, const void* w_down, const void* w_up, void* o, float* lse,
                       void* ws, const PrefillWs& L, bool fast, hipStream_t stream,
                       const void* w_val = nullptr) {
    char* wsb = (char*)ws;
    void* cK = wsb + L.ck_off;
    void* cV = wsb + L.cv_off;
    void* consts = wsb + L.const_off;
    float* cnorm = (float*)(wsb + L.norm_off);
    float* knorm = (float*)(wsb + L.knorm_off);
    hipError_t e;
    if (s->dtype == DAR_BF16) {
        e = launch_prefill_latent<bf16_t>((const bf16_t*)k, (const bf16_t*)v,
                                          (const bf16_t*)w_down, (bf16_t*)cK, (bf16_t*)cV, cnorm,
                                          knorm, (bf16_t*)consts, s->B, s->Hkv, geo, s->d,
                                          s->d_down, s->w, fast, stream);
        if (e != hipSuccess) return e;
        if (fast)
            return launch_prefill_mfma(s, geo, q, k, v, w_down, w_up, o, lse, cK, cV, cnorm, knorm,
                                       consts, stream, w_val);
        return launch_prefill_valu<bf16_t>((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v,
                                           (const bf16_t*)w_down, (const bf16_t*)w_up,
                                           (const bf16_t*)cK, (const bf16_t*)cV, (bf16_t*)o, lse,
                                           s->B, s->Hq, s->Hkv, geo, s->d, s->d_down, s->w,
                                           stream, (const bf16_t*)w_val);
    }
    e = launch_prefill_latent<float>((const float*)k, (const float*)v, (const float*)w_down,
                                     (float*)cK, (float*)cV, cnorm, knorm, (float*)consts, s->B,
                                     s->Hkv, geo, s->d, s->d_down, s->w, false, stream);
    if (e != hipSuccess) return e;
    return launch_prefill_valu<float>((const float*)q, (const float*)k, (const float*)v,
                                      (const float*)w_down, (const float*)w_up, (const float*)cK,
                                      (const float*)cV, (float*)o, lse, s->B, s->Hq, s->Hkv, geo,
                                      s->d, s->d_down, s->w, stream, (const float*)w_val);
}

// Chunked prefill workspace: the context rows (the ring's tokens from kv0 on,
// then the new ones) for K and V, then either (matrix-core shapes, latents
// read in place from the cache) the two block-norm arrays of nblk blocks a
// head, or the prefill workspace of len + n positions; every part 256-byte
// aligned.
struct ChunkWs {
    size_t ctx_k_off, ctx_v_off, pre_off, cnorm_off, knorm_off, bytes;
    PrefillWs pre;
    int kv0, Tc, nblk;
    bool in_place;
};

// Chunked prefill with the rotary embedding: the context rows (from kv0, the
// window's oldest position rounded down to 32 so that key blocks of 32 rows
// are position blocks; with w = 0 there is no window and kv0 = len), the
// rotated queries and context keys, the lifted rotated distant keys and
// lifted values (positions < len + n - w), and the two block-norm arrays.
struct ChunkRopeWs {
    size_t ctx_k_off, ctx_v_off, qr_off, kr_off, kd_off, vd_off, knorm_off, dnorm_off, bytes;
    int kv0, Tc, Td;
};

ChunkRopeWs chunk_rope_ws_layout(const dar_shape* s, int len, int n) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t es = esize_of(s->dtype);
    ChunkRopeWs L{};
    L.kv0 = s->w > 0 ? (len - s->w > 0 ? len - s->w : 0) & ~31 : len;
    L.Tc = len + n - L.kv0;
    const int T = len + n;
    L.Td = T - s->w > 0 ? T - s->w : 0;
    const size_t ctx = al((size_t)s->B * s->Hkv * L.Tc * s->d * es);
    const size_t dist = al((size_t)s->B * s->Hkv * L.Td * s->d * es);
    L.ctx_k_off = 0;
    L.ctx_v_off = ctx;
    L.qr_off = 2 * ctx;
    L.kr_off = L.qr_off + al((size_t)s->B * s->Hq * n * s->d * es);
    L.kd_off = L.kr_off + ctx;
    L.vd_off = L.kd_off + dist;
    L.knorm_off = L.vd_off + dist;
    L.dnorm_off = L.knorm_off + al((size_t)s->B * s->Hkv * ((T + 31) / 32) * sizeof(float));
    L.bytes = L.dnorm_off + al((size_t)s->B * s->Hkv * ((L.Td + 31) / 32 + 1) * sizeof(float));
    return L;
}

ChunkWs chunk_ws_layout(const dar_shape* s, int len, int n) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    ChunkWs L{};
    L.kv0 = len - s->w > 0 ? len - s->w : 0;
    L.Tc = len + n - L.kv0;
    const size_t ctx = al((size_t)s->B * s->Hkv * L.Tc * s->d * esize_of(s->dtype));
    L.ctx_k_off = 0;
    L.ctx_v_off = ctx;
    L.in_place = prefill_mfma_supported(s);
    if (L.in_place) {
        L.nblk = (len + n + 31) / 32;
        const size_t norms = al((size_t)s->B * s->Hkv * L.nblk * sizeof(float));
        L.cnorm_off = 2 * ctx;
        L.knorm_off = L.cnorm_off + norms;
        L.bytes = L.knorm_off + norms;
        return L;
    }
    L.pre_off = 2 * ctx;
    L.pre = prefill_ws_layout(s->B, s->Hkv, len + n, s->d_down, s->w, esize_of(s->dtype));
    L.bytes = L.pre_off + L.pre.bytes;
    return L;
}

// Paged chunked prefill workspace: the context rows of every sequence (w + n
// rows a head), then the two block-norm arrays (a whole sequence's capacity
// of 32-position blocks a head).
struct ChunkPagedWs {
    size_t ctx_k_off, ctx_v_off, cnorm_off, knorm_off, bytes;
    int nblk;
};

// Backward with the rotary embedding: the rotary pre-pass's arrays (bf16:
// rotated queries and keys, lifted and rotated distant keys, lifted values),
// then the fp32 arrays of RopeBwdArgs; every part 256-byte aligned.
struct RopeBwdWs {
    size_t qr, kr, kd, vd, nl2, nd, dqr, dkr, dvw, dkd, dvd, wpart, bytes;
    int nchunk;
};

RopeBwdWs rope_bwd_ws_layout(const dar_shape* s, int T) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    RopeBwdWs L{};
    const size_t B = s->B, Hq = s->Hq, Hkv = s->Hkv, d = s->d, dd = s->d_down;
    const size_t Td = T > s->w ? (size_t)(T - s->w) : 0;
    const size_t Tr = (size_t)round_up(T, 64);
    size_t off = 0;
    auto put = [&](size_t& at, size_t bytes) { at = off; off += al(bytes); };
    put(L.qr, B * Hq * T * d * 2);
    put(L.kr, B * Hkv * T * d * 2);
    put(L.kd, B * Hkv * Td * d * 2);
    put(L.vd, B * Hkv * Td * d * 2);
    put(L.nl2, B * Hq * Tr * 4);
    put(L.nd, B * Hq * Tr * 4);
    put(L.dqr, B * Hq * T * d * 4);
    put(L.dkr, B * Hkv * T * d * 4);
    put(L.dvw, B * Hkv * T * d * 4);
    put(L.dkd, B * Hkv * Td * d * 4);
    put(L.dvd, B * Hkv * Td * d * 4);
    L.nchunk = (int)B * ((T + 31) / 32);  // one share per 32 keys of a sequence
    put(L.wpart, 2 * Hkv * (size_t)L.nchunk * d * dd * 4);
    L.bytes = off;
    return L;
}

ChunkPagedWs chunk_paged_ws_layout(const dar_shape* s, int cap, int n) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    ChunkPagedWs L{};
    const size_t ctx = al((size_t)s->B * s->Hkv * (s->w + n) * s->d * esize_of(s->dtype));
    L.nblk = (int)(((long long)cap + 31) / 32);
    const size_t norms = al((size_t)s->B * s->Hkv * L.nblk * sizeof(float));
    L.ctx_k_off = 0;
    L.ctx_v_off = ctx;
    L.cnorm_off = 2 * ctx;
    L.knorm_off = L.cnorm_off + norms;
    L.bytes = L.knorm_off + norms;
    return L;
}

}  // namespace

extern "C" {

const char* dar_status_string(dar_status st) {
    switch (st) {
        case DAR_OK: return "ok";
        case DAR_E_ARG: return "invalid argument";
        case DAR_E_UNSUPPORTED: return "unsupported shape or dtype";
        case DAR_E_CAPACITY: return "cache capacity exceeded";
        case DAR_E_WORKSPACE: return "workspace missing or too small";
        case DAR_E_HIP: return "HIP launch failure";
    }
    return "unknown status";
}

size_t dar_prefill_workspace_bytes(const dar_shape* s, int T) {
    if (check_shape(s) != DAR_OK || T < 1) return 0;
    return prefill_ws_layout(s->B, s->Hkv, T, s->d_down, s->w, esize_of(s->dtype)).bytes;
}

size_t dar_decode_workspace_bytes(const dar_shape* s, int cap) {
    if (check_shape(s) != DAR_OK || cap < 1 || !group_supported(s)) return 0;
    const int S = decode_max_partials(s->B, s->Hkv, cap, s->w, s->d, s->d_down, s->Hq / s->Hkv);
    // records, then (paged decode) one piece count per (sequence, KV head)
    return (size_t)s->B * s->Hq * S * (2 + s->d_down + s->d) * sizeof(float) +
           (size_t)s->B * s->Hkv * sizeof(int);
}

size_t dar_prefill_chunk_workspace_bytes(const dar_shape* s, int len, int n) {
    if (check_shape(s) != DAR_OK || len < 0 || n < 1) return 0;
    if ((long long)len + n > 0x7fffffffLL) return 0;
    return chunk_ws_layout(s, len, n).bytes;
}

size_t dar_prefill_chunk_rope_workspace_bytes(const dar_shape* s, int len, int n) {
    if (check_shape(s) != DAR_OK || len < 0 || n < 1) return 0;
    if ((long long)len + n > 0x7fffffffLL) return 0;
    return chunk_rope_ws_layout(s, len, n).bytes;
}

size_t dar_prefill_rope_backward_workspace_bytes(const dar_shape* s, int T) {
    if (check_shape(s) != DAR_OK || T < 1) return 0;
    return rope_bwd_ws_layout(s, T).bytes;
}

size_t dar_prefill_rope_workspace_bytes(const dar_shape* s, int T) {
    if (check_shape(s) != DAR_OK || T < 1) return 0;
    return rope_ws_layout(s, T).bytes;
}

dar_status dar_rope_table(int rotary_dim, double base, int n_pos, float* table, hipStream_t stream) {
    if (rotary_dim < 2 || (rotary_dim & 1) || rotary_dim > 256 || n_pos < 1) return DAR_E_ARG;
    if (!(base > 0.0) || base > 1e300) return DAR_E_ARG;
    if (!dev_ok(table)) return DAR_E_ARG;
    if (n_pos > 65535) return DAR_E_UNSUPPORTED;
    clear_hip_error();
    return launch_rope_table(rotary_dim, base, n_pos, table, stream) == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_attn_prefill_rope(const dar_shape* s, int T, int pos0, const dar_rope* rope,
                                 const void* q, const void* k, const void* v, const void* w_down,
                                 const void* w_up, void* o, float* lse, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1 || pos0 < 0 || !rope) return DAR_E_ARG;
    const int r = rope->rotary_dim;
    if (r < 0 || (r & 1) || r > s->d) return DAR_E_ARG;
    if (r > 0 && !dev_ok(rope->table)) return DAR_E_ARG;
    if ((long long)pos0 + T > (long long)rope->n_pos) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    const RopeWs L = rope_ws_layout(s, T);
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    char* wsb = (char*)ws;
    void* qr = wsb + L.qr_off;
    void* kr = wsb + L.kr_off;
    void* kd = wsb + L.kd_off;
    void* vd = wsb + L.vd_off;
    float* knorm = (float*)(wsb + L.knorm_off);
    float* dnorm = (float*)(wsb + L.dnorm_off);
    const bool fast = prefill_mfma_rope_supported(s);
    if (log_enabled())
        fprintf(stderr, "[dar] prefill_rope B=%d Hq=%d Hkv=%d T=%d d=%d dd=%d w=%d r=%d pos0=%d %s path=%s\n",
                s->B, s->Hq, s->Hkv, T, s->d, s->d_down, s->w, r, pos0,
                s->dtype == DAR_BF16 ? "bf16" : "f32", fast ? "mfma" : "valu");
    hipError_t e;
    if (s->dtype == DAR_BF16) {
        e = launch_rope_prepass<bf16_t>((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v,
                                        (const bf16_t*)w_down, (const bf16_t*)w_up, rope->table,
                                        (bf16_t*)qr, (bf16_t*)kr, (bf16_t*)kd, (bf16_t*)vd,
                                        fast ? knorm : nullptr, fast ? dnorm : nullptr, s->B, s->Hq,
                                        s->Hkv, T, s->d, s->d_down, s->w, r, pos0, stream);
        if (e == hipSuccess) {
            if (fast)
                e = launch_prefill_mfma_rope(s, T, qr, kr, v, kd, vd, o, lse, knorm, dnorm, stream);
            else
                e = launch_prefill_rope_valu<bf16_t>((const bf16_t*)qr, (const bf16_t*)kr,
                                                     (const bf16_t*)v, (const bf16_t*)kd,
                                                     (const bf16_t*)vd, (bf16_t*)o, lse, s->B,
                                                     s->Hq, s->Hkv, T, s->d, s->w, stream);
        }
    } else {
        e = launch_rope_prepass<float>((const float*)q, (const float*)k, (const float*)v,
                                       (const float*)w_down, (const float*)w_up, rope->table,
                                       (float*)qr, (float*)kr, (float*)kd, (float*)vd, nullptr,
                                       nullptr, s->B, s->Hq, s->Hkv, T, s->d, s->d_down, s->w, r,
                                       pos0, stream);
        if (e == hipSuccess)
            e = launch_prefill_rope_valu<float>((const float*)qr, (const float*)kr,
                                                (const float*)v, (const float*)kd, (const float*)vd,
                                                (float*)o, lse, s->B, s->Hq, s->Hkv, T, s->d, s->w,
                                                stream);
    }
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

size_t dar_prefill_backward_workspace_bytes(const dar_shape* s, int T) {
    if (check_shape(s) != DAR_OK || T < 1) return 0;
    // enough for either kernel family (DAR_BWD_VALU may pick the generic one)
    const size_t a = bwd_ws_layout(s->B, s->Hq, s->Hkv, T, s->d, s->d_down, false).bytes;
    const size_t b = bwd_ws_layout(s->B, s->Hq, s->Hkv, T, s->d, s->d_down, true).bytes;
    return a > b ? a : b;
}

dar_status dar_attn_prefill(const dar_shape* s, int T, const void* q, const void* k,
                            const void* v, const void* w_down, const void* w_up, void* o,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
    return dar_attn_prefill_lse(s, T, q, k, v, w_down, w_up, o, nullptr, ws, ws_bytes, stream);
}

dar_status dar_attn_prefill_lse(const dar_shape* s, int T, const void* q, const void* k,
                                const void* v, const void* w_down, const void* w_up, void* o,
                                float* lse, void* ws, size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    const PrefillWs L = prefill_ws_layout(s->B, s->Hkv, T, s->d_down, s->w, esize_of(s->dtype));
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    hipError_t e = hipSuccess;
    const bool fast = prefill_mfma_supported(s);
    if (log_enabled())
        fprintf(stderr, "[dar] prefill B=%d Hq=%d Hkv=%d T=%d d=%d dd=%d w=%d %s path=%s\n", s->B,
                s->Hq, s->Hkv, T, s->d, s->d_down, s->w, s->dtype == DAR_BF16 ? "bf16" : "f32",
                fast ? "mfma" : "valu");
    if (s->dtype == DAR_BF16) {
        e = run_prefill(s, whole_sequence(T), q, k, v, w_down, w_up, o, lse, ws, L, fast, stream);
    } else {
        e = run_prefill(s, whole_sequence(T), q, k, v, w_down, w_up, o, lse, ws, L, false, stream);
    }
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_attn_prefill_ragged(const dar_shape* s, int T, const int* seq_lens, const void* q,
                                   const void* k, const void* v, const void* w_down,
                                   const void* w_up, void* o, float* lse, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1 || !seq_lens || ((uintptr_t)seq_lens & 3u)) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    const PrefillWs L = prefill_ws_layout(s->B, s->Hkv, T, s->d_down, s->w, esize_of(s->dtype));
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;
    clear_hip_error();
    PrefillGeo geo = whole_sequence(T);
    geo.seq_lens = seq_lens;
    const bool fast = s->dtype == DAR_BF16 && prefill_mfma_supported(s);
    const hipError_t e = run_prefill(s, geo, q, k, v, w_down, w_up, o, lse, ws, L, fast, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_attn_prefill_backward(const dar_shape* s, int T, const void* q, const void* k,
                                     const void* v, const void* w_down, const void* w_up,
                                     const void* o, const float* lse, const void* dout, void* dq,
                                     void* dk, void* dv, float* dw_down, float* dw_up, void* ws,
                                     size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(w_down) || !dev_ok(o) || !dev_ok(dout) ||
        !dev_ok(lse))
        return DAR_E_ARG;
    if (!dev_ok(dq) || !dev_ok(dk) || !dev_ok(dv) || !dev_ok(dw_down)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if ((w_up == nullptr) != (dw_up == nullptr)) return DAR_E_ARG;
    if (dw_up && !aligned16(dw_up)) return DAR_E_ARG;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    if (ws == nullptr || ws_bytes < dar_prefill_backward_workspace_bytes(s, T))
        return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    if (log_enabled())
        fprintf(stderr, "[dar] prefill_backward B=%d Hq=%d Hkv=%d T=%d d=%d dd=%d w=%d %s path=%s\n",
                s->B, s->Hq, s->Hkv, T, s->d, s->d_down, s->w, s->dtype == DAR_BF16 ? "bf16" : "f32",
                bwd_mfma_supported(s->d, s->d_down, s->dtype == DAR_BF16) && !env_flag("DAR_BWD_VALU")
                    ? "mfma" : "valu");
    hipError_t e;
    const bool fast = bwd_mfma_supported(s->d, s->d_down, s->dtype == DAR_BF16) &&
                      !env_flag("DAR_BWD_VALU");
    const BwdWs L = bwd_ws_layout(s->B, s->Hq, s->Hkv, T, s->d, s->d_down, fast);
    if (fast)
        e = launch_bwd_mfma((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (const bf16_t*)o,
                            lse, (const bf16_t*)dout, (const bf16_t*)w_down, (const bf16_t*)w_up,
                            (bf16_t*)dq, (bf16_t*)dk, (bf16_t*)dv, dw_down, dw_up, (char*)ws, L,
                            s->B, s->Hq, s->Hkv, T, s->d, s->d_down, s->w, stream);
    else if (s->dtype == DAR_BF16)
        e = launch_bwd_valu<bf16_t>((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v,
                                    (const bf16_t*)o, lse, (const bf16_t*)dout, (const bf16_t*)w_down,
                                    (const bf16_t*)w_up, (bf16_t*)dq, (bf16_t*)dk, (bf16_t*)dv,
                                    dw_down, dw_up, (char*)ws, L, s->B, s->Hq, s->Hkv, T, s->d,
                                    s->d_down, s->w, stream);
    else
        e = launch_bwd_valu<float>((const float*)q, (const float*)k, (const float*)v,
                                   (const float*)o, lse, (const float*)dout, (const float*)w_down,
                                   (const float*)w_up, (float*)dq, (float*)dk, (float*)dv,
                                   dw_down, dw_up, (char*)ws, L, s->B, s->Hq, s->Hkv, T, s->d,
                                   s->d_down, s->w, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_attn_prefill_chunk(const dar_shape* s, dar_cache* c, int n, const void* q,
                                  const void* k_new, const void* v_new, const void* w_down,
                                  const void* w_up, void* o, float* lse, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!c || n < 1 || c->cap < 1 || c->len < 0 || c->len > c->cap) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(w_down) || !dev_ok(o))
        return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    if (!dev_ok(c->k_lat) || !dev_ok(c->v_lat)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if ((long long)c->len + n > (long long)c->cap) return DAR_E_CAPACITY;
    if ((long long)s->B * s->Hkv > 65535 || (long long)s->B * s->Hq > 65535)
        return DAR_E_UNSUPPORTED;
    // the context copy moves 4-byte words of whole rows
    if ((s->d * (int)esize_of(s->dtype)) % 4 != 0) return DAR_E_UNSUPPORTED;
    const ChunkWs L = chunk_ws_layout(s, c->len, n);
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    char* wsb = (char*)ws;
    void* ctx_k = wsb + L.ctx_k_off;
    void* ctx_v = wsb + L.ctx_v_off;
    const int len = c->len;
    if (L.in_place) {
        // context rows first (the append below rewrites ring slots), then the
        // append (every distant latent of the chunk's rows is then in the
        // cache), the norms, and the attention reading the latents in place
        const bf16_t* wd = (const bf16_t*)w_down;
        hipError_t e = launch_chunk_gather<bf16_t>((const bf16_t*)c->k_win, (const bf16_t*)c->v_win,
                                                   (const bf16_t*)k_new, (const bf16_t*)v_new,
                                                   (bf16_t*)ctx_k, (bf16_t*)ctx_v, s->B, s->Hkv,
                                                   s->d, s->w, len, n, L.kv0, stream);
        if (e == hipSuccess)
            e = launch_append<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new, wd,
                                      (bf16_t*)c->k_win, (bf16_t*)c->v_win, (bf16_t*)c->k_lat,
                                      (bf16_t*)c->v_lat, s->B, s->Hkv, s->d, s->d_down, s->w,
                                      c->cap, len, n, stream);
        const LatCache lc{(const bf16_t*)c->k_lat, (const bf16_t*)c->v_lat, nullptr, nullptr, nullptr,
                          c->cap, 0, 0, 0, L.nblk, L.nblk};
        float* cnorm = (float*)(wsb + L.cnorm_off);
        float* knorm = (float*)(wsb + L.knorm_off);
        if (e == hipSuccess)
            e = launch_chunk_norms(lc, (const bf16_t*)ctx_k, L.Tc, cnorm, knorm, s->B, s->Hkv, s->d,
                                   s->d_down, s->w, len, n, L.nblk, stream);
        const PrefillGeo geo{len, n, L.kv0, L.Tc, 0, 0, nullptr, nullptr};
        if (e == hipSuccess)
            e = launch_prefill_mfma_cache(s, geo, lc, q, ctx_k, ctx_v, w_down, w_up, o, lse, cnorm,
                                          knorm, stream);
        if (e != hipSuccess) return DAR_E_HIP;
        c->len += n;
        return DAR_OK;
    }
    // rows len..len+n-1; keys/values from the context rows; latents of the
    // tokens that left the window before this chunk from the cache
    const PrefillGeo geo{len, n, L.kv0, L.Tc, L.kv0, c->cap, c->k_lat, c->v_lat};
    const bool fast = prefill_mfma_supported(s);
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_chunk_gather<bf16_t>((const bf16_t*)c->k_win, (const bf16_t*)c->v_win,
                                        (const bf16_t*)k_new, (const bf16_t*)v_new,
                                        (bf16_t*)ctx_k, (bf16_t*)ctx_v, s->B, s->Hkv, s->d, s->w,
                                        len, n, L.kv0, stream);
    else
        e = launch_chunk_gather<float>((const float*)c->k_win, (const float*)c->v_win,
                                       (const float*)k_new, (const float*)v_new, (float*)ctx_k,
                                       (float*)ctx_v, s->B, s->Hkv, s->d, s->w, len, n, L.kv0,
                                       stream);
    if (e == hipSuccess)
        e = run_prefill(s, geo, q, ctx_k, ctx_v, w_down, w_up, o, lse, wsb + L.pre_off, L.pre,
                        fast, stream);
    // the cache update is the append of the same tokens (the attention above
    // reads only the context copy and the workspace)
    if (e == hipSuccess) {
        if (s->dtype == DAR_BF16)
            e = launch_append<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new,
                                      (const bf16_t*)w_down, (bf16_t*)c->k_win,
                                      (bf16_t*)c->v_win, (bf16_t*)c->k_lat, (bf16_t*)c->v_lat,
                                      s->B, s->Hkv, s->d, s->d_down, s->w, c->cap, len, n,
                                      stream);
        else
            e = launch_append<float>((const float*)k_new, (const float*)v_new,
                                     (const float*)w_down, (float*)c->k_win, (float*)c->v_win,
                                     (float*)c->k_lat, (float*)c->v_lat, s->B, s->Hkv, s->d,
                                     s->d_down, s->w, c->cap, len, n, stream);
    }
    if (e != hipSuccess) return DAR_E_HIP;
    c->len += n;
    return DAR_OK;
}

dar_status dar_attn_prefill_chunk_rope(const dar_shape* s, dar_cache* c, const dar_rope* rope,
                                       int n, const void* q, const void* k_new, const void* v_new,
                                       const void* w_down, const void* w_up, void* o, float* lse,
                                       void* ws, size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!c || !rope || n < 1 || c->cap < 1 || c->len < 0 || c->len > c->cap) return DAR_E_ARG;
    const int r = rope->rotary_dim;
    if (r < 0 || (r & 1) || r > s->d) return DAR_E_ARG;
    if (r > 0 && !dev_ok(rope->table)) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(w_down) || !dev_ok(o))
        return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    if (!dev_ok(c->k_lat) || !dev_ok(c->v_lat)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if ((long long)c->len + n > (long long)c->cap) return DAR_E_CAPACITY;
    if ((long long)c->len + n > (long long)rope->n_pos) return DAR_E_ARG;
    if ((long long)s->B * s->Hkv > 65535 || (long long)s->B * s->Hq > 65535)
        return DAR_E_UNSUPPORTED;
    // the matrix-core shapes, rotated in 8-element chunks
    if (!prefill_mfma_rope_supported(s) || r % 16 != 0) return DAR_E_UNSUPPORTED;
    const ChunkRopeWs L = chunk_rope_ws_layout(s, c->len, n);
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    char* wsb = (char*)ws;
    const int len = c->len;
    bf16_t* ctx_k = (bf16_t*)(wsb + L.ctx_k_off);
    bf16_t* ctx_v = (bf16_t*)(wsb + L.ctx_v_off);
    bf16_t* qr = (bf16_t*)(wsb + L.qr_off);
    bf16_t* kr = (bf16_t*)(wsb + L.kr_off);
    bf16_t* kd = (bf16_t*)(wsb + L.kd_off);
    bf16_t* vd = (bf16_t*)(wsb + L.vd_off);
    float* knorm = (float*)(wsb + L.knorm_off);
    float* dnorm = (float*)(wsb + L.dnorm_off);
    hipError_t e = launch_chunk_gather<bf16_t>((const bf16_t*)c->k_win, (const bf16_t*)c->v_win,
                                               (const bf16_t*)k_new, (const bf16_t*)v_new, ctx_k,
                                               ctx_v, s->B, s->Hkv, s->d, s->w, len, n, L.kv0,
                                               stream);
    if (e == hipSuccess)
        e = launch_rope_chunk_prepass<bf16_t>(
            (const bf16_t*)q, ctx_k, ctx_v, (const bf16_t*)c->k_lat, (const bf16_t*)c->v_lat,
            c->cap, (const bf16_t*)w_down, (const bf16_t*)w_up, rope->table, qr, kr, kd, vd, knorm,
            dnorm, s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w, r, len, n, L.kv0, stream);
    // rows len..len+n-1 against the context rows from kv0 and the distant rows
    const PrefillGeo geo{len, n, L.kv0, L.Tc, 0, 0, nullptr, nullptr};
    if (e == hipSuccess)
        e = launch_prefill_mfma_rope_geo(s, geo, qr, kr, ctx_v, kd, vd, o, lse, knorm, dnorm, stream);
    // the cache update: the append of the same (un-rotated) tokens
    if (e == hipSuccess)
        e = launch_append<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new, (const bf16_t*)w_down,
                                  (bf16_t*)c->k_win, (bf16_t*)c->v_win, (bf16_t*)c->k_lat,
                                  (bf16_t*)c->v_lat, s->B, s->Hkv, s->d, s->d_down, s->w, c->cap,
                                  len, n, stream);
    if (e != hipSuccess) return DAR_E_HIP;
    c->len += n;
    return DAR_OK;
}

dar_status dar_cache_append(const dar_shape* s, dar_cache* c, const void* k_new,
                            const void* v_new, int n, const void* w_down, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!c || n < 1 || c->cap < 1 || c->len < 0 || c->len > c->cap) return DAR_E_ARG;
    if (!dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(w_down)) return DAR_E_ARG;
    if (!dev_ok(c->k_lat) || !dev_ok(c->v_lat)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if ((long long)c->len + n > (long long)c->cap) return DAR_E_CAPACITY;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;

    clear_hip_error();
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_append<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new,
                                  (const bf16_t*)w_down, (bf16_t*)c->k_win, (bf16_t*)c->v_win,
                                  (bf16_t*)c->k_lat, (bf16_t*)c->v_lat, s->B, s->Hkv, s->d,
                                  s->d_down, s->w, c->cap, c->len, n, stream);
    else
        e = launch_append<float>((const float*)k_new, (const float*)v_new, (const float*)w_down,
                                 (float*)c->k_win, (float*)c->v_win, (float*)c->k_lat,
                                 (float*)c->v_lat, s->B, s->Hkv, s->d, s->d_down, s->w, c->cap,
                                 c->len, n, stream);
    if (e != hipSuccess) return DAR_E_HIP;
    c->len += n;
    return DAR_OK;
}

}  // extern "C"

namespace {

// Arguments of one decode step over a dense split cache, apart from the
// workspace.
dar_status check_decode(const dar_shape* s, const dar_cache* c, const void* q, const void* w_down,
                        const void* w_up, const void* o) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!c || c->cap < 1 || c->len < 1 || c->len > c->cap) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (!dev_ok(c->k_lat) || !dev_ok(c->v_lat)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if (!group_supported(s)) return DAR_E_UNSUPPORTED;
    const int G = s->Hq / s->Hkv;
    if (decode_max_partials(s->B, s->Hkv, c->cap, s->w, s->d, s->d_down, G) > 1024)
        return DAR_E_UNSUPPORTED;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    return DAR_OK;
}

dar_status run_decode(const dar_shape* s, const dar_cache* c, const void* q, const void* w_down,
                      const void* w_up, void* o, float* part, hipStream_t stream) {
    clear_hip_error();
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_decode<bf16_t>((const bf16_t*)q, (const bf16_t*)w_down, (const bf16_t*)w_up,
                                  (const bf16_t*)c->k_win, (const bf16_t*)c->v_win,
                                  (const bf16_t*)c->k_lat, (const bf16_t*)c->v_lat, (bf16_t*)o,
                                  part, s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w, c->cap,
                                  c->len, stream);
    else
        e = launch_decode<float>((const float*)q, (const float*)w_down, (const float*)w_up,
                                 (const float*)c->k_win, (const float*)c->v_win,
                                 (const float*)c->k_lat, (const float*)c->v_lat, (float*)o, part,
                                 s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w, c->cap, c->len,
                                 stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

// Workspace of dar_attn_decode_noalloc: the partial records of one decode
// call live in this file-scope device array instead of caller memory. Each
// GPU the library runs on holds its own copy until the process ends. In host
// code `scratch` only names the symbol: its device address on the current
// GPU comes from hipGetSymbolAddress, looked up once per device.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_on_device[kMaxDevices];  // null until looked up on that device

hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (scratch_on_device[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        scratch_on_device[dev] = p;
    }
    *out = scratch_on_device[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

dar_status dar_attn_decode(const dar_shape* s, const dar_cache* c, const void* q,
                           const void* w_down, const void* w_up, void* o, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
    const dar_status st = check_decode(s, c, q, w_down, w_up, o);
    if (st != DAR_OK) return st;
    const size_t need = dar_decode_workspace_bytes(s, c->cap);
    if (ws == nullptr || ws_bytes < need) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;
    return run_decode(s, c, q, w_down, w_up, o, (float*)ws, stream);
}

size_t dar_decode_noalloc_max_bytes(void) { return kNoAllocScratchBytes; }

size_t dar_decode_noalloc_bytes(const dar_shape* s, int len) {
    if (check_shape(s) != DAR_OK || len < 1 || !group_supported(s)) return 0;
    const int parts = decode_partials_at(s->B, s->Hkv, len, s->w, s->d, s->d_down, s->Hq / s->Hkv,
                                         s->dtype == DAR_BF16);
    return (size_t)s->B * s->Hq * parts * (2 + s->d_down + s->d) * sizeof(float);
}

dar_status dar_attn_decode_noalloc(const dar_shape* s, const dar_cache* c, const void* q,
                                   const void* w_down, const void* w_up, void* o,
                                   hipStream_t stream) {
    const dar_status st = check_decode(s, c, q, w_down, w_up, o);
    if (st != DAR_OK) return st;
    if (dar_decode_noalloc_bytes(s, c->len) > kNoAllocScratchBytes) return DAR_E_WORKSPACE;
    void* ws = nullptr;
    if (scratch_address(&ws) != hipSuccess) return DAR_E_HIP;
    return run_decode(s, c, q, w_down, w_up, o, (float*)ws, stream);
}

dar_status dar_attn_decode_rope(const dar_shape* s, const dar_cache* c, const dar_rope* rope,
                                const void* q, const void* w_down, const void* w_up, void* o,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!c || c->cap < 1 || c->len < 1 || c->len > c->cap || !rope) return DAR_E_ARG;
    const int r = rope->rotary_dim;
    if (r < 0 || (r & 1) || r > s->d) return DAR_E_ARG;
    if (r > 0 && !dev_ok(rope->table)) return DAR_E_ARG;
    if (c->len > rope->n_pos) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (!dev_ok(c->k_lat) || !dev_ok(c->v_lat)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if (!group_supported(s)) return DAR_E_UNSUPPORTED;
    const int G = s->Hq / s->Hkv;
    if (decode_max_partials(s->B, s->Hkv, c->cap, s->w, s->d, s->d_down, G) > 1024)
        return DAR_E_UNSUPPORTED;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    const size_t need = dar_decode_workspace_bytes(s, c->cap);
    if (ws == nullptr || ws_bytes < need) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    if (log_enabled())
        fprintf(stderr, "[dar] decode_rope B=%d Hq=%d Hkv=%d d=%d dd=%d w=%d r=%d len=%d %s\n", s->B,
                s->Hq, s->Hkv, s->d, s->d_down, s->w, r, c->len,
                s->dtype == DAR_BF16 ? "bf16" : "f32");
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_decode_rope<bf16_t>((const bf16_t*)q, (const bf16_t*)w_down,
                                       (const bf16_t*)w_up, (const bf16_t*)c->k_win,
                                       (const bf16_t*)c->v_win, (const bf16_t*)c->k_lat,
                                       (const bf16_t*)c->v_lat, rope->table, rope->n_pos, (bf16_t*)o,
                                       (float*)ws, s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w,
                                       c->cap, c->len, r, stream);
    else
        e = launch_decode_rope<float>((const float*)q, (const float*)w_down, (const float*)w_up,
                                      (const float*)c->k_win, (const float*)c->v_win,
                                      (const float*)c->k_lat, (const float*)c->v_lat, rope->table,
                                      rope->n_pos, (float*)o, (float*)ws, s->B, s->Hq, s->Hkv, s->d, s->d_down,
                                      s->w, c->cap, c->len, r, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_attn_prefill_shared(const dar_shape* s, int T, const void* q, const void* k,
                                   const void* v, const void* c, const void* u_k, const void* u_v,
                                   void* o, float* lse, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(c) || !dev_ok(u_k) || !dev_ok(u_v) ||
        !dev_ok(o))
        return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    const PrefillWs L = prefill_ws_layout(s->B, s->Hkv, T, s->d_down, s->w, esize_of(s->dtype));
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    // every position's latent is given: the pre-pass reads them (as a chunk
    // reads a cache's) instead of projecting; U_K takes the place of W_up in
    // the query absorption, U_V in the lift of the output. The pre-pass's
    // W_down operand is never used for a projection here (U_K, of the same
    // size, is passed so that its loads stay in bounds).
    const PrefillGeo geo{0, T, 0, T, T, T, c, c};
    const bool fast = s->dtype == DAR_BF16 && prefill_mfma_supported(s);
    if (log_enabled())
        fprintf(stderr, "[dar] prefill_shared B=%d Hq=%d Hkv=%d T=%d d=%d dd=%d w=%d %s path=%s\n",
                s->B, s->Hq, s->Hkv, T, s->d, s->d_down, s->w, s->dtype == DAR_BF16 ? "bf16" : "f32",
                fast ? "mfma" : "valu");
    const hipError_t e = run_prefill(s, geo, q, k, v, u_k, u_k, o, lse, ws, L, fast, stream, u_v);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

dar_status dar_cache_append_shared(const dar_shape* s, dar_cache* cache, const void* k_new,
                                   const void* v_new, const void* c_new, int n,
                                   hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!cache || n < 1 || cache->cap < 1 || cache->len < 0 || cache->len > cache->cap)
        return DAR_E_ARG;
    if (!dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(c_new) || !dev_ok(cache->k_lat))
        return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(cache->k_win) || !dev_ok(cache->v_win))) return DAR_E_ARG;
    if ((long long)cache->len + n > (long long)cache->cap) return DAR_E_CAPACITY;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;

    clear_hip_error();
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_append_shared<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new,
                                         (const bf16_t*)c_new, (bf16_t*)cache->k_win,
                                         (bf16_t*)cache->v_win, (bf16_t*)cache->k_lat, s->B, s->Hkv,
                                         s->d, s->d_down, s->w, cache->cap, cache->len, n, stream);
    else
        e = launch_append_shared<float>((const float*)k_new, (const float*)v_new,
                                        (const float*)c_new, (float*)cache->k_win,
                                        (float*)cache->v_win, (float*)cache->k_lat, s->B, s->Hkv,
                                        s->d, s->d_down, s->w, cache->cap, cache->len, n, stream);
    if (e != hipSuccess) return DAR_E_HIP;
    cache->len += n;
    return DAR_OK;
}

dar_status dar_attn_decode_shared(const dar_shape* s, const dar_cache* cache, const void* q,
                                  const void* u_k, const void* u_v, void* o, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (!cache || cache->cap < 1 || cache->len < 1 || cache->len > cache->cap) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(u_k) || !dev_ok(u_v) || !dev_ok(o) || !dev_ok(cache->k_lat))
        return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(cache->k_win) || !dev_ok(cache->v_win))) return DAR_E_ARG;
    if (!group_supported(s)) return DAR_E_UNSUPPORTED;
    const int G = s->Hq / s->Hkv;
    if (decode_max_partials(s->B, s->Hkv, cache->cap, s->w, s->d, s->d_down, G) > 1024)
        return DAR_E_UNSUPPORTED;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    const size_t need = dar_decode_workspace_bytes(s, cache->cap);
    if (ws == nullptr || ws_bytes < need) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;

    clear_hip_error();
    // keys and values of the distant region read the same latents; U_K is
    // absorbed into the query, U_V lifts the output
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_decode<bf16_t>((const bf16_t*)q, (const bf16_t*)u_k, (const bf16_t*)u_k,
                                  (const bf16_t*)cache->k_win, (const bf16_t*)cache->v_win,
                                  (const bf16_t*)cache->k_lat, (const bf16_t*)cache->k_lat,
                                  (bf16_t*)o, (float*)ws, s->B, s->Hq, s->Hkv, s->d, s->d_down,
                                  s->w, cache->cap, cache->len, stream, (const bf16_t*)u_v);
    else
        e = launch_decode<float>((const float*)q, (const float*)u_k, (const float*)u_k,
                                 (const float*)cache->k_win, (const float*)cache->v_win,
                                 (const float*)cache->k_lat, (const float*)cache->k_lat, (float*)o,
                                 (float*)ws, s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w,
                                 cache->cap, cache->len, stream, (const float*)u_v);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

static dar_status check_paged(const dar_shape* s, const dar_paged_cache* c) {
    if (!c || c->page_size < 32 || (c->page_size & (c->page_size - 1)) || c->max_blocks < 1 ||
        c->n_pages < 1)
        return DAR_E_ARG;
    if ((long long)c->page_size * c->max_blocks > 0x7fffffffLL) return DAR_E_ARG;
    if (!dev_ok(c->k_pool) || !dev_ok(c->v_pool) || !c->block_table || !c->lens) return DAR_E_ARG;
    if (((uintptr_t)c->block_table & 3u) || ((uintptr_t)c->lens & 3u)) return DAR_E_ARG;
    if (s->w > 0 && (!dev_ok(c->k_win) || !dev_ok(c->v_win))) return DAR_E_ARG;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    return DAR_OK;
}

dar_status dar_cache_append_paged(const dar_shape* s, const dar_paged_cache* c, const void* k_new,
                                  const void* v_new, const void* w_down, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    st = check_paged(s, c);
    if (st != DAR_OK) return st;
    if (!dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(w_down)) return DAR_E_ARG;
    clear_hip_error();
    const PagedArgs pg{c->lens, c->block_table, c->page_size, c->max_blocks, c->n_pages,
                       __builtin_ctz((unsigned)c->page_size)};
    hipError_t e;
    if (s->dtype == DAR_BF16)
        e = launch_append_paged<bf16_t>((const bf16_t*)k_new, (const bf16_t*)v_new,
                                        (const bf16_t*)w_down, (bf16_t*)c->k_win, (bf16_t*)c->v_win,
                                        (bf16_t*)c->k_pool, (bf16_t*)c->v_pool, pg, c->lens, s->B,
                                        s->Hkv, s->d, s->d_down, s->w, stream);
    else
        e = launch_append_paged<float>((const float*)k_new, (const float*)v_new,
                                       (const float*)w_down, (float*)c->k_win, (float*)c->v_win,
                                       (float*)c->k_pool, (float*)c->v_pool, pg, c->lens, s->B,
                                       s->Hkv, s->d, s->d_down, s->w, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

}  // extern "C"

namespace {

// The paged decode, without (rope NULL) or with the rotary embedding.
dar_status decode_paged(const dar_shape* s, const dar_paged_cache* c, const dar_rope* rope,
                        const void* q, const void* w_down, const void* w_up, void* o, void* ws,
                        size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    st = check_paged(s, c);
    if (st != DAR_OK) return st;
    if (!dev_ok(q) || !dev_ok(w_down) || !dev_ok(o)) return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (!decode_mfma_supported(s->d, s->d_down, s->Hq / s->Hkv, s->dtype == DAR_BF16) ||
        !group_supported(s))
        return DAR_E_UNSUPPORTED;
    const int cap = c->page_size * c->max_blocks;
    int r = 0;
    if (rope) {
        r = rope->rotary_dim;
        if (r < 0 || (r & 1) || r > s->d) return DAR_E_ARG;
        if (r > 0 && !dev_ok(rope->table)) return DAR_E_ARG;
        // every position a sequence can reach indexes the table
        if (rope->n_pos < cap) return DAR_E_ARG;
        if (r > 0 &&
            !decode_mfma_rope_supported(s->d, s->d_down, s->Hq / s->Hkv, r, s->dtype == DAR_BF16))
            return DAR_E_UNSUPPORTED;
    }
    const size_t need = dar_decode_workspace_bytes(s, cap);
    if (ws == nullptr || ws_bytes < need) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;
    clear_hip_error();
    const PagedArgs pg{c->lens, c->block_table, c->page_size, c->max_blocks, c->n_pages,
                       __builtin_ctz((unsigned)c->page_size)};
    int P = 0;
    int* counts = nullptr;
    hipError_t e = launch_decode_mfma_paged((const bf16_t*)q, (const bf16_t*)w_down,
                                            (const bf16_t*)w_up, (const bf16_t*)c->k_win,
                                            (const bf16_t*)c->v_win, (const bf16_t*)c->k_pool,
                                            (const bf16_t*)c->v_pool, pg, (float*)ws, (bf16_t*)o,
                                            s->B, s->Hq, s->Hkv, s->d, s->d_down, s->w, P, counts,
                                            stream, r > 0 ? rope->table : nullptr,
                                            r > 0 ? rope->n_pos : 0, r);
    // the pairs split over several workgroups, and the empty or overflowed
    // sequences (NaN rows)
    if (e == hipSuccess)
        e = launch_decode_combine<bf16_t>((const float*)ws, (const bf16_t*)w_down,
                                          (const bf16_t*)w_up, (bf16_t*)o, s->B, s->Hq, s->Hkv,
                                          s->d, s->d_down, P, stream, nullptr, c->lens, counts);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

}  // namespace

extern "C" {

dar_status dar_attn_decode_paged(const dar_shape* s, const dar_paged_cache* c, const void* q,
                                 const void* w_down, const void* w_up, void* o, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
    return decode_paged(s, c, nullptr, q, w_down, w_up, o, ws, ws_bytes, stream);
}

dar_status dar_attn_decode_paged_rope(const dar_shape* s, const dar_paged_cache* c,
                                      const dar_rope* rope, const void* q, const void* w_down,
                                      const void* w_up, void* o, void* ws, size_t ws_bytes,
                                      hipStream_t stream) {
    if (!rope) return DAR_E_ARG;
    return decode_paged(s, c, rope, q, w_down, w_up, o, ws, ws_bytes, stream);
}

dar_status dar_attn_prefill_rope_backward(const dar_shape* s, int T, int pos0, const dar_rope* rope,
                                          const void* q, const void* k, const void* v,
                                          const void* w_down, const void* w_up, const void* o,
                                          const float* lse, const void* dout, void* dq, void* dk,
                                          void* dv, float* dw_down, float* dw_up, void* ws,
                                          size_t ws_bytes, hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    if (T < 1 || pos0 < 0 || !rope) return DAR_E_ARG;
    const int r = rope->rotary_dim;
    if (r < 0 || (r & 1) || r > s->d) return DAR_E_ARG;
    if (r > 0 && !dev_ok(rope->table)) return DAR_E_ARG;
    if ((long long)pos0 + T > (long long)rope->n_pos) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k) || !dev_ok(v) || !dev_ok(w_down) || !dev_ok(o) || !dev_ok(lse) ||
        !dev_ok(dout) || !dev_ok(dq) || !dev_ok(dk) || !dev_ok(dv) || !dev_ok(dw_down))
        return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if ((w_up == nullptr) != (dw_up == nullptr)) return DAR_E_ARG;
    if (dw_up && !aligned16(dw_up)) return DAR_E_ARG;
    if (!bwd_rope_mfma_supported(s->d, s->d_down, s->dtype == DAR_BF16)) return DAR_E_UNSUPPORTED;
    if ((long long)s->B * ((T + 31) / 32) > 65535) return DAR_E_UNSUPPORTED;
    if ((long long)s->B * s->Hkv > 65535) return DAR_E_UNSUPPORTED;
    const RopeBwdWs L = rope_bwd_ws_layout(s, T);
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;
    clear_hip_error();
    char* wsb = (char*)ws;
    RopeBwdArgs a{};
    a.q = (const bf16_t*)q;
    a.k = (const bf16_t*)k;
    a.v = (const bf16_t*)v;
    a.o = (const bf16_t*)o;
    a.dout = (const bf16_t*)dout;
    a.wd = (const bf16_t*)w_down;
    a.wu = (const bf16_t*)w_up;
    a.lse = lse;
    a.tab = rope->table;
    a.qr = (const bf16_t*)(wsb + L.qr);
    a.kr = (const bf16_t*)(wsb + L.kr);
    a.kd = (const bf16_t*)(wsb + L.kd);
    a.vd = (const bf16_t*)(wsb + L.vd);
    a.nl2 = (float*)(wsb + L.nl2);
    a.nd = (float*)(wsb + L.nd);
    a.dqr = (float*)(wsb + L.dqr);
    a.dkr = (float*)(wsb + L.dkr);
    a.dvw = (float*)(wsb + L.dvw);
    a.dkd = (float*)(wsb + L.dkd);
    a.dvd = (float*)(wsb + L.dvd);
    a.wpart = (float*)(wsb + L.wpart);
    a.dq = (bf16_t*)dq;
    a.dk = (bf16_t*)dk;
    a.dv = (bf16_t*)dv;
    a.dwd = dw_down;
    a.dwu = dw_up;
    a.L.nchunk = a.L.nchunk_d = a.L.nchunk_u = L.nchunk;
    a.B = s->B;
    a.Hq = s->Hq;
    a.Hkv = s->Hkv;
    a.T = T;
    a.dd = s->d_down;
    a.w = s->w;
    a.r = r;
    a.pos0 = pos0;
    // the forward's rotated and lifted operands, recomputed (no norms needed)
    hipError_t e = launch_rope_prepass<bf16_t>(a.q, a.k, a.v, a.wd, a.wu, rope->table,
                                               (bf16_t*)a.qr, (bf16_t*)a.kr, (bf16_t*)a.kd,
                                               (bf16_t*)a.vd, nullptr, nullptr, s->B, s->Hq,
                                               s->Hkv, T, s->d, s->d_down, s->w, r, pos0, stream);
    if (e == hipSuccess) e = launch_bwd_rope_mfma(a, s->d, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

size_t dar_prefill_chunk_paged_workspace_bytes(const dar_shape* s, int cap, int n) {
    if (check_shape(s) != DAR_OK || cap < 1 || n < 1) return 0;
    return chunk_paged_ws_layout(s, cap, n).bytes;
}

dar_status dar_attn_prefill_chunk_paged(const dar_shape* s, const dar_paged_cache* c, int n,
                                        const int* n_new, const void* q, const void* k_new,
                                        const void* v_new, const void* w_down, const void* w_up,
                                        void* o, float* lse, void* ws, size_t ws_bytes,
                                        hipStream_t stream) {
    dar_status st = check_shape(s);
    if (st != DAR_OK) return st;
    st = check_paged(s, c);
    if (st != DAR_OK) return st;
    if (n < 1) return DAR_E_ARG;
    if (!dev_ok(q) || !dev_ok(k_new) || !dev_ok(v_new) || !dev_ok(w_down) || !dev_ok(o))
        return DAR_E_ARG;
    if (w_up && !aligned16(w_up)) return DAR_E_ARG;
    if (lse && !aligned16(lse)) return DAR_E_ARG;
    if (n_new && ((uintptr_t)n_new & 3u)) return DAR_E_ARG;
    if (!prefill_mfma_supported(s)) return DAR_E_UNSUPPORTED;
    const int cap = c->page_size * c->max_blocks;
    if ((long long)s->w + n > 0x7fffffffLL / 64) return DAR_E_UNSUPPORTED;
    const ChunkPagedWs L = chunk_paged_ws_layout(s, cap, n);
    if (ws == nullptr || ws_bytes < L.bytes) return DAR_E_WORKSPACE;
    if (!aligned16(ws)) return DAR_E_ARG;
    clear_hip_error();
    char* wsb = (char*)ws;
    bf16_t* ctx_k = (bf16_t*)(wsb + L.ctx_k_off);
    bf16_t* ctx_v = (bf16_t*)(wsb + L.ctx_v_off);
    float* cnorm = (float*)(wsb + L.cnorm_off);
    float* knorm = (float*)(wsb + L.knorm_off);
    const LatCache lc{(const bf16_t*)c->k_pool, (const bf16_t*)c->v_pool, c->block_table, c->lens,
                      n_new, cap, c->max_blocks, __builtin_ctz((unsigned)c->page_size), c->n_pages,
                      L.nblk, L.nblk};
    // context rows, then the append, the norms and the attention (each
    // reading lens as it was), then the lengths advance
    hipError_t e = launch_chunk_gather_paged((const bf16_t*)c->k_win, (const bf16_t*)c->v_win,
                                             (const bf16_t*)k_new, (const bf16_t*)v_new, ctx_k,
                                             ctx_v, lc, s->B, s->Hkv, s->d, s->w, n, stream);
    if (e == hipSuccess)
        e = launch_append_chunk_paged((const bf16_t*)k_new, (const bf16_t*)v_new,
                                      (const bf16_t*)w_down, (bf16_t*)c->k_win, (bf16_t*)c->v_win,
                                      (bf16_t*)c->k_pool, (bf16_t*)c->v_pool, lc, s->B, s->Hkv,
                                      s->d, s->d_down, s->w, n, stream);
    if (e == hipSuccess)
        e = launch_chunk_norms(lc, ctx_k, s->w + n, cnorm, knorm, s->B, s->Hkv, s->d, s->d_down,
                               s->w, 0, n, L.nblk, stream);
    const PrefillGeo geo{0, n, 0, s->w + n, 0, 0, nullptr, nullptr};
    if (e == hipSuccess)
        e = launch_prefill_mfma_cache(s, geo, lc, q, ctx_k, ctx_v, w_down, w_up, o, lse, cnorm,
                                      knorm, stream);
    if (e == hipSuccess) e = launch_lens_advance(c->lens, n_new, s->B, cap, n, stream);
    return e == hipSuccess ? DAR_OK : DAR_E_HIP;
}

}  // extern "C"
