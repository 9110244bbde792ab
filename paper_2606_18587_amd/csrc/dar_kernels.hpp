// Launchers of the DAR kernels (host side). All of them enqueue on `st` and
// return the launch status; shapes have been validated by the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dar {

typedef uint16_t bf16_t;

static inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

// Prefill workspace: latents of tokens [0, T - w) per (batch, KV head). The
// token count is padded to Tp = round_up(T - w, 32) + 64 (the padding rows
// are zero, so readers may prefetch two 32-token subtiles past the end):
//   cK     [B*Hkv][Tp][dd]            token-major
//   cVt    [B*Hkv][Tp/32][dd][32]     32-token blocks, transposed in a block
//   cnorm  [B*Hkv][Tp/32] fp32        max L2 norm of the stored c^K rows of each
//                                     32-token block (matrix-core path only)
//   knorm  [B*Hkv][ceil(T/32)] fp32   max L2 norm of the key rows of each 32-token
//                                     block (matrix-core path only)
//   consts 256 bytes; starts with 8 bf16 ones then 8 bf16 zeros (operand rows
//          of the matrix-core kernel that carry no latent column)
// The latent parts are empty when T <= w.
struct PrefillWs {
    size_t ck_off, cv_off, norm_off, knorm_off, const_off, bytes;
};
static inline int prefill_tp(int T, int w) {
    const int Tl = T - w;
    return Tl > 0 ? round_up(Tl, 32) + 64 : 0;
}
PrefillWs prefill_ws_layout(int B, int Hkv, int T, int dd, int w, size_t esize);

// Paged split cache (serving): rings [B][Hkv][w][d] per sequence; latents in
// pages [n_pages][Hkv][ps][dd] (ps tokens of every KV head per page), token e
// of sequence b in page bt[b * maxb + e / ps], row e % ps; lens[b] tokens per
// sequence (device). Page indices outside [0, n_pages) are never read or
// written (such tokens read as zeros and are not stored).
struct PagedArgs {
    const int* lens;
    const int* bt;
    int ps, maxb, n_pages;
    int ps_shift;  // log2(ps): page sizes are powers of two
    int nseq;      // sequences in the batch (B)
    int* counts;   // [B * Hkv]: partial records of each (sequence, KV head) (decode)
};

// Latents that the chunked prefill reads in place, after the chunk's own
// window exits have been appended (so every distant latent is in the cache):
//   dense (bt == nullptr): k, v [B][Hkv][cap][dd], every sequence holding
//     the same number of tokens (the call's len);
//   paged: k, v are the pools [n_pages][Hkv][ps][dd] (ps = 1 << ps_shift),
//     token e of sequence b in page bt[b * maxb + e / ps]; each sequence has
//     its own geometry: lens[b] tokens held before the chunk, n_new[b] new
//     ones (n_new == nullptr: every sequence takes the call's n), capacity cap
//     tokens. A sequence with n_new[b] > 0 and lens[b] < 0 or
//     lens[b] + n_new[b] > cap is not served (its rows are NaN).
// ncb, nkb: 32-position blocks per (batch, KV head) of the latent-key and
// context-key norm arrays the attention reads.
struct LatCache {
    const bf16_t* k;
    const bf16_t* v;
    const int* bt;
    const int* lens;
    const int* n_new;
    int cap;
    int maxb, ps_shift, n_pages;
    int ncb, nkb;
};

// Where the rows, keys/values and latents of a prefill come from. Rows
// r = 0..n_rows-1 are the queries at positions q0 + r (T = q0 + n_rows
// positions in all); k and v row t holds position kv0 + t (t < Tkv); the
// latent of a position below lat0 is read from a split cache (k_lat, v_lat,
// [B*Hkv][cap][dd]) instead of being projected from k and v. A whole-sequence
// prefill has q0 = kv0 = lat0 = 0 and n_rows = Tkv = T; a chunk appended to a
// cache of len tokens has q0 = len, kv0 = max(0, len - w) (the ring's oldest
// token), lat0 = len - w.
// seq_lens (whole-sequence prefill of a ragged batch only): device int [B],
// the length of each sequence of the padded batch; positions at or past a
// sequence's length are neither read nor written (NULL: every sequence is T).
struct PrefillGeo {
    int q0, n_rows, kv0, Tkv, lat0, cap;
    const void* k_lat;
    const void* v_lat;
    const int* seq_lens = nullptr;
    int total() const { return q0 + n_rows; }
};
static inline PrefillGeo whole_sequence(int T) {
    return PrefillGeo{0, T, 0, T, 0, 0, nullptr, nullptr, nullptr};
}
// Rows of a 32-token block of the transposed value latents written by the
// matrix-core pre-pass: d_down, plus a row of ones when d_down == 16 (the
// padding row of the 32-row MFMA operand, which then yields the row sums).
__host__ __device__ inline int cvt_rows(int dd) { return dd == 16 ? 17 : dd; }

// Decode workspace: per (batch, query head, partial) softmax state
// {m, l, acc_lat[dd], acc_win[d]} in fp32.
struct DecodeSplits {
    int chunk_lat, chunk_win;   // tokens per split in each region
    int n_lat_split, n_win_split;
};
DecodeSplits decode_splits(int len, int w, int d, int dd, int G);
int decode_mfma_parts(int B, int Hkv, int len, int w, int d);
int decode_max_partials(int B, int Hkv, int cap, int w, int d, int dd, int G);
// Partial records (each 2 + d_down + d floats per query head) that one
// launch_decode call at cache length len writes: 0 when one workgroup per
// (batch, KV head) finishes the output itself.
int decode_partials_at(int B, int Hkv, int len, int w, int d, int dd, int G, bool bf16);

template <typename T>
hipError_t launch_prefill_latent(const T* k, const T* v, const T* wd, T* cK, T* cVt,
                                 float* cnorm, float* knorm, T* consts, int B, int Hkv,
                                 const PrefillGeo& geo, int d, int dd, int w, bool perm,
                                 hipStream_t st);

// Copies the ring's tokens [kv0, len) and the n new tokens into one row range
// ctx [B*Hkv][len + n - kv0][d] (positions kv0..len+n-1).
template <typename T>
hipError_t launch_chunk_gather(const T* k_win, const T* v_win, const T* k_new, const T* v_new,
                               T* ctx_k, T* ctx_v, int B, int Hkv, int d, int w, int len, int n,
                               int kv0, hipStream_t st);

template <typename T>
hipError_t launch_append(const T* k_new, const T* v_new, const T* wd, T* k_win, T* v_win,
                         T* k_lat, T* v_lat, int B, int Hkv, int d, int dd, int w, int cap, int len,
                         int n, hipStream_t st);

template <typename T>
hipError_t launch_prefill_valu(const T* q, const T* k, const T* v, const T* wd, const T* wu,
                               const T* cK, const T* cVt, T* o, float* lse, int B, int Hq,
                               int Hkv, const PrefillGeo& geo, int d, int dd, int w,
                               hipStream_t st, const T* wv = nullptr);

// Matrix-core decode (bf16, d in {64,128}, d_down in {16,32}, <= 8 query heads
// per KV head); shares decode_combine_kernel with the vector-ALU path.
bool decode_mfma_supported(int d, int dd, int G, bool bf16);
// P = partial records per query head; P == 1: the output is already written.
hipError_t launch_decode_mfma(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                              const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_lat,
                              const bf16_t* v_lat, float* part, bf16_t* o, int B, int Hq, int Hkv,
                              int d, int dd, int w, int cap, int len, int& P, hipStream_t st,
                              const bf16_t* wv = nullptr);

// The same kernel with the rotary embedding of Eq. 3 (d 64 or 128, rotary
// dimension 16, 32 or 64); tab [n_pos][r].
bool decode_mfma_rope_supported(int d, int dd, int G, int r, bool bf16);
hipError_t launch_decode_mfma_rope(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                                   const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_lat,
                                   const bf16_t* v_lat, const float* tab, int n_pos, float* part,
                                   bf16_t* o, int B, int Hq, int Hkv, int dd, int w, int cap,
                                   int len, int r, int& P, hipStream_t st, int d);
// The same kernel over a paged cache with per-sequence lengths (bf16 shapes
// of decode_mfma_supported), as a persistent grid: the batch's cache bytes
// are dealt out in equal shares, one per workgroup. A (sequence, KV head)
// pair that one workgroup covers whole is finished there; the others get one
// partial record per piece (P records per head at most) and their piece
// count in pg.counts, and launch_decode_combine (with lens and counts)
// finishes them. part: P * B * Hq records, then B * Hkv ints (counts).
// With tab (rotary dimension r in {16, 32, 64}, n_pos at least the capacity):
// the rotary embedding of Eq. 3 as launch_decode_mfma_rope applies it.
hipError_t launch_decode_mfma_paged(const bf16_t* q, const bf16_t* wd, const bf16_t* wu,
                                    const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_pool,
                                    const bf16_t* v_pool, const PagedArgs& pg, float* part,
                                    bf16_t* o, int B, int Hq, int Hkv, int d, int dd, int w, int& P,
                                    int*& counts, hipStream_t st, const float* tab = nullptr,
                                    int n_pos = 0, int r = 0);
// Partial records per head of a paged decode (bound over all length mixes).
int decode_paged_slots(int Hkv, int cap, int w, int d, int dd);
// One token per sequence into a paged cache at position lens[b]; the token
// leaving the window is projected (as launch_append projects it) into its
// page slot; lens[b] += 1 for every sequence below capacity.
template <typename T>
hipError_t launch_append_paged(const T* k_new, const T* v_new, const T* wd, T* k_win, T* v_win,
                               T* k_pool, T* v_pool, const PagedArgs& pg, int* lens, int B, int Hkv,
                               int d, int dd, int w, hipStream_t st);
template <typename T>
hipError_t launch_decode(const T* q, const T* wd, const T* wu, const T* k_win, const T* v_win,
                         const T* k_lat, const T* v_lat, T* o, float* part, int B, int Hq, int Hkv,
                         int d, int dd, int w, int cap, int len, hipStream_t st,
                         const T* wv = nullptr);
// Single shared latent: the cache's latent slot of every new token takes its
// given latent (c_new [B][Hkv][n][dd]); the ring takes the newest min(n, w)
// tokens' keys and values. No projection.
template <typename T>
hipError_t launch_append_shared(const T* k_new, const T* v_new, const T* c_new, T* k_win, T* v_win,
                                T* lat, int B, int Hkv, int d, int dd, int w, int cap, int len,
                                int n, hipStream_t st);

// Prefill backward workspace (256-byte aligned parts; Tr = round_up(T, 64)):
//   lse, delta        [B*Hq][Tr] fp32     dO . O per row (matrix-core path: -lse in
//                                         log2 units and -delta)
//   qt, dot           [B*Hq][Tr]          q W_up^T, dO W_up^T: fp32 [dd] per row, or
//                                         on the matrix-core path bf16 [dd] per row
//                                         followed by transposed blocks [Tr/32][32][32]
//                                         (latent rows past dd are zero)
//   rc                [B*Hq][Tr][16] bf16 matrix-core path: -lse and -delta, each as a
//                                         hi + mid + lo bf16 triple (row constants)
//   hk, ol            [B*Hq][T][dd] fp32  sum dS c^K, sum P c^V per row
//   ck, cv            [B*Hkv][Tr]         latents, laid out as qt
//   gk, gv            [B*Hkv][T][dd] fp32 sum dS q~, sum P dO~ per key
//   wpart             [2][Hkv][nchunk][d][dd]  weight-gradient partials per chunk
// (each array region is sized for Tr tokens).
struct BwdWs {
    size_t lse_off, delta_off, qt_off, dot_off, rc_off, hk_off, ol_off, ck_off, cv_off, gk_off,
        gv_off, wpart_off, bytes;
    int nchunk_d, nchunk_u, nchunk;
};
// Row chunks of the weight-gradient reduction: about 256 rows each, at most 128.
static inline int bwd_nchunk(long long rows) {
    long long n = (rows + 255) / 256;
    return (int)(n < 1 ? 1 : (n > 128 ? 128 : n));
}
// mfma: chunks of the weight-gradient shares are the matrix-core kernels'
// workgroups (else row chunks of the vector-ALU reduction).
BwdWs bwd_ws_layout(int B, int Hq, int Hkv, int T, int d, int dd, bool mfma);
hipError_t launch_bwd_wreduce(const float* part, float* dwd, float* dwu, int Hkv, int d, int dd,
                              const BwdWs& L, hipStream_t st);

template <typename T>
hipError_t launch_bwd_prep(const T* q, const T* k, const T* v, const T* o, const T* dout,
                           const T* wd, const T* wu, float* ck, float* cv, float* qt, float* dot,
                           float* delta, int B, int Hq, int Hkv, int T_, int d, int dd,
                           hipStream_t st);
template <typename T>
hipError_t launch_bwd_weights(const T* q, const T* k, const T* v, const T* dout, const float* gk,
                              const float* gv, const float* hk, const float* ol, float* part,
                              float* dwd, float* dwu, int B, int Hq, int Hkv, int T_, int d,
                              int dd, const BwdWs& L, hipStream_t st);
// Matrix-core backward (bf16, d in {64, 128}, d_down in {16, 32}).
bool bwd_mfma_supported(int d, int dd, bool bf16);
hipError_t launch_bwd_mfma(const bf16_t* q, const bf16_t* k, const bf16_t* v, const bf16_t* o,
                           const float* lse, const bf16_t* dout, const bf16_t* wd,
                           const bf16_t* wu, bf16_t* dq, bf16_t* dk, bf16_t* dv, float* dwd,
                           float* dwu, char* ws, const BwdWs& L, int B, int Hq, int Hkv, int T,
                           int d, int dd, int w, hipStream_t st);
template <typename T>
hipError_t launch_bwd_valu(const T* q, const T* k, const T* v, const T* o, const float* lse,
                           const T* dout, const T* wd, const T* wu, T* dq, T* dk, T* dv,
                           float* dwd, float* dwu, char* ws, const BwdWs& L, int B, int Hq,
                           int Hkv, int T_, int d, int dd, int w, hipStream_t st);

// Backward of the prefill with the rotary embedding (backward_mfma.hip;
// bf16, d in {64, 128}, any d_down). Inputs: q, k, v, o, dout, wd, wu (NULL:
// tied), lse (the forward's, natural log), tab [n_pos][r]; qr, kr, kd, vd:
// the rotary pre-pass of the same inputs (rotated queries and keys, lifted
// and rotated distant keys and lifted values of positions < T - w).
// Workspace arrays (fp32): nl2, nd [B*Hq][Tr] (Tr = round_up(T, 64)); dqr
// [B*Hq][T][d]; dkr, dvw [B*Hkv][T][d]; dkd, dvd [B*Hkv][T - w][d]; wpart
// [2][Hkv][L.nchunk][d][dd] with L.nchunk = B * ceil(T / 32).
struct RopeBwdArgs {
    const bf16_t *q, *k, *v, *o, *dout, *wd, *wu;
    const float* lse;
    const float* tab;
    const bf16_t *qr, *kr, *kd, *vd;
    float *nl2, *nd, *dqr, *dkr, *dvw, *dkd, *dvd, *wpart;
    bf16_t *dq, *dk, *dv;
    float *dwd, *dwu;
    BwdWs L;
    int B, Hq, Hkv, T, dd, w, r, pos0;
};
bool bwd_rope_mfma_supported(int d, int dd, bool bf16);
hipError_t launch_bwd_rope_mfma(const RopeBwdArgs& a, int d, hipStream_t st);

// Rotary embedding inside Eq. 3 (rope.hip): the angle table [n_pos][r] (cos
// of the r/2 angles of a position, then their sin; fp32 from fp64), the
// prefill pre-pass (rotated queries and keys; lifted, rotated distant keys
// and lifted values of positions < T - w; block norms when knorm/dnorm are
// given) and the generic attention over those arrays.
hipError_t launch_rope_table(int r, double base, int n_pos, float* tab, hipStream_t st);
template <typename T>
hipError_t launch_rope_prepass(const T* q, const T* k, const T* v, const T* wd, const T* wu,
                               const float* tab, T* qr, T* kr, T* kd, T* vd, float* knorm,
                               float* dnorm, int B, int Hq, int Hkv, int T_, int d, int dd, int w,
                               int r, int pos0, hipStream_t st);
// Pre-pass of a chunked prefill with the rotary embedding (n new tokens at
// positions len.., context rows ctx_k / ctx_v of positions kv0..len+n-1, kv0
// a multiple of 32): the rotated queries and context keys, the lifted and
// rotated distant keys and lifted values of positions < len + n - w (below
// len - w from the cache's latents, k_lat / v_lat with cap rows a head, the
// rest projected from the context rows), and the block norms of both key
// arrays in the matrix-core kernel's position-block layout.
template <typename T>
hipError_t launch_rope_chunk_prepass(const T* q, const T* ctx_k, const T* ctx_v, const T* k_lat,
                                     const T* v_lat, int cap, const T* wd, const T* wu,
                                     const float* tab, T* qr, T* kr, T* kd, T* vd, float* knorm,
                                     float* dnorm, int B, int Hq, int Hkv, int d, int dd, int w,
                                     int r, int len, int n, int kv0, hipStream_t st);
// Chunked prefill reading the cached latents in place (bf16, the shapes of
// prefill_mfma_supported). Per (batch, KV head) and 32-position block, the
// largest L2 norm of the stored key latents of positions [0, T - w) (cnorm,
// lc.ncb blocks a head) and of the context key rows of positions [kv0, T)
// (knorm, lc.nkb blocks), where T = len + n and kv0 = max(0, len - w) (paged:
// each sequence's own len and n); ctx_k row t of a head (kst rows a head)
// holds position kv0 + t. nblk: blocks to cover (the largest T over 32).
hipError_t launch_chunk_norms(const LatCache& lc, const bf16_t* ctx_k, int kst, float* cnorm,
                              float* knorm, int B, int Hkv, int d, int dd, int w, int len, int n,
                              int nblk, hipStream_t st);
// Paged chunk: context rows of sequence b (the ring's tokens from
// max(0, lens[b] - w), then its n_new[b] new ones; w + n rows a head).
hipError_t launch_chunk_gather_paged(const bf16_t* k_win, const bf16_t* v_win, const bf16_t* k_new,
                                     const bf16_t* v_new, bf16_t* ctx_k, bf16_t* ctx_v,
                                     const LatCache& lc, int B, int Hkv, int d, int w, int n,
                                     hipStream_t st);
// Paged chunk append: the n_new[b] tokens of sequence b at positions
// lens[b].., each window exit projected into its page slot (the arithmetic
// of launch_append), the newest min(n_new[b], w) tokens into the ring. lens
// is not changed (launch_lens_advance does it after the attention).
hipError_t launch_append_chunk_paged(const bf16_t* k_new, const bf16_t* v_new, const bf16_t* wd,
                                     bf16_t* k_win, bf16_t* v_win, bf16_t* k_pool, bf16_t* v_pool,
                                     const LatCache& lc, int B, int Hkv, int d, int dd, int w, int n,
                                     hipStream_t st);
// lens[b] += n_new[b] (n_new == nullptr: n) for each sequence it fits; one that
// does not fit (or was overflowed before) is marked -1 - lens[b].
hipError_t launch_lens_advance(int* lens, const int* n_new, int B, int cap, int n, hipStream_t st);
// Second stage of the split decodes: merges the S partial records of each
// (batch, query head) and lifts the latent part (decode_combine_kernel).
template <typename T>
hipError_t launch_decode_combine(const float* part, const T* wd, const T* wu, T* o, int B, int Hq,
                                 int Hkv, int d, int dd, int S, hipStream_t st,
                                 const T* wv = nullptr, const int* lens = nullptr,
                                 const int* counts = nullptr);
// Decode with the rotary embedding of Eq. 3 (query at position len - 1, cache
// token e at position e; positions < len index the table).
template <typename T>
hipError_t launch_decode_rope(const T* q, const T* wd, const T* wu, const T* k_win, const T* v_win,
                              const T* k_lat, const T* v_lat, const float* tab, int n_pos, T* o,
                              float* part, int B, int Hq, int Hkv, int d, int dd, int w, int cap,
                              int len, int r, hipStream_t st);
template <typename T>
hipError_t launch_prefill_rope_valu(const T* qr, const T* kr, const T* v, const T* kd, const T* vd,
                                    T* o, float* lse, int B, int Hq, int Hkv, int T_, int d, int w,
                                    hipStream_t st);
}  // namespace dar
