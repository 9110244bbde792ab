/*
 * dar.h — C ABI of libdar, Distance-Adaptive Representation (DAR) attention
 * on AMD Instinct MI355X (gfx950).
 *
 * Method (arXiv 2606.18587, "Dual Dimensionality for Local and Global
 * Attention", Section 2):
 *   Eq. 1  a token's bottleneck representation is c_j = x_j W_down (d -> d_down);
 *   Eq. 2  it is lifted back with W_up (d_down -> d) before use;
 *   Eq. 3  for query position i, token j <= i is used at full dimension if
 *          i - j < w (the window includes the current token) and in lifted
 *          form otherwise, for keys and for values alike;
 *   Eq. 4  o_i = softmax_j(q_i . k_j / sqrt(d)) v_j over j = 0..i, one softmax
 *          for both regions, d being the full per-head key dimension.
 * The Limitations section's efficient cache is what this library keeps for
 * decoding: full-dimension K/V for the last w tokens, the d_down latent for
 * every older token, with W_up absorbed into the query and the output:
 *   q . ((k W_down) W_up) = (q W_up^T) . (k W_down),
 *   sum_j p_j (c_j W_up) = (sum_j p_j c_j) W_up.
 *
 * Conventions for every entry point
 *   - Bottleneck per KV head: W_down [Hkv][d][d_down] maps each KV head's key
 *     and value (one matrix shared by K and V); W_up [Hkv][d_down][d], or NULL
 *     for the tied form W_up = W_down^T.
 *   - GQA: query head h reads KV head h / (Hq / Hkv).
 *   - Layout: row-major, contiguous, [B][H][T][d]. Every tensor of a call has
 *     the dtype of the shape (fp32 or bf16), except the weight gradients of
 *     the backward, which are fp32; bf16 runs accumulate in fp32.
 *   - Positions are 0-based and implicit (prefill: 0..T-1; decode: the query
 *     sits at position len-1 of the cache). The entry points without "rope"
 *     in their name take q and k as they are (a caller may rotate them first:
 *     then the distant key is the lift of the rotated key); the "rope" entry
 *     points apply the rotary embedding where Eq. 3 does.
 *   - Ownership: every tensor pointer is device memory owned by the caller.
 *     The library allocates nothing and keeps no state between calls beyond
 *     one-time per-device kernel attributes; calls on different streams with
 *     disjoint buffers may run concurrently.
 *   - Asynchrony: work is enqueued on `stream` (NULL = the default stream) and
 *     the call returns without synchronising. Kernel faults surface at the
 *     caller's next synchronisation.
 *   - Errors: arguments are validated before anything is enqueued; on any
 *     error status nothing has been written and the cache length is unchanged.
 *     Device pointers must be non-NULL and 16-byte aligned (W_up may be NULL).
 *     No exception crosses the ABI.
 */
#ifndef DAR_H
#define DAR_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DAR_OK = 0,
    DAR_E_ARG = 1,          /* bad shape, NULL or misaligned pointer          */
    DAR_E_UNSUPPORTED = 2,  /* valid, but outside what the kernels implement  */
    DAR_E_CAPACITY = 3,     /* cache append would exceed its capacity         */
    DAR_E_WORKSPACE = 4,    /* workspace missing or smaller than required     */
    DAR_E_HIP = 5           /* the HIP runtime refused a launch               */
} dar_status;

typedef enum { DAR_F32 = 0, DAR_BF16 = 1 } dar_dtype;

/* B batch, Hq query heads, Hkv KV heads (Hq % Hkv == 0), d head dimension,
 * d_down bottleneck dimension (1 <= d_down <= d), w window (w >= 0; w = 0
 * puts every token, including the query's own, in the bottleneck form). */
typedef struct {
    int B, Hq, Hkv, d, d_down, w;
    dar_dtype dtype;
} dar_shape;

/* Split KV cache (device buffers owned by the caller, this struct on the host).
 *   k_win, v_win [B][Hkv][w][d]       ring: token p lives in slot p % w while
 *                                       p >= len - w (unused when w == 0)
 *   k_lat, v_lat [B][Hkv][cap][d_down] latent of token e (= x_e W_down) in
 *                                       slot e for every e < len - w
 *   cap   maximum number of tokens     len   tokens appended so far          */
typedef struct {
    void *k_win, *v_win, *k_lat, *v_lat;
    int cap;
    int len;
} dar_cache;

/* Paged split cache with one length per sequence (serving: sequences of
 * different lengths in one batch, memory handed out in pages). Device
 * buffers owned by the caller, this struct on the host.
 *   k_win, v_win  [B][Hkv][w][d]      ring per sequence, token p in slot p % w
 *                                     while p >= lens[b] - w
 *   k_pool, v_pool [n_pages][Hkv][page_size][d_down]  latent pages: token e
 *                 of sequence b (e < lens[b] - w) in page
 *                 block_table[b * max_blocks + e / page_size], row
 *                 e % page_size (every KV head of the token in that page)
 *   block_table   device int [B][max_blocks] (caller-managed; an entry
 *                 outside [0, n_pages) is never read or written through:
 *                 such tokens are not stored and read as zeros)
 *   lens          device int [B], tokens held per sequence (the append
 *                 advances it on the device; the library never reads it on
 *                 the host). A negative entry -1 - n marks a sequence that
 *                 held n tokens when an append found it at capacity
 *                 (overflowed: not appended to or attended any more)
 *   page_size     a power of two, at least 32; capacity max_blocks *
 *                 page_size tokens per sequence */
typedef struct {
    void *k_win, *v_win, *k_pool, *v_pool;
    const int* block_table;
    int* lens;
    int page_size, max_blocks, n_pages;
} dar_paged_cache;

/* Causal prefill over positions 0..T-1 (Eq. 3-4 for every row).
 *   q [B][Hq][T][d], k, v [B][Hkv][T][d], w_down [Hkv][d][d_down],
 *   w_up [Hkv][d_down][d] or NULL (tied), o [B][Hq][T][d] (output).
 *   ws: device workspace of at least dar_prefill_workspace_bytes(s, T) bytes
 *   (never NULL; caller-owned, overwritten by the call): latents of the
 *   tokens that are distant for some row (Eq. 1), per-32-token norm maxima
 *   and constant operand rows. T >= 1.
 * Supported: fp32 with d <= 256; bf16 with d <= 256 (d in {64, 128} with
 * d_down in {16, 32} take the matrix-core path). */
dar_status dar_attn_prefill(const dar_shape* s, int T, const void* q, const void* k,
                            const void* v, const void* w_down, const void* w_up, void* o,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* dar_attn_prefill that also writes each row's softmax statistics for a
 * backward pass (Section 2.3 trains through this attention):
 *   lse: NULL (then identical to dar_attn_prefill), or fp32 [B][Hq][T]
 *   (output): the natural log of each row's softmax denominator,
 *   log sum_j exp(S_ij) with S_ij the scaled score of Eq. 4;
 *   dar_attn_prefill_backward takes it.
 * Every other argument, the output o and the support are those of
 * dar_attn_prefill; asking for lse changes no bit of o. */
dar_status dar_attn_prefill_lse(const dar_shape* s, int T, const void* q, const void* k,
                                const void* v, const void* w_down, const void* w_up, void* o,
                                float* lse, void* ws, size_t ws_bytes, hipStream_t stream);

/* Causal prefill of a ragged batch: sequence b of the padded batch holds
 * seq_lens[b] tokens (device int [B], each in [0, T]); q, k, v, o, lse are laid
 * out as for dar_attn_prefill with T the padded length. Row i of sequence b,
 * i < seq_lens[b], is Eq. 3-4 over that sequence's positions 0..i; positions
 * at or past seq_lens[b] are never read (their contents do not matter) and
 * those rows of o and lse are not written. Workspace and support as for
 * dar_attn_prefill. */
dar_status dar_attn_prefill_ragged(const dar_shape* s, int T, const int* seq_lens, const void* q,
                                   const void* k, const void* v, const void* w_down,
                                   const void* w_up, void* o, float* lse, void* ws,
                                   size_t ws_bytes, hipStream_t stream);

/* Append n >= 1 tokens k_new, v_new [B][Hkv][n][d] at positions len..len+n-1.
 * Every token that leaves the window (position len+t-w for t < n) is
 * down-projected with W_down (Eq. 1, fp32 accumulation, rounded to the cache
 * dtype) into its latent slot; the newest min(n, w) tokens are written to the
 * ring. The result is bit-identical to n single-token appends. On success
 * c->len += n (host side, at enqueue time). Fails with DAR_E_CAPACITY if
 * len + n > cap. */
dar_status dar_cache_append(const dar_shape* s, dar_cache* c, const void* k_new,
                            const void* v_new, int n, const void* w_down, hipStream_t stream);

/* Chunked prefill into a split cache (serving: a prompt arriving in pieces, or
 * a batch of new tokens appended at once). The n >= 1 new tokens sit at
 * positions len..len+n-1 (len = c->len) with queries q [B][Hq][n][d] and keys
 * and values k_new, v_new [B][Hkv][n][d]. Every new row i attends to the
 * positions 0..i under Eq. 3-4 exactly as row i of dar_attn_prefill over the
 * whole sequence 0..len+n-1 would: the window tokens come from the cache's
 * ring and from k_new/v_new at full dimension, older tokens from the cache's
 * latents (Eq. 1, absorbed as in dar_attn_prefill). The cache is then
 * extended by the n tokens exactly as dar_cache_append(s, c, k_new, v_new, n,
 * w_down) extends it (bit-identical ring and latents; c->len += n at enqueue
 * time).
 *   o [B][Hq][n][d] (output); lse: NULL or fp32 [B][Hq][n] (output, as for
 *   dar_attn_prefill); w_up: [Hkv][d_down][d] or NULL (tied).
 *   ws: device workspace of at least dar_prefill_chunk_workspace_bytes(s, len,
 *   n) bytes (caller-owned, overwritten): a copy of the ring's tokens and the
 *   new ones, and, on the matrix-core shapes (bf16, d in {64, 128}, d_down in
 *   {16, 32}), the block norms of the keys (the cache's latents are read in
 *   place), else a prefill workspace of len + n positions (the cache's
 *   latents are re-laid out into it).
 * Fails with DAR_E_CAPACITY if len + n > cap (nothing is enqueued). Supported:
 * as dar_attn_prefill, with d * (element size) a multiple of 4 bytes. */
dar_status dar_attn_prefill_chunk(const dar_shape* s, dar_cache* c, int n, const void* q,
                                  const void* k_new, const void* v_new, const void* w_down,
                                  const void* w_up, void* o, float* lse, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/* Rotary position embedding inside Eq. 3. Eq. 3 rotates the key of both
 * paths: the window key is RoPE(k_j), the distant key is RoPE of the lifted
 * key, RoPE((k_j W_down) W_up); values are not rotated; the query is rotated
 * at its own position. Rotate-half pairing: for m < r/2 the pair
 * (x[m], x[m + r/2]) of a row at position p turns by the angle
 * p * base^(-2m/r); elements r..d-1 are left as they are.
 *   rotary_dim  r: even, 0 <= r <= d (0: no rotation)
 *   n_pos       positions the table covers (0..n_pos-1)
 *   table       device fp32 [n_pos][r]: cos of the r/2 angles of position p,
 *               then their sin (dar_rope_table writes it; caller-owned) */
typedef struct {
    int rotary_dim;
    int n_pos;
    const float* table;
} dar_rope;

/* Fills table [n_pos][rotary_dim] (device, caller-owned) for the base
 * frequency `base` (10000 in the original rotary embedding), computing each
 * angle and its cos/sin in fp64 and rounding to fp32. rotary_dim even in
 * [2, 256], 1 <= n_pos <= 65535, base > 0. */
dar_status dar_rope_table(int rotary_dim, double base, int n_pos, float* table, hipStream_t stream);

/* Causal prefill with the rotary embedding of Eq. 3: rows at positions
 * pos0..pos0+T-1 (pos0 >= 0, pos0 + T <= rope->n_pos). q, k are the
 * un-rotated queries and keys (q = h W_Q, k = h W_K); everything else as for
 * dar_attn_prefill (lse included). Because the rotation does not commute with
 * W_up, the distant keys are lifted and rotated to full d in the workspace
 * (not absorbed into the query), so the attention costs as much as full
 * causal attention; the cache the decode keeps is unchanged (latents of the
 * un-rotated keys).
 *   ws: at least dar_prefill_rope_workspace_bytes(s, T) bytes (caller-owned,
 *   overwritten): rotated queries and keys, lifted distant keys and values,
 *   and block norms.
 * Supported: fp32 and bf16 with d <= 256 (bf16 with d in {64, 128}, any
 * d_down, takes the matrix-core path). */
dar_status dar_attn_prefill_rope(const dar_shape* s, int T, int pos0, const dar_rope* rope,
                                 const void* q, const void* k, const void* v, const void* w_down,
                                 const void* w_up, void* o, float* lse, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* Chunked prefill (as dar_attn_prefill_chunk) with the rotary embedding of
 * Eq. 3 (as dar_attn_prefill_rope): the n new tokens at positions
 * len..len+n-1 (len = c->len, len + n <= rope->n_pos) with un-rotated q,
 * k_new, v_new; window keys are rotated at their positions, distant keys are
 * lifted and then rotated: those below len - w from the cache's latents
 * (c^K W_up), the others projected from the ring or the chunk
 * ((k W_down) W_up), as the decode with rotation treats them. The cache is
 * extended by the un-rotated tokens exactly as dar_cache_append extends it
 * (c->len += n at enqueue time).
 *   o [B][Hq][n][d] (output); lse: NULL or fp32 [B][Hq][n].
 *   ws: at least dar_prefill_chunk_rope_workspace_bytes(s, len, n) bytes
 *   (caller-owned, overwritten): the window's and the chunk's rows, rotated
 *   queries and keys, lifted distant keys and values of positions below
 *   len + n - w (full d), and block norms.
 * Fails with DAR_E_CAPACITY if len + n > cap. Supported: the matrix-core
 * shapes (bf16, d in {64, 128}, any d_down) with rotary_dim a multiple of
 * 16; other shapes return DAR_E_UNSUPPORTED. */
dar_status dar_attn_prefill_chunk_rope(const dar_shape* s, dar_cache* c, const dar_rope* rope,
                                       int n, const void* q, const void* k_new, const void* v_new,
                                       const void* w_down, const void* w_up, void* o, float* lse,
                                       void* ws, size_t ws_bytes, hipStream_t stream);

/* One decode step for the query q [B][Hq][d] at position c->len - 1, whose own
 * key and value must already have been appended. o [B][Hq][d] (output).
 * ws: device workspace of at least dar_decode_workspace_bytes(s, c->cap)
 * bytes. Requires c->len >= 1. */
dar_status dar_attn_decode(const dar_shape* s, const dar_cache* c, const void* q,
                           const void* w_down, const void* w_up, void* o, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* dar_attn_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, hosts that forbid allocation): no
 * workspace argument. The partial records a call may need live in a
 * fixed device array inside the library, dar_decode_noalloc_max_bytes()
 * bytes (16 MiB) per GPU, created when the library is loaded on that GPU and
 * held until the process ends; the call allocates nothing.
 *   dar_decode_noalloc_bytes(s, len): bytes of that array a call at cache
 *   length len uses (0 when one workgroup per (batch, KV head) finishes the
 *   output itself, as at B32 Hkv8); 0 also on an invalid shape.
 * Arguments, output and support as dar_attn_decode. Fails with
 * DAR_E_WORKSPACE, before anything is enqueued, when the call would need
 * more than dar_decode_noalloc_max_bytes(). Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (different streams
 * without ordering between them) race and must not be issued; calls in one
 * stream are ordered and safe. Nothing in the array needs to start at zero
 * (every record a call reads, that call writes first). */
dar_status dar_attn_decode_noalloc(const dar_shape* s, const dar_cache* c, const void* q,
                                   const void* w_down, const void* w_up, void* o,
                                   hipStream_t stream);
size_t dar_decode_noalloc_bytes(const dar_shape* s, int len);
size_t dar_decode_noalloc_max_bytes(void);

/* One decode step with the rotary embedding of Eq. 3: the query q [B][Hq][d]
 * (un-rotated) sits at position c->len - 1 and cache token e at position e
 * (c->len <= rope->n_pos). The cache is the one dar_cache_append keeps (ring
 * of un-rotated keys and values, latents of the un-rotated keys): each ring
 * key is rotated at its position, each distant key is lifted from its latent
 * to full d and rotated (Eq. 3; the rotation does not commute with W_up, so
 * W_up cannot be absorbed into the query for the keys); the distant values
 * are summed in d_down space and lifted once. ws, o and the other arguments
 * as for dar_attn_decode (same workspace size). */
dar_status dar_attn_decode_rope(const dar_shape* s, const dar_cache* c, const dar_rope* rope,
                                const void* q, const void* w_down, const void* w_up, void* o,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/* One token per sequence appended to a paged cache: k_new, v_new
 * [B][Hkv][d] at position lens[b] of each sequence. The token leaving the
 * window (position lens[b] - w) is projected with W_down (Eq. 1, the same
 * arithmetic as dar_cache_append, bit-identical latents) into its page slot;
 * the new token goes to the ring; then lens[b] += 1 on the device (stream
 * order). A sequence found at capacity (lens[b] == max_blocks * page_size)
 * stores nothing and is marked overflowed: lens[b] becomes -1 - lens[b]
 * (the caller may read it back to detect the overflow); an overflowed
 * sequence stays as it is under later appends. The pages of the blocks being
 * written must be mapped in block_table. */
dar_status dar_cache_append_paged(const dar_shape* s, const dar_paged_cache* c, const void* k_new,
                                  const void* v_new, const void* w_down, hipStream_t stream);

/* One decode step over a paged cache: the query q [B][Hq][d] of sequence b
 * sits at position lens[b] - 1 (its own key and value already appended;
 * lens[b] >= 1). A sequence with lens[b] < 1 (empty, or marked overflowed by
 * the append) has no query position: its rows of o are written as NaN, the
 * other sequences' are unaffected. As dar_attn_decode otherwise; ws: at least
 * dar_decode_workspace_bytes(s, max_blocks * page_size) bytes. Supported:
 * the matrix-core shapes (bf16, d in {64, 128}, d_down in {16, 32},
 * Hq / Hkv in {1, 2, 4, 8}). */
dar_status dar_attn_decode_paged(const dar_shape* s, const dar_paged_cache* c, const void* q,
                                 const void* w_down, const void* w_up, void* o, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* dar_attn_decode_paged with the rotary embedding of Eq. 3, applied as
 * dar_attn_decode_rope applies it (query of sequence b at position
 * lens[b] - 1, cache token e at position e). rope->n_pos must be at least
 * the capacity max_blocks * page_size (every position a sequence can reach
 * indexes the table), else DAR_E_ARG; rope NULL, an odd rotary_dim or one
 * above d: DAR_E_ARG. Supported: the shapes of dar_attn_decode_paged with
 * rotary_dim 16, 32 or 64 (0: no rotation, the table is not read); others
 * return DAR_E_UNSUPPORTED. Workspace, output and empty or overflowed
 * sequences as for dar_attn_decode_paged. */
dar_status dar_attn_decode_paged_rope(const dar_shape* s, const dar_paged_cache* c,
                                      const dar_rope* rope, const void* q, const void* w_down,
                                      const void* w_up, void* o, void* ws, size_t ws_bytes,
                                      hipStream_t stream);

/* Chunked prefill over a paged cache (serving: several sequences of different
 * lengths taking their next prompt tokens in one call). Sequence b takes
 * n_b = n_new[b] new tokens (n_new: device int [B], each clamped to [0, n];
 * NULL: every sequence takes n) at positions lens[b]..lens[b]+n_b-1, with
 * queries q [B][Hq][n][d] and keys and values k_new, v_new [B][Hkv][n][d]
 * (rows at or past n_b are never read). Every new row of sequence b attends
 * to that sequence's positions 0..i under Eq. 3-4 exactly as row i of
 * dar_attn_prefill over its whole sequence would (window tokens from its
 * ring and the chunk at full dimension, older ones from its latent pages,
 * Eq. 1, absorbed). The cache is extended as n_b single-token
 * dar_cache_append_paged calls would extend it (bit-identical ring and
 * latent pages), then lens[b] += n_b on the device.
 *   o [B][Hq][n][d] (output; rows at or past n_b are not written); lse: NULL
 *   or fp32 [B][Hq][n] (output, as for dar_attn_prefill).
 *   A sequence with n_b > 0 whose chunk does not fit (lens[b] < 0, or
 *   lens[b] + n_b > max_blocks * page_size) stores nothing, gets NaN rows
 *   and is marked overflowed (lens[b] = -1 - lens[b] if it was >= 0).
 *   The pages of every block written must be mapped in block_table.
 *   ws: at least dar_prefill_chunk_paged_workspace_bytes(s, max_blocks *
 *   page_size, n) bytes (caller-owned, overwritten): the window's and the
 *   chunk's rows of every sequence and the block norms.
 * The latent pages are read in place (nothing is copied out of them).
 * Supported: the matrix-core shapes (bf16, d in {64, 128}, d_down in {16,
 * 32}); others return DAR_E_UNSUPPORTED. */
dar_status dar_attn_prefill_chunk_paged(const dar_shape* s, const dar_paged_cache* c, int n,
                                        const int* n_new, const void* q, const void* k_new,
                                        const void* v_new, const void* w_down, const void* w_up,
                                        void* o, float* lse, void* ws, size_t ws_bytes,
                                        hipStream_t stream);

/* Single shared latent (the Limitations section's cache): one d_down latent
 * per token and KV head, c_j = h_j W_down of Eq. 1, from which both the
 * distant key and the distant value are computed. With the lift of Eq. 2
 * followed by the key and value projections, distant key = c_j U_K and
 * distant value = c_j U_V, where U_K = W_up W_K and U_V = W_up W_V per KV head
 * ([Hkv][d_down][d] each). The latent is an input, projected from the hidden
 * state by the caller like q, k and v; window keys and values are k, v (Eq. 3).
 * The distant cache is one latent array instead of two.
 *   Prefill: c [B][Hkv][T][d_down]; other arguments as dar_attn_prefill (same
 *   workspace size, dar_prefill_workspace_bytes). Supported as dar_attn_prefill.
 *   Append: the latent slot of each of the n new tokens (positions
 *   len..len+n-1) takes c_new [B][Hkv][n][d_down] as given (every token, the
 *   window's included); the ring takes the newest min(n, w) tokens of k_new,
 *   v_new. c->k_lat holds the latents; c->v_lat is not used (may be NULL).
 *   Fails with DAR_E_CAPACITY if len + n > cap.
 *   Decode: as dar_attn_decode over such a cache (same workspace size). */
dar_status dar_attn_prefill_shared(const dar_shape* s, int T, const void* q, const void* k,
                                   const void* v, const void* c, const void* u_k, const void* u_v,
                                   void* o, float* lse, void* ws, size_t ws_bytes,
                                   hipStream_t stream);
dar_status dar_cache_append_shared(const dar_shape* s, dar_cache* cache, const void* k_new,
                                   const void* v_new, const void* c_new, int n,
                                   hipStream_t stream);
dar_status dar_attn_decode_shared(const dar_shape* s, const dar_cache* cache, const void* q,
                                  const void* u_k, const void* u_v, void* o, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/* Backward of dar_attn_prefill: the gradients of L = sum(dout * o) with
 * respect to q, k, v, W_down and W_up (the training setting of Section 2.3,
 * whose objective is Eq. 5; the bottleneck weights receive gradient only
 * through the pairs whose query takes the distant path).
 *   q, k, v, w_down, w_up: the forward's inputs (w_up NULL = tied);
 *   o [B][Hq][T][d]: the forward's output (used for delta_i = dout_i . o_i);
 *   lse fp32 [B][Hq][T]: the log-sum-exp the forward call wrote (its lse
 *   argument); the softmax is recomputed against it, not re-normalised;
 *   dout [B][Hq][T][d]: the incoming gradient;
 *   dq [B][Hq][T][d], dk, dv [B][Hkv][T][d]: outputs in the shape's dtype;
 *   dw_down [Hkv][d][d_down], dw_up [Hkv][d_down][d]: fp32 outputs whatever
 *   the shape's dtype (sums over every row of the batch). Tied (w_up NULL):
 *   dw_up must be NULL and dw_down receives the gradient of the shared matrix,
 *   dW_down + dW_up^T. Untied: dw_up must be non-NULL.
 *   Every output is overwritten (not accumulated into).
 *   ws: device workspace of at least dar_prefill_backward_workspace_bytes(s, T)
 *   bytes (caller-owned, overwritten). The result does not depend on the
 *   stream or on timing: every reduction runs in a fixed order.
 * Supported: as dar_attn_prefill. */
dar_status dar_attn_prefill_backward(const dar_shape* s, int T, const void* q, const void* k,
                                     const void* v, const void* w_down, const void* w_up,
                                     const void* o, const float* lse, const void* dout, void* dq,
                                     void* dk, void* dv, float* dw_down, float* dw_up, void* ws,
                                     size_t ws_bytes, hipStream_t stream);

/* Backward of dar_attn_prefill_rope: the gradients of L = sum(dout * o) with
 * respect to the un-rotated q, k, v and W_down, W_up (Section 2.3 trains
 * through the attention, Eq. 3 puts the rotation inside it). The window keys
 * are R_j k_j, the distant keys R_j ((k_j W_down) W_up), so a distant pair's
 * key gradient is rotated back (R_j^T) before it goes through the lift.
 *   T, pos0, rope: as for the forward call; q, k, v, w_down, w_up, o, lse:
 *   its inputs, its output and the log-sum-exp it wrote; dout [B][Hq][T][d].
 *   Outputs as for dar_attn_prefill_backward (dq, dk, dv in bf16; dw_down,
 *   dw_up fp32, dw_up NULL exactly when w_up is NULL, the tied case then in
 *   dw_down); every output is overwritten, every reduction runs in a fixed
 *   order.
 *   ws: at least dar_prefill_rope_backward_workspace_bytes(s, T) bytes
 *   (caller-owned, overwritten): the rotated and lifted operands and fp32
 *   gradient arrays of the full-d distant keys.
 * Supported: bf16 with d in {64, 128}, any rotary_dim, d_down up to d (up to
 * 64 at d = 128); other shapes return DAR_E_UNSUPPORTED. */
dar_status dar_attn_prefill_rope_backward(const dar_shape* s, int T, int pos0, const dar_rope* rope,
                                          const void* q, const void* k, const void* v,
                                          const void* w_down, const void* w_up, const void* o,
                                          const float* lse, const void* dout, void* dq, void* dk,
                                          void* dv, float* dw_down, float* dw_up, void* ws,
                                          size_t ws_bytes, hipStream_t stream);

/* Workspace sizes (0 on an invalid shape). */
size_t dar_prefill_workspace_bytes(const dar_shape* s, int T);
size_t dar_decode_workspace_bytes(const dar_shape* s, int cap);
size_t dar_prefill_backward_workspace_bytes(const dar_shape* s, int T);
size_t dar_prefill_chunk_workspace_bytes(const dar_shape* s, int len, int n);
size_t dar_prefill_rope_workspace_bytes(const dar_shape* s, int T);
size_t dar_prefill_chunk_rope_workspace_bytes(const dar_shape* s, int len, int n);
size_t dar_prefill_chunk_paged_workspace_bytes(const dar_shape* s, int cap, int n);
size_t dar_prefill_rope_backward_workspace_bytes(const dar_shape* s, int T);

/* Static English text for a status code. */
const char* dar_status_string(dar_status st);

#ifdef __cplusplus
}
#endif
#endif /* DAR_H */
