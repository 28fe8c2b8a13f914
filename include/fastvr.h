/*
 * fastvr.h -- C ABI of the chunk-wise causal attention library (libfastvr.so).
 *
 * The operation is the chunk-wise causal self-attention of FastVR
 * (arXiv 2609.36757, Sec. 3.1, Eq. 1 and the paragraph that follows it):
 * latent tokens, flattened frame-major, are grouped into temporal chunks of
 * `chunk_len` tokens; a query in chunk c sees every key of chunks
 * c - window_chunks .. c (bidirectional inside a chunk, nothing from later
 * chunks).  Eq. 1 is window_chunks = 1; window_chunks = -1 lifts the lower
 * bound (an unbounded causal prefix of chunks).  The same call serves the
 * parallel form over a whole sequence and the streaming form, where one new
 * query chunk attends to a KV cache (q_chunk_offset = that chunk's index
 * relative to the first cached chunk; only chunk differences matter).
 *
 *   LSE_i = ln sum_{j visible to i} exp(scale * q_i . k_j)
 *   O_i   = sum_{j visible to i} exp(scale * q_i . k_j - LSE_i) * v_j
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The library
 *    allocates nothing and keeps no pointer after returning.  Its only global
 *    state is a thread-local error string, caches (guarded, safe for concurrent
 *    callers) of each device's CU count and of the last few work plans of the
 *    forward, and the per-device static array of fastvr_chunk_attn_bwd_noalloc.
 *    Every entry point except that one is re-entrant.
 *  - `stream` is a hipStream_t passed as void*; NULL is the null stream.  Calls
 *    return after enqueueing; work is ordered on `stream`.  Faults during
 *    execution surface at the caller's next synchronisation of that stream.
 *  - Every argument is validated on the host BEFORE any HIP call.  A failing
 *    check returns a non-zero status, enqueues nothing, and leaves a message
 *    for fastvr_last_error().  No entry point throws or aborts.
 *  - Element types: bf16 inputs (16-bit brain float, round-to-nearest-even
 *    produced by the caller), fp32 outputs.
 */
#ifndef FASTVR_H
#define FASTVR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FASTVR_ABI_VERSION 7

typedef enum {
  FASTVR_OK = 0,
  FASTVR_ERR_INVALID_ARGUMENT = 1, /* null/misaligned pointer, bad size, offset, window, stride or scale */
  FASTVR_ERR_UNSUPPORTED = 2,      /* head_dim not in {64, 128}, or a problem too large for one launch */
  FASTVR_ERR_CAPACITY = 3,         /* a KV append would overflow the cache */
  FASTVR_ERR_HIP = 4               /* the HIP runtime refused a launch */
} fastvr_status;

/*
 * Chunk-causal attention forward (Sec. 3.1, Eq. 1; streaming form: last
 * paragraph of Sec. 3.1).
 *
 *   q   bf16 [B, Nq,  H, d] contiguous     query rows
 *   k   bf16 [B, Nkv, H, d] contiguous     key rows
 *   v   bf16 [B, Nkv, H, d] contiguous     value rows
 *   o   fp32 [B, Nq,  H, d] contiguous     output, fully overwritten
 *   lse fp32 [B, H, Nq]     contiguous     natural-log sum-exp per row, or NULL
 *
 * Query row i lies in chunk q_chunk_offset + i / chunk_len; key row j in chunk
 * j / chunk_len.  Keys of later chunks may be present in k/v; they are masked.
 *
 * Preconditions (else FASTVR_ERR_INVALID_ARGUMENT unless noted):
 *  - q, k, v, o non-NULL and 16-byte aligned; lse NULL or 4-byte aligned;
 *    o does not overlap q, k or v;
 *  - B, H, Nq, Nkv, chunk_len >= 0 and q_chunk_offset >= 0, with
 *    q_chunk_offset * chunk_len + Nq <= Nkv (every query sees its own key, so
 *    no softmax row is empty) and chunk_len >= 1 when Nq > 0;
 *  - d in {64, 128} (else FASTVR_ERR_UNSUPPORTED);
 *  - window_chunks >= -1;  scale finite;
 *  - no element count overflows int64.
 * B, H or Nq equal to 0 is an empty problem: FASTVR_OK, nothing enqueued.
 */
fastvr_status fastvr_chunk_attn_fwd(const void* q, const void* k, const void* v, float* o,
                                    float* lse, int64_t B, int64_t H, int64_t Nq, int64_t Nkv,
                                    int64_t d, int64_t chunk_len, int64_t q_chunk_offset,
                                    int64_t window_chunks, float scale, void* stream);

/*
 * Same operation with explicit element strides, for tensors that are views
 * (e.g. a KV cache [B, capacity, H, d] with capacity > Nkv and B > 1), and a
 * choice of output type: o_bf16 = 0 stores O as fp32, o_bf16 = 1 as bf16 (the
 * fp32 value rounded to nearest even).  Within a token, heads are contiguous
 * with stride d and head_dim elements are contiguous.  Strides are in elements:
 * *_sb between batches, *_st between tokens.  The bf16 strides must be
 * multiples of 8 and the fp32 ones of 4 (16-byte rows), and each must be
 * >= H * d.  lse is [B, H, Nq] contiguous.  o_bf16 not in {0, 1}:
 * FASTVR_ERR_INVALID_ARGUMENT.
 */
fastvr_status fastvr_chunk_attn_fwd_ex(const void* q, int64_t q_sb, int64_t q_st,
                                       const void* k, int64_t k_sb, int64_t k_st,
                                       const void* v, int64_t v_sb, int64_t v_st,
                                       void* o, int64_t o_sb, int64_t o_st, int32_t o_bf16, float* lse,
                                       int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                                       int64_t chunk_len, int64_t q_chunk_offset,
                                       int64_t window_chunks, float scale, void* stream);

/*
 * KV-cache append for streaming inference with KV caching (Sec. 3.1, last
 * paragraph): copies the new chunk's keys and values
 *   k_new, v_new  bf16 [B, n_new, H, d] contiguous
 * into the caches
 *   k_cache, v_cache  bf16 [B, capacity, H, d] contiguous
 * at token offset cache_len (tokens cache_len .. cache_len + n_new - 1 of each
 * batch).  Nothing is evicted; the caller tracks cache_len.
 * Preconditions: pointers non-NULL and 16-byte aligned, caches not overlapping
 * the new tensors; B, H, capacity, cache_len, n_new >= 0; d in {64, 128};
 * cache_len + n_new <= capacity (else FASTVR_ERR_CAPACITY).
 * n_new, B or H equal to 0: FASTVR_OK, nothing enqueued.
 */
fastvr_status fastvr_kv_cache_append(void* k_cache, void* v_cache, const void* k_new,
                                     const void* v_new, int64_t B, int64_t H, int64_t d,
                                     int64_t capacity, int64_t cache_len, int64_t n_new,
                                     void* stream);

/*
 * Streaming step with a bounded ring KV cache (Sec. 3.1, last paragraph:
 * streaming inference with KV caching, whose cache size stays O(k) for a
 * fixed chunk size k, independent of the video length).  The ring holds
 * W + 1 chunk slots, W = window_chunks (Eq. 1 is W = 1):
 *   k_ring, v_ring  bf16 [B, (W + 1) * chunk_len, H, d] contiguous
 * Chunk c of the stream occupies token rows s * chunk_len .. s * chunk_len +
 * chunk_len - 1 of slot s = c mod (W + 1).  For the new chunk c = chunk_index,
 * given
 *   q_new, k_new, v_new  bf16 [B, n_new, H, d] contiguous   its tokens,
 * one kernel
 *   1. computes the attention of q_new over the keys and values of chunks
 *      max(0, c - W) .. c in chunk order: chunk c from k_new / v_new, the earlier
 *      ones from their ring slots (they must be full chunks written by the
 *      previous steps of the same stream);
 *   2. writes k_new / v_new into slot c mod (W + 1) (the append, fused into the
 *      same launch; the slot held chunk c - W - 1, which chunk c does not see).
 * Outputs o fp32 [B, n_new, H, d] and lse fp32 [B, H, n_new] (or NULL) equal,
 * for the rows of chunk c, those of fastvr_chunk_attn_fwd over the whole
 * sequence with the same window_chunks.
 *
 * Preconditions (else FASTVR_ERR_INVALID_ARGUMENT unless noted):
 *  - all pointers except lse non-NULL and 16-byte aligned, lse NULL or 4-byte
 *    aligned; the ring, o and lse overlap no other argument;
 *  - B, H >= 0; 1 <= n_new <= chunk_len; chunk_index >= 0; 0 <= W;
 *  - W <= 7, d in {64, 128} and chunk_len a multiple of 4 (d = 128) or 8
 *    (d = 64), so that no DMA row group of the kernel straddles two chunks
 *    (else FASTVR_ERR_UNSUPPORTED);
 *  - scale finite; no element count overflows int64.
 * B or H equal to 0: FASTVR_OK, nothing enqueued.
 */
fastvr_status fastvr_chunk_attn_ring_step(const void* q_new, const void* k_new, const void* v_new,
                                          void* k_ring, void* v_ring, float* o, float* lse, int64_t B,
                                          int64_t H, int64_t n_new, int64_t d, int64_t chunk_len,
                                          int64_t chunk_index, int64_t window_chunks, float scale,
                                          void* stream);

/*
 * Backward of fastvr_chunk_attn_fwd (gradients for training with the
 * chunk-causal mask over the whole sequence, Sec. 3.1, Eq. 1), reusing the
 * forward's output and LSE.  With P_ij = exp(scale * q_i . k_j - LSE_i) on
 * visible pairs (0 elsewhere), D_i = sum_c dO_ic O_ic and
 * dS_ij = P_ij (dO_i . v_j - D_i):
 *   dV = P^T dO,   dQ = scale * dS K,   dK = scale * dS^T Q.
 *
 *   q, dout     bf16 [B, Nq,  H, d] contiguous   queries, upstream gradient dL/dO
 *   k, v        bf16 [B, Nkv, H, d] contiguous
 *   o           fp32 [B, Nq,  H, d] contiguous   forward output for (q, k, v)
 *   lse         fp32 [B, H, Nq]     contiguous   forward natural-log LSE
 *   dq          fp32 [B, Nq,  H, d] contiguous   output, fully overwritten
 *   dk, dv      fp32 [B, Nkv, H, d] contiguous   outputs, fully overwritten (zero for
 *                                                keys no query sees)
 *   row_stats   fp32 [B, H, 2, Nq]  contiguous   caller-owned workspace, written by
 *                                                the call: plane 0 LSE_i * log2 e,
 *                                                plane 1 -D_i
 * Mask arguments (chunk_len, q_chunk_offset, window_chunks) and scale are those
 * of the forward call that produced o and lse.  Two kernels run in order on
 * `stream`; sums run in a fixed order, so results are reproducible bit for bit.
 *
 * Preconditions (else FASTVR_ERR_INVALID_ARGUMENT unless noted):
 *  - q, k, v, dout, o, dq, dk, dv non-NULL and 16-byte aligned (q, dout, o, dq
 *    may be NULL when Nq = 0); lse and row_stats non-NULL and 4-byte aligned
 *    when Nq > 0;
 *  - dq, dk, dv and row_stats overlap no argument;
 *  - size, offset, window and scale rules of fastvr_chunk_attn_fwd, and
 *    H * d < 2^22 (else FASTVR_ERR_UNSUPPORTED).
 * B, H or Nkv equal to 0 (then Nq must be 0): FASTVR_OK, nothing enqueued.
 * Nq = 0 with Nkv > 0 sets dk and dv to zero.
 */
fastvr_status fastvr_chunk_attn_bwd(const void* q, const void* k, const void* v, const float* o, const float* lse,
                                    const void* dout, float* dq, float* dk, float* dv, float* row_stats, int64_t B,
                                    int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len,
                                    int64_t q_chunk_offset, int64_t window_chunks, float scale, void* stream);

/*
 * fastvr_chunk_attn_bwd without the row_stats workspace argument, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving or training loops, harnesses that forbid allocation).  The row
 * statistics go to a static array of the library instead, 32 MiB
 * (FASTVR_BWD_NOALLOC_MAX_FLOATS floats) that each device holds from the first
 * call until the process ends; the call itself allocates nothing (no hipMalloc,
 * no allocating library routine).  The caller still passes every input and
 * output, with the same meaning, layout and preconditions as in
 * fastvr_chunk_attn_bwd; outputs are identical bit for bit.
 *
 * Limit: 2 * B * H * Nq <= FASTVR_BWD_NOALLOC_MAX_FLOATS, else
 * FASTVR_ERR_UNSUPPORTED (the 1080p sequence needs 1.6 M floats, the 24-head
 * sliding-window sequence 6.7 M).  Every call on one device shares the array:
 * calls that may overlap in time on the same device (different streams or host
 * threads) race and must be serialised by the caller.  FASTVR_ERR_HIP if the
 * array's device address cannot be obtained.
 */
#define FASTVR_BWD_NOALLOC_MAX_FLOATS (8 * 1024 * 1024)
fastvr_status fastvr_chunk_attn_bwd_noalloc(const void* q, const void* k, const void* v, const float* o,
                                            const float* lse, const void* dout, float* dq, float* dk, float* dv,
                                            int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                                            int64_t chunk_len, int64_t q_chunk_offset, int64_t window_chunks,
                                            float scale, void* stream);

/*
 * One-step latent update (Sec. 3.2, Eq. 9, the update used at inference, Sec.
 * 4.1): z_hat = z_lq - sigma * v, element by element over n elements.
 *
 *   z_lq    bf16 [n]   the LQ latent z_LQ (any layout; v and z_hat share it)
 *   v       bf16 [n]   the velocity the DiT predicts at (z_LQ, tau)
 *   z_hat   fp32 [n] (out_bf16 = 0) or bf16 [n] (out_bf16 = 1)   output
 *   sigma   sigma_tau, the noise level of the starting timestep tau
 * Each element is fma(-sigma, v, z_lq) in fp32 (the exact value rounded once);
 * with out_bf16 = 1 that value is rounded to bf16 (nearest even).
 *
 * Preconditions (else FASTVR_ERR_INVALID_ARGUMENT): n >= 0; pointers non-NULL
 * and 16-byte aligned; sigma finite; out_bf16 in {0, 1}; z_hat overlaps neither
 * input, except that with out_bf16 = 1 it may be exactly z_lq or v (in place).
 * n = 0: FASTVR_OK, nothing enqueued.
 */
fastvr_status fastvr_one_step_update(const void* z_lq, const void* v, void* z_hat, int64_t n, float sigma,
                                     int32_t out_bf16, void* stream);

/*
 * Spatial tiles for tiled inference (Sec. 3 overview: one DiT pass per temporal
 * chunk and spatial tile; Sec. 4.1, Inference: overlapping 64 x 64 latent tiles).
 * The paper does not state the overlap, the placement or the blend; this library
 * takes the following, for fields laid out channels-last x[b, t, y, x, c] over a
 * grid of Hg x Wg positions and T frames (tiles span every frame and cut both
 * spatial axes the same way):
 *  - along an axis of `size` positions: tile length L = min(tile, size);
 *    n = 1 if size <= tile, else ceil((size - overlap) / (tile - overlap)) tiles
 *    at origins a_k = (k (size - L) + (n - 1) / 2) / (n - 1) (integer division):
 *    evenly spaced, a_0 = 0, a_{n-1} = size - L, neighbours overlapping by at
 *    least `overlap`;
 *  - tile (ty, tx) has index ty * nx + tx; a tile tensor is
 *    [B, ny * nx, T, Ly, Lx, C], so a tile batch feeds fastvr_chunk_attn_fwd
 *    directly (batch B * ny * nx, Nq = T * Ly * Lx tokens, chunk_len =
 *    frames per chunk * Ly * Lx);
 *  - blend: position i of a tile has the axis weight min(i + 1, L - i, R),
 *    R = max(overlap, 1); a tile's weight is the product of its two axis
 *    weights, and the blended value is the weight-normalised sum over the tiles
 *    that cover the position (fp32, tiles in index order).
 * Common preconditions (else FASTVR_ERR_INVALID_ARGUMENT unless noted): sizes
 * >= 0; tile >= 1 and 0 <= overlap < tile; tile <= 4096 (else
 * FASTVR_ERR_UNSUPPORTED); Wg * C < 2^31 (else FASTVR_ERR_UNSUPPORTED); tensors
 * contiguous, pointers 16-byte aligned (z_lq: 8-byte); outputs overlap no
 * input.  An empty field (any size 0): FASTVR_OK, nothing enqueued.
 */

/* Host only: number of tiles and tile length along one axis of `size` >= 1. */
fastvr_status fastvr_tile_axis(int64_t size, int64_t tile, int64_t overlap, int64_t* n_tiles, int64_t* tile_len);

/* tiles bf16 [B, ny*nx, T, Ly, Lx, C] <- x bf16 [B, T, Hg, Wg, C]; C a multiple of 8. */
fastvr_status fastvr_tile_gather(const void* x, void* tiles, int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C,
                                 int64_t tile, int64_t overlap, void* stream);

/* out fp32 [B, T, Hg, Wg, C] <- blend of tiles fp32 [B, ny*nx, T, Ly, Lx, C]; C a multiple of 4. */
fastvr_status fastvr_tile_blend(const float* tiles, float* out, int64_t B, int64_t T, int64_t Hg, int64_t Wg,
                                int64_t C, int64_t tile, int64_t overlap, void* stream);

/* The blend fused with the one-step update of Eq. 9 (Sec. 3.2):
 * z_hat fp32 [B, T, Hg, Wg, C] = z_lq - sigma * blend(v_tiles), z_lq bf16 of the
 * same shape (each element fma(-sigma, blend, z) in fp32); sigma finite. */
fastvr_status fastvr_tile_blend_update(const float* v_tiles, const void* z_lq, float* z_hat, float sigma, int64_t B,
                                       int64_t T, int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t overlap,
                                       void* stream);

/* Static string naming a status code ("FASTVR_OK", ...); never NULL. */
const char* fastvr_status_string(fastvr_status s);

/* Detail of the last failing call on this thread ("" if none).  The pointer is
   valid until the next library call on the same thread. */
const char* fastvr_last_error(void);

/* FASTVR_ABI_VERSION of the built library. */
int fastvr_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FASTVR_H */
