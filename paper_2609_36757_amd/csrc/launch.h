// Internal launch interface between the C-ABI layer and the HIP kernels.
// Arguments reaching these functions have already been validated.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "fastvr.h"

namespace fastvr {

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;               // fp32, or bf16 when o_bf16
  float* lse;            // may be null
  int64_t q_sb, q_st;    // element strides: batch, token (bf16)
  int64_t k_sb, k_st;
  int64_t v_sb, v_st;
  int64_t o_sb, o_st;    // fp32
  int64_t B, H, nq, nkv, d;
  int64_t chunk_len, q_chunk_offset, window_chunks;
  float scale;
  bool o_bf16 = false;
  // Ring step (k_ring != nullptr): k / v are the new chunk, the earlier visible
  // chunks come from the ring; the kernel also writes k / v into new_slot.
  void* k_ring = nullptr;
  void* v_ring = nullptr;
  int64_t ring_sb = 0;      // batch stride of the ring (elements)
  int64_t ring_slots = 0;   // window_chunks + 1
  int64_t ring_first = 0;   // slot of the oldest visible chunk
  int64_t n_seg = 0;        // visible chunks (the new one included)
  int64_t new_slot = 0;     // slot of the new chunk
};
constexpr int64_t kMaxRingWindow = 7;  // window_chunks of a ring step

// Work decomposition of one forward call (host side, also used for checks).
struct FwdGrid {
  int64_t n_local_chunks;  // query chunks touched by the call
  int64_t tiles_full;      // query tiles of a full chunk
  int64_t tiles_last;      // query tiles of the last (possibly ragged) chunk
  int64_t n_items;         // workgroups
};

constexpr int kFwdThreads = 512;  // 8 wave64 per workgroup
constexpr int kFwdRowsPerItem = 256;
constexpr int64_t kMaxFwdItems = (int64_t(1) << 32) / kFwdThreads - 1;
// 32-bit buffer offsets of a 256-row tile: token strides stay below 2^22 elements
constexpr int64_t kMaxTokenStride = int64_t(1) << 22;

FwdGrid fwd_grid(int64_t B, int64_t H, int64_t nq, int64_t chunk_len);
hipError_t launch_chunk_attn_fwd(const FwdArgs& a, hipStream_t stream);

// Backward of one chunk-causal attention call.  All tensors are contiguous
// [B, N, H, d] (lse and the row statistics [B, H, Nq]).
struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;    // bf16 upstream gradient dL/dO
  const float* o;      // forward output
  const float* lse;    // forward natural-log LSE
  float* dq;
  float* dk;
  float* dv;
  float* row_stats;    // [B, H, 2, Nq] workspace: lse * log2 e, then -rowsum(dO * O)
  int64_t B, H, nq, nkv, d;
  int64_t chunk_len, q_chunk_offset, window_chunks;
  float scale;
};

struct BwdGrid {
  FwdGrid q;               // dQ kernel: query tiles, as in the forward
  int64_t n_kchunks;       // key chunks of the key range
  int64_t kblocks_full;    // key blocks of a full chunk
  int64_t kblocks_last;    // key blocks of the last (possibly ragged) chunk
  int64_t n_kv_items;      // workgroups of the dK/dV kernel
};

constexpr int kBwdDqThreads = 512;   // 8 wave64, 32 queries each
constexpr int kBwdDkvThreads = 512;  // 8 wave64: 4 pairs, 32 keys each
constexpr int kBwdKeysPerItem = 128;

BwdGrid bwd_grid(int64_t B, int64_t H, int64_t nq, int64_t nkv, int64_t chunk_len);
hipError_t launch_chunk_attn_bwd(const BwdArgs& a, hipStream_t stream);

// The allocation-free backward keeps its row statistics (2 * B * H * Nq
// floats) in a static device array of this many floats (32 MiB) per device.
constexpr int64_t kBwdScratchFloats = FASTVR_BWD_NOALLOC_MAX_FLOATS;
// Device address of the current device's array (looked up once per device).
hipError_t bwd_scratch(float** out);

hipError_t launch_one_step(const void* z_lq, const void* v, void* z_hat, int64_t n, float sigma, bool out_bf16,
                           hipStream_t stream);

// Spatial tiles: tiles and tile length along one axis (host side, shared by the
// C ABI's checks and the launchers); n = 0 for an invalid geometry.
struct TileAxis {
  int64_t n, len;
};
constexpr int64_t kMaxTile = 4096;  // integer blend weights up to kMaxTile^2 stay exact in fp32
TileAxis tile_axis(int64_t size, int64_t tile, int64_t overlap);
hipError_t launch_tile_gather(const void* x, void* tiles, int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C,
                              int64_t tile, int64_t overlap, hipStream_t stream);
hipError_t launch_tile_blend(const float* tiles, const void* z_lq, float* out, float sigma, int64_t B, int64_t T,
                             int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t overlap, hipStream_t stream);

hipError_t launch_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new,
                            int64_t B, int64_t H, int64_t d, int64_t capacity, int64_t cache_len,
                            int64_t n_new, hipStream_t stream);

}  // namespace fastvr
