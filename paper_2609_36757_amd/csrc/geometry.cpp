// Work decomposition and tile placement on the host (plain C++, no HIP calls):
// shared by the C ABI's argument checks and the kernel launchers, and built
// on its own for the sanitizer check of the host layer.
#include "launch.h"

namespace fastvr {

// Forward: one work item per (batch, head, query chunk, query tile of
// kFwdRowsPerItem rows); tiles never straddle a chunk.
FwdGrid fwd_grid(int64_t B, int64_t H, int64_t nq, int64_t chunk_len) {
  FwdGrid g{};
  if (B <= 0 || H <= 0 || nq <= 0 || chunk_len <= 0) return g;
  g.n_local_chunks = (nq + chunk_len - 1) / chunk_len;
  const int64_t last_rows = nq - (g.n_local_chunks - 1) * chunk_len;
  g.tiles_last = (last_rows + kFwdRowsPerItem - 1) / kFwdRowsPerItem;
  g.tiles_full = g.n_local_chunks > 1 ? (chunk_len + kFwdRowsPerItem - 1) / kFwdRowsPerItem : g.tiles_last;
  g.n_items = B * H * (g.tiles_last + g.tiles_full * (g.n_local_chunks - 1));
  return g;
}

// Backward: the dQ kernel uses the forward's items; the dK/dV kernel one item
// per (batch, head, key chunk, block of kBwdKeysPerItem keys).
BwdGrid bwd_grid(int64_t B, int64_t H, int64_t nq, int64_t nkv, int64_t chunk_len) {
  BwdGrid g{};
  const int64_t L = chunk_len > nkv ? nkv : chunk_len;
  g.q = fwd_grid(B, H, nq, L);
  if (B <= 0 || H <= 0 || nkv <= 0 || L <= 0) return g;
  g.n_kchunks = (nkv + L - 1) / L;
  const int64_t last_keys = nkv - (g.n_kchunks - 1) * L;
  g.kblocks_last = (last_keys + kBwdKeysPerItem - 1) / kBwdKeysPerItem;
  g.kblocks_full = g.n_kchunks > 1 ? (L + kBwdKeysPerItem - 1) / kBwdKeysPerItem : g.kblocks_last;
  g.n_kv_items = B * H * (g.kblocks_last + g.kblocks_full * (g.n_kchunks - 1));
  return g;
}

// Tiles along one axis: length min(tile, size), and the fewest tiles at evenly
// spaced origins that cover the axis with neighbours overlapping by at least
// `overlap` positions (one tile when the axis fits in one).
TileAxis tile_axis(int64_t size, int64_t tile, int64_t overlap) {
  TileAxis a{};
  if (size < 1 || tile < 1 || overlap < 0 || overlap >= tile) return a;
  a.len = size < tile ? size : tile;
  a.n = size <= tile ? 1 : (size - overlap + (tile - overlap) - 1) / (tile - overlap);
  return a;
}

}  // namespace fastvr
