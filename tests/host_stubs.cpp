// Stand-ins for the kernel launchers, linked with the C-ABI layer
// (fastvr_api.cpp) and the host geometry (geometry.cpp) into a host-only
// library for the address- and undefined-behaviour-sanitizer check
// (tests/test_host_sanitizers.py).  They launch nothing and touch no memory:
// each counts the call and checks the argument invariants the real launcher
// relies on (validation happened before).
#include <hip/hip_runtime_api.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>

#include "launch.h"

namespace {
std::atomic<int64_t> g_launches{0};

hipError_t record(bool invariants_hold) {
  if (!invariants_hold) std::abort();  // a validated call reached a launcher with bad arguments
  g_launches.fetch_add(1);
  return hipSuccess;
}
}  // namespace

extern "C" int64_t fastvr_stub_launch_count(void) { return g_launches.load(); }

extern "C" const char* hipGetErrorString(hipError_t) { return "stub"; }

namespace fastvr {

hipError_t launch_chunk_attn_fwd(const FwdArgs& a, hipStream_t) {
  const FwdGrid g = fwd_grid(a.B, a.H, a.nq, a.chunk_len > a.nkv ? a.nkv : a.chunk_len);
  return record(a.q && a.k && a.v && a.o && a.B > 0 && a.H > 0 && a.nq > 0 && a.nkv >= a.nq &&
                (a.d == 64 || a.d == 128) && g.n_items > 0 && g.n_items <= kMaxFwdItems &&
                a.q_st < kMaxTokenStride && a.k_st < kMaxTokenStride && a.v_st < kMaxTokenStride &&
                a.o_st < kMaxTokenStride && (a.k_ring == nullptr || (a.ring_slots >= 1 && a.n_seg >= 1)));
}

hipError_t launch_chunk_attn_bwd(const BwdArgs& a, hipStream_t) {
  const BwdGrid g = bwd_grid(a.B, a.H, a.nq, a.nkv, a.chunk_len);
  return record(a.k && a.v && a.dk && a.dv && a.B > 0 && a.H > 0 && a.nkv > 0 && a.nq >= 0 &&
                (a.nq == 0 || (a.q && a.dout && a.o && a.lse && a.dq && a.row_stats)) && g.n_kv_items > 0 &&
                g.n_kv_items <= kMaxFwdItems);
}

// a fake, aligned device address: the stand-in launchers never touch memory
hipError_t bwd_scratch(float** out) {
  *out = reinterpret_cast<float*>(uintptr_t(1) << 44);
  return hipSuccess;
}

hipError_t launch_one_step(const void* z_lq, const void* v, void* z_hat, int64_t n, float, bool, hipStream_t) {
  return record(z_lq && v && z_hat && n > 0);
}

hipError_t launch_tile_gather(const void* x, void* tiles, int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C,
                              int64_t tile, int64_t overlap, hipStream_t) {
  const TileAxis ay = tile_axis(Hg, tile, overlap), ax = tile_axis(Wg, tile, overlap);
  return record(x && tiles && B > 0 && T > 0 && C % 8 == 0 && ay.n > 0 && ax.n > 0);
}

hipError_t launch_tile_blend(const float* tiles, const void*, float* out, float, int64_t B, int64_t T, int64_t Hg,
                             int64_t Wg, int64_t C, int64_t tile, int64_t overlap, hipStream_t) {
  const TileAxis ay = tile_axis(Hg, tile, overlap), ax = tile_axis(Wg, tile, overlap);
  return record(tiles && out && B > 0 && T > 0 && C % 4 == 0 && ay.n > 0 && ax.n > 0);
}

hipError_t launch_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new, int64_t B, int64_t H,
                            int64_t d, int64_t capacity, int64_t cache_len, int64_t n_new, hipStream_t) {
  return record(k_cache && v_cache && k_new && v_new && B > 0 && H > 0 && (d == 64 || d == 128) && n_new > 0 &&
                cache_len + n_new <= capacity);
}

}  // namespace fastvr
