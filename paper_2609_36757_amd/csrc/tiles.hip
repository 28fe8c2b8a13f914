// Spatial tiling of the latent for tiled inference (FastVR, Sec. 3 overview and
// Sec. 4.1: the DiT runs once per temporal chunk and overlapping 64 x 64 latent
// tile).  Fields are channels-last, x[b, t, y, x, c]; tiles span every frame and
// cut the two spatial axes identically:
//  * placement along an axis of `size`: tile length L = min(tile, size),
//    n = 1 if size <= tile else ceil((size - overlap) / (tile - overlap)) tiles
//    at evenly spaced origins a_k = (k (size - L) + (n - 1) / 2) / (n - 1)
//    (integer division), so a_0 = 0, a_{n-1} = size - L and neighbours overlap
//    by at least `overlap`;
//  * gather: tiles[b, ty * nx + tx, t, iy, ix, c] = x[b, t, a_ty + iy, a_tx + ix, c];
//  * blend: axis weight of tile position i is min(i + 1, L - i, R), R =
//    max(overlap, 1); a tile's weight at a position is the product of its two
//    axis weights, and the field is the weight-normalised sum over the tiles
//    covering the position.  Optionally fused with the one-step update of
//    Eq. 9: z_hat = z_LQ - sigma * blend(v tiles).
// Both kernels are bound by HBM bandwidth.  The gather copies each tile row (a
// contiguous run in source and destination) with 16-byte vectors; the blend
// gathers, for each output element, the few tiles covering it (no atomics), with
// the covering tiles of a run of positions found in closed form.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gfx950_ops.h"
#include "launch.h"

namespace fastvr {
namespace {

using namespace dev;

constexpr int kThreads = 256;

struct Axis {
  int n, L, span;  // tiles, tile length, size - L
};

__device__ __forceinline__ int origin(const Axis& a, int k) {
  return a.n == 1 ? 0 : (int)(((int64_t)k * a.span + (a.n - 1) / 2) / (a.n - 1));
}

__device__ __forceinline__ int axis_weight(int i, int L, int R) {
  const int m = (i + 1 < L - i) ? i + 1 : L - i;
  return m < R ? m : R;
}

// One tile row (b, tile, t, iy) per loop step of a workgroup; 16-byte units.
__global__ __launch_bounds__(kThreads) void tile_gather_kernel(const u32x4* __restrict__ x, u32x4* __restrict__ tiles,
                                                               int T, int Hg, int Wg, int C16, Axis ay, Axis ax,
                                                               int64_t n_rows) {
  const int64_t row_units = (int64_t)ax.L * C16;
  for (int64_t r = blockIdx.x; r < n_rows; r += gridDim.x) {
    // r = ((b * nt + tile) * T + t) * Ly + iy  (wave-uniform)
    int64_t q = r;
    const int iy = (int)(q % ay.L);
    q /= ay.L;
    const int t = (int)(q % T);
    q /= T;
    const int nt = ay.n * ax.n;
    const int tile = (int)(q % nt);
    const int64_t b = q / nt;
    const int ty = tile / ax.n, tx = tile - ty * ax.n;
    const int y = origin(ay, ty) + iy, x0 = origin(ax, tx);
    const u32x4* src = x + (((b * T + t) * Hg + y) * (int64_t)Wg + x0) * C16;
    u32x4* dst = tiles + r * row_units;
    for (int64_t u = threadIdx.x; u < row_units; u += kThreads) __builtin_nontemporal_store(src[u], dst + u);
  }
}

// Index arithmetic of the blend in type I: uint32_t when every numerator below
// fits (the usual case), uint64_t otherwise.
template <typename I>
__device__ __forceinline__ int origin_t(const Axis& a, int k) {
  return a.n == 1 ? 0 : (int)(((I)k * (I)a.span + (I)((a.n - 1) / 2)) / (I)(a.n - 1));
}

// Last tile starting at or before position p: the largest k with origin(k) <= p.
// origin(k) <= p  <=>  k * span + (n - 1) / 2 < (p + 1)(n - 1), solved for k.
template <typename I>
__device__ __forceinline__ int last_start_le(const Axis& a, int p) {
  if (a.n == 1) return 0;
  const I num = (I)(p + 1) * (I)(a.n - 1) - (I)((a.n - 1) / 2) - 1;
  const I k = num / (I)a.span;  // span > 0 whenever n > 1
  return k < (I)(a.n - 1) ? (int)k : a.n - 1;
}

// First tile ending after position p: the smallest k with origin(k) + L > p,
// i.e. one past the last tile starting at or before p - L.
template <typename I>
__device__ __forceinline__ int first_end_gt(const Axis& a, int p) {
  const int m = p - a.L;
  return m < 0 ? 0 : last_start_le<I>(a, m) + 1;
}

// Work item = (output row r = (b * T + t) * Hg + y, segment of kThreads * U
// consecutive units of that row); a unit is 4 channels of one position (16 bytes
// of fp32).  The tiles covering the row (along y) and the segment's positions
// (along x) are two index ranges found in closed form once per item; a thread
// then forms its U units (kThreads apart), issuing the loads of all U units
// from one tile before using any.  With Z (fused Eq. 9) the output is
// z - sigma * blend, z bf16.
#ifndef FASTVR_BLEND_UNITS
#define FASTVR_BLEND_UNITS 4
#endif
constexpr int kBlendUnits = FASTVR_BLEND_UNITS;
template <bool Z, typename I>
__global__ __launch_bounds__(kThreads) void tile_blend_kernel(const float* __restrict__ tiles,
                                                              const uint16_t* __restrict__ z, float* __restrict__ out,
                                                              float neg_sigma, int T, int Hg, int Wg, int C, Axis ay,
                                                              Axis ax, int R, int64_t n_rows) {
  constexpr int U = kBlendUnits;
  const int C4 = C / 4;
  const int row_units = Wg * C4;
  const int nt = ay.n * ax.n;
  const int64_t tile_rows = (int64_t)T * ay.L;  // rows of one tile
  const int u_begin = blockIdx.x * (kThreads * U);
  const int u_end = min(u_begin + kThreads * U, row_units);
  int xg[U], c4[U];
  bool ok[U];
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = u_begin + k * kThreads + (int)threadIdx.x;
    ok[k] = u < u_end;
    xg[k] = ok[k] ? u / C4 : 0;
    c4[k] = u - xg[k] * C4;
  }
  const int tx_lo = first_end_gt<I>(ax, u_begin / C4), tx_hi = last_start_le<I>(ax, (u_end - 1) / C4);
  for (int64_t r = blockIdx.y; r < n_rows; r += gridDim.y) {
    const I rr = (I)r;
    const int y = (int)(rr % (I)Hg);
    const I bt = rr / (I)Hg;
    const int t = (int)(bt % (I)T);
    const int64_t b = (int64_t)(bt / (I)T);
    f32x4 acc[U];
    float wsum[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
      wsum[k] = 0.f;
    }
    const int ty_hi = last_start_le<I>(ay, y);
    for (int ty = first_end_gt<I>(ay, y); ty <= ty_hi; ++ty) {
      const int iy = y - origin_t<I>(ay, ty);
      const int wy = axis_weight(iy, ay.L, R);
      const int64_t row0 = ((b * nt + ty * ax.n) * T + t) * ay.L + iy;  // tile row for tx = 0
      for (int tx = tx_lo; tx <= tx_hi; ++tx) {
        const int ox = origin_t<I>(ax, tx);
        const float* trow = tiles + (row0 + (int64_t)tx * tile_rows) * ax.L * C;
        f32x4 val[U];
        float w[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
          const int ix = xg[k] - ox;
          val[k] = f32x4{0.f, 0.f, 0.f, 0.f};
          w[k] = 0.f;
          if (ok[k] && ix >= 0 && ix < ax.L) {
            w[k] = (float)(wy * axis_weight(ix, ax.L, R));
            // each tile element is read exactly once: stream it past the caches
            val[k] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(trow + (int64_t)ix * C + 4 * c4[k]));
          }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
          acc[k].x = __builtin_fmaf(w[k], val[k].x, acc[k].x);
          acc[k].y = __builtin_fmaf(w[k], val[k].y, acc[k].y);
          acc[k].z = __builtin_fmaf(w[k], val[k].z, acc[k].z);
          acc[k].w = __builtin_fmaf(w[k], val[k].w, acc[k].w);
          wsum[k] += w[k];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      if (!ok[k]) continue;
      f32x4 res = {acc[k].x / wsum[k], acc[k].y / wsum[k], acc[k].z / wsum[k], acc[k].w / wsum[k]};
      const int64_t o = (r * Wg + xg[k]) * C + 4 * c4[k];
      if (Z) {
        const uint64_t zz = *reinterpret_cast<const uint64_t*>(z + o);
        const __bf16* zb = reinterpret_cast<const __bf16*>(&zz);
        res.x = __builtin_fmaf(neg_sigma, res.x, (float)zb[0]);
        res.y = __builtin_fmaf(neg_sigma, res.y, (float)zb[1]);
        res.z = __builtin_fmaf(neg_sigma, res.z, (float)zb[2]);
        res.w = __builtin_fmaf(neg_sigma, res.w, (float)zb[3]);
      }
      __builtin_nontemporal_store(res, reinterpret_cast<f32x4*>(out + o));
    }
  }
}

Axis make_axis(int64_t size, int64_t tile, int64_t overlap) {
  const TileAxis t = tile_axis(size, tile, overlap);
  return Axis{(int)t.n, (int)t.len, (int)(size - t.len)};
}

unsigned grid_for(int64_t rows) { return (unsigned)(rows < 8192 ? (rows < 1 ? 1 : rows) : 8192); }

}  // namespace

hipError_t launch_tile_gather(const void* x, void* tiles, int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C,
                              int64_t tile, int64_t overlap, hipStream_t stream) {
  const Axis ay = make_axis(Hg, tile, overlap), ax = make_axis(Wg, tile, overlap);
  const int64_t rows = B * ay.n * ax.n * T * ay.L;
  hipLaunchKernelGGL(tile_gather_kernel, dim3(grid_for(rows)), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(x), static_cast<u32x4*>(tiles), (int)T, (int)Hg, (int)Wg, (int)(C / 8),
                     ay, ax, rows);
  return hipGetLastError();
}

hipError_t launch_tile_blend(const float* tiles, const void* z_lq, float* out, float sigma, int64_t B, int64_t T,
                             int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t overlap, hipStream_t stream) {
  const Axis ay = make_axis(Hg, tile, overlap), ax = make_axis(Wg, tile, overlap);
  const int64_t rows = B * T * Hg;
  const int R = overlap > 1 ? (int)overlap : 1;
  const int64_t row_units = Wg * (C / 4);
  const dim3 grid((unsigned)((row_units + kThreads * kBlendUnits - 1) / (kThreads * kBlendUnits)),
                  (unsigned)(rows < 65535 ? rows : 65535));
  // 32-bit index arithmetic when the row index and every origin numerator
  // (below n * size along each axis) stay below 2^32
  const int64_t lim = int64_t(1) << 32;
  const bool narrow = rows < lim && (int64_t)ay.n * Hg < lim && (int64_t)ax.n * Wg < lim;
  const uint16_t* zp = static_cast<const uint16_t*>(z_lq);
  const float ns = z_lq != nullptr ? -sigma : 0.f;
#define FASTVR_BLEND_LAUNCH(ZV, IT)                                                                              \
  hipLaunchKernelGGL((tile_blend_kernel<ZV, IT>), grid, dim3(kThreads), 0, stream, tiles, zp, out, ns, (int)T, \
                     (int)Hg, (int)Wg, (int)C, ay, ax, R, rows)
  if (z_lq != nullptr) {
    if (narrow) FASTVR_BLEND_LAUNCH(true, uint32_t);
    else FASTVR_BLEND_LAUNCH(true, uint64_t);
  } else {
    if (narrow) FASTVR_BLEND_LAUNCH(false, uint32_t);
    else FASTVR_BLEND_LAUNCH(false, uint64_t);
  }
#undef FASTVR_BLEND_LAUNCH
  return hipGetLastError();
}

}  // namespace fastvr
