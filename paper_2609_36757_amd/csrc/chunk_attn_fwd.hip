// Chunk-wise causal attention forward for CDNA4 (gfx950).
//
// Operation (FastVR, Sec. 3.1, Eq. 1): query row i of chunk cq sees every key
// of chunks cq - W .. cq; O = softmax(scale * Q K^T + mask) V and the natural-log
// LSE per row.  Because a key's chunk index is monotone in the key index, the
// visible keys of one query chunk are a single contiguous interval [lo, hi),
// so masked chunks are never visited and the only element mask is the ragged
// end of that interval.
//
// Work decomposition: one workgroup (8 wave64, 512 threads) per
// (batch, head, query chunk, 256-row query tile); tiles never straddle a chunk.
// Each wave owns 32 query rows.  Scores are computed transposed,
// S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the accumulator puts one query per
// lane (column) and 16 keys per lane (rows), so row max / row sum are in-lane
// plus one exchange between the two 32-lane halves.  The same registers,
// converted to bf16, are the B operand of O^T = V^T P^T; V is staged
// transposed in LDS with its keys permuted so that every A-operand read is one
// 16-byte LDS load.  K and V^T tiles (64 keys) are double-buffered in LDS with
// XOR swizzles; the next K tile's scores are issued before the current tile's
// softmax so the matrix cores and the vector ALU overlap.
//
// Online softmax runs in the log2 domain: t = s * scale * log2(e), running
// maximum m, running sum l; the output is rescaled only when the maximum grows
// by more than 2^8 (values of P stay below 256, exact rearrangement).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace fastvr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = kFwdThreads / 64;  // 8
constexpr int kBQ = 32 * kWaves;          // 256 query rows per workgroup
constexpr int kBK = 64;                   // keys per KV tile
constexpr float kRescaleLog2 = 8.0f;      // lazy rescale threshold (log2 units)
constexpr float kLn2 = 0.693147180559945309f;
static_assert(kBQ == kFwdRowsPerItem, "tile height mismatch");

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* o;
  float* lse;
  int64_t q_sb, q_st, k_sb, k_st, v_sb, v_st, o_sb, o_st;
  int64_t nq, nkv, chunk_len, q_chunk_offset, window;
  int32_t B, H, n_local_chunks, tiles_full, tiles_last, n_items;
  float c;  // scale * log2(e)
};

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// LDS layouts
//   K tile   [kBK rows][D]   bf16, 16-byte chunk index XOR (row & swz)
//   V^T tile [D rows][kBK]   bf16, key order permuted inside each group of 16
//            (swap of key bits 2 and 3), 16-byte chunk index XOR vswz(d)
// ---------------------------------------------------------------------------
template <int D>
struct Lds {
  static constexpr int kKStage = kBK * D;
  static constexpr int kVStage = D * kBK;
  static constexpr int kElems = 2 * kKStage + 2 * kVStage;
  static constexpr int kKSwz = (D / 8 - 1) & 15;
  static __device__ __forceinline__ int k_off(int row, int chunk) {
    return row * D + ((chunk ^ (row & kKSwz)) << 3);
  }
};

__device__ __forceinline__ int vswz(int d) { return (d & 7) ^ ((d >> 3) & 1); }
__device__ __forceinline__ int vt_off(int d, int chunk) { return d * kBK + ((chunk ^ vswz(d)) << 3); }

// Global -> register -> LDS copy of one K tile (512 threads, 16 bytes each).
template <int D>
struct KTile {
  static constexpr int kChunksPerRow = D / 8;
  static constexpr int kPer = kBK * kChunksPerRow / kFwdThreads;
  u32x4 r[kPer];
  __device__ __forceinline__ void load(const uint16_t* kb, int64_t k_st, int64_t t0, int64_t hi, int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int cid = tid + i * kFwdThreads;
      const int row = cid / kChunksPerRow, ch = cid % kChunksPerRow;
      const int64_t kr = t0 + row;
      r[i] = (kr < hi) ? *reinterpret_cast<const u32x4*>(kb + kr * k_st + ch * 8) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(uint16_t* ks, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int cid = tid + i * kFwdThreads;
      const int row = cid / kChunksPerRow, ch = cid % kChunksPerRow;
      *reinterpret_cast<u32x4*>(ks + Lds<D>::k_off(row, ch)) = r[i];
    }
  }
};

// Global -> register -> transposed LDS copy of one V tile.  Thread t < 4*D owns
// the 4x4 block of keys 4*kq..4*kq+3 (kq = t % 16) and dims 4*dq..4*dq+3
// (dq = t / 16); it transposes the block in registers and writes 4 rows of V^T.
template <int D>
struct VTile {
  static constexpr int kBlocks = (kBK / 4) * (D / 4);
  u32x2 r[4];
  __device__ __forceinline__ void load(const uint16_t* vb, int64_t v_st, int64_t t0, int64_t hi, int tid) {
    if (tid < kBlocks) {
      const int kq = tid & 15, dq = tid >> 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t row = t0 + kq * 4 + e;
        r[e] = (row < hi) ? *reinterpret_cast<const u32x2*>(vb + row * v_st + dq * 4) : u32x2{0u, 0u};
      }
    }
  }
  __device__ __forceinline__ void store(uint16_t* vt, int tid) const {
    if (tid < kBlocks) {
      const int kq = tid & 15, dq = tid >> 4;
      // keys 4kq..4kq+3 land at permuted positions: 16-byte chunk and 8-byte half
      const int chunk = ((kq >> 2) << 1) | (kq & 1);
      const int half = (kq >> 1) & 1;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int d = dq * 4 + x;
        const uint32_t w0 = (x < 2) ? r[0].x : r[0].y, w1 = (x < 2) ? r[1].x : r[1].y;
        const uint32_t w2 = (x < 2) ? r[2].x : r[2].y, w3 = (x < 2) ? r[3].x : r[3].y;
        u32x2 out;
        if (x & 1) {
          out.x = (w0 >> 16) | (w1 & 0xffff0000u);
          out.y = (w2 >> 16) | (w3 & 0xffff0000u);
        } else {
          out.x = (w0 & 0xffffu) | (w1 << 16);
          out.y = (w2 & 0xffffu) | (w3 << 16);
        }
        *reinterpret_cast<u32x2*>(vt + vt_off(d, chunk) + half * 4) = out;
      }
    }
  }
};

// blockIdx -> (local query chunk, batch*head, tile).  Workgroups are handed to
// the 8 XCDs round-robin; within each full round of 256 workgroups the
// mapping gives XCD x a run of 32 consecutive items (same batch, head and
// chunk, i.e. the same K/V stream) so they share that XCD's L2.  Items are
// ordered by query chunk, last chunk first: under the causal mask later chunks
// see at least as many keys, so the longest items start first.
__device__ __forceinline__ void decode_item(const Params& p, int i, int& cl, int& bh, int& t) {
  constexpr int kRound = 256;
  int vi = i;
  const int full = (p.n_items / kRound) * kRound;
  if (i < full) {
    const int r = i / kRound, w = i % kRound;
    vi = r * kRound + (w & 7) * 32 + (w >> 3);
  }
  const int BH = p.B * p.H;
  const int n_last = BH * p.tiles_last;
  if (vi < n_last) {
    cl = p.n_local_chunks - 1;
    bh = vi / p.tiles_last;
    t = vi - bh * p.tiles_last;
  } else {
    const int v2 = vi - n_last;
    const int per = BH * p.tiles_full;
    const int rank = v2 / per;
    const int rem = v2 - rank * per;
    cl = p.n_local_chunks - 2 - rank;
    bh = rem / p.tiles_full;
    t = rem - bh * p.tiles_full;
  }
}

// S^T for one K tile: s[mb] holds keys mb*32 + 8*(v/4) + 4*hh + v%4 of query n.
template <int D>
__device__ __forceinline__ void qk_tile(const uint16_t* ks, const int* koff, const u32x4* qf, f32x16 (&s)[2]) {
  s[0] = f32x16{};
  s[1] = f32x16{};
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(ks + koff[kk] + mb * 32 * D);
      s[mb] = mfma32(a, qf[kk], s[mb]);
    }
  }
}

// O^T += V^T P^T for one tile.
template <int D>
__device__ __forceinline__ void pv_tile(const uint16_t* vt, const int* voff, const u32x4 (&pf)[4], f32x16* o) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(vt + voff[g] + dm * 32 * kBK);
      o[dm] = mfma32(a, pf[g], o[dm]);
    }
  }
}

// Online-softmax update for one tile.  NEG: scale < 0 (the largest t = s*c
// comes from the smallest s).  MASK: keys at tile positions >= n_valid are
// outside the visible interval.
template <int D, bool NEG, bool MASK>
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[2], u32x4 (&pf)[4], float& m_run, float& l_run,
                                             f32x16* o, float c, int hh, int n_valid) {
  constexpr float kInf = __builtin_inff();
  if (MASK) {
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
        if (key >= n_valid) s[mb][v] = NEG ? kInf : -kInf;
      }
  }
  float mx = s[0][0];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = NEG ? __builtin_fminf(mx, s[mb][v]) : __builtin_fmaxf(mx, s[mb][v]);
  const float other = __shfl_xor(mx, 32);
  mx = NEG ? __builtin_fminf(mx, other) : __builtin_fmaxf(mx, other);
  const float mt = mx * c;
  const float m_new = (mt > m_run + kRescaleLog2) ? mt : m_run;
  const bool upd = m_new != m_run;
  const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
  m_run = m_new;
  const float nm = -m_new;
  float psum = 0.f;
  float pr[2][16];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][v], c, nm));
      if (MASK) {
        const int key = mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
        pv = (key < n_valid) ? pv : 0.f;
      }
      pr[mb][v] = pv;
      psum += pv;
    }
  l_run = l_run * alpha + psum;
  if (__builtin_amdgcn_ballot_w64(upd)) {
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm) o[dm] *= alpha;
  }
  // B operand of O^T += V^T P^T: group g = 2*mb + half uses accumulators 8*half .. 8*half+7
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    bf16x8 b;
#pragma unroll
    for (int r = 0; r < 8; ++r) b[r] = (__bf16)pr[g >> 1][8 * (g & 1) + r];
    pf[g] = __builtin_bit_cast(u32x4, b);
  }
}

template <int D, bool NEG>
__global__ __launch_bounds__(kFwdThreads) void chunk_attn_fwd_kernel(const Params p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[Lds<D>::kElems];
  uint16_t* const ks_base = smem;
  uint16_t* const vt_base = smem + 2 * Lds<D>::kKStage;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;

  int cl, bh, t;
  decode_item(p, blockIdx.x, cl, bh, t);
  const int b = bh / p.H, h = bh - (bh / p.H) * p.H;

  const int64_t L = p.chunk_len;
  const int64_t chunk_q0 = (int64_t)cl * L;
  const int64_t q_end = (chunk_q0 + L < p.nq) ? chunk_q0 + L : p.nq;
  const int64_t q0 = chunk_q0 + (int64_t)t * kBQ;
  const int64_t cg = p.q_chunk_offset + cl;
  int64_t lo = 0;
  if (p.window >= 0) lo = (cg - p.window > 0 ? cg - p.window : 0) * L;
  const int64_t hi = ((cg + 1) * L < p.nkv) ? (cg + 1) * L : p.nkv;
  const int n_tiles = (int)((hi - lo + kBK - 1) / kBK);

  const int64_t row = q0 + wave * 32 + n;
  const bool active = (q0 + wave * 32) < q_end;  // wave-uniform

  const uint16_t* qb = p.q + (int64_t)b * p.q_sb + (int64_t)h * D;
  const uint16_t* kb = p.k + (int64_t)b * p.k_sb + (int64_t)h * D;
  const uint16_t* vb = p.v + (int64_t)b * p.v_sb + (int64_t)h * D;

  // Q fragments (B operand of S^T = K Q^T): lane (n, hh) holds row n, dims 16kk + 8hh .. +7
  u32x4 qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk)
    qf[kk] = (row < q_end) ? *reinterpret_cast<const u32x4*>(qb + row * p.q_st + kk * 16 + hh * 8)
                           : u32x4{0u, 0u, 0u, 0u};

  // loop-invariant LDS offsets of this lane's operand reads
  int koff[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) koff[kk] = Lds<D>::k_off(n, 2 * kk + hh);
  int voff[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) voff[g] = vt_off(n, 2 * g + hh);

  KTile<D> kt;
  VTile<D> vtl;
  kt.load(kb, p.k_st, lo, hi, tid);
  kt.store(ks_base, tid);
  if (n_tiles > 1) {
    kt.load(kb, p.k_st, lo + kBK, hi, tid);
    kt.store(ks_base + Lds<D>::kKStage, tid);
  }
  vtl.load(vb, p.v_st, lo, hi, tid);
  vtl.store(vt_base, tid);
  __syncthreads();

  f32x16 o[D / 32];
#pragma unroll
  for (int dm = 0; dm < D / 32; ++dm) o[dm] = f32x16{};
  float m_run = -__builtin_inff(), l_run = 0.f;
  f32x16 s[2];
  u32x4 pf[4];
  if (active) qk_tile<D>(ks_base, koff, qf, s);

  for (int j = 0; j + 1 < n_tiles; ++j) {
    const bool k_ahead = j + 2 < n_tiles;
    if (k_ahead) kt.load(kb, p.k_st, lo + (int64_t)(j + 2) * kBK, hi, tid);
    vtl.load(vb, p.v_st, lo + (int64_t)(j + 1) * kBK, hi, tid);
    if (active) {
      f32x16 sn[2];
      qk_tile<D>(ks_base + ((j + 1) & 1) * Lds<D>::kKStage, koff, qf, sn);
      softmax_tile<D, NEG, false>(s, pf, m_run, l_run, o, p.c, hh, kBK);
      pv_tile<D>(vt_base + (j & 1) * Lds<D>::kVStage, voff, pf, o);
      s[0] = sn[0];
      s[1] = sn[1];
    }
    if (k_ahead) kt.store(ks_base + (j & 1) * Lds<D>::kKStage, tid);
    vtl.store(vt_base + ((j + 1) & 1) * Lds<D>::kVStage, tid);
    __syncthreads();
  }

  if (!active) return;
  const int jl = n_tiles - 1;
  const int n_valid = (int)(hi - (lo + (int64_t)jl * kBK));
  if (n_valid < kBK)
    softmax_tile<D, NEG, true>(s, pf, m_run, l_run, o, p.c, hh, n_valid);
  else
    softmax_tile<D, NEG, false>(s, pf, m_run, l_run, o, p.c, hh, kBK);
  pv_tile<D>(vt_base + (jl & 1) * Lds<D>::kVStage, voff, pf, o);

  // epilogue: the two halves of the wave hold partial sums over disjoint keys
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (row < q_end) {
    const float inv = 1.0f / l_tot;
    float* ob = p.o + (int64_t)b * p.o_sb + row * p.o_st + (int64_t)h * D;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 val;
        val.x = o[dm][4 * g + 0] * inv;
        val.y = o[dm][4 * g + 1] * inv;
        val.z = o[dm][4 * g + 2] * inv;
        val.w = o[dm][4 * g + 3] * inv;
        *reinterpret_cast<f32x4*>(ob + dm * 32 + g * 8 + hh * 4) = val;
      }
    if (hh == 0 && p.lse != nullptr)
      p.lse[((int64_t)b * p.H + h) * p.nq + row] = (m_run + __builtin_log2f(l_tot)) * kLn2;
  }
}

template <int D, bool NEG>
hipError_t launch_t(const Params& p, int64_t n_items, hipStream_t stream) {
  hipLaunchKernelGGL((chunk_attn_fwd_kernel<D, NEG>), dim3((unsigned)n_items), dim3(kFwdThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

FwdGrid fwd_grid(int64_t B, int64_t H, int64_t nq, int64_t chunk_len) {
  FwdGrid g{};
  if (B <= 0 || H <= 0 || nq <= 0 || chunk_len <= 0) return g;
  g.n_local_chunks = (nq + chunk_len - 1) / chunk_len;
  const int64_t last_rows = nq - (g.n_local_chunks - 1) * chunk_len;
  g.tiles_last = (last_rows + kBQ - 1) / kBQ;
  g.tiles_full = g.n_local_chunks > 1 ? (chunk_len + kBQ - 1) / kBQ : g.tiles_last;
  g.n_items = B * H * (g.tiles_last + g.tiles_full * (g.n_local_chunks - 1));
  return g;
}

hipError_t launch_chunk_attn_fwd(const FwdArgs& a, hipStream_t stream) {
  const FwdGrid g = fwd_grid(a.B, a.H, a.nq, a.chunk_len);
  Params p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = a.o;
  p.lse = a.lse;
  p.q_sb = a.q_sb; p.q_st = a.q_st;
  p.k_sb = a.k_sb; p.k_st = a.k_st;
  p.v_sb = a.v_sb; p.v_st = a.v_st;
  p.o_sb = a.o_sb; p.o_st = a.o_st;
  p.nq = a.nq;
  p.nkv = a.nkv;
  p.chunk_len = a.chunk_len;
  p.q_chunk_offset = a.q_chunk_offset;
  p.window = a.window_chunks;
  p.B = (int32_t)a.B;
  p.H = (int32_t)a.H;
  p.n_local_chunks = (int32_t)g.n_local_chunks;
  p.tiles_full = (int32_t)g.tiles_full;
  p.tiles_last = (int32_t)g.tiles_last;
  p.n_items = (int32_t)g.n_items;
  p.c = a.scale * 1.44269504088896340736f;
  const bool neg = p.c < 0.f;
  if (a.d == 128) return neg ? launch_t<128, true>(p, g.n_items, stream) : launch_t<128, false>(p, g.n_items, stream);
  return neg ? launch_t<64, true>(p, g.n_items, stream) : launch_t<64, false>(p, g.n_items, stream);
}

}  // namespace fastvr
