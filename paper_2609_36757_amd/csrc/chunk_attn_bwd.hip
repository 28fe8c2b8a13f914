// Chunk-wise causal attention backward for CDNA4 (gfx950).
//
// Gradients of O = softmax(scale * Q K^T + M) V (FastVR, Sec. 3.1, Eq. 1; M the
// chunk-causal mask) for an upstream gradient dO, reusing the forward's LSE:
//   P   = exp(scale * Q K^T - LSE)            recomputed per tile, never stored
//   D_i = sum_d dO_id * O_id
//   dV  = P^T dO,   dP = dO V^T,   dS = P o (dP - D),
//   dQ  = scale * dS K,   dK = scale * dS^T Q.
// As in the forward, the keys a query chunk sees form one contiguous interval
// and the queries that see a key chunk form one contiguous interval, so masked
// chunk pairs are never visited.
//
// Two kernels, no atomics, so every gradient is a fixed-order sum (results are
// reproducible bit for bit):
//  * dQ kernel (query-stationary, the forward's grid): 8 waves, 32 queries each,
//    Q and dO fragments in registers.  It first writes LSE * log2 e and -D of its
//    rows to a workspace, then per 64-key tile computes S^T = K Q^T and
//    dP^T = V dO^T (one query per lane, 16 keys per lane), P^T and dS^T in
//    registers, and dQ^T += K^T dS^T.
//  * dK/dV kernel (key-stationary): a workgroup owns 128 keys of one chunk
//    and walks the 64-query tiles of the queries that see that chunk.  Each
//    32 keys belong to a wave pair: one wave holds K, computes S = Q K^T (one
//    key per lane, 16 queries per lane), P, and dV^T += dO^T P; the other holds
//    V, computes dP = dO V^T and dS = P (dP - D) from the first wave's P, and
//    dK^T += Q^T dS.
// All products are v_mfma_f32_32x32x16_bf16 with fp32 accumulation; P and dS
// are rounded to bf16 as MFMA operands.
//
// Streamed tiles (K and V, or Q and dO: 64 rows of d bf16) travel by DMA from
// HBM straight into LDS (buffer_load ... lds), triple-buffered and issued two
// tiles ahead.  Every row offset is in the per-lane VGPR offset, which the
// buffer range check covers, so rows past a tile's valid end read as zero.
// In LDS a row keeps its 16-byte chunks with the chunk index XOR bswz(row);
// the same tile is read both by rows (ds_read_b128, MFMA operands K, V, Q, dO)
// and transposed (ds_read_b64_tr_b16, operands K^T, Q^T, dO^T), and bswz keeps
// both free of LDS bank conflicts.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "gfx950_ops.h"
#include "launch.h"

namespace fastvr {
namespace {

using namespace dev;

#ifndef FASTVR_BWD_AHEAD
#define FASTVR_BWD_AHEAD 4  // dK/dV kernel: MFMA operand reads kept in flight ahead (0: the compiler places them)
#endif
#ifndef FASTVR_DQ_AHEAD
#define FASTVR_DQ_AHEAD 4  // dQ kernel: MFMA operand reads kept in flight ahead (0: the compiler places them)
#endif
#ifndef FASTVR_PRIO
#define FASTVR_PRIO 1  // raise the wave priority during matrix-core slots
#endif


constexpr int kTile = 64;  // rows per staged tile: keys (dQ) or queries (dK/dV)
constexpr int kStages = 3;
constexpr int kDqWaves = kBwdDqThreads / 64;    // 8
constexpr int kDkvWaves = kBwdDkvThreads / 64;  // 8 (two groups of 4)
constexpr int kDqRows = 32 * kDqWaves;          // 256 queries per dQ workgroup
static_assert(kDqRows == kFwdRowsPerItem, "the dQ grid is the forward's");
static_assert(32 * (kDkvWaves / 2) == kBwdKeysPerItem, "32 keys per dK/dV wave pair");

struct BwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* dout;
  const float* o;
  const float* lse;
  float* dq;
  float* dk;
  float* dv;
  float* rs;             // row statistics [B, H, 2, nq]: LSE log2 e, then -D
  int64_t q_sb, kv_sb;   // batch strides (elements) of the query-side and key-side tensors
  int32_t st;            // token stride H * d (elements), all tensors
  int32_t nq, nkv, chunk_len, q_chunk_offset, window;  // window -1 = unbounded
  int32_t B, H;
  int32_t n_local_chunks, tiles_full, tiles_last, n_q_items;
  int32_t n_kchunks, kblocks_full, kblocks_last, n_kv_items;
  float c;      // scale * log2(e)
  float scale;
};

// XOR applied to the 16-byte chunk index of row r of a staged tile.
//  * Row reads: 16 lanes read one logical chunk of 16 consecutive rows, so
//    bswz must be one-to-one on r mod 16 (d = 128: a row is one 256-byte bank
//    row of 16 chunk slots; d = 64: two rows share a bank row, one-to-one per
//    row parity).
//  * Transposed reads: 32 lanes read rows 4a .. 4a+3 and logical chunks
//    4m .. 4m+3, so the four rows must fall into four different chunk quads
//    (d = 128), or two per row parity (d = 64).
template <int D>
__device__ __forceinline__ int bswz(int r) {
  return D >= 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}

// Staged tile of 64 rows x D bf16 filled by NW waves.
template <int D, int NW>
struct TileDma {
  static constexpr int kChunks = D / 8;                    // 16-byte chunks per row
  static constexpr int kElems = kTile * D;                 // bf16 per stage
  static constexpr int kRowsPerInst = 64 / kChunks;        // rows one wave instruction fills
  static constexpr int kPer = kTile * kChunks / (64 * NW); // instructions per wave per tile
  static_assert(kPer >= 1 && (NW * kRowsPerInst) % 16 == 0, "row swizzle must repeat per instruction");
  uint32_t off;   // this lane's byte offset in the source tile, instruction 0
  uint32_t step;  // byte offset between consecutive instructions

  // Instruction i of wave w fills LDS chunk slots (i * NW + w) * 64 + lane: row
  // P / kChunks, physical chunk P % kChunks, read from logical chunk
  // phys ^ bswz(row).  Rows advance by NW * kRowsPerInst (a multiple of 16)
  // per instruction, so the swizzle of a lane's row does not depend on i.
  __device__ __forceinline__ void init(int wave, int lane, int st) {
    const int P = wave * 64 + lane;
    const int row = P / kChunks, phys = P % kChunks;
    off = (uint32_t)(row * st + (phys ^ bswz<D>(row)) * 8) * 2u;
    step = (uint32_t)(NW * kRowsPerInst * st) * 2u;
  }
  // DMA of a tile whose first row is `base` and whose `rows` first rows are
  // valid (rows past them, all of them when rows <= 0, read as zero).
  __device__ __forceinline__ void load(const uint16_t* base, int rows, int st, uint16_t* dst, int wave) const {
    const i32x4 rsrc = make_vsharp(base, rows > 0 ? (int64_t)rows * st * 2 : 0);
    const uint32_t la = lds_addr(dst) + (uint32_t)(wave * 64 * 16);
#pragma unroll
    for (int i = 0; i < kPer; ++i) dma16(la + (uint32_t)(i * NW * 64 * 16), off + (uint32_t)i * step, rsrc, 0);
  }
};

// Operand reads from a staged tile, for lane (n = lane % 32, hh = lane / 32).
template <int D>
struct TileReads {
  int row_rd[D / 16];     // row reads: row n, logical chunk 2 kk + hh
  int tr_rd[D / 32][2];   // transposed reads, rows 4 hh + (i >> 2) (+ 8)

  __device__ __forceinline__ void init(int lane) {
    const int n = lane & 31, hh = lane >> 5;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) row_rd[kk] = n * (D * 2) + (((2 * kk + hh) ^ bswz<D>(n)) * 16);
    // 16-lane block b = lane / 16, i = lane % 16: the lane addresses row
    // 4 hh + (i >> 2) (and 8 rows further), dims dm * 32 + 16 (b & 1) + 4 (i & 3)
    // .. + 3, and receives rows 4 hh + 0..3 of dim dm * 32 + 16 (b & 1) + i.
    const int i = lane & 15, b = lane >> 4;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int h8 = 0; h8 < 2; ++h8) {
        const int row = hh * 4 + (i >> 2) + 8 * h8;
        const int logical = dm * 4 + 2 * (b & 1) + ((i >> 1) & 1);
        tr_rd[dm][h8] = row * (D * 2) + ((logical ^ bswz<D>(row)) * 16) + (i & 1) * 8;
      }
  }
  // A operand rows mb * 32 + n, dims 16 kk + 8 hh .. + 7
  __device__ __forceinline__ u32x4 row(const char* t, int mb, int kk) const {
    return *reinterpret_cast<const u32x4*>(t + row_rd[kk] + mb * 32 * (D * 2));
  }
  // A operand of T^T for k-step g (tile rows 16 g .. 16 g + 15) and dims
  // dm * 32 .. + 31: lane (i_A, hh) gets T[16 g + 4 hh + {0..3, 8..11}][dm * 32 + i_A]
  __device__ __forceinline__ u32x4 tr(const char* t, int g, int dm) const {
    const char* base = t + g * 16 * (D * 2);
    const i16x4 lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + tr_rd[dm][0]));
    const i16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + tr_rd[dm][1]));
    return __builtin_bit_cast(u32x4, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
  }
};

// bf16 B-operand fragments of a 32-row accumulator a (rows 8 (v >> 2) +
// 4 hh + (v & 3)): k-step gg covers rows 16 gg .. 16 gg + 15 in the order the
// transposed reads deliver them.
__device__ __forceinline__ void pack_bf16_half(const f32x16& a, u32x4 (&f)[2]) {
#pragma unroll
  for (int gg = 0; gg < 2; ++gg) {
    bf16x8 b;
#pragma unroll
    for (int r = 0; r < 8; ++r) b[r] = (__bf16)a[8 * gg + r];
    f[gg] = __builtin_bit_cast(u32x4, b);
  }
}
// The same for a 64-row pair a[0], a[1] (rows 32 mb + ...): k-step g covers
// rows 16 g .. 16 g + 15.
__device__ __forceinline__ void pack_bf16(const f32x16 (&a)[2], u32x4 (&f)[4]) {
  u32x4 f0[2], f1[2];
  pack_bf16_half(a[0], f0);
  pack_bf16_half(a[1], f1);
  f[0] = f0[0];
  f[1] = f0[1];
  f[2] = f1[0];
  f[3] = f1[1];
}

// Workgroups go to the 8 XCDs round-robin; within each full round of 256,
// XCD x gets 32 consecutive items (neighbouring tiles of one stream share its L2).
__device__ __forceinline__ int xcd_item(int i, int n_items) {
  constexpr int kRound = 256;
  const int full = (n_items / kRound) * kRound;
  if (i >= full) return i;
  const int r = i / kRound, w = i % kRound;
  return r * kRound + (w & 7) * 32 + (w >> 3);
}

// ---------------------------------------------------------------- dQ kernel

template <int D>
__global__ __launch_bounds__(kBwdDqThreads) void chunk_attn_bwd_dq_kernel(const BwdParams p) {
  using Dma = TileDma<D, kDqWaves>;
  constexpr int kStage = Dma::kElems;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * kStages * kStage];
  uint16_t* ks = smem;
  uint16_t* vs = smem + kStages * kStage;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;

  // item -> (local query chunk, batch*head, tile), last chunk first (longest)
  int cl, bh, t;
  {
    const int vi = xcd_item(blockIdx.x, p.n_q_items);
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
  const int b = bh / p.H, h = bh - (bh / p.H) * p.H;
  const int L = p.chunk_len;
  const int chunk_q0 = cl * L;
  const int q_end = (L < p.nq - chunk_q0) ? chunk_q0 + L : p.nq;
  const int q0 = chunk_q0 + t * kDqRows;
  const int cg = p.q_chunk_offset + cl;
  const int lo = (p.window >= 0 && cg > p.window) ? (cg - p.window) * L : 0;
  const int hi = (L < p.nkv - cg * L) ? (cg + 1) * L : p.nkv;
  const int n_tiles = (hi - lo + kTile - 1) / kTile;
  const int st = p.st;
  const uint16_t* kb = p.k + (int64_t)b * p.kv_sb + (int64_t)h * D;
  const uint16_t* vb = p.v + (int64_t)b * p.kv_sb + (int64_t)h * D;

  Dma dma;
  dma.init(wave, lane, st);
  TileReads<D> rd;
  rd.init(lane);
  auto tile_rows = [&](int j) { return hi - (lo + j * kTile); };

  // prologue: K and V tiles 0 and 1 to LDS
  dma.load(kb + (int64_t)lo * st, tile_rows(0), st, ks, wave);
  dma.load(vb + (int64_t)lo * st, tile_rows(0), st, vs, wave);
  dma.load(kb + (int64_t)(lo + kTile) * st, tile_rows(1), st, ks + kStage, wave);
  dma.load(vb + (int64_t)(lo + kTile) * st, tile_rows(1), st, vs + kStage, wave);

  // this wave's 32 query rows: Q and dO fragments (B operands Q^T, dO^T), the
  // row statistics, written to the workspace for the dK/dV kernel
  const int row = q0 + wave * 32 + n;
  const bool row_ok = row < q_end;
  u32x4 qf[D / 16], dof[D / 16];
  float lse2, dlt;
  {
    const int rows = q_end - (q0 + wave * 32);  // valid rows of this wave (may be <= 0)
    const int64_t qoff = (int64_t)b * p.q_sb + (int64_t)(q0 + wave * 32) * st + (int64_t)h * D;
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(p.q + qoff, rows > 0 ? (int64_t)rows * st * 2 : 0);
    const __amdgpu_buffer_rsrc_t rdo = make_rsrc(p.dout + qoff, rows > 0 ? (int64_t)rows * st * 2 : 0);
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.o + qoff, rows > 0 ? (int64_t)rows * st * 4 : 0);
    float dpart = 0.f;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const uint32_t e = (uint32_t)(n * st + kk * 16 + hh * 8);  // element offset of dims 16 kk + 8 hh
      qf[kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, e * 2u, 0, 0));
      dof[kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rdo, e * 2u, 0, 0));
      const f32x4 o0 = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ro, e * 4u, 0, 0));
      const f32x4 o1 = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ro, e * 4u + 16u, 0, 0));
      const bf16x8 d8 = __builtin_bit_cast(bf16x8, dof[kk]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dpart = __builtin_fmaf((float)d8[r], o0[r], dpart);
        dpart = __builtin_fmaf((float)d8[4 + r], o1[r], dpart);
      }
    }
    float dother;
    const float dmine = swap_halves(dpart, &dother);
    dlt = dmine + dother;  // the same sum in both halves
    const float lse = row_ok ? p.lse[((int64_t)b * p.H + h) * p.nq + row] : 0.f;
    lse2 = row_ok ? lse * 1.44269504088896340736f : 0.f;
    dlt = row_ok ? dlt : 0.f;
    if (row_ok && hh == 0) {
      float* rs = p.rs + ((int64_t)b * p.H + h) * 2 * p.nq + row;
      rs[0] = lse2;
      rs[p.nq] = -dlt;
    }
  }
  f32x16 acc[D / 32];
#pragma unroll
  for (int dm = 0; dm < D / 32; ++dm) acc[dm] = f32x16{};
  wait_vmcnt<0>();
  __builtin_amdgcn_s_waitcnt(0x0F70);
  barrier();

  const float c = p.c;
  const int last_valid = hi - (lo + (n_tiles - 1) * kTile);
  int s_cur = 0, s_next = 1, s_free = 2;
  for (int j = 0; j < n_tiles; ++j) {
    const char* kst = reinterpret_cast<const char*>(ks + s_cur * kStage);
    const char* vst = reinterpret_cast<const char*>(vs + s_cur * kStage);
    // The tile's two 32-key halves one after the other (register budget of
    // two waves per SIMD).
    const int lim = (j + 1 == n_tiles) ? last_valid - 4 * hh : kTile;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      // S^T = K Q^T and dP^T = V dO^T: lane = query n, 16 keys per lane
      f32x16 s, dp;
      if (FASTVR_DQ_AHEAD > 0) {
        // MFMA i: k-step i / 2, S^T (even i, K rows) or dP^T (odd i, V rows)
        constexpr int kN = D / 8;
        constexpr int kA = FASTVR_DQ_AHEAD < kN ? FASTVR_DQ_AHEAD : kN;
        u32x4 f[kN];
#pragma unroll
        for (int i = 0; i < kA; ++i) f[i] = rd.row((i & 1) ? vst : kst, mb, i >> 1);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          if (i + kA < kN) f[i + kA] = rd.row(((i + kA) & 1) ? vst : kst, mb, (i + kA) >> 1);
          const int kk = i >> 1;
          if (i & 1)
            dp = mfma32(f[i], dof[kk], kk == 0 ? f32x16{} : dp);
          else
            s = mfma32(f[i], qf[kk], kk == 0 ? f32x16{} : s);
        }
        __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, kA, 0);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
          if (i + kA < kN) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      } else {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          s = mfma32(rd.row(kst, mb, kk), qf[kk], kk == 0 ? f32x16{} : s);
          dp = mfma32(rd.row(vst, mb, kk), dof[kk], kk == 0 ? f32x16{} : dp);
        }
      }
      // P^T = exp2(S^T c - LSE log2 e); dS^T = P^T (dP^T - D).  Keys past the
      // interval (last tile only) get P = 0.
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = mb * 32 + 8 * (v >> 2) + (v & 3);
        float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], c, -lse2));
        pv = key < lim ? pv : 0.f;
        s[v] = pv * (dp[v] - dlt);
      }
      u32x4 dsf[2];
      pack_bf16_half(s, dsf);
      // dQ^T += K^T dS^T over keys 32 mb .. 32 mb + 31, at a raised priority:
      // the other wave of the SIMD is then most often in its S / dP MFMAs or
      // its exp2, and these transposed-read MFMAs go first (the whole
      // backward 0.5% faster; raising the S / dP MFMAs as well is not)
#if FASTVR_PRIO
      __builtin_amdgcn_s_setprio(1);
#endif
      if (FASTVR_DQ_AHEAD > 0) {
        constexpr int kN = 2 * (D / 32);
        constexpr int kA = FASTVR_DQ_AHEAD < kN ? FASTVR_DQ_AHEAD : kN;
        u32x4 f[kN];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < kA; ++i) f[i] = rd.tr(kst, 2 * mb + i / (D / 32), i % (D / 32));
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          if (i + kA < kN) f[i + kA] = rd.tr(kst, 2 * mb + (i + kA) / (D / 32), (i + kA) % (D / 32));
          const int gg = i / (D / 32), dm = i % (D / 32);
          acc[dm] = mfma32(f[i], dsf[gg], acc[dm]);
        }
        __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2 * kA, 0);
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          if (i + kA < kN) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2, 0);
          __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      } else {
#pragma unroll
        for (int gg = 0; gg < 2; ++gg)
#pragma unroll
          for (int dm = 0; dm < D / 32; ++dm) acc[dm] = mfma32(rd.tr(kst, 2 * mb + gg, dm), dsf[gg], acc[dm]);
      }
#if FASTVR_PRIO
      __builtin_amdgcn_s_setprio(0);
#endif
      if (mb == 0) {
        // tile j + 2 into the stage tile j - 1 used (zero rows past the
        // interval), issued between the halves: each DMA instruction holds
        // the wave for over a hundred cycles, which costs least here (0.4%
        // faster than at the top of the tile)
        dma.load(kb + (int64_t)(lo + (j + 2) * kTile) * st, tile_rows(j + 2), st, ks + s_free * kStage, wave);
        dma.load(vb + (int64_t)(lo + (j + 2) * kTile) * st, tile_rows(j + 2), st, vs + s_free * kStage, wave);
      }
    }
    wait_vmcnt<2 * Dma::kPer>();
    barrier();
    const int s_old = s_cur;
    s_cur = s_next;
    s_next = s_free;
    s_free = s_old;
  }
  wait_vmcnt<0>();

  // dQ = scale * dQ^T: lane n holds dims dm * 32 + 8 g + 4 hh + 0..3 of its row
  if (row_ok) {
    float* out = p.dq + (int64_t)b * p.q_sb + (int64_t)row * st + (int64_t)h * D;
    const float sc = p.scale;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 val;
        val.x = acc[dm][4 * g + 0] * sc;
        val.y = acc[dm][4 * g + 1] * sc;
        val.z = acc[dm][4 * g + 2] * sc;
        val.w = acc[dm][4 * g + 3] * sc;
        *reinterpret_cast<f32x4*>(out + dm * 32 + g * 8 + hh * 4) = val;
      }
  }
}

// -------------------------------------------------------------- dK/dV kernel
//
// Eight waves in two groups that share the four SIMDs one-to-one.  Wave pair
// (a, a + 4) owns 32 keys: group A (waves 0-3) computes S = Q K^T, P and
// dV^T += dO^T P; group B (waves 4-7) computes dP - D = dO V^T - D, dS = P (dP - D)
// and dK^T += Q^T dS, taking P from group A through LDS as bf16 fragments.
// Time is cut into slots separated by workgroup barriers, and the two groups
// swap between a matrix-core slot and a vector-ALU slot every slot:
//   slot 2t:   A  S(t) and dV += dO^T(t-1) P(t-1)       B  dS(t-1); DMA of Q(t+2), row stats(t+2)
//   slot 2t+1: A  DMA dO(t+2); P(t) (exp2), P(t) to LDS  B  dP(t) - D and dK += Q^T(t-1) dS(t-1)
// A tile is read from slot 2t to slot 2t+3, so the LDS holds four stages.
// The dP accumulator starts from -D (read from the row statistics), so
// dP - D comes out of the MFMAs.

constexpr int kDkvStages = 4;

template <int D>
struct Dkv {
  using Dma = TileDma<D, kDkvWaves / 2>;  // one group issues each operand
  static constexpr int kStage = Dma::kElems;
  static constexpr int kRs = 2 * kTile;  // floats per row-statistics stage: LSE log2 e, then -D
  int lane, wave, pair, n, hh;
  float c;
  uint16_t* qs;
  uint16_t* dos;
  float* rss;
  u32x4* pex;  // P exchange of this pair: [4 fragments][64 lanes]
  TileReads<D> rd;
  u32x4 kvf[D / 16];  // A: K fragments (B operand K^T); B: V fragments (V^T)
  f32x16 acc[D / 32]; // A: dV^T; B: dK^T
  f32x16 sp[2];       // A: S, then P; B: dP - D
  u32x4 frag[4];      // A: bf16 P; B: bf16 dS

  __device__ __forceinline__ const char* q_stage(int t) const {
    return reinterpret_cast<const char*>(qs + (t & (kDkvStages - 1)) * kStage);
  }
  __device__ __forceinline__ const char* do_stage(int t) const {
    return reinterpret_cast<const char*>(dos + (t & (kDkvStages - 1)) * kStage);
  }
  __device__ __forceinline__ const float* rs_stage(int t) const { return rss + (t & (kDkvStages - 1)) * kRs; }

  // sp[mb] (+)= rows 32 mb + n of stage st times kvf (D/16 k-steps x 2 row
  // blocks), operand reads kA MFMAs ahead
  template <bool ZERO>
  __device__ __forceinline__ void row_products(const char* st) {
    constexpr int kN = D / 8;
    constexpr int kA = FASTVR_BWD_AHEAD < kN ? FASTVR_BWD_AHEAD : kN;
    u32x4 f[kN];
#pragma unroll
    for (int i = 0; i < kA; ++i) f[i] = rd.row(st, i & 1, i >> 1);
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      if (i + kA < kN) f[i + kA] = rd.row(st, (i + kA) & 1, (i + kA) >> 1);
      const int kk = i >> 1, mb = i & 1;
      sp[mb] = mfma32(f[i], kvf[kk], (ZERO && kk == 0) ? f32x16{} : sp[mb]);
    }
    __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, kA, 0);
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      if (i + kA < kN) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  // acc[dm] += (stage st)^T k-step g, dims dm * 32 .. times frag[g], operand
  // reads kA MFMAs ahead
  __device__ __forceinline__ void tr_products(const char* st) {
    constexpr int kN = 4 * (D / 32);
    constexpr int kA = FASTVR_BWD_AHEAD < kN ? FASTVR_BWD_AHEAD : kN;
    u32x4 f[kN];
#pragma unroll
    for (int i = 0; i < kA; ++i) f[i] = rd.tr(st, i / (D / 32), i % (D / 32));
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      if (i + kA < kN) f[i + kA] = rd.tr(st, (i + kA) / (D / 32), (i + kA) % (D / 32));
      const int g = i / (D / 32), dm = i % (D / 32);
      acc[dm] = mfma32(f[i], frag[g], acc[dm]);
    }
    __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2 * kA, 0);
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      if (i + kA < kN) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // Group A, matrix-core slot: S(t) = Q K^T (when S_T) and dV^T += dO^T(t-1) P(t-1) (when PV)
  template <bool S_T, bool PV>
  __device__ __forceinline__ void a_mfma(int t) {
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(1);
#endif
    if (FASTVR_BWD_AHEAD > 0) {
      if (S_T) row_products<true>(q_stage(t));
      if (PV) tr_products(do_stage(t - 1));
    } else {
      if (S_T) {
        const char* qst = q_stage(t);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) sp[mb] = mfma32(rd.row(qst, mb, kk), kvf[kk], kk == 0 ? f32x16{} : sp[mb]);
      }
      if (PV) {
        const char* dost = do_stage(t - 1);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int dm = 0; dm < D / 32; ++dm) acc[dm] = mfma32(rd.tr(dost, g, dm), frag[g], acc[dm]);
      }
    }
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(0);
#endif
  }
  // Group A, vector-ALU slot: P(t) = exp2(S c - LSE log2 e) for query rows
  // 32 mb + 8 g + 4 hh + r, rounded to bf16 fragments, and handed to group B.
  // Rows past the query range have Q = 0 and zero statistics, so P = 1 there,
  // and dO = 0 and -D = 0 make their dV and dS terms vanish.
  __device__ __forceinline__ void a_valu(int t) {
    const float* l2 = rs_stage(t);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(l2 + 32 * mb + 8 * g + 4 * hh);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sp[mb][4 * g + r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sp[mb][4 * g + r], c, -l4[r]));
      }
    pack_bf16(sp, frag);
#pragma unroll
    for (int g = 0; g < 4; ++g) pex[g * 64 + lane] = frag[g];
  }
  // Group B, matrix-core slot: dP(t) - D = dO V^T - D (when DP) and dK^T +=
  // Q^T(t-1) dS(t-1) (when DK)
  template <bool DP, bool DK>
  __device__ __forceinline__ void b_mfma(int t) {
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(1);
#endif
    if (DP) {
      const char* dost = do_stage(t);
      const float* nd = rs_stage(t) + kTile;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(nd + 32 * mb + 8 * g + 4 * hh);
#pragma unroll
          for (int r = 0; r < 4; ++r) sp[mb][4 * g + r] = d4[r];
        }
      if (FASTVR_BWD_AHEAD > 0) {
        __builtin_amdgcn_sched_barrier(0);
        row_products<false>(dost);
      } else {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) sp[mb] = mfma32(rd.row(dost, mb, kk), kvf[kk], sp[mb]);
      }
    }
    if (DK) {
      if (FASTVR_BWD_AHEAD > 0) {
        tr_products(q_stage(t - 1));
      } else {
        const char* qst = q_stage(t - 1);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int dm = 0; dm < D / 32; ++dm) acc[dm] = mfma32(rd.tr(qst, g, dm), frag[g], acc[dm]);
      }
    }
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(0);
#endif
  }
  // Group B, vector-ALU slot: dS(t) = P(t) (dP - D), rounded to bf16 fragments
  __device__ __forceinline__ void b_valu() {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const bf16x8 p8 = __builtin_bit_cast(bf16x8, pex[g * 64 + lane]);
#pragma unroll
      for (int r = 0; r < 8; ++r) sp[g >> 1][8 * (g & 1) + r] *= (float)p8[r];
    }
    pack_bf16(sp, frag);
  }
};

template <int D>
__global__ __launch_bounds__(kBwdDkvThreads) void chunk_attn_bwd_dkv_kernel(const BwdParams p) {
  using K = Dkv<D>;
  using Dma = typename K::Dma;
  constexpr int kStage = K::kStage;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * kDkvStages * kStage];
  __shared__ __attribute__((aligned(16))) float rss[kDkvStages * K::kRs];
  __shared__ __attribute__((aligned(16))) u32x4 pex[(kDkvWaves / 2) * 4 * 64];
  K a;
  a.qs = smem;
  a.dos = smem + kDkvStages * kStage;
  a.rss = rss;
  const int tid = threadIdx.x;
  a.lane = tid & 63;
  a.wave = tid >> 6;
  a.pair = a.wave & 3;
  const int group = a.wave >> 2;  // 0: A (S, P, dV), 1: B (dP, dS, dK)
  a.n = a.lane & 31;
  a.hh = a.lane >> 5;
  a.c = p.c;
  a.pex = pex + a.pair * 4 * 64;

  // item -> (key chunk, batch*head, key block), first chunk first: with an
  // unbounded window the earliest keys are seen by the most queries
  int ck, bh, kblk;
  {
    const int vi = xcd_item(blockIdx.x, p.n_kv_items);
    const int BH = p.B * p.H;
    const int n_full = (p.n_kchunks - 1) * BH * p.kblocks_full;
    if (vi < n_full) {
      const int per = BH * p.kblocks_full;
      ck = vi / per;
      const int rem = vi - ck * per;
      bh = rem / p.kblocks_full;
      kblk = rem - bh * p.kblocks_full;
    } else {
      const int v2 = vi - n_full;
      ck = p.n_kchunks - 1;
      bh = v2 / p.kblocks_last;
      kblk = v2 - bh * p.kblocks_last;
    }
  }
  const int b = bh / p.H, h = bh - (bh / p.H) * p.H;
  const int L = p.chunk_len;
  const int key_end = (L < p.nkv - ck * L) ? (ck + 1) * L : p.nkv;
  const int key0 = ck * L + kblk * kBwdKeysPerItem + a.pair * 32;  // this pair's first key
  const int key = key0 + a.n;
  // queries that see key chunk ck: local chunks [ck - q_off, ck + W - q_off]
  int cl_lo = ck - p.q_chunk_offset;
  if (cl_lo < 0) cl_lo = 0;
  int cl_hi = p.n_local_chunks;  // exclusive
  if (p.window >= 0 && ck + p.window - p.q_chunk_offset + 1 < cl_hi) cl_hi = ck + p.window - p.q_chunk_offset + 1;
  const int qlo = cl_lo * L;
  int qhi = cl_hi * L;
  if (qhi > p.nq) qhi = p.nq;
  const int n_tiles = qhi > qlo ? (qhi - qlo + kTile - 1) / kTile : 0;
  const int st = p.st;
  const uint16_t* qb = p.q + (int64_t)b * p.q_sb + (int64_t)h * D;
  const uint16_t* dob = p.dout + (int64_t)b * p.q_sb + (int64_t)h * D;
  const float* rsb = p.rs + ((int64_t)b * p.H + h) * 2 * p.nq;  // planes: LSE log2 e, -D

  Dma dma;
  dma.init(a.pair, a.lane, st);
  a.rd.init(a.lane);
  auto tile_rows = [&](int t) { return qhi - (qlo + t * kTile); };
  // Group B: Q tile t and its row statistics (wave pair w: plane w >> 1, rows
  // 32 (w & 1) .. + 31, 4 bytes per lane from 32 exec-masked lanes; the tile
  // may start at an odd row)
  auto load_b = [&](int t) {
    dma.load(qb + (int64_t)(qlo + t * kTile) * st, tile_rows(t), st, a.qs + (t & (kDkvStages - 1)) * kStage, a.pair);
    if (a.lane < 32) {
      const int r0 = 32 * (a.pair & 1);
      int rows = tile_rows(t) - r0;
      rows = rows < 0 ? 0 : (rows > 32 ? 32 : rows);
      const float* src = rsb + (int64_t)(a.pair >> 1) * p.nq + qlo + t * kTile + r0;
      const i32x4 rsrc = make_vsharp(src, (int64_t)rows * 4);
      const uint32_t la = lds_addr(rss + (t & (kDkvStages - 1)) * K::kRs) + (uint32_t)(a.pair * 32 * 4);
      dma4(la, (uint32_t)(a.lane * 4), rsrc, 0);
    }
  };
  // Group A: dO tile t
  auto load_a = [&](int t) {
    dma.load(dob + (int64_t)(qlo + t * kTile) * st, tile_rows(t), st, a.dos + (t & (kDkvStages - 1)) * kStage,
             a.pair);
  };
  if (n_tiles > 0) {
    if (group == 0) {
      load_a(0);
      load_a(1);
    } else {
      load_b(0);
      load_b(1);
    }
  }
  // K (group A) or V (group B) fragments of this pair's 32 keys
  {
    const int rows = key_end - key0;
    const int64_t koff = (int64_t)b * p.kv_sb + (int64_t)key0 * st + (int64_t)h * D;
    const __amdgpu_buffer_rsrc_t rkv =
        make_rsrc((group == 0 ? p.k : p.v) + koff, rows > 0 ? (int64_t)rows * st * 2 : 0);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const uint32_t e = (uint32_t)(a.n * st + kk * 16 + a.hh * 8);
      a.kvf[kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rkv, e * 2u, 0, 0));
    }
  }
#pragma unroll
  for (int dm = 0; dm < D / 32; ++dm) a.acc[dm] = f32x16{};
  wait_vmcnt<0>();
  __builtin_amdgcn_s_waitcnt(0x0F70);
  barrier();

  // In its vector-ALU slot group B issues the DMA of Q(t + 2) after forming
  // dS, group A that of dO(t + 2) before forming P: 1% faster than the other
  // three orders (one process, alternated turns, identical gradients).
  const int n = n_tiles;
  for (int t = 0; t < n; ++t) {
    // ---- slot 2t ----
    if (group == 0) {
      if (t == 0)
        a.template a_mfma<true, false>(t);
      else
        a.template a_mfma<true, true>(t);
    } else {
      if (t > 0) a.b_valu();
      load_b(t + 2);
    }
    barrier();
    // ---- slot 2t+1 ----
    if (group == 0) {
      load_a(t + 2);
      a.a_valu(t);
      wait_vmcnt<Dma::kPer>();
    } else {
      if (t == 0)
        a.template b_mfma<true, false>(t);
      else
        a.template b_mfma<true, true>(t);
      wait_vmcnt<Dma::kPer + 1>();
    }
    barrier();
  }
  if (n > 0) {
    // ---- slot 2n: dV(n-1), dS(n-1) ----
    if (group == 0)
      a.template a_mfma<false, true>(n);
    else
      a.b_valu();
    barrier();
    // ---- slot 2n+1: dK(n-1) ----
    if (group == 1) a.template b_mfma<false, true>(n);
  }
  wait_vmcnt<0>();

  // dV = dV^T (group A), dK = scale * dK^T (group B): lane n holds dims
  // dm * 32 + 8 g + 4 hh + 0..3 of key n
  if (key < key_end) {
    const int64_t off = (int64_t)b * p.kv_sb + (int64_t)key * st + (int64_t)h * D;
    float* out = (group == 0 ? p.dv : p.dk) + off;
    const float sc = group == 0 ? 1.0f : p.scale;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 val;
        val.x = a.acc[dm][4 * g + 0] * sc;
        val.y = a.acc[dm][4 * g + 1] * sc;
        val.z = a.acc[dm][4 * g + 2] * sc;
        val.w = a.acc[dm][4 * g + 3] * sc;
        *reinterpret_cast<f32x4*>(out + dm * 32 + g * 8 + a.hh * 4) = val;
      }
  }
}

template <int D>
hipError_t launch_bwd_t(const BwdParams& p, hipStream_t stream) {
  if (p.n_q_items > 0)
    hipLaunchKernelGGL((chunk_attn_bwd_dq_kernel<D>), dim3((unsigned)p.n_q_items), dim3(kBwdDqThreads), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.n_kv_items > 0)
    hipLaunchKernelGGL((chunk_attn_bwd_dkv_kernel<D>), dim3((unsigned)p.n_kv_items), dim3(kBwdDkvThreads), 0, stream,
                       p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_chunk_attn_bwd(const BwdArgs& a, hipStream_t stream) {
  const BwdGrid g = bwd_grid(a.B, a.H, a.nq, a.nkv, a.chunk_len);
  BwdParams p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.dout = static_cast<const uint16_t*>(a.dout);
  p.o = a.o;
  p.lse = a.lse;
  p.dq = a.dq;
  p.dk = a.dk;
  p.dv = a.dv;
  p.rs = a.row_stats;
  p.st = (int32_t)(a.H * a.d);
  p.q_sb = a.nq * a.H * a.d;
  p.kv_sb = a.nkv * a.H * a.d;
  // a chunk longer than the key range (only with q_chunk_offset = 0) is the
  // same as a chunk of exactly Nkv tokens
  const int64_t L = (a.chunk_len > a.nkv) ? a.nkv : a.chunk_len;
  p.nq = (int32_t)a.nq;
  p.nkv = (int32_t)a.nkv;
  p.chunk_len = (int32_t)L;
  p.q_chunk_offset = (int32_t)a.q_chunk_offset;
  p.window = (int32_t)((a.window_chunks < 0 || a.window_chunks > a.nkv) ? -1 : a.window_chunks);
  p.B = (int32_t)a.B;
  p.H = (int32_t)a.H;
  p.n_local_chunks = (int32_t)g.q.n_local_chunks;
  p.tiles_full = (int32_t)g.q.tiles_full;
  p.tiles_last = (int32_t)g.q.tiles_last;
  p.n_q_items = (int32_t)g.q.n_items;
  p.n_kchunks = (int32_t)g.n_kchunks;
  p.kblocks_full = (int32_t)g.kblocks_full;
  p.kblocks_last = (int32_t)g.kblocks_last;
  p.n_kv_items = (int32_t)g.n_kv_items;
  p.c = a.scale * 1.44269504088896340736f;
  p.scale = a.scale;
  if (a.d == 128) return launch_bwd_t<128>(p, stream);
  return launch_bwd_t<64>(p, stream);
}

// Workspace of the allocation-free backward (fastvr_chunk_attn_bwd_noalloc):
// the row statistics [B, H, 2, Nq] live in this array instead of caller
// memory.  Each device holds its own copy from the first load of the library's
// code object until the process ends; every call on a device shares it.  The
// dQ kernel writes every entry the dK/dV kernel reads before it reads them
// (same stream), so nothing has to start at zero.
static __device__ __align__(256) float scratch[kBwdScratchFloats];

// Device address of this device's copy of `scratch` (host code must not use
// the array's name as an address): looked up once per device, with that
// device current, and kept.
hipError_t bwd_scratch(float** out) {
  constexpr int kMaxDevices = 64;
  static std::atomic<float*> addr[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  float* p = addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

}  // namespace fastvr
