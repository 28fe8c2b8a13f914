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
// Items are dispatched longest first; when they are few per CU and uneven, the
// host instead packs them into one list per CU and launches one workgroup per
// CU that runs its list (item_lists.h).  Each wave owns 32 query rows.  Scores are computed transposed,
// S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the accumulator puts one query per
// lane (column) and 16 keys per lane (rows), so row max and row sum are in-lane
// plus one exchange between the two 32-lane halves.  The same registers,
// rounded to bf16, are the B operand of O^T = V^T P^T.
//
// Matrix-core / vector-ALU ping-pong: waves 0-3 (group A) and 4-7 (group B)
// share the four SIMDs one-to-one.  Time is cut into slots separated by
// workgroup barriers, and the two groups swap roles every slot:
//  * matrix-core slot: the QK MFMAs of key tile j (24 for 96 keys and
//    d = 128), then as many P.V MFMAs of tile j-1, with the row statistics of
//    the new scores (running maximum, rescale factor, s * c - m) issued
//    between them, so that this wave's vector-ALU work hides under its own
//    matrix-core time;
//  * vector-ALU slot: exp2, row sums, bf16 rounding of P and the rescale of O,
//    plus the DMA of the next K or V tile.
// Each SIMD therefore always has a matrix-core wave and a vector-ALU wave side
// by side.
//
// Memory: all K and V tiles (96 keys) travel by DMA straight from HBM into LDS
// (buffer_load ... lds, per-tile buffer descriptors: rows outside the visible
// interval read as zero), triple-buffered and issued two tiles ahead, K in the
// even slots and V in the odd ones.  Both tiles are stored row-major, K with
// its 16-byte chunk index XOR (row & 15), V with it XOR vswz(row & 3), so one
// DMA instruction moves four whole key rows; V^T operands are read with
// ds_read_b64_tr_b16, which transposes 4x16 blocks across 16 lanes.
// Both layouts keep the operand reads free of LDS bank conflicts (64 banks,
// 32 lanes served per cycle).
//
// Online softmax in the log2 domain: t = s * scale * log2(e), exact running
// maximum m, running sum l; O is rescaled only when a row's maximum grows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "gfx950_ops.h"
#include "item_lists.h"
#include "launch.h"

namespace fastvr {
namespace {

using namespace dev;

constexpr int kWaves = kFwdThreads / 64;  // 8
constexpr int kBQ = 32 * kWaves;          // 256 query rows per workgroup
#ifndef FASTVR_BK
#define FASTVR_BK 96
#endif
constexpr int kBK = FASTVR_BK;            // keys per KV tile (FASTVR_BK: 64 or 96)
constexpr int kKB = kBK / 32;             // 32-key blocks of a tile (score accumulators)
constexpr int kKG = kBK / 16;             // 16-key groups of a tile (P fragments)
// 96 keys: 48 MFMAs per matrix-core slot instead of 32 spread each slot's fixed
// costs (operand-read ramp, barrier skew) over more work; three stages of K and
// V then take 144 KB of LDS (d = 128), so 128 keys would not fit
static_assert(kBK == 64 || kBK == 96, "key tile of 64 or 96 keys");
constexpr int kStages = 3;                // LDS buffers per operand
// Tuning switches (compile time):
//  FASTVR_SCHED      order MFMAs, LDS reads and vector-ALU work with scheduling groups
//  FASTVR_PRIO       raise the wave priority during matrix-core slots
//  FASTVR_AHEAD      MFMA operand reads kept in flight ahead of their MFMA
//  FASTVR_VALU_PER   row-statistics instructions placed after each P.V MFMA
//  FASTVR_DMA_SPLIT  1: the four vector-ALU waves of a slot issue its DMA; 0: all eight
//                    (with 96-key tiles only for head_dim 128: a d = 64 tile is 12
//                    DMA instructions, not a multiple of eight)
#ifndef FASTVR_SCHED
#define FASTVR_SCHED 1
#endif
#ifndef FASTVR_PRIO
#define FASTVR_PRIO 1
#endif
#ifndef FASTVR_AHEAD
#define FASTVR_AHEAD 8
#endif
#ifndef FASTVR_VALU_PER
#define FASTVR_VALU_PER 4
#endif
#ifndef FASTVR_DMA_SPLIT
#define FASTVR_DMA_SPLIT 1
#endif
static_assert(kBQ == kFwdRowsPerItem, "tile height mismatch");

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  void* o;        // fp32, or bf16 when o_bf16
  float* lse;
  int64_t q_sb, k_sb, v_sb, o_sb;  // batch strides (elements)
  int32_t q_st, k_st, v_st, o_st;  // token strides (elements, < 2^22)
  int32_t nq, nkv, chunk_len, q_chunk_offset, window;  // window -1 = unbounded
  int32_t B, H, n_local_chunks, tiles_full, tiles_last, n_items;
  float c;  // scale * log2(e)
  int32_t o_bf16;  // 1: O stored as bf16 (round to nearest even), 0: fp32
  // Bounded ring cache (ring step only): key rows are virtual rows over the
  // visible chunks in chunk order; chunk s < n_seg - 1 is read from ring slot
  // (ring_first + s) mod ring_slots, the last (new) one from k / v above.
  uint16_t* rk;
  uint16_t* rv;
  int64_t ring_sb;  // batch stride of the ring (elements); token stride = k_st
  int32_t ring_slots, ring_first, n_seg, new_slot, ring_chunk;  // ring_chunk: tokens per slot
};
constexpr int kMaxRingSlots = 8;

// XOR applied to the 16-byte chunk index of V row r (u = r & 3).  A transpose
// read by lanes 0-31 touches rows u = 0..3 and the chunks 4*dm + (0..3); the
// pattern 0, 6, 12, 10 spreads those 16 chunks over all 64 banks (and any 16
// lanes over 8 distinct chunk slots).  With 8 chunks per row (head_dim 64) the
// pattern 2u keeps them within the row.
template <int D>
__device__ __forceinline__ int vswz(int u) {
  return D >= 128 ? (((u & 1) * 6) ^ ((u >> 1) * 12)) : 2 * u;
}

// Item index vi -> (local query chunk, batch*head, tile).  Items are ordered by
// query chunk, last chunk first: under the causal mask later chunks see at
// least as many keys, so the longest items start first.  (The host's item-list
// planner decodes item indices the same way.)
__device__ __forceinline__ void decode_item(const Params& p, int vi, int& cl, int& bh, int& t) {
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

// blockIdx -> item index.  Workgroups are handed to the 8 XCDs round-robin;
// within each full round of 256 workgroups the mapping gives XCD x a run of 32
// consecutive items (same batch, head and chunk, i.e. the same K/V stream) so
// they share that XCD's L2.
__device__ __forceinline__ int item_of_block(const Params& p, int i) {
  constexpr int kRound = 256;
  const int full = (p.n_items / kRound) * kRound;
  if (i < full) {
    const int r = i / kRound, w = i % kRound;
    return r * kRound + (w & 7) * 32 + (w >> 3);
  }
  return i;
}

// SPLIT: the matrix-core slot takes only each lane's row maximum of the fresh
// scores; the exchange between the halves, the running maximum and s * c - m
// move into the following vector-ALU slot (fused with the exp2).  Same
// arithmetic either way (outputs are bit-identical).  The per-CU list kernel
// uses it: it moves work out of the matrix-core slot, which helps the short
// items of those calls, and it keeps that kernel within its registers.
template <int D, bool NEG, bool RING, bool SPLIT = false>
struct Attn {
  static constexpr int kChunks = D / 8;                        // 16-byte chunks per key row
  static constexpr int kStage = kBK * D;                       // bf16 elements per stage (K or V)
  // Waves issuing the DMA of one tile: all 8, or (split) the 4 waves that run
  // the softmax in that slot, each with twice the instructions.
  static constexpr int kDmaWaves = FASTVR_DMA_SPLIT ? kWaves / 2 : kWaves;
  static constexpr int kDmaPer = kBK * kChunks / (64 * kDmaWaves);  // DMA instructions per issuing wave per tile
  static constexpr int kLdsElems = 2 * kStages * kStage;
  static_assert(kDmaPer >= 1 && kChunks >= 8, "head_dim must be 64 or 128");
  static_assert((kBK * kChunks) % (64 * kDmaWaves) == 0, "a tile is a whole number of DMA instructions per wave");

  int lane, wave, n, hh;
  int lo, hi, n_tiles;
  float c;
  uint16_t* ks;  // K stages (chunk-major)
  uint16_t* vs;  // V stages (row-major, swizzled)
  const uint16_t* kb;
  const uint16_t* vb;
  int k_st, v_st;
  uint32_t k_dma_off, v_dma_off;  // per-lane byte offsets of this wave's DMA rows
  // ring step: ring bases of this (batch, head), chunk length, slots
  const uint16_t* rkb;
  const uint16_t* rvb;
  int ring_L, ring_slots, ring_first, n_seg, n_last;
  int k_rd[D / 16];                // byte offsets of this lane's K operand reads (row n, chunk 2kk + hh)
  int v_rd[D / 32];                // byte offsets of this lane's V^T transpose reads
  u32x4 qf[D / 16];
  f32x16 o[D / 32];
  f32x16 s[kKB];
  u32x4 pf[kKG];
  float m_run, l_run;
  float alpha;  // rescale factor of the tile whose statistics were taken last
  float pmax;   // this lane's maximum of the fresh scores (before the exchange between halves)

  // XOR applied to the 16-byte chunk index of K row r: 16 consecutive rows read
  // the same logical chunk from 16 distinct bank groups
  static __device__ __forceinline__ int kswz(int row) { return row & (kChunks - 1) & 15; }

  __device__ __forceinline__ void init_offsets() {
    // DMA instruction i of wave w fills LDS chunk slots (i * 8 + w) * 64 + lane of
    // a stage: row P / kChunks, physical chunk P % kChunks.  The row offset i * 8 * 64
    // / kChunks goes into the scalar offset; row & 15 does not depend on i.
    {
      const int P = (wave % kDmaWaves) * 64 + lane;
      const int row = P / kChunks, phys = P % kChunks;
      k_dma_off = (uint32_t)(row * k_st + (phys ^ kswz(row)) * 8) * 2u;
      v_dma_off = (uint32_t)(row * v_st + (phys ^ vswz<D>(row & 3)) * 8) * 2u;
    }
    // K operand (A of S^T = K Q^T): row mb*32 + n, chunk 2*kk + hh (mb adds 32 rows)
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) k_rd[kk] = n * (D * 2) + (((2 * kk + hh) ^ kswz(n)) * 16);
    // V^T operand via transpose reads: 16-lane block b = lane / 16 reads rows
    // hh*4 + (i >> 2) (+ 16 g + 8 rho), dims dm*32 + 16*(b & 1) + 4*(i & 3) .. + 3
    const int i = lane & 15, b = lane >> 4;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm) {
      const int row = hh * 4 + (i >> 2);
      const int logical = dm * 4 + 2 * (b & 1) + ((i >> 1) & 1);
      const int phys = logical ^ vswz<D>(row & 3);
      v_rd[dm] = row * (D * 2) + phys * 16 + (i & 1) * 8;
    }
  }

  // DMA of one K (or V) tile: `base` points at the tile's first key row, `rows`
  // valid rows (0 past the end of the interval: the stage is filled with zeros).
  // A tile is kDmaPer instructions per issuing wave; a DmaJob holds what they share.
  struct DmaJob {
    i32x4 rsrc;
    uint32_t lds;
  };
  template <bool IS_K>
  __device__ __forceinline__ DmaJob dma_job(const uint16_t* base, int rows, int stage) const {
    const int st = IS_K ? k_st : v_st;
    return DmaJob{make_vsharp(base, (int64_t)rows * st * 2), lds_addr((IS_K ? ks : vs) + stage * kStage)};
  }
  template <bool IS_K>
  __device__ __forceinline__ void dma_inst(const DmaJob& jb, int i) const {
    constexpr int kRowsPerInst = 64 / kChunks;  // rows covered by one wave instruction
    const int slot0 = (i * kDmaWaves + wave % kDmaWaves) * 64;
    const int st = IS_K ? k_st : v_st;
    dma16(jb.lds + slot0 * 16, IS_K ? k_dma_off : v_dma_off, jb.rsrc, i * kDmaWaves * kRowsPerInst * st * 2);
  }
  __device__ __forceinline__ void dma_k(const uint16_t* base, int rows, int stage) {
    const DmaJob jb = dma_job<true>(base, rows, stage);
#pragma unroll
    for (int i = 0; i < kDmaPer; ++i) dma_inst<true>(jb, i);
  }
  __device__ __forceinline__ void dma_v(const uint16_t* base, int rows, int stage) {
    const DmaJob jb = dma_job<false>(base, rows, stage);
#pragma unroll
    for (int i = 0; i < kDmaPer; ++i) dma_inst<false>(jb, i);
  }
  // Ring step.  Virtual key rows run over the visible chunks in chunk order;
  // chunk seg < n_seg - 1 lives in ring slot (ring_first + seg) mod ring_slots,
  // the last one is the new chunk in k / v.
  struct RingSeg {
    const uint16_t* base;  // row 0 of the chunk
    int start;             // virtual row of its first key
    int len;               // keys it holds
  };
  template <bool IS_K>
  __device__ __forceinline__ RingSeg ring_seg(int seg) const {
    if (seg >= n_seg - 1) return RingSeg{IS_K ? kb : vb, (n_seg - 1) * ring_L, n_last};
    int slot = ring_first + seg;
    if (slot >= ring_slots) slot -= ring_slots;
    return RingSeg{(IS_K ? rkb : rvb) + (int64_t)slot * ring_L * (IS_K ? k_st : v_st), seg * ring_L, ring_L};
  }
  __device__ __forceinline__ int ring_seg_of(int r) const {
    // chunks are consecutive runs of ring_L virtual rows (scalar loop, n_seg <= 8)
    int seg = 0, bound = ring_L;
    while (seg + 1 < n_seg && r >= bound) {
      ++seg;
      bound += ring_L;
    }
    return seg;
  }

  // DMA instruction i of the tile starting at virtual row t0, whose rows all
  // lie in chunk sg (the host requires chunk_len to be a multiple of the
  // instruction's kRowsPerInst rows): one buffer descriptor over the rest of
  // that chunk, so rows past its end read as zero.
  template <bool IS_K>
  __device__ __forceinline__ void dma_inst_ring(const RingSeg& sg, int r0, int stage, int i) const {
    constexpr int kRowsPerInst = 64 / kChunks;
    const int st = IS_K ? k_st : v_st;
    const int in_seg = r0 - sg.start;
    // only this instruction's rows matter: clamp to [0, kRowsPerInst] so the
    // byte count stays a small 32-bit value
    int rows = sg.len - in_seg;
    rows = rows < 0 ? 0 : (rows > kRowsPerInst ? kRowsPerInst : rows);
    const uint64_t a = (uint64_t)(sg.base + (int64_t)in_seg * st);
    const i32x4 r = {(int)(uint32_t)a, (int)((a >> 32) & 0xffff), rows * st * 2, kBufFlags};
    // per-lane offset within the instruction's rows: drop this wave's row offset
    const uint32_t off = (IS_K ? k_dma_off : v_dma_off) - (uint32_t)((wave % kDmaWaves) * kRowsPerInst * st * 2);
    const uint32_t la = lds_addr((IS_K ? ks : vs) + stage * kStage) +
                        (uint32_t)((i * kDmaWaves + wave % kDmaWaves) * 64 * 16);
    dma16(la, off, r, 0);
  }

  // One K or V tile of a ring step.  With chunks of at least one tile the tile
  // touches at most two chunks, looked up once per tile; shorter chunks take
  // the lookup per instruction.
  template <bool IS_K>
  __device__ __forceinline__ void load_ring(int j, int stage) {
    constexpr int kRowsPerInst = 64 / kChunks;
    const int t0 = __builtin_amdgcn_readfirstlane(lo + j * kBK);
    // wave-uniform offset of this wave's rows in the tile (scalar register)
    const int w0 = __builtin_amdgcn_readfirstlane((wave % kDmaWaves) * kRowsPerInst);
    if (ring_L >= kBK) {
      const int seg0 = ring_seg_of(t0);
      const RingSeg s0 = ring_seg<IS_K>(seg0);
      if (seg0 + 1 >= n_seg || t0 + kBK <= (seg0 + 1) * ring_L) {
        // the whole tile lies in one chunk (all but one tile per chunk
        // boundary): the plain tile DMA from that chunk
        const int in_seg = t0 - s0.start;
        const int rows = s0.len - in_seg;
        if (IS_K)
          dma_k(s0.base + (int64_t)in_seg * k_st, rows < 0 ? 0 : (rows > kBK ? kBK : rows), stage);
        else
          dma_v(s0.base + (int64_t)in_seg * v_st, rows < 0 ? 0 : (rows > kBK ? kBK : rows), stage);
        return;
      }
      const RingSeg s1 = ring_seg<IS_K>(seg0 + 1);
#pragma unroll
      for (int i = 0; i < kDmaPer; ++i) {
        const int r0 = t0 + i * kDmaWaves * kRowsPerInst + w0;
        dma_inst_ring<IS_K>(r0 >= s1.start ? s1 : s0, r0, stage, i);
      }
    } else {
#pragma unroll
      for (int i = 0; i < kDmaPer; ++i) {
        const int r0 = t0 + i * kDmaWaves * kRowsPerInst + w0;
        dma_inst_ring<IS_K>(ring_seg<IS_K>(ring_seg_of(r0)), r0, stage, i);
      }
    }
  }

  // DMA of K (or V) tile j (kBK keys from lo + kBK j) into LDS stage `stage`
  __device__ __forceinline__ void load_k(int j, int stage) {
    if (RING) {
      load_ring<true>(j, stage);
    } else {
      dma_k(kb + (int64_t)(lo + j * kBK) * k_st, tile_rows(j), stage);
    }
  }
  __device__ __forceinline__ void load_v(int j, int stage) {
    if (RING) {
      load_ring<false>(j, stage);
    } else {
      dma_v(vb + (int64_t)(lo + j * kBK) * v_st, tile_rows(j), stage);
    }
  }

  __device__ __forceinline__ int tile_rows(int j) const {
    const int r = hi - (lo + j * kBK);
    return r <= 0 ? 0 : (r < kBK ? r : kBK);
  }

  __device__ __forceinline__ u32x4 read_k(const char* kst, int i) const {
    const int kk = i / kKB, mb = i % kKB;
    return *reinterpret_cast<const u32x4*>(kst + k_rd[kk] + mb * 32 * (D * 2));
  }

  __device__ __forceinline__ i16x8 read_vt(const char* vst, int i) const {
    const int g = i / (D / 32), dm = i % (D / 32);
    const char* base = vst + v_rd[dm] + g * 16 * (D * 2);
    const i16x4 lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 8 * (D * 2)));
    return __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
  }

  // Row statistics of the fresh scores s[] (tile positions >= n_valid lie
  // outside the visible interval): running maximum m (log2 domain), alpha =
  // 2^(m_old - m), and s <- s * c - m in place, ready for exp2.
  template <bool MASK>
  __device__ __forceinline__ void row_stats(int n_valid) {
    constexpr float kInf = __builtin_inff();
    // keys of this lane: mb * 32 + 8 * (v >> 2) + (v & 3) + 4 * hh; the limit is
    // made opaque so that the compares are not shared with another call site
    // and kept alive across the main loop
    int lim = n_valid - 4 * hh;
    if (MASK) asm volatile("" : "+v"(lim));
    float part[4] = {NEG ? kInf : -kInf, NEG ? kInf : -kInf, NEG ? kInf : -kInf, NEG ? kInf : -kInf};
#pragma unroll
    for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = s[mb][v];
        if (MASK) {
          const int key = mb * 32 + 8 * (v >> 2) + (v & 3);
          x = (key < lim) ? x : (NEG ? kInf : -kInf);
        }
        float& pm = part[v & 3];
        pm = NEG ? __builtin_fminf(pm, x) : __builtin_fmaxf(pm, x);
      }
    float mx = NEG ? __builtin_fminf(__builtin_fminf(part[0], part[1]), __builtin_fminf(part[2], part[3]))
                   : __builtin_fmaxf(__builtin_fmaxf(part[0], part[1]), __builtin_fmaxf(part[2], part[3]));
    float other;
    const float mine = swap_halves(mx, &other);
    mx = NEG ? __builtin_fminf(mine, other) : __builtin_fmaxf(mine, other);
    const float m_new = __builtin_fmaxf(m_run, mx * c);
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first tile (m_run = -inf)
    m_run = m_new;
    const float nm = -m_new;
#pragma unroll
    for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float t = __builtin_fmaf(s[mb][v], c, nm);
        if (MASK) {
          const int key = mb * 32 + 8 * (v >> 2) + (v & 3);
          t = (key < lim) ? t : -kInf;
        }
        s[mb][v] = t;
      }
  }

  // First half of the statistics of unmasked fresh scores: this lane's maximum
  // (or minimum for a negative scale) only, with no dependency chain, so that
  // it interleaves freely with MFMAs.
  __device__ __forceinline__ void row_max_partial() {
    constexpr float kInf = __builtin_inff();
    float part[4] = {NEG ? kInf : -kInf, NEG ? kInf : -kInf, NEG ? kInf : -kInf, NEG ? kInf : -kInf};
#pragma unroll
    for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float& pm = part[v & 3];
        pm = NEG ? __builtin_fminf(pm, s[mb][v]) : __builtin_fmaxf(pm, s[mb][v]);
      }
    pmax = NEG ? __builtin_fminf(__builtin_fminf(part[0], part[1]), __builtin_fminf(part[2], part[3]))
               : __builtin_fmaxf(__builtin_fmaxf(part[0], part[1]), __builtin_fmaxf(part[2], part[3]));
  }

  // Second half: the exchange between the halves, the running maximum and
  // alpha, then P = exp2(s * c - m) in one pass.  Same arithmetic as row_stats
  // followed by the exp2 of softmax_rest.
  __device__ __forceinline__ void row_max_finish_exp() {
    float other;
    const float mine = swap_halves(pmax, &other);
    const float mx = NEG ? __builtin_fminf(mine, other) : __builtin_fmaxf(mine, other);
    const float m_new = __builtin_fmaxf(m_run, mx * c);
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    const float nm = -m_new;
#pragma unroll
    for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[mb][v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][v], c, nm));
  }

  // The rest of the online softmax once row_stats has run: P = exp2(t) rounded
  // to bf16 fragments, l = l * alpha + rowsum(P), O *= alpha.  With split
  // statistics (EXP_DONE) the exp2 was already taken by row_max_finish_exp.
  template <bool EXP_DONE = false>
  __device__ __forceinline__ void softmax_rest() {
    if (!EXP_DONE) {
#pragma unroll
      for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
        for (int v = 0; v < 16; ++v) s[mb][v] = __builtin_amdgcn_exp2f(s[mb][v]);
    }
    float ps[4] = {s[0][0], s[0][1], s[0][2], s[0][3]};
#pragma unroll
    for (int mb = 0; mb < kKB; ++mb)
#pragma unroll
      for (int v = (mb == 0 ? 4 : 0); v < 16; ++v) ps[v & 3] += s[mb][v];
    l_run = l_run * alpha + ((ps[0] + ps[1]) + (ps[2] + ps[3]));
#pragma unroll
    for (int g = 0; g < kKG; ++g) {
      bf16x8 b;
#pragma unroll
      for (int r = 0; r < 8; ++r) b[r] = (__bf16)s[g >> 1][8 * (g & 1) + r];
      pf[g] = __builtin_bit_cast(u32x4, b);
    }
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
      for (int dm = 0; dm < D / 32; ++dm) o[dm] *= alpha;
    }
  }

  // One matrix-core slot: S^T(tile in st_k) = K Q^T (QK), then
  // O^T += V^T P^T (tile in st_v, PV) with, when STATS, the row statistics of
  // the new scores interleaved (FASTVR_VALU_PER vector-ALU instructions after
  // each P.V MFMA).  The two phases are separate scheduling regions; K and V^T
  // operand reads run kAhead MFMAs ahead, and the first V^T reads are issued
  // during the last QK MFMAs.  K fragments: one 16-byte read; V^T fragments:
  // two transpose reads of 4 keys each.
  template <bool QK, bool PV, bool STATS>
  __device__ __forceinline__ void mfma_slot(int st_k, int st_v) {
    constexpr int kN = D * kBK / 512;  // MFMAs of each kind (QK: D/16 x kKB key blocks; PV: kKG key groups x D/32)
    constexpr int kAhead = FASTVR_AHEAD < kN ? FASTVR_AHEAD : kN;
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(1);
#endif
    const char* kst = reinterpret_cast<const char*>(ks + st_k * kStage);
    const char* vst = reinterpret_cast<const char*>(vs + st_v * kStage);
    i16x8 vt[kN];
    u32x4 kf[kN];
    if (QK) {
#pragma unroll
      for (int i = 0; i < kAhead; ++i) kf[i] = read_k(kst, i);
#pragma unroll
      for (int i = 0; i < kN; ++i) {
        if (i + kAhead < kN)
          kf[i + kAhead] = read_k(kst, i + kAhead);
        else if (PV)
          vt[i + kAhead - kN] = read_vt(vst, i + kAhead - kN);
        const int kk = i / kKB, mb = i % kKB;
        s[mb] = (kk == 0) ? mfma32(kf[i], qf[kk], f32x16{}) : mfma32(kf[i], qf[kk], s[mb]);
      }
#if FASTVR_SCHED
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, kAhead, 0);
#pragma unroll
      for (int i = 0; i < kN; ++i) {
        __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
        if (i + kAhead < kN)
          __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
        else if (PV)
          __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2, 0);
      }
#endif
      __builtin_amdgcn_sched_barrier(0);
    } else if (PV) {
#pragma unroll
      for (int i = 0; i < kAhead; ++i) vt[i] = read_vt(vst, i);
    }
    if (PV) {
#pragma unroll
      for (int i = 0; i < kN; ++i) {
        if (i + kAhead < kN) vt[i + kAhead] = read_vt(vst, i + kAhead);
        const int g = i / (D / 32), dm = i % (D / 32);
        o[dm] = mfma32(__builtin_bit_cast(u32x4, vt[i]), pf[g], o[dm]);
      }
    }
    if (STATS) {
      if (SPLIT)
        row_max_partial();
      else
        row_stats<false>(kBK);
    }
#if FASTVR_SCHED
    if (PV) {
      if (!QK) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2 * kAhead, 0);
#pragma unroll
      for (int i = 0; i < kN; ++i) {
        if (i + kAhead < kN) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 2, 0);
        __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
        if (STATS) __builtin_amdgcn_sched_group_barrier(SCHED_VALU, FASTVR_VALU_PER, 0);
      }
    }
#endif
#if FASTVR_PRIO
    __builtin_amdgcn_s_setprio(0);
#endif
  }

  // The vector-ALU slot after a matrix-core slot that took the statistics.
  __device__ __forceinline__ void softmax_after_stats() {
    if (SPLIT) {
      row_max_finish_exp();
      softmax_rest<true>();
    } else {
      softmax_rest();
    }
  }

  // Online softmax of the last tile (the only one that can be ragged): its
  // statistics, masked when the tile holds fewer than kBK visible keys, are
  // taken here rather than in the matrix-core slot.
  __device__ __forceinline__ void softmax_last(int last_valid) {
    if (last_valid < kBK)
      row_stats<true>(last_valid);
    else
      row_stats<false>(kBK);
    softmax_rest();
  }
};

// One work item (a query tile of one batch, head and query chunk) from its
// decode to its epilogue, run by the whole workgroup; smem is the workgroup's
// LDS.  Waves without query rows leave before the epilogue.
template <int D, bool NEG, bool RING, bool SPLIT = false>
__device__ __forceinline__ void fwd_item(const Params& p, int vi, uint16_t* smem) {
  using A = Attn<D, NEG, RING, SPLIT>;
  A a;
  a.ks = smem;
  a.vs = smem + kStages * A::kStage;
  const int tid = threadIdx.x;
  a.lane = tid & 63;
  a.wave = tid >> 6;
  a.n = a.lane & 31;
  a.hh = a.lane >> 5;
  a.c = p.c;
  const int group = a.wave >> 2;  // 0: waves 0-3, 1: waves 4-7 (one wave of each per SIMD)

  int cl, bh, t;
  decode_item(p, vi, cl, bh, t);
  const int b = bh / p.H, h = bh - (bh / p.H) * p.H;

  const int L = p.chunk_len;
  const int chunk_q0 = cl * L;
  const int q_end = (L < p.nq - chunk_q0) ? chunk_q0 + L : p.nq;
  const int q0 = chunk_q0 + t * kBQ;
  const int cg = p.q_chunk_offset + cl;  // global chunk of this query tile
  a.lo = (p.window >= 0 && cg > p.window) ? (cg - p.window) * L : 0;
  a.hi = (L < p.nkv - cg * L) ? (cg + 1) * L : p.nkv;
  a.n_tiles = (a.hi - a.lo + kBK - 1) / kBK;
  a.kb = p.k + (int64_t)b * p.k_sb + (int64_t)h * D;
  a.vb = p.v + (int64_t)b * p.v_sb + (int64_t)h * D;
  a.k_st = p.k_st;
  a.v_st = p.v_st;
  if (RING) {
    a.rkb = p.rk + (int64_t)b * p.ring_sb + (int64_t)h * D;
    a.rvb = p.rv + (int64_t)b * p.ring_sb + (int64_t)h * D;
    a.ring_L = p.ring_chunk;
    a.ring_slots = p.ring_slots;
    a.ring_first = p.ring_first;
    a.n_seg = p.n_seg;
    a.n_last = p.nq;  // the new chunk: as many keys as queries
  }
  a.init_offsets();

  const int row = q0 + a.wave * 32 + a.n;
  const bool active = (q0 + a.wave * 32) < q_end;  // wave-uniform
  const int n = a.n_tiles;
  const int last_valid = a.hi - (a.lo + (n - 1) * kBK);  // keys in the last tile

  // prologue: K(0), K(1), V(0) to LDS, Q fragments to registers
  // K DMA is issued by group B (or everyone), V DMA by group A (or everyone):
  // the group in its vector-ALU slot
  const bool k_issuer = !FASTVR_DMA_SPLIT || group == 1;
  const bool v_issuer = !FASTVR_DMA_SPLIT || group == 0;
  if (k_issuer) {
    a.load_k(0, 0);
    a.load_k(1, 1);
  }
  if (v_issuer) a.load_v(0, 0);
  {
    const int rows = (q_end - q0 < kBQ) ? q_end - q0 : kBQ;
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(p.q + (int64_t)b * p.q_sb + (int64_t)q0 * p.q_st + (int64_t)h * D,
                                                (int64_t)rows * p.q_st * 2);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      a.qf[kk] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     rq, (uint32_t)((a.wave * 32 + a.n) * p.q_st + kk * 16 + a.hh * 8) * 2u, 0, 0));
  }
#pragma unroll
  for (int dm = 0; dm < D / 32; ++dm) a.o[dm] = f32x16{};
  a.m_run = -__builtin_inff();
  a.l_run = 0.f;
  wait_vmcnt<0>();
  // the same wait through the builtin, so the compiler's own bookkeeping also
  // sees the Q loads complete and inserts no further vmcnt waits for them
  __builtin_amdgcn_s_waitcnt(0x0F70);
  barrier();

  // DMA instructions a wave issues per iteration (one K and one V tile, or one of them when split)
  constexpr int kBatch = FASTVR_DMA_SPLIT ? A::kDmaPer : 2 * A::kDmaPer;

  // Slot 2j: group A runs the matrix-core slot of tile j (S(j), P(j-1).V(j-1),
  // statistics of S(j)); group B the vector-ALU slot of tile j-1.
  // Slot 2j+1: group A the vector-ALU slot of tile j; group B the matrix-core
  // slot of tile j.
  // Slot 2j starts the DMA of K(j+2), slot 2j+1 that of V(j+1) (zeros past the
  // end); the barrier closing slot 2j+1 waits for the pair issued two slots
  // earlier.  Tile j lives in LDS stage j % 3, so K(j+2) reuses the stage of
  // tile j-1 and V(j+1) the third one.  The first tile, the last tile (the
  // only one that can be ragged; its statistics are taken in the vector-ALU
  // slot) and the drain (j = n) are peeled out of the loop.
  int st_cur = 0, st_prev = 2, st_next = 1;  // stages of tiles j, j-1 (== j+2) and j+1
  // j = 0
  if (k_issuer) a.load_k(2, st_prev);
  if (active && group == 0) {
    if (n == 1)
      a.template mfma_slot<true, false, false>(st_cur, 0);
    else
      a.template mfma_slot<true, false, true>(st_cur, 0);
  }
  barrier();
  if (v_issuer) a.load_v(1, st_next);
  if (active) {
    if (group == 0) {
      if (n == 1)
        a.softmax_last(last_valid);
      else
        a.softmax_after_stats();
    } else {
      if (n == 1)
        a.template mfma_slot<true, false, false>(st_cur, 0);
      else
        a.template mfma_slot<true, false, true>(st_cur, 0);
    }
  }
  wait_vmcnt<kBatch>();
  barrier();
  if (n >= 2) {
    st_prev = st_cur;
    st_cur = st_next;
    st_next = (st_next == 2) ? 0 : st_next + 1;
    for (int j = 1; j + 1 < n; ++j) {
      // ---- slot 2j ----
      if (k_issuer) a.load_k(j + 2, st_prev);
      if (active) {
        if (group == 0)
          a.template mfma_slot<true, true, true>(st_cur, st_prev);
        else
          a.softmax_after_stats();
      }
      barrier();
      // ---- slot 2j+1 ----
      if (v_issuer) a.load_v(j + 1, st_next);
      if (active) {
        if (group == 0)
          a.softmax_after_stats();
        else
          a.template mfma_slot<true, true, true>(st_cur, st_prev);
      }
      wait_vmcnt<kBatch>();
      barrier();
      st_prev = st_cur;
      st_cur = st_next;
      st_next = (st_next == 2) ? 0 : st_next + 1;
    }
    // j = n - 1: last tile (no further DMA)
    if (active) {
      if (group == 0)
        a.template mfma_slot<true, true, false>(st_cur, st_prev);
      else
        a.softmax_after_stats();
    }
    barrier();
    if (active) {
      if (group == 0)
        a.softmax_last(last_valid);
      else
        a.template mfma_slot<true, true, false>(st_cur, st_prev);
    }
  }
  wait_vmcnt<0>();
  barrier();
  // j = n: drain, P(n-1).V(n-1)
  if (active) {
    if (group == 0)
      a.template mfma_slot<false, true, false>(0, st_cur);
    else
      a.softmax_last(last_valid);
  }
  barrier();
  if (active && group == 1) a.template mfma_slot<false, true, false>(0, st_cur);
  if (RING) {
    // fused append: this workgroup's share of the new chunk's K and V goes to
    // ring slot new_slot (a slot no query of this call reads)
    const int64_t hd8 = (int64_t)p.H * D / 8;        // 16-byte units per token
    const int64_t per_b = (int64_t)p.nq * hd8;        // units per batch row
    const int64_t total = per_b * p.B;
    const int64_t share = (total + p.n_items - 1) / p.n_items;
    const int64_t u0 = (int64_t)blockIdx.x * share;
    const int64_t u1 = (u0 + share < total) ? u0 + share : total;
    for (int bb = 0; bb < p.B; ++bb) {
      const int64_t lo_u = (u0 > bb * per_b) ? u0 : bb * per_b;
      const int64_t hi_u = (u1 < (bb + 1) * per_b) ? u1 : (bb + 1) * per_b;
      if (lo_u >= hi_u) continue;
      const u32x4* ksrc = reinterpret_cast<const u32x4*>(p.k + (int64_t)bb * p.k_sb);
      const u32x4* vsrc = reinterpret_cast<const u32x4*>(p.v + (int64_t)bb * p.v_sb);
      const int64_t dst = (int64_t)bb * p.ring_sb + (int64_t)p.new_slot * p.ring_chunk * p.k_st;
      u32x4* kd = reinterpret_cast<u32x4*>(p.rk + dst);
      u32x4* vd = reinterpret_cast<u32x4*>(p.rv + dst);
      for (int64_t u = lo_u - bb * per_b + tid; u < hi_u - bb * per_b; u += kFwdThreads) {
        kd[u] = ksrc[u];
        vd[u] = vsrc[u];
      }
    }
  }
  if (!active) return;

  // epilogue: the two halves of the wave hold partial sums over disjoint keys
  float l_other;
  const float l_mine = swap_halves(a.l_run, &l_other);
  const float l_tot = l_mine + l_other;
  if (row < q_end) {
    const float inv = 1.0f / l_tot;
    const int64_t oo = (int64_t)b * p.o_sb + (int64_t)row * p.o_st + (int64_t)h * D;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 val;
        val.x = a.o[dm][4 * g + 0] * inv;
        val.y = a.o[dm][4 * g + 1] * inv;
        val.z = a.o[dm][4 * g + 2] * inv;
        val.w = a.o[dm][4 * g + 3] * inv;
        const int64_t e = oo + dm * 32 + g * 8 + a.hh * 4;
        if (p.o_bf16) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          const bf16x4 r = {(__bf16)val.x, (__bf16)val.y, (__bf16)val.z, (__bf16)val.w};
          *reinterpret_cast<bf16x4*>(static_cast<uint16_t*>(p.o) + e) = r;
        } else {
          *reinterpret_cast<f32x4*>(static_cast<float*>(p.o) + e) = val;
        }
      }
    if (a.hh == 0 && p.lse != nullptr)
      p.lse[((int64_t)b * p.H + h) * p.nq + row] = (a.m_run + __builtin_log2f(l_tot)) * kLn2;
  }
}

// One workgroup per item, dispatched in item order (longest first).
template <int D, bool NEG, bool RING>
__global__ __launch_bounds__(kFwdThreads) void chunk_attn_fwd_kernel(const Params p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[Attn<D, NEG, RING>::kLdsElems];
  fwd_item<D, NEG, RING>(p, item_of_block(p, blockIdx.x), smem);
}

// One workgroup per CU, each running the items of its own list one after the
// other (lists planned on the host to even out the CUs' total work).
template <int D, bool NEG>
__global__ __launch_bounds__(kFwdThreads) void chunk_attn_fwd_list_kernel(const Params p, const ItemLists lst) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[Attn<D, NEG, false>::kLdsElems];
  const int g = blockIdx.x;
  for (int u = lst.start[g]; u < lst.start[g + 1]; ++u) {
    fwd_item<D, NEG, false, true>(p, lst.item[u], smem);
    // every wave is done with the item's LDS stages before the next item's DMA
    barrier();
  }
}

template <int D, bool NEG>
hipError_t launch_t(const Params& p, bool ring, int64_t n_items, const ItemLists* lists, int n_groups,
                    hipStream_t stream) {
  if (ring)
    hipLaunchKernelGGL((chunk_attn_fwd_kernel<D, NEG, true>), dim3((unsigned)n_items), dim3(kFwdThreads), 0, stream,
                       p);
  else if (lists != nullptr)
    hipLaunchKernelGGL((chunk_attn_fwd_list_kernel<D, NEG>), dim3((unsigned)n_groups), dim3(kFwdThreads), 0, stream,
                       p, *lists);
  else
    hipLaunchKernelGGL((chunk_attn_fwd_kernel<D, NEG, false>), dim3((unsigned)n_items), dim3(kFwdThreads), 0, stream,
                       p);
  return hipGetLastError();
}

// CU count of the current device, queried once per device (0 if it cannot be read)
int device_cu_count() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cus[kMaxDevices];  // 0: not queried yet, -1: query failed
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev >= kMaxDevices) {
    int n = 0;
    return hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess ? n : 0;
  }
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = -1;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n > 0 ? n : 0;
}

}  // namespace

hipError_t launch_chunk_attn_fwd(const FwdArgs& a, hipStream_t stream) {
  const FwdGrid g = fwd_grid(a.B, a.H, a.nq, a.chunk_len > a.nkv ? a.nkv : a.chunk_len);
  Params p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = a.o;
  p.o_bf16 = a.o_bf16 ? 1 : 0;
  p.lse = a.lse;
  // Validated by the caller: sizes < 2^31, token strides < 2^22.  A chunk longer
  // than the key range (only possible with q_chunk_offset = 0) is the same as a
  // chunk of exactly Nkv tokens.
  const int64_t L = (a.chunk_len > a.nkv) ? a.nkv : a.chunk_len;
  p.q_sb = a.q_sb; p.q_st = (int32_t)a.q_st;
  p.k_sb = a.k_sb; p.k_st = (int32_t)a.k_st;
  p.v_sb = a.v_sb; p.v_st = (int32_t)a.v_st;
  p.o_sb = a.o_sb; p.o_st = (int32_t)a.o_st;
  p.nq = (int32_t)a.nq;
  p.nkv = (int32_t)a.nkv;
  p.chunk_len = (int32_t)L;
  p.q_chunk_offset = (int32_t)a.q_chunk_offset;
  // a window reaching past the first chunk is unbounded
  p.window = (int32_t)((a.window_chunks < 0 || a.window_chunks > a.nkv) ? -1 : a.window_chunks);
  p.B = (int32_t)a.B;
  p.H = (int32_t)a.H;
  p.n_local_chunks = (int32_t)g.n_local_chunks;
  p.tiles_full = (int32_t)g.tiles_full;
  p.tiles_last = (int32_t)g.tiles_last;
  p.n_items = (int32_t)g.n_items;
  p.c = a.scale * 1.44269504088896340736f;
  const bool ring = a.k_ring != nullptr;
  p.rk = static_cast<uint16_t*>(a.k_ring);
  p.rv = static_cast<uint16_t*>(a.v_ring);
  p.ring_sb = a.ring_sb;
  p.ring_slots = (int32_t)a.ring_slots;
  p.ring_first = (int32_t)a.ring_first;
  p.n_seg = (int32_t)a.n_seg;
  p.new_slot = (int32_t)a.new_slot;
  p.ring_chunk = (int32_t)a.chunk_len;
  const bool neg = p.c < 0.f;
  // a few uneven items per CU: per-CU item lists (the CU count of the current
  // device; any failure to query it keeps plain dispatch)
  ItemLists lists;
  const ItemLists* use_lists = nullptr;
  int n_groups = 0;
  int n_cu = 0;
  if (!ring && g.n_items > 0 && g.n_items <= kListMaxItems && (n_cu = device_cu_count()) > 0) {
    const ItemShape shape{(int64_t)p.B * p.H, p.n_local_chunks, p.tiles_full, p.tiles_last, p.chunk_len,
                          p.q_chunk_offset, p.window, p.nkv, kBK};
    static PlanCache plans;
    if (plans.plan(shape, (int)g.n_items, n_cu, &lists, &n_groups)) use_lists = &lists;
  }
  if (a.d == 128)
    return neg ? launch_t<128, true>(p, ring, g.n_items, use_lists, n_groups, stream)
               : launch_t<128, false>(p, ring, g.n_items, use_lists, n_groups, stream);
  return neg ? launch_t<64, true>(p, ring, g.n_items, use_lists, n_groups, stream)
             : launch_t<64, false>(p, ring, g.n_items, use_lists, n_groups, stream);
}

}  // namespace fastvr
