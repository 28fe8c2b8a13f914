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
// Each wave owns 32 query rows; two waves share each SIMD.  Scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the accumulator puts
// one query per lane (column) and 16 keys per lane (rows), so row max and row
// sum are in-lane plus one exchange between the two 32-lane halves.  The same
// registers, rounded to bf16, are the B operand of O^T = V^T P^T; V is staged
// transposed in LDS with its keys permuted so that every A-operand read is one
// 16-byte LDS load.
//
// Memory: buffer loads with per-tile descriptors (out-of-range rows read as
// zero, no per-lane bounds checks); K tiles go straight from HBM into
// XOR-swizzled LDS (buffer_load ... lds); V tiles pass through registers for
// the 4x4 transpose.  K and V^T tiles of 64 keys are double-buffered.
//
// Pipeline per KV tile j (one barrier per tile):
//   phase A: MFMA  S(j+1) = K(j+1) Q^T          | VALU  P(j) = exp2(t(j)), bf16 pack, half of rowsum
//   (rare)  rescale O by alpha(j) if any row's running maximum grew
//   phase B: MFMA  O^T += V(j)^T P(j)^T          | VALU  rest of rowsum, max of S(j+1), t(j+1) = S*c - m
// with t = s * scale * log2(e) - m (log2 domain, exact running maximum m).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

#ifndef FASTVR_SETPRIO
#define FASTVR_SETPRIO 0
#endif
#ifndef FASTVR_SCHED
#define FASTVR_SCHED 0
#endif

namespace fastvr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kWaves = kFwdThreads / 64;  // 8
constexpr int kBQ = 32 * kWaves;          // 256 query rows per workgroup
constexpr int kBK = 64;                   // keys per KV tile
constexpr float kLn2 = 0.693147180559945309f;
constexpr int kBufFlags = 0x00020000;     // raw buffer, 32-bit data format (gfx9 family)
static_assert(kBQ == kFwdRowsPerItem, "tile height mismatch");

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* o;
  float* lse;
  int64_t q_sb, k_sb, v_sb, o_sb;  // batch strides (elements)
  int32_t q_st, k_st, v_st, o_st;  // token strides (elements, < 2^22)
  int32_t nq, nkv, chunk_len, q_chunk_offset, window;  // window -1 = unbounded
  int32_t B, H, n_local_chunks, tiles_full, tiles_last, n_items;
  float c;  // scale * log2(e)
};

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kBufFlags);
}

// value of the other 32-lane half of the wave, combined with this lane's
__device__ __forceinline__ float swap_halves(float x, float* other) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                  false, false);
  *other = __builtin_bit_cast(float, (uint32_t)r[1]);
  return __builtin_bit_cast(float, (uint32_t)r[0]);
}

// instruction-group ordering hints for the scheduler (sched_group_barrier masks)
#define FASTVR_SCHED_VALU 0x002
#define FASTVR_SCHED_MFMA 0x008
#define FASTVR_SCHED_DS_READ 0x100
#if FASTVR_SCHED
#define SCHED(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
#else
#define SCHED(mask, n) ((void)0)
#endif
#if FASTVR_SETPRIO
#define SETPRIO(p) __builtin_amdgcn_s_setprio(p)
#else
#define SETPRIO(p) ((void)0)
#endif

// ---------------------------------------------------------------------------
// LDS layouts
//   K tile   [D/8 chunks][kBK rows][8] bf16: 16-byte chunk c of key row r at
//            (c * kBK + r) * 16 bytes, so lanes reading consecutive rows of one
//            chunk touch consecutive 16-byte slots (no bank conflicts) and a lane's
//            reads for different chunks differ by compile-time offsets
//   V^T tile [D rows][kBK]   bf16, key order permuted inside each group of 16
//            (swap of key bits 2 and 3), 16-byte chunk index XOR vswz(d)
// ---------------------------------------------------------------------------
template <int D>
struct Lds {
  static constexpr int kKStage = kBK * D;
  static constexpr int kVStage = D * kBK;
  static constexpr int kElems = 2 * kKStage + 2 * kVStage;
  static __device__ __forceinline__ int k_off(int row, int chunk) { return (chunk * kBK + row) * 8; }
};

__device__ __forceinline__ int vswz(int d) { return (d & 7) ^ ((d >> 3) & 1); }
__device__ __forceinline__ int vt_off(int d, int chunk) { return d * kBK + ((chunk ^ vswz(d)) << 3); }

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

// s_waitcnt vmcnt(0) (gfx9 encoding, other counters left at their maximum):
// direct-to-LDS loads must have landed before the barrier that publishes them.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int D, bool NEG>
struct Attn {
  static constexpr int kKPer = kBK * (D / 8) / kFwdThreads;  // 16-byte K chunks per thread per tile
  static constexpr int kVBlocks = (kBK / 4) * (D / 4);       // 4x4 V blocks per tile

  // geometry
  int tid, lane, wave, n, hh;
  int lo, hi;  // visible key interval [lo, hi)
  int n_tiles;
  float c;
  uint16_t* ks;  // K stages
  uint16_t* vt;  // V^T stages
  const uint16_t* kb;
  const uint16_t* vb;
  int k_st, v_st;
  // per-lane constant offsets
  uint32_t k_voff;  // byte offset of this lane's K row (+16 * chunk)
  uint32_t v_voff;  // byte offset of this lane's first V row (+ e * row stride via soffset)
  int vst_off[4];
  int koff;         // element offset of this lane's K operand row, chunk hh
  int voff[4];
  // state
  u32x4 qf[D / 16];
  f32x16 o[D / 32];
  f32x16 s[2];  // raw scores of the next tile
  f32x16 t[2];  // current tile: s*c - m, then exp2 of it in place
  u32x4 pf[4];  // bf16 P fragments of the current tile
  u32x2 vr[4];  // V tile in flight (registers)
  float m_run, l_run, alpha, psum;

  __device__ __forceinline__ void init_offsets() {
    // K: wave w, round i loads chunk c = i * 8 + w of all 64 rows; lane = row
    k_voff = (uint32_t)(lane * k_st + wave * 8) * 2u;
    // V: thread owns keys 4kq..4kq+3 x dims 4dq..4dq+3; in V^T those keys sit in
    // 16-byte chunk `chunk`, 8-byte half `half` of rows 4dq..4dq+3
    const int kq = tid & 15, dq = tid >> 4;
    v_voff = (uint32_t)(kq * 4 * v_st + dq * 4) * 2u;
    const int chunk = ((kq >> 2) << 1) | (kq & 1), half = (kq >> 1) & 1;
#pragma unroll
    for (int x = 0; x < 4; ++x) vst_off[x] = vt_off(dq * 4 + x, chunk) + half * 4;
    koff = Lds<D>::k_off(n, hh);
#pragma unroll
    for (int g = 0; g < 4; ++g) voff[g] = vt_off(n, 2 * g + hh);
  }

  // K tile j -> LDS stage (direct buffer -> LDS, rows >= hi read as zero)
  __device__ __forceinline__ void load_k(int j, int stage) {
    const int t0 = lo + j * kBK;
    const int rows = (hi - t0 < kBK) ? hi - t0 : kBK;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(kb + (int64_t)t0 * k_st, (int64_t)rows * k_st * 2);
#pragma unroll
    for (int i = 0; i < kKPer; ++i) {
      const int c = i * kWaves + wave;
      uint16_t* dst = ks + stage * Lds<D>::kKStage + c * kBK * 8;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, k_voff, i * kWaves * 16, 0, 0);
    }
  }

  // V tile j -> registers (rows >= hi read as zero)
  __device__ __forceinline__ void load_v(int j) {
    if (tid < kVBlocks) {
      const int t0 = lo + j * kBK;
      const int rows = (hi - t0 < kBK) ? hi - t0 : kBK;
      const __amdgpu_buffer_rsrc_t r = make_rsrc(vb + (int64_t)t0 * v_st, (int64_t)rows * v_st * 2);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        vr[e] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, v_voff, e * v_st * 2, 0));
    }
  }

  // registers -> transposed V^T stage: row 4dq+x gets keys 4kq..4kq+3 of dim x
  __device__ __forceinline__ void store_v(int stage) {
    if (tid < kVBlocks) {
      uint16_t* base = vt + stage * Lds<D>::kVStage;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const uint32_t w0 = (x < 2) ? vr[0].x : vr[0].y, w1 = (x < 2) ? vr[1].x : vr[1].y;
        const uint32_t w2 = (x < 2) ? vr[2].x : vr[2].y, w3 = (x < 2) ? vr[3].x : vr[3].y;
        const uint32_t sel = (x & 1) ? 0x07060302u : 0x05040100u;  // high or low bf16 of each word
        u32x2 out;
        out.x = __builtin_amdgcn_perm(w1, w0, sel);
        out.y = __builtin_amdgcn_perm(w3, w2, sel);
        *reinterpret_cast<u32x2*>(base + vst_off[x]) = out;
      }
    }
  }

  // S^T(tile in stage) = K Q^T : 16 MFMAs, raw scores land in s[]
  __device__ __forceinline__ void qk(int stage) {
    const uint16_t* kst = ks + stage * Lds<D>::kKStage;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(kst + koff + Lds<D>::k_off(mb * 32, 2 * kk));
        s[mb] = (kk == 0) ? mfma32(a, qf[kk], f32x16{}) : mfma32(a, qf[kk], s[mb]);
      }
    }
  }

  // O^T += V^T P^T : 16 MFMAs
  __device__ __forceinline__ void pv(int stage) {
    const uint16_t* vst = vt + stage * Lds<D>::kVStage;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
#pragma unroll
      for (int dm = 0; dm < D / 32; ++dm) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(vst + voff[g] + dm * 32 * kBK);
        o[dm] = mfma32(a, pf[g], o[dm]);
      }
    }
  }

  // Row maximum of the raw scores in s[] (MASK: keys at tile positions >= n_valid
  // are outside the visible interval), new running maximum, alpha = 2^(m_old - m_new)
  // and t = s*c - m_new (-inf for masked keys).
  template <bool MASK>
  __device__ __forceinline__ void row_max_and_shift(int n_valid) {
    constexpr float kInf = __builtin_inff();
    float mx = NEG ? kInf : -kInf;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = s[mb][v];
        if (MASK) {
          const int key = mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
          x = (key < n_valid) ? x : (NEG ? kInf : -kInf);
        }
        mx = NEG ? __builtin_fminf(mx, x) : __builtin_fmaxf(mx, x);
      }
    float other;
    const float mine = swap_halves(mx, &other);
    mx = NEG ? __builtin_fminf(mine, other) : __builtin_fmaxf(mine, other);
    const float m_new = __builtin_fmaxf(m_run, mx * c);
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first tile (m_run = -inf)
    m_run = m_new;
    const float nm = -m_new;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = __builtin_fmaf(s[mb][v], c, nm);
        if (MASK) {
          const int key = mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
          x = (key < n_valid) ? x : -kInf;
        }
        t[mb][v] = x;
      }
  }

  // P = exp2(t) in place, bf16 fragments, first half of the row sum
  __device__ __forceinline__ void exp_and_pack() {
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) t[mb][v] = __builtin_amdgcn_exp2f(t[mb][v]);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x8 b;
#pragma unroll
      for (int r = 0; r < 8; ++r) b[r] = (__bf16)t[g >> 1][8 * (g & 1) + r];
      pf[g] = __builtin_bit_cast(u32x4, b);
    }
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) ps += t[0][v];
    psum = ps;
  }

  __device__ __forceinline__ void finish_sum() {
    float ps = psum;
#pragma unroll
    for (int v = 0; v < 16; ++v) ps += t[1][v];
    l_run = l_run * alpha + ps;
  }

  __device__ __forceinline__ void rescale_o() {
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f)) {
#pragma unroll
      for (int dm = 0; dm < D / 32; ++dm) o[dm] *= alpha;
    }
  }

  __device__ __forceinline__ void sched_phase() {
    // 16 MFMAs, each followed by ~4 VALU ops; LDS operand reads run 4 ahead
    SCHED(FASTVR_SCHED_DS_READ, 4);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      SCHED(FASTVR_SCHED_MFMA, 1);
      SCHED(FASTVR_SCHED_VALU, 4);
      if (i < 12) SCHED(FASTVR_SCHED_DS_READ, 1);
    }
  }

  // one pipelined KV tile: j in [0, n_tiles - 2]; t[] holds tile j, s[] receives tile j+1
  template <bool MASK_NEXT>
  __device__ __forceinline__ void step(int j, int n_valid_next) {
    const int cur = j & 1, nxt = (j + 1) & 1;
    load_v(j + 1);
    if (j + 2 < n_tiles) load_k(j + 2, cur);
    // phase A: scores of tile j+1 on the matrix cores, exp2 of tile j on the VALU
    SETPRIO(1);
    qk(nxt);
    exp_and_pack();
    sched_phase();
    SETPRIO(0);
    rescale_o();
    // phase B: O += P V on the matrix cores, row statistics of tile j+1 on the VALU
    SETPRIO(1);
    pv(cur);
    finish_sum();
    row_max_and_shift<MASK_NEXT>(n_valid_next);
    sched_phase();
    SETPRIO(0);
    store_v(nxt);
    wait_vmem();
    __syncthreads();
  }

  // same loads, stores and barriers as step() for a wave whose rows are all padding
  __device__ __forceinline__ void step_idle(int j) {
    load_v(j + 1);
    if (j + 2 < n_tiles) load_k(j + 2, j & 1);
    store_v((j + 1) & 1);
    wait_vmem();
    __syncthreads();
  }
};

template <int D, bool NEG>
__global__ __launch_bounds__(kFwdThreads) void chunk_attn_fwd_kernel(const Params p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[Lds<D>::kElems];
  Attn<D, NEG> a;
  a.ks = smem;
  a.vt = smem + 2 * Lds<D>::kKStage;
  a.tid = threadIdx.x;
  a.lane = a.tid & 63;
  a.wave = a.tid >> 6;
  a.n = a.lane & 31;
  a.hh = a.lane >> 5;
  a.c = p.c;

  int cl, bh, t;
  decode_item(p, blockIdx.x, cl, bh, t);
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
  a.init_offsets();

  const int row = q0 + a.wave * 32 + a.n;
  const bool active = (q0 + a.wave * 32) < q_end;  // wave-uniform
  const int last_valid = a.hi - (a.lo + (a.n_tiles - 1) * kBK);  // keys in the last tile

  // prologue: V(0) to registers, K(0), K(1) to LDS, Q fragments
  a.load_v(0);
  a.load_k(0, 0);
  if (a.n_tiles > 1) a.load_k(1, 1);
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
  a.store_v(0);
  wait_vmem();
  __syncthreads();

  if (active) {
    a.qk(0);
    if (a.n_tiles == 1 && last_valid < kBK)
      a.template row_max_and_shift<true>(last_valid);
    else
      a.template row_max_and_shift<false>(kBK);
  }
  __syncthreads();  // every wave has read K stage 0 before it is refilled
  for (int j = 0; j + 2 < a.n_tiles; ++j) {
    if (active)
      a.template step<false>(j, kBK);
    else
      a.step_idle(j);
  }
  if (a.n_tiles >= 2) {
    const int j = a.n_tiles - 2;
    if (!active)
      a.step_idle(j);
    else if (last_valid < kBK)
      a.template step<true>(j, last_valid);
    else
      a.template step<false>(j, kBK);
  }
  if (!active) return;

  // last tile
  const int jl = a.n_tiles - 1;
  a.exp_and_pack();
  a.rescale_o();
  a.pv(jl & 1);
  a.finish_sum();

  // epilogue: the two halves of the wave hold partial sums over disjoint keys
  float l_other;
  const float l_mine = swap_halves(a.l_run, &l_other);
  const float l_tot = l_mine + l_other;
  if (row < q_end) {
    const float inv = 1.0f / l_tot;
    float* ob = p.o + (int64_t)b * p.o_sb + (int64_t)row * p.o_st + (int64_t)h * D;
#pragma unroll
    for (int dm = 0; dm < D / 32; ++dm)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 val;
        val.x = a.o[dm][4 * g + 0] * inv;
        val.y = a.o[dm][4 * g + 1] * inv;
        val.z = a.o[dm][4 * g + 2] * inv;
        val.w = a.o[dm][4 * g + 3] * inv;
        *reinterpret_cast<f32x4*>(ob + dm * 32 + g * 8 + a.hh * 4) = val;
      }
    if (a.hh == 0 && p.lse != nullptr)
      p.lse[((int64_t)b * p.H + h) * p.nq + row] = (a.m_run + __builtin_log2f(l_tot)) * kLn2;
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
  const FwdGrid g = fwd_grid(a.B, a.H, a.nq, a.chunk_len > a.nkv ? a.nkv : a.chunk_len);
  Params p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = a.o;
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
  const bool neg = p.c < 0.f;
  if (a.d == 128) return neg ? launch_t<128, true>(p, g.n_items, stream) : launch_t<128, false>(p, g.n_items, stream);
  return neg ? launch_t<64, true>(p, g.n_items, stream) : launch_t<64, false>(p, g.n_items, stream);
}

}  // namespace fastvr
