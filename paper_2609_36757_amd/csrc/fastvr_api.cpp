// C ABI of libfastvr.so: argument validation (entirely on the host, before any
// HIP call), status strings, the thread-local error detail, and dispatch to
// the kernel launchers.  Declarations and the contract: include/fastvr.h.
#include "fastvr.h"

#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "launch.h"

namespace {

thread_local std::string g_last_error;

fastvr_status fail(fastvr_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

fastvr_status ok() {
  g_last_error.clear();
  return FASTVR_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// a * b with an overflow check on non-negative int64
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

bool add_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0 || a > INT64_MAX - b) return false;
  *out = a + b;
  return true;
}

// Byte extent of a [B, N, H*d] view with element strides (sb, st): the last
// element touched is (B-1)*sb + (N-1)*st + H*d - 1.
bool extent_bytes(int64_t B, int64_t N, int64_t sb, int64_t st, int64_t hd, int64_t elem, int64_t* out) {
  int64_t a, b, c;
  if (!mul_ok(B - 1, sb, &a) || !mul_ok(N - 1, st, &b) || !add_ok(a, b, &c) || !add_ok(c, hd, &c)) return false;
  return mul_ok(c, elem, out);
}

bool overlap(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + static_cast<uintptr_t>(nb) && y < x + static_cast<uintptr_t>(na);
}

struct View {
  const char* name;
  const void* ptr;
  int64_t sb, st, n;
  int64_t elem;  // bytes per element
};

fastvr_status check_view(const View& w, int64_t B, int64_t hd, int64_t* bytes) {
  if (w.ptr == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is NULL", w.name);
  if (!aligned(w.ptr, 16)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", w.name);
  const int64_t unit = 16 / w.elem;
  if (w.st < hd) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s token stride %lld < H*d = %lld", w.name,
                             (long long)w.st, (long long)hd);
  if (w.st % unit != 0 || w.sb % unit != 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s strides must be multiples of %lld elements", w.name, (long long)unit);
  if (B > 1) {
    int64_t span;
    if (!mul_ok(w.n, w.st, &span)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s size overflows int64", w.name);
    if (w.sb < span)
      return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s batch stride %lld < N * token stride = %lld", w.name,
                  (long long)w.sb, (long long)span);
  }
  if (!extent_bytes(B, w.n, w.sb, w.st, hd, w.elem, bytes))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s size overflows int64", w.name);
  return FASTVR_OK;
}

struct Ring {
  void* k = nullptr;
  void* v = nullptr;
  int64_t sb = 0, slots = 0, first = 0, n_seg = 0, new_slot = 0, bytes = 0;
};

fastvr_status fwd_impl(const void* q, int64_t q_sb, int64_t q_st, const void* k, int64_t k_sb, int64_t k_st,
                       const void* v, int64_t v_sb, int64_t v_st, void* o, int64_t o_sb, int64_t o_st, int o_bf16,
                       float* lse,
                       int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len,
                       int64_t q_chunk_offset, int64_t window_chunks, float scale, void* stream,
                       const Ring& ring = Ring()) {
  if (B < 0 || H < 0 || Nq < 0 || Nkv < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size (B=%lld H=%lld Nq=%lld Nkv=%lld)", (long long)B,
                (long long)H, (long long)Nq, (long long)Nkv);
  if (d != 64 && d != 128) return fail(FASTVR_ERR_UNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)d);
  if (q_chunk_offset < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "q_chunk_offset %lld < 0", (long long)q_chunk_offset);
  if (window_chunks < -1)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "window_chunks %lld < -1", (long long)window_chunks);
  if (!std::isfinite(scale)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "scale is not finite");
  if (B == 0 || H == 0 || Nq == 0) return ok();  // empty problem
  if (chunk_len < 1) return fail(FASTVR_ERR_INVALID_ARGUMENT, "chunk_len %lld < 1", (long long)chunk_len);
  int64_t first_q, last_q;
  if (!mul_ok(q_chunk_offset, chunk_len, &first_q) || !add_ok(first_q, Nq, &last_q))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "q_chunk_offset * chunk_len + Nq overflows int64");
  if (last_q > Nkv)
    return fail(FASTVR_ERR_INVALID_ARGUMENT,
                "q_chunk_offset * chunk_len + Nq = %lld > Nkv = %lld (a query would not see its own key)",
                (long long)last_q, (long long)Nkv);
  if (Nkv > INT32_MAX || Nq > INT32_MAX || B > INT32_MAX || H > INT32_MAX)
    return fail(FASTVR_ERR_UNSUPPORTED, "sizes must be below 2^31");
  int64_t hd, bh;
  if (!mul_ok(H, d, &hd) || !mul_ok(B, H, &bh)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");

  int64_t qb, kb, vb, ob;
  fastvr_status s;
  if ((s = check_view({"q", q, q_sb, q_st, Nq, 2}, B, hd, &qb)) != FASTVR_OK) return s;
  // k / v rows in memory: all Nkv key rows, or in a ring step only the new chunk
  const int64_t kv_rows = ring.k != nullptr ? Nq : Nkv;
  if ((s = check_view({"k", k, k_sb, k_st, kv_rows, 2}, B, hd, &kb)) != FASTVR_OK) return s;
  if ((s = check_view({"v", v, v_sb, v_st, kv_rows, 2}, B, hd, &vb)) != FASTVR_OK) return s;
  if (o_bf16 != 0 && o_bf16 != 1)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "o_bf16 must be 0 or 1 (got %d)", o_bf16);
  if ((s = check_view({"o", o, o_sb, o_st, Nq, o_bf16 ? 2 : 4}, B, hd, &ob)) != FASTVR_OK) return s;
  if (q_st >= fastvr::kMaxTokenStride || k_st >= fastvr::kMaxTokenStride || v_st >= fastvr::kMaxTokenStride ||
      o_st >= fastvr::kMaxTokenStride)
    return fail(FASTVR_ERR_UNSUPPORTED, "token strides must be below %lld elements",
                (long long)fastvr::kMaxTokenStride);
  int64_t lb = 0;
  if (lse != nullptr) {
    if (!aligned(lse, 4)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse is not 4-byte aligned");
    if (!mul_ok(bh, Nq, &lb) || !mul_ok(lb, 4, &lb)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse size overflows");
  }
  if (overlap(o, ob, q, qb) || overlap(o, ob, k, kb) || overlap(o, ob, v, vb))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "o overlaps q, k or v");
  if (lse != nullptr && (overlap(lse, lb, q, qb) || overlap(lse, lb, k, kb) || overlap(lse, lb, v, vb) ||
                         overlap(lse, lb, o, ob)))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse overlaps q, k, v or o");
  if (ring.k != nullptr) {
    const void* others[5] = {q, k, v, o, lse};
    const int64_t sizes[5] = {qb, kb, vb, ob, lb};
    for (int i = 0; i < 5; ++i)
      if (others[i] != nullptr && (overlap(ring.k, ring.bytes, others[i], sizes[i]) ||
                                   overlap(ring.v, ring.bytes, others[i], sizes[i])))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "the ring overlaps q_new, k_new, v_new, o or lse");
    if (overlap(ring.k, ring.bytes, ring.v, ring.bytes))
      return fail(FASTVR_ERR_INVALID_ARGUMENT, "k_ring and v_ring overlap");
  }

  const fastvr::FwdGrid g = fastvr::fwd_grid(B, H, Nq, chunk_len);
  if (g.n_items > fastvr::kMaxFwdItems)
    return fail(FASTVR_ERR_UNSUPPORTED, "problem needs %lld workgroups (> %lld)", (long long)g.n_items,
                (long long)fastvr::kMaxFwdItems);

  fastvr::FwdArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse;
  a.o_bf16 = o_bf16 == 1;
  a.q_sb = q_sb; a.q_st = q_st;
  a.k_sb = k_sb; a.k_st = k_st;
  a.v_sb = v_sb; a.v_st = v_st;
  a.o_sb = o_sb; a.o_st = o_st;
  a.B = B; a.H = H; a.nq = Nq; a.nkv = Nkv; a.d = d;
  a.chunk_len = chunk_len;
  a.q_chunk_offset = q_chunk_offset;
  a.window_chunks = window_chunks;
  a.scale = scale;
  a.k_ring = ring.k;
  a.v_ring = ring.v;
  a.ring_sb = ring.sb;
  a.ring_slots = ring.slots;
  a.ring_first = ring.first;
  a.n_seg = ring.n_seg;
  a.new_slot = ring.new_slot;
  const hipError_t e = fastvr::launch_chunk_attn_fwd(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "chunk_attn_fwd launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

fastvr_status fastvr_chunk_attn_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int64_t B,
                                    int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len,
                                    int64_t q_chunk_offset, int64_t window_chunks, float scale, void* stream) {
  int64_t hd = 0, sq = 0, skv = 0;
  if (H >= 0 && d >= 0 && Nq >= 0 && Nkv >= 0 &&
      (!mul_ok(H, d, &hd) || !mul_ok(Nq, hd, &sq) || !mul_ok(Nkv, hd, &skv)))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  return fwd_impl(q, sq, hd, k, skv, hd, v, skv, hd, o, sq, hd, 0, lse, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
                  window_chunks, scale, stream);
}

fastvr_status fastvr_chunk_attn_fwd_ex(const void* q, int64_t q_sb, int64_t q_st, const void* k, int64_t k_sb,
                                       int64_t k_st, const void* v, int64_t v_sb, int64_t v_st, void* o,
                                       int64_t o_sb, int64_t o_st, int32_t o_bf16, float* lse, int64_t B, int64_t H,
                                       int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len, int64_t q_chunk_offset,
                                       int64_t window_chunks, float scale, void* stream) {
  return fwd_impl(q, q_sb, q_st, k, k_sb, k_st, v, v_sb, v_st, o, o_sb, o_st, o_bf16, lse, B, H, Nq, Nkv, d,
                  chunk_len, q_chunk_offset, window_chunks, scale, stream);
}

fastvr_status fastvr_chunk_attn_ring_step(const void* q_new, const void* k_new, const void* v_new, void* k_ring,
                                          void* v_ring, float* o, float* lse, int64_t B, int64_t H, int64_t n_new,
                                          int64_t d, int64_t chunk_len, int64_t chunk_index, int64_t window_chunks,
                                          float scale, void* stream) {
  if (B < 0 || H < 0 || n_new < 0 || chunk_len < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size (B=%lld H=%lld n_new=%lld chunk_len=%lld)",
                (long long)B, (long long)H, (long long)n_new, (long long)chunk_len);
  if (chunk_index < 0) return fail(FASTVR_ERR_INVALID_ARGUMENT, "chunk_index %lld < 0", (long long)chunk_index);
  if (window_chunks < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "a ring cache needs window_chunks >= 0 (got %lld)",
                (long long)window_chunks);
  if (window_chunks > fastvr::kMaxRingWindow)
    return fail(FASTVR_ERR_UNSUPPORTED, "window_chunks %lld > %lld", (long long)window_chunks,
                (long long)fastvr::kMaxRingWindow);
  if (d != 64 && d != 128) return fail(FASTVR_ERR_UNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)d);
  if (n_new < 1 || n_new > chunk_len)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "n_new = %lld must be in 1 .. chunk_len = %lld", (long long)n_new,
                (long long)chunk_len);
  const int64_t rows_per_dma = d == 128 ? 4 : 8;
  if (chunk_len % rows_per_dma != 0)
    return fail(FASTVR_ERR_UNSUPPORTED, "chunk_len %lld is not a multiple of %lld (head_dim %lld)",
                (long long)chunk_len, (long long)rows_per_dma, (long long)d);
  if (k_ring == nullptr || v_ring == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "k_ring or v_ring is NULL");
  if (!aligned(k_ring, 16) || !aligned(v_ring, 16))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "k_ring or v_ring is not 16-byte aligned");
  Ring r;
  r.slots = window_chunks + 1;
  int64_t hd, ring_rows, n_prev, nkv;
  if (!mul_ok(H, d, &hd) || !mul_ok(r.slots, chunk_len, &ring_rows) || !mul_ok(ring_rows, hd, &r.sb) ||
      !mul_ok(B, r.sb, &r.bytes) || !mul_ok(r.bytes, 2, &r.bytes))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  n_prev = chunk_index < window_chunks ? chunk_index : window_chunks;  // earlier visible chunks
  if (!mul_ok(n_prev, chunk_len, &nkv) || !add_ok(nkv, n_new, &nkv))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  if (ring_rows > INT32_MAX) return fail(FASTVR_ERR_UNSUPPORTED, "ring rows must be below 2^31");
  r.k = k_ring;
  r.v = v_ring;
  r.n_seg = n_prev + 1;
  r.new_slot = chunk_index % r.slots;
  r.first = (chunk_index - n_prev) % r.slots;
  int64_t sn = 0;
  if (!mul_ok(n_new, hd, &sn)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  // queries: the new chunk, which is chunk n_prev of the visible sequence; keys:
  // the visible chunks, virtual rows 0 .. nkv - 1 (the kernel reads the earlier
  // ones from the ring and the new one from k_new / v_new)
  return fwd_impl(q_new, sn, hd, k_new, sn, hd, v_new, sn, hd, o, sn, hd, 0, lse, B, H, n_new, nkv, d, chunk_len,
                  n_prev, window_chunks, scale, stream, r);
}

}  // extern "C"

namespace {

// The backward's checks and launch.  own_ws: row_stats is ignored and the
// row statistics go to the library's static per-device array (looked up after
// every check has passed).
fastvr_status bwd_impl(const void* q, const void* k, const void* v, const float* o, const float* lse,
                       const void* dout, float* dq, float* dk, float* dv, float* row_stats, int64_t B, int64_t H,
                       int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len, int64_t q_chunk_offset,
                       int64_t window_chunks, float scale, void* stream, bool own_ws) {
  if (B < 0 || H < 0 || Nq < 0 || Nkv < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size (B=%lld H=%lld Nq=%lld Nkv=%lld)", (long long)B,
                (long long)H, (long long)Nq, (long long)Nkv);
  if (d != 64 && d != 128) return fail(FASTVR_ERR_UNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)d);
  if (q_chunk_offset < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "q_chunk_offset %lld < 0", (long long)q_chunk_offset);
  if (window_chunks < -1)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "window_chunks %lld < -1", (long long)window_chunks);
  if (!std::isfinite(scale)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "scale is not finite");
  if (B == 0 || H == 0 || Nkv == 0) {
    if (Nq > 0 && B > 0 && H > 0)
      return fail(FASTVR_ERR_INVALID_ARGUMENT, "Nq = %lld queries but no keys", (long long)Nq);
    return ok();  // nothing to write
  }
  if (chunk_len < 1) return fail(FASTVR_ERR_INVALID_ARGUMENT, "chunk_len %lld < 1", (long long)chunk_len);
  int64_t first_q, last_q;
  if (!mul_ok(q_chunk_offset, chunk_len, &first_q) || !add_ok(first_q, Nq, &last_q))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "q_chunk_offset * chunk_len + Nq overflows int64");
  if (last_q > Nkv)
    return fail(FASTVR_ERR_INVALID_ARGUMENT,
                "q_chunk_offset * chunk_len + Nq = %lld > Nkv = %lld (a query would not see its own key)",
                (long long)last_q, (long long)Nkv);
  if (Nkv > INT32_MAX || Nq > INT32_MAX || B > INT32_MAX || H > INT32_MAX)
    return fail(FASTVR_ERR_UNSUPPORTED, "sizes must be below 2^31");
  int64_t hd, bh, nrows;
  if (!mul_ok(H, d, &hd) || !mul_ok(B, H, &bh) || !mul_ok(bh, Nq, &nrows))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  if (hd >= fastvr::kMaxTokenStride)
    return fail(FASTVR_ERR_UNSUPPORTED, "H * d = %lld must be below %lld", (long long)hd,
                (long long)fastvr::kMaxTokenStride);
  int64_t sq, skv;
  if (!mul_ok(Nq, hd, &sq) || !mul_ok(Nkv, hd, &skv)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  // every tensor is contiguous; views give the byte extents for the overlap checks
  const View views[8] = {{"q", q, sq, hd, Nq, 2},         {"dout", dout, sq, hd, Nq, 2},
                         {"o", o, sq, hd, Nq, 4},         {"dq", dq, sq, hd, Nq, 4},
                         {"k", k, skv, hd, Nkv, 2},       {"v", v, skv, hd, Nkv, 2},
                         {"dk", dk, skv, hd, Nkv, 4},     {"dv", dv, skv, hd, Nkv, 4}};
  int64_t bytes[10] = {0};
  fastvr_status s;
  for (int i = 0; i < 8; ++i) {
    if (views[i].n == 0) {
      // Nq = 0: the query-side tensors are not read; dK and dV become zero
      if (views[i].ptr != nullptr && !aligned(views[i].ptr, 16))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", views[i].name);
      continue;
    }
    if ((s = check_view(views[i], B, hd, &bytes[i])) != FASTVR_OK) return s;
  }
  const void* lse_ptr = lse;
  const void* rs_ptr = own_ws ? nullptr : row_stats;
  if (Nq > 0) {
    if (own_ws) {
      if (lse == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse is NULL");
      if (!aligned(lse, 4)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse is not 4-byte aligned");
      if (!mul_ok(nrows, 4, &bytes[8])) return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
      if (nrows > fastvr::kBwdScratchFloats / 2)
        return fail(FASTVR_ERR_UNSUPPORTED,
                    "row statistics need 2 * B * H * Nq = %lld floats; the allocation-free backward holds at most "
                    "%lld",
                    (long long)(2 * nrows), (long long)fastvr::kBwdScratchFloats);
    } else {
      if (lse == nullptr || row_stats == nullptr)
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse or row_stats is NULL");
      if (!aligned(lse, 4) || !aligned(row_stats, 4))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "lse or row_stats is not 4-byte aligned");
      if (!mul_ok(nrows, 4, &bytes[8]) || !mul_ok(nrows, 8, &bytes[9]))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
    }
  }
  // outputs (dq, dk, dv, row_stats) overlap nothing else
  const void* ptrs[10] = {q, dout, o, dq, k, v, dk, dv, lse_ptr, rs_ptr};
  const int outs[4] = {3, 6, 7, 9};
  for (int oi = 0; oi < 4; ++oi)
    for (int i = 0; i < 10; ++i) {
      const int w = outs[oi];
      if (i == w || bytes[w] == 0 || bytes[i] == 0) continue;
      if (overlap(ptrs[w], bytes[w], ptrs[i], bytes[i]))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s overlaps %s", w == 9 ? "row_stats" : views[w].name,
                    i == 8 ? "lse" : (i == 9 ? "row_stats" : views[i].name));
    }

  const fastvr::BwdGrid g = fastvr::bwd_grid(B, H, Nq, Nkv, chunk_len);
  if (g.q.n_items > fastvr::kMaxFwdItems || g.n_kv_items > fastvr::kMaxFwdItems)
    return fail(FASTVR_ERR_UNSUPPORTED, "problem needs too many workgroups");

  if (own_ws && Nq > 0) {
    const hipError_t e = fastvr::bwd_scratch(&row_stats);
    if (e != hipSuccess)
      return fail(FASTVR_ERR_HIP, "workspace of the allocation-free backward: %s", hipGetErrorString(e));
  }
  fastvr::BwdArgs a;
  a.q = q; a.k = k; a.v = v; a.dout = dout; a.o = o; a.lse = lse;
  a.dq = dq; a.dk = dk; a.dv = dv; a.row_stats = row_stats;
  a.B = B; a.H = H; a.nq = Nq; a.nkv = Nkv; a.d = d;
  a.chunk_len = chunk_len;
  a.q_chunk_offset = q_chunk_offset;
  a.window_chunks = window_chunks;
  a.scale = scale;
  const hipError_t e = fastvr::launch_chunk_attn_bwd(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "chunk_attn_bwd launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

fastvr_status fastvr_chunk_attn_bwd(const void* q, const void* k, const void* v, const float* o, const float* lse,
                                    const void* dout, float* dq, float* dk, float* dv, float* row_stats, int64_t B,
                                    int64_t H, int64_t Nq, int64_t Nkv, int64_t d, int64_t chunk_len,
                                    int64_t q_chunk_offset, int64_t window_chunks, float scale, void* stream) {
  return bwd_impl(q, k, v, o, lse, dout, dq, dk, dv, row_stats, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
                  window_chunks, scale, stream, false);
}

fastvr_status fastvr_chunk_attn_bwd_noalloc(const void* q, const void* k, const void* v, const float* o,
                                            const float* lse, const void* dout, float* dq, float* dk, float* dv,
                                            int64_t B, int64_t H, int64_t Nq, int64_t Nkv, int64_t d,
                                            int64_t chunk_len, int64_t q_chunk_offset, int64_t window_chunks,
                                            float scale, void* stream) {
  return bwd_impl(q, k, v, o, lse, dout, dq, dk, dv, nullptr, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
                  window_chunks, scale, stream, true);
}

fastvr_status fastvr_kv_cache_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new, int64_t B,
                                     int64_t H, int64_t d, int64_t capacity, int64_t cache_len, int64_t n_new,
                                     void* stream) {
  if (B < 0 || H < 0 || capacity < 0 || cache_len < 0 || n_new < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size");
  if (d != 64 && d != 128) return fail(FASTVR_ERR_UNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)d);
  int64_t end;
  if (!add_ok(cache_len, n_new, &end)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "cache_len + n_new overflows");
  if (end > capacity)
    return fail(FASTVR_ERR_CAPACITY, "cache_len + n_new = %lld > capacity = %lld", (long long)end,
                (long long)capacity);
  if (B == 0 || H == 0 || n_new == 0) return ok();
  if (B > 65535) return fail(FASTVR_ERR_UNSUPPORTED, "B = %lld > 65535", (long long)B);
  const void* ptrs[4] = {k_cache, v_cache, k_new, v_new};
  const char* names[4] = {"k_cache", "v_cache", "k_new", "v_new"};
  for (int i = 0; i < 4; ++i) {
    if (ptrs[i] == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is NULL", names[i]);
    if (!aligned(ptrs[i], 16)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", names[i]);
  }
  int64_t hd, cache_bytes, new_bytes;
  if (!mul_ok(H, d, &hd) || !mul_ok(B, capacity, &cache_bytes) || !mul_ok(cache_bytes, hd, &cache_bytes) ||
      !mul_ok(cache_bytes, 2, &cache_bytes) || !mul_ok(B, n_new, &new_bytes) || !mul_ok(new_bytes, hd, &new_bytes) ||
      !mul_ok(new_bytes, 2, &new_bytes))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  if (overlap(k_cache, cache_bytes, v_cache, cache_bytes))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "k_cache and v_cache overlap");
  for (int c = 0; c < 2; ++c)
    for (int n = 2; n < 4; ++n)
      if (overlap(ptrs[c], cache_bytes, ptrs[n], new_bytes))
        return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s overlaps %s", names[c], names[n]);
  const hipError_t e = fastvr::launch_kv_append(k_cache, v_cache, k_new, v_new, B, H, d, capacity, cache_len, n_new,
                                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "kv_append launch failed: %s", hipGetErrorString(e));
  return ok();
}

fastvr_status fastvr_one_step_update(const void* z_lq, const void* v, void* z_hat, int64_t n, float sigma,
                                     int32_t out_bf16, void* stream) {
  if (n < 0) return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size n = %lld", (long long)n);
  if (!std::isfinite(sigma)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "sigma is not finite");
  if (out_bf16 != 0 && out_bf16 != 1)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "out_bf16 must be 0 or 1 (got %d)", (int)out_bf16);
  if (n == 0) return ok();
  const void* ptrs[3] = {z_lq, v, z_hat};
  const char* names[3] = {"z_lq", "v", "z_hat"};
  for (int i = 0; i < 3; ++i) {
    if (ptrs[i] == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is NULL", names[i]);
    if (!aligned(ptrs[i], 16)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", names[i]);
  }
  int64_t in_bytes, out_bytes;
  if (!mul_ok(n, 2, &in_bytes) || !mul_ok(n, out_bf16 ? 2 : 4, &out_bytes))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  // in place is allowed when the output has the input's element size and
  // starts exactly at z_lq or v (each element is read before it is written)
  for (int i = 0; i < 2; ++i) {
    if (out_bf16 && z_hat == ptrs[i]) continue;
    if (overlap(z_hat, out_bytes, ptrs[i], in_bytes))
      return fail(FASTVR_ERR_INVALID_ARGUMENT, "z_hat overlaps %s", names[i]);
  }
  const hipError_t e = fastvr::launch_one_step(z_lq, v, z_hat, n, sigma, out_bf16 != 0,
                                               static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "one_step launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

namespace {

// Shared checks of the tile entry points; fills the two axes and the element
// counts of the field and of the tile tensor.
fastvr_status tile_check(int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t tile_overlap,
                         int64_t c_multiple, fastvr::TileAxis* ay, fastvr::TileAxis* ax, int64_t* field_elems,
                         int64_t* tile_elems) {
  if (B < 0 || T < 0 || Hg < 0 || Wg < 0 || C < 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "negative size (B=%lld T=%lld Hg=%lld Wg=%lld C=%lld)", (long long)B,
                (long long)T, (long long)Hg, (long long)Wg, (long long)C);
  if (tile < 1 || tile_overlap < 0 || tile_overlap >= tile)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "need tile >= 1 and 0 <= overlap < tile (tile=%lld overlap=%lld)",
                (long long)tile, (long long)tile_overlap);
  if (tile > fastvr::kMaxTile)
    return fail(FASTVR_ERR_UNSUPPORTED, "tile %lld > %lld", (long long)tile, (long long)fastvr::kMaxTile);
  if (C % c_multiple != 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "C = %lld is not a multiple of %lld", (long long)C, (long long)c_multiple);
  *field_elems = 0;
  *tile_elems = 0;
  if (B == 0 || T == 0 || Hg == 0 || Wg == 0 || C == 0) return FASTVR_OK;
  *ay = fastvr::tile_axis(Hg, tile, tile_overlap);
  *ax = fastvr::tile_axis(Wg, tile, tile_overlap);
  int64_t f, t;
  if (!mul_ok(B, T, &f) || !mul_ok(f, Hg, &f) || !mul_ok(f, Wg, &f) || !mul_ok(f, C, &f) ||
      !mul_ok(B, ay->n * ax->n, &t) || !mul_ok(t, T, &t) || !mul_ok(t, ay->len * ax->len, &t) || !mul_ok(t, C, &t) ||
      !mul_ok(t, 4, &t) || !mul_ok(f, 4, &f))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "size overflows int64");
  if (Hg > INT32_MAX || Wg > INT32_MAX || T > INT32_MAX || Wg * C > INT32_MAX)
    return fail(FASTVR_ERR_UNSUPPORTED, "a grid row must hold fewer than 2^31 elements");
  *field_elems = f / 4;
  *tile_elems = t / 4;
  return FASTVR_OK;
}

}  // namespace

extern "C" {

fastvr_status fastvr_tile_axis(int64_t size, int64_t tile, int64_t tile_overlap, int64_t* n_tiles, int64_t* tile_len) {
  if (n_tiles == nullptr || tile_len == nullptr)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "n_tiles or tile_len is NULL");
  if (size < 1 || tile < 1 || tile_overlap < 0 || tile_overlap >= tile)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "need size >= 1, tile >= 1 and 0 <= overlap < tile");
  const fastvr::TileAxis a = fastvr::tile_axis(size, tile, tile_overlap);
  *n_tiles = a.n;
  *tile_len = a.len;
  return ok();
}

fastvr_status fastvr_tile_gather(const void* x, void* tiles, int64_t B, int64_t T, int64_t Hg, int64_t Wg, int64_t C,
                                 int64_t tile, int64_t tile_overlap, void* stream) {
  fastvr::TileAxis ay{}, ax{};
  int64_t fe, te;
  fastvr_status s = tile_check(B, T, Hg, Wg, C, tile, tile_overlap, 8, &ay, &ax, &fe, &te);
  if (s != FASTVR_OK) return s;
  if (fe == 0) return ok();
  if (x == nullptr || tiles == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "x or tiles is NULL");
  if (!aligned(x, 16) || !aligned(tiles, 16))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "x or tiles is not 16-byte aligned");
  if (overlap(x, fe * 2, tiles, te * 2)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "tiles overlaps x");
  const hipError_t e =
      fastvr::launch_tile_gather(x, tiles, B, T, Hg, Wg, C, tile, tile_overlap, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "tile_gather launch failed: %s", hipGetErrorString(e));
  return ok();
}

static fastvr_status blend_impl(const float* tiles, const void* z_lq, float* out, float sigma, int64_t B, int64_t T,
                                int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t tile_overlap, void* stream) {
  fastvr::TileAxis ay{}, ax{};
  int64_t fe, te;
  fastvr_status s = tile_check(B, T, Hg, Wg, C, tile, tile_overlap, 4, &ay, &ax, &fe, &te);
  if (s != FASTVR_OK) return s;
  if (!std::isfinite(sigma)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "sigma is not finite");
  if (fe == 0) return ok();
  if (tiles == nullptr || out == nullptr) return fail(FASTVR_ERR_INVALID_ARGUMENT, "tiles or out is NULL");
  if (!aligned(tiles, 16) || !aligned(out, 16))
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "tiles or out is not 16-byte aligned");
  if (overlap(out, fe * 4, tiles, te * 4)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "out overlaps tiles");
  if (z_lq != nullptr) {
    if (!aligned(z_lq, 8)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "z_lq is not 8-byte aligned");
    if (overlap(out, fe * 4, z_lq, fe * 2)) return fail(FASTVR_ERR_INVALID_ARGUMENT, "out overlaps z_lq");
  }
  const hipError_t e = fastvr::launch_tile_blend(tiles, z_lq, out, sigma, B, T, Hg, Wg, C, tile, tile_overlap,
                                                 static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FASTVR_ERR_HIP, "tile_blend launch failed: %s", hipGetErrorString(e));
  return ok();
}

fastvr_status fastvr_tile_blend(const float* tiles, float* out, int64_t B, int64_t T, int64_t Hg, int64_t Wg,
                                int64_t C, int64_t tile, int64_t tile_overlap, void* stream) {
  return blend_impl(tiles, nullptr, out, 0.f, B, T, Hg, Wg, C, tile, tile_overlap, stream);
}

fastvr_status fastvr_tile_blend_update(const float* v_tiles, const void* z_lq, float* z_hat, float sigma, int64_t B,
                                       int64_t T, int64_t Hg, int64_t Wg, int64_t C, int64_t tile, int64_t tile_overlap,
                                       void* stream) {
  if (z_lq == nullptr && B > 0 && T > 0 && Hg > 0 && Wg > 0 && C > 0)
    return fail(FASTVR_ERR_INVALID_ARGUMENT, "z_lq is NULL");
  return blend_impl(v_tiles, z_lq, z_hat, sigma, B, T, Hg, Wg, C, tile, tile_overlap, stream);
}

const char* fastvr_status_string(fastvr_status s) {
  switch (s) {
    case FASTVR_OK: return "FASTVR_OK";
    case FASTVR_ERR_INVALID_ARGUMENT: return "FASTVR_ERR_INVALID_ARGUMENT";
    case FASTVR_ERR_UNSUPPORTED: return "FASTVR_ERR_UNSUPPORTED";
    case FASTVR_ERR_CAPACITY: return "FASTVR_ERR_CAPACITY";
    case FASTVR_ERR_HIP: return "FASTVR_ERR_HIP";
  }
  return "FASTVR_ERR_UNKNOWN";
}

const char* fastvr_last_error(void) { return g_last_error.c_str(); }

int fastvr_abi_version(void) { return FASTVR_ABI_VERSION; }

}  // extern "C"
