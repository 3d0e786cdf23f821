// Host side of the Kamera C ABI: argument validation (no HIP call happens
// before every check has passed), translation into kernel parameters, launch.
// The operator itself is defined in include/kamera.h.

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cstdint>
#include <initializer_list>
#include <vector>

#include "kamera.h"
#include "kamera_launch.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return KAMERA_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr double kTwoPi = 6.283185307179586476925286766559;

// ---------------------------------------------------------------------------
// RoPE descriptor
// ---------------------------------------------------------------------------

int check_rope(const kamera_rope& r, int32_t head_dim, const char* who) {
  if (!(r.theta > 0.0) || !isfinite(r.theta))
    return fail(KAMERA_ERR_SHAPE, "%s: rope.theta must be a finite positive number (got %g)", who, r.theta);
  if (r.rope_dim <= 0 || (r.rope_dim & 1))
    return fail(KAMERA_ERR_SHAPE, "%s: rope.rope_dim must be positive and even (got %d)", who, r.rope_dim);
  if (r.rope_dim > KAMERA_MAX_ROPE_DIM)
    return fail(KAMERA_ERR_RANGE, "%s: rope.rope_dim %d exceeds %d", who, r.rope_dim, KAMERA_MAX_ROPE_DIM);
  if (r.rope_offset < 0 || (int64_t)r.rope_offset + r.rope_dim > head_dim)
    return fail(KAMERA_ERR_SHAPE, "%s: rope band [%d, %lld) lies outside the %d-column row", who,
                r.rope_offset, (long long)r.rope_offset + r.rope_dim, head_dim);
  if (r.pairing != KAMERA_PAIR_NEOX && r.pairing != KAMERA_PAIR_INTERLEAVED)
    return fail(KAMERA_ERR_SHAPE, "%s: unknown rope.pairing %d", who, r.pairing);
  if (r.n_sections != 1 && r.n_sections != 3)
    return fail(KAMERA_ERR_SHAPE, "%s: rope.n_sections must be 1 or 3 (got %d)", who, r.n_sections);
  if (r.n_sections == 3) {
    if (r.sections[0] < 0 || r.sections[1] < 0 || r.sections[2] < 0 ||
        r.sections[0] + r.sections[1] + r.sections[2] != r.rope_dim / 2)
      return fail(KAMERA_ERR_SHAPE, "%s: sections %d/%d/%d must be >= 0 and sum to rope_dim/2 = %d", who,
                  r.sections[0], r.sections[1], r.sections[2], r.rope_dim / 2);
    if (r.section_order != KAMERA_SECTIONS_BLOCKED && r.section_order != KAMERA_SECTIONS_INTERLEAVED)
      return fail(KAMERA_ERR_SHAPE, "%s: unknown rope.section_order %d", who, r.section_order);
  }
  return KAMERA_OK;
}

// Frequencies in revolutions per position step, and the (t, h, w) coordinate
// of each pair.
void fill_rope(const kamera_rope& r, kamera::RopeParams& o) {
  memset(&o, 0, sizeof(o));
  const int half = r.rope_dim / 2;
  for (int j = 0; j < half; ++j) o.rev_freq[j] = pow(r.theta, -2.0 * j / (double)r.rope_dim) / kTwoPi;
  if (r.n_sections == 3) {
    if (r.section_order == KAMERA_SECTIONS_BLOCKED) {
      for (int j = 0; j < half; ++j)
        o.coord[j] = (int8_t)(j < r.sections[0] ? 0 : (j < r.sections[0] + r.sections[1] ? 1 : 2));
    } else {
      int left[3] = {r.sections[0], r.sections[1], r.sections[2]};
      int j = 0;
      while (j < half) {
        for (int s = 0; s < 3 && j < half; ++s)
          if (left[s] > 0) {
            o.coord[j++] = (int8_t)s;
            --left[s];
          }
      }
    }
  }
  o.rope_offset = r.rope_offset;
  o.rope_dim = r.rope_dim;
  o.pairing = r.pairing;
}

// ---------------------------------------------------------------------------
// placement (dense rows or paged slots)
// ---------------------------------------------------------------------------

int check_paging(int32_t paged, const int32_t* page_table, int32_t pt_stride, int32_t page_size,
                 int32_t n_pool_pages, int32_t n_tokens, const char* who) {
  if (paged != 0 && paged != 1) return fail(KAMERA_ERR_SHAPE, "%s: paged must be 0 or 1", who);
  if (!paged) return KAMERA_OK;
  if (page_table == nullptr) return fail(KAMERA_ERR_NULL, "%s: paged output needs a page_table", who);
  if (page_size <= 0) return fail(KAMERA_ERR_SHAPE, "%s: page_size must be positive (got %d)", who, page_size);
  if (n_pool_pages <= 0) return fail(KAMERA_ERR_SHAPE, "%s: n_pool_pages must be positive", who);
  if (pt_stride < ceil_div(n_tokens, page_size))
    return fail(KAMERA_ERR_SHAPE, "%s: pt_stride %d < %lld pages needed for %d tokens", who, pt_stride,
                (long long)ceil_div(n_tokens, page_size), n_tokens);
  return KAMERA_OK;
}

void fill_place(kamera::Placement& pl, int32_t n_tokens, const int32_t* chunk_tokens, int32_t paged,
                const int32_t* row_base, const int32_t* page_table, int32_t pt_stride, int32_t page_size,
                int32_t n_pool_pages, uint32_t* status) {
  memset(&pl, 0, sizeof(pl));
  pl.n_tokens = n_tokens;
  pl.paged = paged;
  pl.chunk_tokens = chunk_tokens;
  pl.row_base = paged ? nullptr : row_base;
  pl.page_table = paged ? page_table : nullptr;
  pl.pt_stride = pt_stride;
  pl.page_size = paged ? page_size : 1;
  pl.n_pool_pages = n_pool_pages;
  pl.status = status;
}

bool strides_ok(const int64_t* s, int n) {
  for (int k = 0; k < n; ++k)
    if (s[k] % 8 != 0) return false;
  return true;
}

// Largest work a call may describe (elements, rows or tasks): far beyond any
// device, and small enough that the host arithmetic on it cannot overflow.
constexpr int64_t kMaxWork = (int64_t)1 << 50;

// product of non-negative factors, or -1 once it exceeds kMaxWork
int64_t bounded_product(std::initializer_list<int64_t> factors) {
  __int128 p = 1;
  for (const int64_t f : factors) {
    if (f < 0) return -1;
    p *= f;
    if (p > kMaxWork) return -1;
  }
  return (int64_t)p;
}

// byte range [lo, hi) of an n-D strided view (element strides, elem_bytes
// each) whose innermost rows are row_elems contiguous elements; false when
// the range does not fit in the address space (the arithmetic is 128-bit)
bool span(const void* base, const int64_t* s, const int64_t* ext, int nd, int64_t row_elems, int elem_bytes,
          uintptr_t& lo, uintptr_t& hi) {
  __int128 a = 0, b = 0;
  for (int k = 0; k < nd; ++k) {
    if (ext[k] <= 0) continue;
    const __int128 d = (__int128)(ext[k] - 1) * s[k];
    if (d < 0) a += d; else b += d;
  }
  const __int128 p = (__int128)reinterpret_cast<uintptr_t>(base);
  const __int128 l = p + a * elem_bytes, h = p + (b + row_elems) * elem_bytes;
  if (l < 0 || h > (__int128)UINTPTR_MAX) return false;
  lo = (uintptr_t)l;
  hi = (uintptr_t)h;
  return true;
}

// the same for a 4-D bf16 view
bool extent(const void* base, const int64_t* s, const int64_t* ext, int64_t row_elems, uintptr_t& lo,
            uintptr_t& hi) {
  return span(base, s, ext, 4, row_elems, 2, lo, hi);
}

bool overlap(uintptr_t a0, uintptr_t a1, uintptr_t b0, uintptr_t b1) { return a0 < b1 && b0 < a1; }

int pick_grid(int64_t n_tasks, int32_t& per_xcd, const char* who) {
  const int64_t px = ceil_div(n_tasks, 8);
  // the dispatch packet counts work-items in 32 bits
  if (px * 8 * kamera::kThreads > 0xFFFFFFFFLL)
    return fail(KAMERA_ERR_RANGE, "%s: %lld workgroup tasks exceed one launch", who, (long long)n_tasks);
  per_xcd = (int32_t)px;
  return KAMERA_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// kamera_rehydrate
// ---------------------------------------------------------------------------

// Two row sets of one call, each at base + c*s[0] + l*s[1] + row*s[2] + h*s[3]
// + [0, head_dim) (s[0] unused for a pool), interleave without sharing an
// element: the same strides (none negative); every offset is a multiple of the
// row stride r plus a position inside one row's span (all heads of the row);
// the bases are d elements apart with span <= |d| <= r - span, so a row of one
// set lies in the gap between two rows of the other.  This admits two planes
// written into one tensor [.., row, K|V, head, dim], also in place.
static bool interleaved_rows(const kamera_rehydrate_args* a, const void* b0, const int64_t* s0, const void* b1,
                             const int64_t* s1, bool chunk_stride_used) {
  if (memcmp(s0, s1, 4 * sizeof(int64_t)) != 0) return false;
  for (int k = 0; k < 4; ++k)
    if (s0[k] < 0) return false;
  const int64_t r = s0[2];
  if (r <= 0 || s0[1] % r != 0 || (chunk_stride_used && s0[0] % r != 0)) return false;
  const __int128 row_span = (__int128)(a->n_heads - 1) * s0[3] + a->head_dim;
  const uintptr_t p0 = (uintptr_t)b0, p1 = (uintptr_t)b1;
  const uintptr_t gap = p0 > p1 ? p0 - p1 : p1 - p0;
  if (gap % 2 != 0) return false;
  const __int128 d = (__int128)(gap / 2);
  return row_span <= d && d + row_span <= r;
}

// Validation and kernel parameters of a rehydrate call; *launch is false for
// an empty call (nothing to do).
static int build_rehydrate(const kamera_rehydrate_args* a, kamera::RehydrateParams& P, bool& launch) {
  const char* who = "kamera_rehydrate";
  launch = false;
  if (a == nullptr) return fail(KAMERA_ERR_NULL, "%s: args is NULL", who);
  if (a->n_chunks < 0 || a->n_layers < 0 || a->n_heads < 0 || a->n_tokens < 0)
    return fail(KAMERA_ERR_SHAPE, "%s: negative n_chunks/n_layers/n_heads/n_tokens", who);
  if (a->head_dim <= 0 || a->head_dim % 32 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: head_dim must be a positive multiple of 32 (got %d)", who, a->head_dim);
  if (a->head_dim > KAMERA_MAX_HEAD_DIM)
    return fail(KAMERA_ERR_RANGE, "%s: head_dim %d exceeds %d", who, a->head_dim, KAMERA_MAX_HEAD_DIM);
  if (a->n_planes != 1 && a->n_planes != 2)
    return fail(KAMERA_ERR_SHAPE, "%s: n_planes must be 1 or 2 (got %d)", who, a->n_planes);
  if (a->kernel < KAMERA_KERNEL_AUTO || a->kernel > KAMERA_KERNEL_ROW_GROUP4)
    return fail(KAMERA_ERR_SHAPE, "%s: unknown kernel choice %d", who, a->kernel);
  if (a->max_workgroups < 0)
    return fail(KAMERA_ERR_SHAPE, "%s: max_workgroups must be >= 0 (got %d)", who, a->max_workgroups);
  if (a->schedule < KAMERA_SCHEDULE_AUTO || a->schedule > KAMERA_SCHEDULE_BLOCKS)
    return fail(KAMERA_ERR_SHAPE, "%s: unknown schedule %d", who, a->schedule);
  if (a->schedule == KAMERA_SCHEDULE_BLOCKS && a->max_workgroups > 0)
    return fail(KAMERA_ERR_SHAPE, "%s: max_workgroups caps the persistent schedule only", who);
  if (a->patch_frame != KAMERA_PATCH_PRE_ROPE && a->patch_frame != KAMERA_PATCH_POST_ROPE)
    return fail(KAMERA_ERR_SHAPE, "%s: unknown patch_frame %d", who, a->patch_frame);
  bool any_rot = false;
  for (int p = 0; p < a->n_planes; ++p) any_rot = any_rot || a->plane[p].rotate;
  if (any_rot) {
    int rc = check_rope(a->rope, a->head_dim, who);
    if (rc) return rc;
    const kamera_rope& r = a->rope;
    if (r.rope_offset % 32 != 0 || r.rope_dim % 32 != 0)
      return fail(KAMERA_ERR_UNSUPPORTED, "%s: the rope band must start and end on a multiple of 32 columns", who);
    if (r.pairing == KAMERA_PAIR_NEOX && r.rope_dim % 64 != 0)
      return fail(KAMERA_ERR_UNSUPPORTED, "%s: NeoX pairing needs rope_dim %% 64 == 0 (got %d)", who, r.rope_dim);
    if (a->pos_mode != KAMERA_POS_LINEAR && a->pos_mode != KAMERA_POS_GRID3 && a->pos_mode != KAMERA_POS_EXPLICIT)
      return fail(KAMERA_ERR_SHAPE, "%s: unknown pos_mode %d", who, a->pos_mode);
    if (a->pos_mode == KAMERA_POS_GRID3 && a->grid_w <= 0)
      return fail(KAMERA_ERR_SHAPE, "%s: GRID3 positions need grid_w > 0", who);
    if (a->pos_mode == KAMERA_POS_EXPLICIT && a->explicit_chunk_stride < 0)
      return fail(KAMERA_ERR_SHAPE, "%s: explicit_chunk_stride must be >= 0", who);
  }
  for (int p = 0; p < a->n_planes; ++p) {
    const kamera_plane& q = a->plane[p];
    int cb = q.col_begin, ce = q.col_end;
    if (cb == 0 && ce == 0) ce = a->head_dim;
    if (cb < 0 || ce > a->head_dim || cb >= ce)
      return fail(KAMERA_ERR_SHAPE, "%s: plane %d columns [%d, %d) outside the %d-column row", who, p, cb, ce,
                  a->head_dim);
    if (cb % 32 != 0 || ce % 32 != 0)
      return fail(KAMERA_ERR_UNSUPPORTED, "%s: plane %d column range must start/end on multiples of 32", who, p);
    if (q.rotate && (a->rope.rope_offset < cb || a->rope.rope_offset + a->rope.rope_dim > ce))
      return fail(KAMERA_ERR_SHAPE, "%s: plane %d rotates but its columns [%d, %d) do not hold the rope band",
                  who, p, cb, ce);
    if (q.m > 0 && (q.patch_offset < cb || (int64_t)q.patch_offset + q.patch_dim > ce))
      return fail(KAMERA_ERR_SHAPE, "%s: plane %d patch columns lie outside its column range", who, p);
    if (q.m < 0 || q.m > KAMERA_MAX_RANK)
      return fail(KAMERA_ERR_RANGE, "%s: plane %d rank m = %d outside [0, %d]", who, p, q.m, KAMERA_MAX_RANK);
    if (q.rotate != 0 && q.rotate != 1) return fail(KAMERA_ERR_SHAPE, "%s: plane %d rotate must be 0 or 1", who, p);
    if (q.m > 0) {
      if (q.patch_offset < 0 || q.patch_dim <= 0 || (int64_t)q.patch_offset + q.patch_dim > a->head_dim)
        return fail(KAMERA_ERR_SHAPE, "%s: plane %d patch columns [%d, %lld) outside the %d-column row", who, p,
                    q.patch_offset, (long long)q.patch_offset + q.patch_dim, a->head_dim);
      if (q.patch_offset % 8 != 0 || q.patch_dim % 8 != 0)
        return fail(KAMERA_ERR_UNSUPPORTED, "%s: plane %d patch columns must start/end on multiples of 8", who, p);
    }
  }
  int rc = check_paging(a->paged, a->page_table, a->pt_stride, a->page_size, a->n_pool_pages, a->n_tokens, who);
  if (rc) return rc;

  const int64_t work = bounded_product({a->n_chunks, a->n_layers, a->n_heads, a->n_tokens});
  if (work < 0) return fail(KAMERA_ERR_RANGE, "%s: chunks x layers x heads x tokens exceeds 2^50", who);
  if (work == 0) return KAMERA_OK;  // empty call: nothing to read or write

  if (any_rot && a->pos_mode != KAMERA_POS_EXPLICIT && a->chunk_pos == nullptr)
    return fail(KAMERA_ERR_NULL, "%s: chunk_pos is NULL", who);
  if (any_rot && a->pos_mode == KAMERA_POS_EXPLICIT && a->explicit_pos == nullptr)
    return fail(KAMERA_ERR_NULL, "%s: explicit_pos is NULL", who);
  for (int p = 0; p < a->n_planes; ++p) {
    const kamera_plane& q = a->plane[p];
    if (q.in == nullptr || q.out == nullptr) return fail(KAMERA_ERR_NULL, "%s: plane %d in/out is NULL", who, p);
    if (q.m > 0 && (q.U == nullptr || q.W == nullptr))
      return fail(KAMERA_ERR_NULL, "%s: plane %d has m = %d but U or W is NULL", who, p, q.m);
    if (!aligned16(q.in) || !aligned16(q.out) || !strides_ok(q.in_stride, 4) || !strides_ok(q.out_stride, 4))
      return fail(KAMERA_ERR_ALIGN, "%s: plane %d in/out rows must be 16-byte aligned (base %% 16, strides %% 8)",
                  who, p);
  }
  // inputs must not be overwritten while other workgroups still read them
  for (int p = 0; p < a->n_planes; ++p) {
    const kamera_plane& q = a->plane[p];
    const int64_t ein[4] = {a->n_chunks, a->n_layers, a->n_tokens, a->n_heads};
    uintptr_t ilo, ihi;
    if (!extent(q.in, q.in_stride, ein, a->head_dim, ilo, ihi))
      return fail(KAMERA_ERR_RANGE, "%s: plane %d input strides span more than the address space", who, p);
    for (int o = 0; o < a->n_planes; ++o) {
      const kamera_plane& r = a->plane[o];
      uintptr_t olo, ohi;
      const int64_t eo[4] = {1, a->n_layers, (int64_t)a->n_pool_pages * a->page_size, a->n_heads};
      if (!extent(r.out, r.out_stride, a->paged ? eo : ein, a->head_dim, olo, ohi))
        return fail(KAMERA_ERR_RANGE, "%s: plane %d output strides span more than the address space", who, o);
      // Exact in place is allowed: same base and strides, dense rows, no row
      // base -- every element is then read and written by the workgroup that
      // owns it, provided two different planes cover disjoint columns.
      const bool same_map = !a->paged && a->row_base == nullptr && r.out == q.in &&
                            memcmp(r.out_stride, q.in_stride, sizeof(q.in_stride)) == 0;
      if (same_map) {
        const int qb = q.col_begin, qe = (q.col_begin == 0 && q.col_end == 0) ? a->head_dim : q.col_end;
        const int rb = r.col_begin, re = (r.col_begin == 0 && r.col_end == 0) ? a->head_dim : r.col_end;
        if (o == p || qe <= rb || re <= qb) continue;
      }
      // the other plane's input may interleave with this output by rows (one
      // tensor [.., row, K|V, head, dim] rehydrated in place)
      if (o != p && !a->paged && interleaved_rows(a, r.out, r.out_stride, q.in, q.in_stride, true)) continue;
      if (overlap(ilo, ihi, olo, ohi))
        return fail(KAMERA_ERR_ALIAS, "%s: output of plane %d overlaps the input of plane %d", who, o, p);
    }
  }
  // two planes may write one tensor only through the same mapping on disjoint
  // columns, or with interleaved rows (interleaved_rows)
  if (a->n_planes == 2) {
    const kamera_plane& q0 = a->plane[0];
    const kamera_plane& q1 = a->plane[1];
    const int64_t e_dense[4] = {a->n_chunks, a->n_layers, a->n_tokens, a->n_heads};
    const int64_t e_pool[4] = {1, a->n_layers, (int64_t)a->n_pool_pages * a->page_size, a->n_heads};
    uintptr_t lo0 = 0, hi0 = 0, lo1 = 0, hi1 = 0;
    if (!extent(q0.out, q0.out_stride, a->paged ? e_pool : e_dense, a->head_dim, lo0, hi0) ||
        !extent(q1.out, q1.out_stride, a->paged ? e_pool : e_dense, a->head_dim, lo1, hi1))
      return fail(KAMERA_ERR_RANGE, "%s: output strides span more than the address space", who);
    if (overlap(lo0, hi0, lo1, hi1)) {
      const bool same_map = q0.out == q1.out && memcmp(q0.out_stride, q1.out_stride, sizeof(q0.out_stride)) == 0;
      const int b0 = q0.col_begin, e0 = (q0.col_begin == 0 && q0.col_end == 0) ? a->head_dim : q0.col_end;
      const int b1 = q1.col_begin, e1 = (q1.col_begin == 0 && q1.col_end == 0) ? a->head_dim : q1.col_end;
      if ((!same_map || !(e0 <= b1 || e1 <= b0)) &&
          !interleaved_rows(a, q0.out, q0.out_stride, q1.out, q1.out_stride, !a->paged))
        return fail(KAMERA_ERR_ALIAS, "%s: the two planes' outputs overlap", who);
    }
  }

  memset(&P, 0, sizeof(P));
  if (any_rot) fill_rope(a->rope, P.rope);
  fill_place(P.place, a->n_tokens, a->chunk_tokens, a->paged, a->row_base, a->page_table, a->pt_stride,
             a->page_size, a->n_pool_pages, a->status);
  P.chunk_pos = a->chunk_pos;
  P.explicit_pos = a->explicit_pos;
  P.delta = any_rot ? a->delta : nullptr;
  P.explicit_cs = a->explicit_chunk_stride;
  P.pos_mode = a->pos_mode;
  P.grid_w = a->grid_w > 0 ? a->grid_w : 1;
  P.patch_post_rope = a->patch_frame == KAMERA_PATCH_POST_ROPE;
  P.n_planes = a->n_planes;
  P.n_chunks = a->n_chunks;
  P.n_layers = a->n_layers;
  P.n_heads = a->n_heads;
  P.max_wgs = a->max_workgroups;

  int64_t units = 0;
  for (int p = 0; p < a->n_planes; ++p) {
    const kamera_plane& q = a->plane[p];
    kamera::PlaneParams& o = P.plane[p];
    o.in = static_cast<const uint16_t*>(q.in);
    o.out = static_cast<uint16_t*>(q.out);
    o.U = static_cast<const uint16_t*>(q.U);
    o.W = static_cast<const uint16_t*>(q.W);
    memcpy(o.in_s, q.in_stride, sizeof(o.in_s));
    memcpy(o.out_s, q.out_stride, sizeof(o.out_s));
    memcpy(o.u_s, q.u_stride, sizeof(o.u_s));
    memcpy(o.w_s, q.w_stride, sizeof(o.w_s));
    o.m = q.m;
    o.m_steps = (q.m + 31) / 32;
    o.layer_rank = q.layer_rank;
    o.patch_lo = q.m > 0 ? q.patch_offset : 0;
    o.patch_hi = q.m > 0 ? q.patch_offset + q.patch_dim : 0;
    o.u_vec = q.m % 8 == 0 && aligned16(q.U) && strides_ok(q.u_stride, 4);
    o.w_vec = aligned16(q.W) && strides_ok(q.w_stride, 4);
    // column blocks: the rotated band as one block, the rest in <= 128-column pieces
    std::pair<int, int> segs[3];  // [col0, col1): before the band, the band, after it
    int nseg = 0;
    const int cb = q.col_begin, ce = (q.col_begin == 0 && q.col_end == 0) ? a->head_dim : q.col_end;
    if (q.rotate) {
      const int r0 = a->rope.rope_offset, r1 = r0 + a->rope.rope_dim;
      if (r0 > cb) segs[nseg++] = {cb, r0};
      segs[nseg++] = {r0, r1};
      if (r1 < ce) segs[nseg++] = {r1, ce};
    } else {
      segs[nseg++] = {cb, ce};
    }
    int nb = 0;
    for (int si = 0; si < nseg; ++si) {
      const std::pair<int, int>& sg = segs[si];
      const bool band = q.rotate && sg.first == a->rope.rope_offset;
      for (int c0 = sg.first; c0 < sg.second; c0 += 128) {
        const int w = band ? sg.second - sg.first : std::min(128, sg.second - c0);
        if (nb >= kamera::kMaxBlocks) return fail(KAMERA_ERR_RANGE, "%s: too many column blocks", who);
        kamera::ColBlock& b = o.blk[nb++];
        b.col0 = (int16_t)(c0 / 8);
        b.nq = (int8_t)(w / 32);
        int flags = 0;
        if (band) flags |= kamera::kBlkRotate;
        if (q.m > 0 && c0 < o.patch_hi && c0 + w > o.patch_lo) flags |= kamera::kBlkPatch;
        b.flags = (int8_t)flags;
        if (band) break;
      }
    }
    o.n_blocks = nb;
    units += (int64_t)a->n_chunks * a->n_layers * a->n_heads * nb;
  }
  // Rows of <= 8 heads of 128 columns, one block per head and rank <= 64 can
  // take the row-group kernel: a workgroup takes hw = 4 or 8 heads of a token
  // row, so it writes them as one contiguous run (a whole pool page at 8
  // heads).  AUTO follows where it measured faster than the per-head kernel,
  // over three placements of the buffers in HBM each: rows of 4 or 8 heads
  // and chunks of >= 256 tokens take groups of 4 heads (two workgroups per CU)
  // from 2^19 rows in all (planes x chunks x layers x tokens x heads) on --
  // the row-group kernel's equal shares of tiles and its two tiles in flight
  // beat the per-head kernel's small tasks there -- except dense outputs at
  // rank <= 32 with 2^21 .. 2^23 rows, where the per-head kernel's token
  // blocks are long enough and its four workgroups per CU keep more bytes in
  // flight.  8-head groups never led 4-head ones by more than the spread of
  // placements and trail them when relocating (they run out of registers).
  // Tiny calls, shorter chunks and other head counts keep the per-head kernel.
  const double n_rows = (double)a->n_planes * a->n_chunks * a->n_layers * a->n_tokens * a->n_heads;
  int hw = 0;
  if (a->kernel == KAMERA_KERNEL_ROW_GROUP) {
    hw = a->n_heads <= 4 ? 4 : 8;
  } else if (a->kernel == KAMERA_KERNEL_ROW_GROUP4) {
    hw = 4;
  } else if (a->kernel == KAMERA_KERNEL_AUTO) {
    int max_rank = 0;
    for (int p = 0; p < a->n_planes; ++p) max_rank = std::max(max_rank, (int)a->plane[p].m);
    const bool dense_window = !a->paged && max_rank <= 32 && n_rows >= 2097152.0 && n_rows < 8388608.0;
    hw = (a->n_heads == 4 || a->n_heads == 8) && a->n_tokens >= 256 && n_rows >= 524288.0 && !dense_window ? 4 : 0;
  }
  bool rows = hw > 0 && a->n_heads <= kamera::kRgMaxHeads && a->head_dim == 128 &&
              (!any_rot || a->pos_mode != KAMERA_POS_EXPLICIT);
  for (int p = 0; p < a->n_planes && rows; ++p) {
    kamera::PlaneParams& o = P.plane[p];
    const kamera::ColBlock& b = o.blk[0];
    rows = o.n_blocks == 1 && b.col0 == 0 && b.nq == 4 && o.m_steps <= 2 &&
           (o.m == 0 || (o.patch_lo == 0 && o.patch_hi == 128 && o.u_vec));
    for (int d = 0; d < 4 && rows; ++d) rows = o.in_s[d] >= 0 && o.out_s[d] >= 0 && (o.m == 0 || o.u_s[d] >= 0);
    if (!rows) break;
    // the buffer instructions of that kernel take 32-bit byte offsets within
    // one (chunk, layer) slab (dense output: from the chunk's row base on), or
    // within one layer of the pool
    const __int128 n1 = a->n_tokens - 1, h1 = a->n_heads - 1;
    const __int128 in_rec = (n1 * o.in_s[2] + h1 * o.in_s[3] + 128) * 2;
    const __int128 u_rec = o.m > 0 ? (h1 * o.u_s[2] + n1 * o.u_s[3] + o.m) * 2 : 0;
    const __int128 rows_out = a->paged ? (__int128)a->n_pool_pages * a->page_size - 1 : n1;
    const __int128 out_rec = (rows_out * o.out_s[2] + h1 * o.out_s[3] + 128) * 2;
    const __int128 lim = 0x7ffffff0;
    rows = in_rec <= lim && u_rec <= lim && out_rec <= lim;
    o.in_rec = (int32_t)in_rec;
    o.u_rec = (int32_t)u_rec;
    o.out_rec = (int32_t)out_rec;
  }
  if (rows) {
    // a workgroup takes 4 heads (two workgroups per CU) or 8 (one per CU).
    // Token blocks: up to 1024 tokens, shrunk (to >= 64) until the launch has
    // 4096 of them (2048 with 8-head groups).  Where they stay >= 512 tokens
    // one workgroup per block, handed out by the hardware, ran faster than
    // the persistent schedule on the same buffers (the 80-layer recall by
    // 3-9%, its deep half by 14%, the 32-layer recalls and the relocation by
    // 1-5%); with shorter blocks the persistent schedule pays a unit's set-up
    // once per long range instead of once per block (the 28-layer reorder:
    // 7-13% faster than per-head, 25-32% faster than 64-token blocks).
    P.row_group = hw;
    P.n_hgroups = (int32_t)ceil_div(a->n_heads, hw);
    P.unit_tiles = (int32_t)ceil_div(a->n_tokens, kamera::kTileTokens);
    P.blocks_per_group = a->n_planes;
    const int64_t lanes_units = (int64_t)a->n_planes * P.n_hgroups * a->n_chunks * a->n_layers;
    const int64_t target = hw == 4 ? 4096 : 2048;
    int bt = 1024 / kamera::kTileTokens;
    while (bt > 4 && lanes_units * ceil_div(P.unit_tiles, bt) < target) bt /= 2;
    const bool blocks = a->schedule == KAMERA_SCHEDULE_BLOCKS ||
                        (a->schedule == KAMERA_SCHEDULE_AUTO && a->max_workgroups == 0 && bt >= 512 / kamera::kTileTokens);
    P.block_tiles = blocks ? bt : 0;
    P.n_tasks = lanes_units * P.unit_tiles;
    // the dispatch packet counts work-items in 32 bits (64 * hw per block)
    if (lanes_units * ceil_div(P.unit_tiles, bt) * 64 * hw > 0xFFFFFFFFLL)
      return fail(KAMERA_ERR_RANGE, "%s: %lld token blocks exceed one launch", who,
                  (long long)(lanes_units * ceil_div(P.unit_tiles, bt)));
    launch = true;
    return KAMERA_OK;
  }
  // token block: as large as possible while keeping >= 32 workgroups per CU
  // (the MLA workloads ran 3-5% faster than at 16 per CU, the 28-layer one
  // as fast; all slower at 64 or 8)
  int tb = 1024;
  while (tb > 64 && units * ceil_div(a->n_tokens, tb) < 8192) tb /= 2;
  tb = (int)std::min<int64_t>(tb, ceil_div(a->n_tokens, 64) * 64);
  P.token_block = tb;
  P.n_tblk = (int32_t)ceil_div(a->n_tokens, tb);
  int32_t nb_all = 0;
  for (int p = 0; p < a->n_planes; ++p) {
    P.plane[p].block_base = nb_all;
    nb_all += P.plane[p].n_blocks;
  }
  P.blocks_per_group = nb_all;
  const int64_t n_tasks = (int64_t)a->n_chunks * a->n_layers * a->n_heads * P.n_tblk * nb_all;
  if (n_tasks >= (int64_t)1 << 31)
    return fail(KAMERA_ERR_RANGE, "%s: %lld tasks exceed one launch", who, (long long)n_tasks);
  P.n_tasks = n_tasks;
  P.fd_bpg = kamera::make_fast_div((uint32_t)std::max(1, nb_all));
  P.fd_tblk = kamera::make_fast_div((uint32_t)std::max(1, P.n_tblk));
  P.fd_heads = kamera::make_fast_div((uint32_t)std::max(1, a->n_heads));
  P.fd_layers = kamera::make_fast_div((uint32_t)std::max(1, a->n_layers));
  rc = pick_grid(P.n_tasks, P.per_xcd, who);
  if (rc) return rc;
  launch = true;
  return KAMERA_OK;
}

extern "C" int kamera_rehydrate(const kamera_rehydrate_args* a, void* stream) {
  static thread_local kamera::RehydrateParams P;
  bool launch = false;
  const int rc = build_rehydrate(a, P, launch);
  if (rc) return rc;
  if (launch) {
    const hipError_t e = kamera::launch_rehydrate(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(KAMERA_ERR_HIP, "kamera_rehydrate: launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

// ---------------------------------------------------------------------------
// kamera_shift
// ---------------------------------------------------------------------------

static int build_shift(const kamera_shift_args* a, kamera::ShiftParams& P, bool& launch) {
  const char* who = "kamera_shift";
  launch = false;
  if (a == nullptr) return fail(KAMERA_ERR_NULL, "%s: args is NULL", who);
  if (a->n_chunks < 0 || a->n_layers < 0 || a->n_heads < 0 || a->n_tokens < 0)
    return fail(KAMERA_ERR_SHAPE, "%s: negative n_chunks/n_layers/n_heads/n_tokens", who);
  if (a->head_dim <= 0 || a->head_dim % 8 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: head_dim must be a positive multiple of 8 (got %d)", who, a->head_dim);
  if (a->head_dim > KAMERA_MAX_HEAD_DIM)
    return fail(KAMERA_ERR_RANGE, "%s: head_dim %d exceeds %d", who, a->head_dim, KAMERA_MAX_HEAD_DIM);
  int rc = check_rope(a->rope, a->head_dim, who);
  if (rc) return rc;
  const kamera_rope& r = a->rope;
  if (r.rope_offset % 8 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: rope_offset must be a multiple of 8", who);
  if (r.pairing == KAMERA_PAIR_NEOX && r.rope_dim % 16 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: NeoX pairing needs rope_dim %% 16 == 0", who);
  if (r.pairing == KAMERA_PAIR_INTERLEAVED && r.rope_dim % 8 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: interleaved pairing needs rope_dim %% 8 == 0", who);
  rc = check_paging(a->paged, a->page_table, a->pt_stride, a->page_size, a->n_pool_pages, a->n_tokens, who);
  if (rc) return rc;
  const int64_t work = bounded_product({a->n_chunks, a->n_layers, a->n_heads, a->n_tokens});
  if (work < 0) return fail(KAMERA_ERR_RANGE, "%s: chunks x layers x heads x tokens exceeds 2^50", who);
  if (work == 0) return KAMERA_OK;
  if (a->k == nullptr) return fail(KAMERA_ERR_NULL, "%s: k is NULL", who);
  if (a->delta == nullptr) return fail(KAMERA_ERR_NULL, "%s: delta is NULL", who);
  if (!aligned16(a->k) || !strides_ok(a->k_stride, 4))
    return fail(KAMERA_ERR_ALIGN, "%s: k rows must be 16-byte aligned (base %% 16, strides %% 8)", who);

  memset(&P, 0, sizeof(P));
  fill_rope(r, P.rope);
  fill_place(P.place, a->n_tokens, a->chunk_tokens, a->paged, a->row_base, a->page_table, a->pt_stride,
             a->page_size, a->n_pool_pages, a->status);
  P.delta = a->delta;
  P.k = static_cast<uint16_t*>(a->k);
  memcpy(P.k_s, a->k_stride, sizeof(P.k_s));
  P.n_chunks = a->n_chunks;
  P.n_layers = a->n_layers;
  P.n_heads = a->n_heads;
  P.vec_per_row = r.pairing == KAMERA_PAIR_NEOX ? r.rope_dim / 16 : r.rope_dim / 8;
  // about 512 rows per task, at least 2048 tasks when the call is large enough
  int tb = 16;
  while (tb < 1024 && (int64_t)tb * a->n_heads < 512) tb *= 2;
  while (tb > 16 && (int64_t)a->n_chunks * a->n_layers * ceil_div(a->n_tokens, tb) < 2048) tb /= 2;
  P.token_block = tb;
  P.n_tblk = (int32_t)ceil_div(a->n_tokens, tb);
  P.n_tasks = (int64_t)a->n_chunks * a->n_layers * P.n_tblk;
  P.fd_tblk = kamera::make_fast_div((uint32_t)std::max(1, P.n_tblk));
  P.fd_layers = kamera::make_fast_div((uint32_t)std::max(1, a->n_layers));
  rc = pick_grid(P.n_tasks, P.per_xcd, who);
  if (rc) return rc;
  launch = true;
  return KAMERA_OK;
}

extern "C" int kamera_shift(const kamera_shift_args* a, void* stream) {
  static thread_local kamera::ShiftParams P;
  bool launch = false;
  const int rc = build_shift(a, P, launch);
  if (rc) return rc;
  if (launch) {
    const hipError_t e = kamera::launch_shift(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(KAMERA_ERR_HIP, "kamera_shift: launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

// ---------------------------------------------------------------------------
// kamera_scatter_paged
// ---------------------------------------------------------------------------

static int build_scatter(const kamera_scatter_args* a, kamera::ScatterParams& P, bool& launch, bool gather) {
  const char* who = gather ? "kamera_gather_paged" : "kamera_scatter_paged";
  launch = false;
  if (a == nullptr) return fail(KAMERA_ERR_NULL, "%s: args is NULL", who);
  if (a->n_chunks < 0 || a->n_layers < 0 || a->n_tokens < 0)
    return fail(KAMERA_ERR_SHAPE, "%s: negative n_chunks/n_layers/n_tokens", who);
  if (a->row_bytes <= 0 || a->row_bytes % 16 != 0)
    return fail(KAMERA_ERR_ALIGN, "%s: row_bytes must be a positive multiple of 16", who);
  int rc = check_paging(1, a->page_table, a->pt_stride, a->page_size, a->n_pool_pages, a->n_tokens, who);
  if (rc) return rc;
  const int64_t work = bounded_product({a->n_chunks, a->n_layers, a->n_tokens, a->row_bytes / 16});
  if (work < 0) return fail(KAMERA_ERR_RANGE, "%s: chunks x layers x tokens x row vectors exceeds 2^50", who);
  if (work == 0) return KAMERA_OK;
  if (a->rows == nullptr || a->pool == nullptr) return fail(KAMERA_ERR_NULL, "%s: rows or pool is NULL", who);
  for (int k = 0; k < 3; ++k)
    if (a->rows_stride_bytes[k] % 16 != 0) return fail(KAMERA_ERR_ALIGN, "%s: row strides must be multiples of 16", who);
  for (int k = 0; k < 2; ++k)
    if (a->pool_stride_bytes[k] % 16 != 0) return fail(KAMERA_ERR_ALIGN, "%s: pool strides must be multiples of 16", who);
  if (!aligned16(a->rows) || !aligned16(a->pool)) return fail(KAMERA_ERR_ALIGN, "%s: rows/pool must be 16-byte aligned", who);
  {
    // the dense rows and the pool must be different memory (byte strides)
    const int64_t ext[3] = {a->n_chunks, a->n_layers, a->n_tokens};
    const int64_t pext[2] = {a->n_layers, (int64_t)a->n_pool_pages * a->page_size};
    uintptr_t slo, shi, plo, phi;
    if (!span(a->rows, a->rows_stride_bytes, ext, 3, a->row_bytes, 1, slo, shi) ||
        !span(a->pool, a->pool_stride_bytes, pext, 2, a->row_bytes, 1, plo, phi))
      return fail(KAMERA_ERR_RANGE, "%s: strides span more than the address space", who);
    if (overlap(slo, shi, plo, phi)) return fail(KAMERA_ERR_ALIAS, "%s: the dense rows overlap the pool", who);
  }

  memset(&P, 0, sizeof(P));
  fill_place(P.place, a->n_tokens, a->chunk_tokens, 1, nullptr, a->page_table, a->pt_stride, a->page_size,
             a->n_pool_pages, a->status);
  P.rows = static_cast<uint8_t*>(a->rows);
  P.pool = static_cast<uint8_t*>(a->pool);
  P.gather = gather ? 1 : 0;
  memcpy(P.rows_s, a->rows_stride_bytes, sizeof(P.rows_s));
  memcpy(P.pool_s, a->pool_stride_bytes, sizeof(P.pool_s));
  P.row_vecs = a->row_bytes / 16;
  P.n_chunks = a->n_chunks;
  P.n_layers = a->n_layers;
  // about 16K 16-byte vectors (256 KiB) per task
  int tb = 16;
  while (tb < 1024 && (int64_t)tb * P.row_vecs < 16384) tb *= 2;
  while (tb > 16 && (int64_t)a->n_chunks * a->n_layers * ceil_div(a->n_tokens, tb) < 2048) tb /= 2;
  P.token_block = tb;
  P.n_tblk = (int32_t)ceil_div(a->n_tokens, tb);
  P.n_tasks = (int64_t)a->n_chunks * a->n_layers * P.n_tblk;
  P.fd_tblk = kamera::make_fast_div((uint32_t)std::max(1, P.n_tblk));
  P.fd_layers = kamera::make_fast_div((uint32_t)std::max(1, a->n_layers));
  rc = pick_grid(P.n_tasks, P.per_xcd, who);
  if (rc) return rc;
  launch = true;
  return KAMERA_OK;
}

static int scatter_or_gather(const kamera_scatter_args* a, void* stream, bool gather) {
  static thread_local kamera::ScatterParams P;
  bool launch = false;
  const int rc = build_scatter(a, P, launch, gather);
  if (rc) return rc;
  if (launch) {
    const hipError_t e = kamera::launch_scatter(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
      return fail(KAMERA_ERR_HIP, "%s: launch failed: %s", gather ? "kamera_gather_paged" : "kamera_scatter_paged",
                  hipGetErrorString(e));
  }
  return ok();
}

extern "C" int kamera_scatter_paged(const kamera_scatter_args* a, void* stream) {
  return scatter_or_gather(a, stream, false);
}

extern "C" int kamera_gather_paged(const kamera_scatter_args* a, void* stream) {
  return scatter_or_gather(a, stream, true);
}

// ---------------------------------------------------------------------------
// kamera_form_patch
// ---------------------------------------------------------------------------

static int build_form(const kamera_form_args* a, kamera::FormParams& P, bool& launch) {
  const char* who = "kamera_form_patch";
  launch = false;
  if (a == nullptr) return fail(KAMERA_ERR_NULL, "%s: args is NULL", who);
  if (a->n_chunks < 0 || a->n_layers < 0 || a->n_heads < 0 || a->n_tokens < 0)
    return fail(KAMERA_ERR_SHAPE, "%s: negative sizes", who);
  if (a->dim <= 0 || a->dim % 4 != 0)
    return fail(KAMERA_ERR_UNSUPPORTED, "%s: dim must be a positive multiple of 4 (got %d)", who, a->dim);
  if (a->dim > KAMERA_FORM_MAX_DIM)
    return fail(KAMERA_ERR_RANGE, "%s: dim %d exceeds %d", who, a->dim, KAMERA_FORM_MAX_DIM);
  if (a->m < 1 || a->m > a->dim) return fail(KAMERA_ERR_RANGE, "%s: m = %d outside [1, dim]", who, a->m);
  if (a->sweeps < 0) return fail(KAMERA_ERR_SHAPE, "%s: sweeps must be >= 0", who);
  if (a->n_orbit < 0) return fail(KAMERA_ERR_SHAPE, "%s: n_orbit must be >= 0", who);
  const int64_t units = bounded_product({a->n_chunks, a->n_layers, a->n_heads});
  if (units < 0 || units > 0x7fffffff) return fail(KAMERA_ERR_RANGE, "%s: too many units", who);
  if (units == 0 || a->n_tokens == 0) return KAMERA_OK;
  // the dispatch packets count work-items in 32 bits: 1024 per unit for the
  // eigensolver kernel, 256 per 256 token rows of a unit for the U kernel
  // (its grid rounded up to a multiple of 8)
  if (units * 1024 > 0xFFFFFFFFLL || (ceil_div(ceil_div(a->n_tokens, 256) * units, 8) * 8) * 256 > 0xFFFFFFFFLL)
    return fail(KAMERA_ERR_RANGE, "%s: %lld units of %d tokens exceed one launch", who, (long long)units,
                a->n_tokens);
  if (a->delta == nullptr || a->U == nullptr || a->W == nullptr)
    return fail(KAMERA_ERR_NULL, "%s: delta, U and W are required", who);
  if (!aligned16(a->delta))
    return fail(KAMERA_ERR_ALIGN, "%s: delta must be 16-byte aligned", who);
  for (int k = 0; k < 4; ++k)
    if (a->delta_stride[k] % 4 != 0)
      return fail(KAMERA_ERR_ALIGN, "%s: delta strides must be multiples of 4 floats", who);
  const int32_t n_orbit = a->n_orbit > 1 ? a->n_orbit : 1;
  if (n_orbit > 1 && a->orbit_stride % 4 != 0)
    return fail(KAMERA_ERR_ALIGN, "%s: orbit_stride must be a multiple of 4 floats", who);
  {
    // outputs must not overlap any deficit that is read
    const int64_t ext_d[5] = {a->n_chunks, a->n_layers, a->n_heads, a->n_tokens, n_orbit};
    const int64_t s_d[5] = {a->delta_stride[0], a->delta_stride[1], a->delta_stride[2], a->delta_stride[3],
                            n_orbit > 1 ? a->orbit_stride : 0};
    uintptr_t d0, d1;
    const int64_t ext_u[4] = {a->n_chunks, a->n_layers, a->n_heads, a->n_tokens};
    const int64_t ext_w[4] = {a->n_chunks, a->n_layers, a->n_heads, a->m};
    uintptr_t u0, u1, w0, w1;
    if (!span(a->delta, s_d, ext_d, 5, a->dim, 4, d0, d1) || !span(a->U, a->u_stride, ext_u, 4, a->m, 2, u0, u1) ||
        !span(a->W, a->w_stride, ext_w, 4, a->dim, 2, w0, w1))
      return fail(KAMERA_ERR_RANGE, "%s: strides span more than the address space", who);
    if (overlap(u0, u1, d0, d1) || overlap(w0, w1, d0, d1))
      return fail(KAMERA_ERR_ALIAS, "%s: U and W must not overlap the deficits", who);
    if (overlap(u0, u1, w0, w1)) return fail(KAMERA_ERR_ALIAS, "%s: U must not overlap W (U is formed from W)", who);
    if (a->sigma != nullptr) {
      const int64_t ext_s[3] = {a->n_chunks, a->n_layers, a->n_heads};
      uintptr_t s0, s1;
      if (!span(a->sigma, a->sigma_stride, ext_s, 3, a->m, 4, s0, s1))
        return fail(KAMERA_ERR_RANGE, "%s: sigma strides span more than the address space", who);
      if (overlap(s0, s1, d0, d1)) return fail(KAMERA_ERR_ALIAS, "%s: sigma must not overlap the deficits", who);
    }
    if (a->sweeps_done != nullptr) {
      const uintptr_t c0 = reinterpret_cast<uintptr_t>(a->sweeps_done);
      if (overlap(c0, c0 + 4 * (uintptr_t)units, d0, d1))
        return fail(KAMERA_ERR_ALIAS, "%s: sweeps_done must not overlap the deficits", who);
    }
  }
  memset(&P, 0, sizeof(P));
  P.delta = a->delta;
  P.U = static_cast<uint16_t*>(a->U);
  P.W = static_cast<uint16_t*>(a->W);
  P.sigma = a->sigma;
  P.sweeps_done = a->sweeps_done;
  memcpy(P.delta_s, a->delta_stride, sizeof(P.delta_s));
  memcpy(P.u_s, a->u_stride, sizeof(P.u_s));
  memcpy(P.w_s, a->w_stride, sizeof(P.w_s));
  memcpy(P.sigma_s, a->sigma_stride, sizeof(P.sigma_s));
  P.n_chunks = a->n_chunks;
  P.n_layers = a->n_layers;
  P.n_heads = a->n_heads;
  P.n_tokens = a->n_tokens;
  P.dim = a->dim;
  P.m = a->m;
  P.sweeps = a->sweeps;                        // 0: tridiagonal solver
  P.n_units = (int32_t)units;
  P.n_orbit = n_orbit;
  P.orbit_s = n_orbit > 1 ? a->orbit_stride : 0;
  P.inv_orbit = 1.0f / (float)n_orbit;
  {
    bool wv = reinterpret_cast<uintptr_t>(a->W) % 16 == 0, up = reinterpret_cast<uintptr_t>(a->U) % 4 == 0;
    for (int k = 0; k < 4; ++k) {
      wv = wv && a->w_stride[k] % 8 == 0;
      up = up && a->u_stride[k] % 2 == 0;
    }
    P.w_vec = wv ? 1 : 0;
    P.u_pair = up ? 1 : 0;
  }
  launch = true;
  return KAMERA_OK;
}

extern "C" int kamera_form_patch(const kamera_form_args* a, void* stream) {
  static thread_local kamera::FormParams P;
  bool launch = false;
  const int rc = build_form(a, P, launch);
  if (rc) return rc;
  if (launch) {
    const hipError_t e = kamera::launch_form_patch(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(KAMERA_ERR_HIP, "kamera_form_patch: launch failed: %s", hipGetErrorString(e));
  }
  return ok();
}

extern "C" int kamera_validate(int32_t which, const void* args) {
  bool launch = false;
  int rc;
  switch (which) {
    case 0: { static thread_local kamera::RehydrateParams P; rc = build_rehydrate(static_cast<const kamera_rehydrate_args*>(args), P, launch); break; }
    case 1: { static thread_local kamera::ShiftParams P; rc = build_shift(static_cast<const kamera_shift_args*>(args), P, launch); break; }
    case 2:
    case 3: {
      static thread_local kamera::ScatterParams P;
      rc = build_scatter(static_cast<const kamera_scatter_args*>(args), P, launch, which == 3);
      break;
    }
    case 4: {
      static thread_local kamera::FormParams P;
      rc = build_form(static_cast<const kamera_form_args*>(args), P, launch);
      break;
    }
    default: return fail(KAMERA_ERR_SHAPE, "kamera_validate: unknown entry point %d", which);
  }
  return rc ? rc : ok();
}

extern "C" int kamera_rehydrate_plan(const kamera_rehydrate_args* a) {
  static thread_local kamera::RehydrateParams P;
  bool launch = false;
  const int rc = build_rehydrate(a, P, launch);
  if (rc) return rc;
  ok();
  if (!launch) return KAMERA_PLAN_NONE;
  if (P.row_group == 0) return KAMERA_PLAN_PER_HEAD;
  return P.row_group == 4 ? KAMERA_PLAN_ROW_GROUP4 : KAMERA_PLAN_ROW_GROUP;
}

extern "C" int kamera_rehydrate_schedule(const kamera_rehydrate_args* a) {
  static thread_local kamera::RehydrateParams P;
  bool launch = false;
  const int rc = build_rehydrate(a, P, launch);
  if (rc) return rc;
  ok();
  if (!launch || P.row_group == 0) return 0;
  return P.block_tiles > 0 ? KAMERA_SCHEDULE_BLOCKS : KAMERA_SCHEDULE_PERSISTENT;
}

// ---------------------------------------------------------------------------
// small exports
// ---------------------------------------------------------------------------

extern "C" int kamera_check_page_table(const int32_t* pt, int32_t n_chunks, int32_t pt_stride, int32_t n_tokens,
                                       int32_t page_size, int32_t n_pool_pages) {
  const char* who = "kamera_check_page_table";
  if (n_chunks < 0 || n_tokens < 0) return fail(KAMERA_ERR_SHAPE, "%s: negative sizes", who);
  if (n_chunks == 0 || n_tokens == 0) return ok();
  if (pt == nullptr) return fail(KAMERA_ERR_NULL, "%s: page table is NULL", who);
  if (page_size <= 0 || n_pool_pages <= 0) return fail(KAMERA_ERR_SHAPE, "%s: page_size and n_pool_pages must be > 0", who);
  const int64_t used = ceil_div(n_tokens, page_size);
  if (pt_stride < used) return fail(KAMERA_ERR_SHAPE, "%s: pt_stride %d < %lld pages per chunk", who, pt_stride, (long long)used);
  std::vector<uint8_t> seen((size_t)n_pool_pages, 0);
  for (int64_t c = 0; c < n_chunks; ++c)
    for (int64_t k = 0; k < used; ++k) {
      const int32_t pg = pt[c * pt_stride + k];
      if (pg < 0 || pg >= n_pool_pages)
        return fail(KAMERA_ERR_RANGE, "%s: chunk %lld page %lld = %d outside [0, %d)", who, (long long)c,
                    (long long)k, pg, n_pool_pages);
      if (seen[(size_t)pg]) return fail(KAMERA_ERR_ALIAS, "%s: pool page %d is used twice", who, pg);
      seen[(size_t)pg] = 1;
    }
  return ok();
}

extern "C" const char* kamera_last_error(void) { return g_err; }

extern "C" int kamera_abi_version(void) { return KAMERA_ABI_VERSION; }

extern "C" int64_t kamera_struct_size(int32_t which) {
  switch (which) {
    case 0: return (int64_t)sizeof(kamera_rehydrate_args);
    case 1: return (int64_t)sizeof(kamera_shift_args);
    case 2: return (int64_t)sizeof(kamera_scatter_args);
    case 3: return (int64_t)sizeof(kamera_plane);
    case 4: return (int64_t)sizeof(kamera_rope);
    case 5: return (int64_t)sizeof(kamera_form_args);
    default: return -1;
  }
}
