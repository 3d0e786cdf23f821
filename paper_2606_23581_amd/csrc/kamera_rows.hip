// gfx950 row-group rehydrate kernel of the Kamera operator:
// K' = R(pos)(K + U W), V' = V + U_v W_v  (Eq. eq:operator, Sec. 3; serve
// step of App. A) for rows of <= 8 heads: workgroups each owning one (plane,
// group of heads) and a contiguous range of its (chunk, layer, 16-token tile)
// space (long ranges on persistent workgroups, or one token block each),
// writing their heads of a token row together.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kamera_device.h"

namespace kamera {

// ---------------------------------------------------------------------------
// Rows of <= 8 heads of 128 columns with one 128-column block per head (the
// rope band, if any, is the whole head), rank <= 64, positions linear or on a
// grid, with or without the relocation of already-rotated keys.  A workgroup
// of HW = 4 or 8 waves walks segments of one (plane, chunk, layer) unit's
// tiles for its group of HW heads; wave h computes head h of the group
// in the register layout of the per-head kernel (kamera_kernels.hip: lane
// (g, t) holds chunks g, g+4, g+8, g+12 of token t).  Per 16-token tile the
// group's heads move
//   HBM -> registers (two tiles in flight) -> LDS -> MFMA layout -> LDS -> HBM
// and the store phase writes every token's row of the group's heads: with 8
// heads a pool page of 16 tokens is one contiguous 32 KiB run instead of one
// 256-byte piece per head.  W^T of every head sits in registers for the whole
// segment, and the segment's page numbers in LDS.  Tile loads and stores are
// buffer instructions whose out-of-range lanes (ragged tails, missing heads,
// pages outside the pool) read zeros or write nothing, so the tile loop issues
// the same memory instructions on every path.
// ---------------------------------------------------------------------------

// HW (4 or 8) heads per workgroup, one wave each: 64 * HW threads.
constexpr int kRgDepth = 2;                                // tiles in flight per thread
constexpr int kRgKRow = 256 + kRowPad;                     // LDS bytes per (head, token) K row
__host__ __device__ constexpr int rg_u_row(int ms) { return 64 * ms + kRowPad; }
__host__ __device__ constexpr int rg_buf_bytes(int ms, int hw) {
  return hw * kTileTokens * (kRgKRow + rg_u_row(ms));
}
// W^T staging row of one column: 32 * ms ranks + pad (a round stages 4 heads)
__host__ __device__ constexpr int rg_wt_row(int ms) { return 64 * ms + kRowPad; }
__host__ __device__ constexpr int rg_wt_bytes(int ms) { return ms > 0 ? 4 * 128 * rg_wt_row(ms) : 0; }
constexpr int kRgMaxBlock = 1024;                          // tokens per row-group segment
__host__ __device__ constexpr int rg_lds_bytes(int ms, int hw) {
  return (2 * rg_buf_bytes(ms, hw) > rg_wt_bytes(ms) ? 2 * rg_buf_bytes(ms, hw) : rg_wt_bytes(ms)) +
         kRgMaxBlock * 4;
}
// waves per SIMD the launch bounds ask for: three 4-head workgroups per CU
// without a patch (40 KiB of LDS each), else two (one with 8 heads); at rank
// 32 three would spill registers
__host__ __device__ constexpr int rg_min_waves(int ms, int hw) { return hw == 4 && ms == 0 ? 3 : 8 / hw; }

// per thread and tile: HW * 16 tokens * 16 K chunks over 64 * HW threads,
// and HW * 16 tokens * (up to 8) U chunks
constexpr int kRgKVec = 4;
// U vectors per thread and tile at MS rank steps (HW * 16 tokens * 4 MS
// chunks over 64 * HW threads)
__host__ __device__ constexpr int rg_u_vec(int ms) { return ms > 0 ? ms : 1; }

template <int MS>
struct RgRegs {              // one tile's global loads, in flight until the LDS write
  u32x4 k[kRgKVec];
  u32x4 u[rg_u_vec(MS)];
};

constexpr uint32_t kRgOob = 0x7ffffff0u;                    // byte offset past every buffer extent
constexpr int kRgBufWord3 = 0x00020000;                    // raw buffer, 32-bit data format

struct RgTask {
  const PlaneParams* Q;
  int c, l, n_c;
  int H;                     // heads of this workgroup (<= HW)
  int h0;                    // their first head in the row
  int m, m_steps;            // rank at this layer
  int t_end;                 // end of the task's token block
  bool in_head_major;        // rows of one head lie closer together than the heads
  bool out_head_major;
  int s_in2, s_in3;          // input token / head strides (elements)
  int s_u3, s_u2;            // U token / head strides
  int s_o2, s_o3;            // output row (slot) / head strides
  double cp0, cp1, cp2;      // chunk position (t, h, w) of token 0
  double dt, dh, dw;         // relocation: the chunk's move of already-rotated keys
  __amdgpu_buffer_rsrc_t rin, ru, rout;   // (chunk, layer) slabs of input, U and output
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rg_rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kRgBufWord3);
}

// 16-byte vector v of a tile (16 tokens x H heads x 16 chunks) -> (head, token),
// heads counted from the workgroup's first
__device__ __forceinline__ void rg_vec(int v, int H, bool head_major, int& h, int& t) {
  if (head_major) {
    h = v >> 8;
    t = (v >> 4) & 15;
  } else {
    t = v / (16 * H);
    h = (v >> 4) % H;
  }
}

template <int MS, int HW>
__device__ __forceinline__ void rg_load(const RgTask& T, int tid, int i0, RgRegs<MS>& R) {
  constexpr int NT = 64 * HW;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + NT * k;
    int h, t;
    rg_vec(v, T.H, T.in_head_major, h, t);
    const int i = i0 + t;
    const uint32_t off = (v < nv && i < T.t_end) ? 2u * (uint32_t)(i * T.s_in2 + h * T.s_in3 + 8 * (v & 15)) : kRgOob;
    R.k[k] = __builtin_amdgcn_raw_buffer_load_b128(T.rin, (int)off, 0, 2);
  }
  if constexpr (MS > 0) {
    const int cpr = 4 * (T.m_steps > 0 ? T.m_steps : 1);   // 16-byte chunks per U row (rank padded to 32)
#pragma unroll
    for (int k = 0; k < rg_u_vec(MS); ++k) {
      const int v = tid + NT * k;
      const int h = v / (kTileTokens * cpr), t = (v / cpr) % kTileTokens, c = v % cpr;
      const int i = i0 + t;
      const uint32_t off = (h < T.H && 8 * c < T.m && i < T.t_end)
                               ? 2u * (uint32_t)(h * T.s_u2 + i * T.s_u3 + 8 * c) : kRgOob;
      R.u[k] = __builtin_amdgcn_raw_buffer_load_b128(T.ru, (int)off, 0, 2);
    }
  }
}

template <int MS, int HW>
__device__ __forceinline__ void rg_to_lds(const RgTask& T, int tid, const RgRegs<MS>& R, uint8_t* buf) {
  constexpr int NT = 64 * HW;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + NT * k;
    int h, t;
    rg_vec(v, T.H, T.in_head_major, h, t);
    if (v < nv) *reinterpret_cast<u32x4*>(buf + (h * kTileTokens + t) * kRgKRow + 16 * (v & 15)) = R.k[k];
  }
  if constexpr (MS > 0) {
    if (T.m_steps > 0) {
      const int cpr = 4 * T.m_steps;
#pragma unroll
      for (int k = 0; k < rg_u_vec(MS); ++k) {
        const int v = tid + NT * k;
        const int h = v / (kTileTokens * cpr), t = (v / cpr) % kTileTokens, c = v % cpr;
        // a layer rank that is not a multiple of 8 ends inside a chunk: the
        // ranks past it are cleared (the plane's U rows hold m >= 8c + 8 ranks)
        u32x4 u = R.u[k];
        const int rem = T.m - 8 * c;
        if (rem < 8) {
          uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            wv[e] &= (2 * e < rem ? 0x0000ffffu : 0u) | (2 * e + 1 < rem ? 0xffff0000u : 0u);
          u = u32x4{wv[0], wv[1], wv[2], wv[3]};
        }
        if (h < T.H)
          *reinterpret_cast<u32x4*>(buf + HW * kTileTokens * kRgKRow + (h * kTileTokens + t) * rg_u_row(MS) +
                                    16 * c) = u;
      }
    }
  }
}

// rotation of one head's tile: lane (g, t) holds chunks g + 4q of token t in
// acc[2q], acc[2q + 1].  The frequencies and coordinates are re-read from LDS
// on every tile: the empty asm hides that their index is loop-invariant, so
// the compiler does not keep them live across the tile loop.
template <int ROT>
__device__ __forceinline__ void rg_rotate(f32x4 (&acc)[8], int g, const double* s_freq, const int* s_coord,
                                          double pt, double ph, double pw) {
  int jb = 8 * g;
  asm volatile("" : "+v"(jb));
  if constexpr (ROT == 1) {                     // NeoX: chunk q pairs with chunk q + 8
#pragma unroll
    for (int q = 0; q < 2; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = jb + 32 * q + e;
        const int sc = s_coord[j];
        const double pos = sc == 0 ? pt : (sc == 1 ? ph : pw);
        float sn, cs;
        sincos_rev(pos, s_freq[j], sn, cs);
        const int ax = 2 * q + (e >> 2), ay = 2 * (q + 2) + (e >> 2), k = e & 3;
        const float x = acc[ax][k];
        const float y = acc[ay][k];
        acc[ax][k] = x * cs - y * sn;
        acc[ay][k] = x * sn + y * cs;
      }
    }
  } else if constexpr (ROT == 2) {              // interleaved: adjacent elements
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
#pragma unroll
      for (int k = 0; k < 4; k += 2) {
        const int j = (jb >> 1) + 16 * (mt >> 1) + 2 * (mt & 1) + (k >> 1);
        const int sc = s_coord[j];
        const double pos = sc == 0 ? pt : (sc == 1 ? ph : pw);
        float sn, cs;
        sincos_rev(pos, s_freq[j], sn, cs);
        const float x = acc[mt][k];
        const float y = acc[mt][k + 1];
        acc[mt][k] = x * cs - y * sn;
        acc[mt][k + 1] = x * sn + y * cs;
      }
    }
  }
}

// relocation: acc += R(delta) K for the head row at krow, with the chunk's
// (cos, sin) of delta per pair from s_dcs (R(delta) is the same for every
// token of the chunk); the element-to-pair layout is that of rg_rotate
template <int ROT>
__device__ __forceinline__ void rg_add_turned(f32x4 (&acc)[8], int g, const uint8_t* krow, const float* s_dcs) {
  u32x4 kc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) kc[q] = *reinterpret_cast<const u32x4*>(krow + 16 * (g + 4 * q));
  auto kv = [&](int mt, int k) -> float {
    const u32x4& w = kc[mt >> 1];
    const uint32_t u = (mt & 1) ? (k < 2 ? w.z : w.w) : (k < 2 ? w.x : w.y);
    return (k & 1) ? bf_hi(u) : bf_lo(u);
  };
  int jb = 8 * g;
  asm volatile("" : "+v"(jb));
  if constexpr (ROT == 0) {
#pragma unroll
    for (int mt = 0; mt < 8; ++mt)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[mt][k] += kv(mt, k);
  } else if constexpr (ROT == 1) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = jb + 32 * q + e;
        const float cs = s_dcs[2 * j], sn = s_dcs[2 * j + 1];
        const int ax = 2 * q + (e >> 2), ay = 2 * (q + 2) + (e >> 2), k = e & 3;
        const float x = kv(ax, k), y = kv(ay, k);
        acc[ax][k] += x * cs - y * sn;
        acc[ay][k] += x * sn + y * cs;
      }
    }
  } else {
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
#pragma unroll
      for (int k = 0; k < 4; k += 2) {
        const int j = (jb >> 1) + 16 * (mt >> 1) + 2 * (mt & 1) + (k >> 1);
        const float cs = s_dcs[2 * j], sn = s_dcs[2 * j + 1];
        const float x = kv(mt, k), y = kv(mt, k + 1);
        acc[mt][k] += x * cs - y * sn;
        acc[mt][k + 1] += x * sn + y * cs;
      }
    }
  }
}

// one wave: head h of the tile in LDS, result written back in place
template <int MS, int ROT, int HW, bool RELOC>
__device__ __forceinline__ void rg_compute(const RehydrateParams& P, const RgTask& T, int tid, int i0, int h,
                                           const u32x4 (&wa)[8][MS > 0 ? MS : 1], uint8_t* buf,
                                           const double* s_freq, const int* s_coord, const float* s_dcs) {
  const int lane = tid & 63;
  const int g = lane >> 4, t = lane & 15;
  uint8_t* krow = buf + (h * kTileTokens + t) * kRgKRow;
  f32x4 acc[8];
  if constexpr (RELOC) {
    // the patch accumulates alone; the keys are added, turned, at the end
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
    u32x4 kc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) kc[q] = *reinterpret_cast<const u32x4*>(krow + 16 * (g + 4 * q));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc[2 * q][0] = bf_lo(kc[q].x);
      acc[2 * q][1] = bf_hi(kc[q].x);
      acc[2 * q][2] = bf_lo(kc[q].y);
      acc[2 * q][3] = bf_hi(kc[q].y);
      acc[2 * q + 1][0] = bf_lo(kc[q].z);
      acc[2 * q + 1][1] = bf_hi(kc[q].z);
      acc[2 * q + 1][2] = bf_lo(kc[q].w);
      acc[2 * q + 1][3] = bf_hi(kc[q].w);
    }
  }
  const int i = i0 + t;
  double pt = 0.0, ph = 0.0, pw = 0.0;
  if constexpr (ROT != 0) {
    if (P.pos_mode == 0) {
      pt = ph = pw = T.cp0 + (double)i;
    } else {
      pt = T.cp0;
      ph = T.cp1 + (double)(i / P.grid_w);
      pw = T.cp2 + (double)(i % P.grid_w);
    }
    // post-rope frame: R(p) K before the patch (+ U W after)
    if constexpr (!RELOC) {
      if (P.patch_post_rope) rg_rotate<ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
    }
  }
  if constexpr (MS > 0) {
    const uint8_t* urow = buf + HW * kTileTokens * kRgKRow + (h * kTileTokens + t) * rg_u_row(MS);
#pragma unroll
    for (int k = 0; k < MS; ++k) {
      if (k < T.m_steps) {
        const bf16x8 b = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(urow + 64 * k + 16 * g));
#pragma unroll
        for (int mt = 0; mt < 8; ++mt)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[mt][k]), b, acc[mt], 0, 0, 0);
      }
    }
  }
  if constexpr (RELOC) {
    // relocation of keys already turned to p - delta (Sec. 5):
    //   stored frame:    R(p) (R(delta - p) K + U W) = R(delta) K + R(p) U W
    //   post-rope frame: R(delta) K + U W
    // so the only per-token angles are those of the patch term
    if constexpr (ROT != 0) {
      if (!P.patch_post_rope && MS > 0 && T.m_steps > 0) rg_rotate<ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
    }
    rg_add_turned<ROT>(acc, g, krow, s_dcs);
  } else if constexpr (ROT != 0) {
    if (!P.patch_post_rope) rg_rotate<ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    u32x4 o;
    o.x = pack_bf16x2(acc[2 * q][0], acc[2 * q][1]);
    o.y = pack_bf16x2(acc[2 * q][2], acc[2 * q][3]);
    o.z = pack_bf16x2(acc[2 * q + 1][0], acc[2 * q + 1][1]);
    o.w = pack_bf16x2(acc[2 * q + 1][2], acc[2 * q + 1][3]);
    *reinterpret_cast<u32x4*>(krow + 16 * (g + 4 * q)) = o;
  }
}

// store phase: every thread writes four 16-byte pieces of the tile's rows;
// s_page holds the pool page of every token of the block (-1: not written)
template <int HW>
__device__ __forceinline__ void rg_store(const RehydrateParams& P, const RgTask& T, int tid, int t_begin, int i0,
                                         const uint8_t* buf, const int* s_page) {
  constexpr int NT = 64 * HW;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + NT * k;
    int h, t;
    rg_vec(v, T.H, T.out_head_major, h, t);
    const int i = i0 + t;
    bool ok = v < nv && i < T.n_c;
    int row = i;
    if (P.place.paged) {
      const int page = ok ? s_page[i - t_begin] : -1;
      ok = ok && page >= 0;
      row = page * P.place.page_size + i % P.place.page_size;
    }
    const uint32_t off = ok ? 2u * (uint32_t)(row * T.s_o2 + h * T.s_o3 + 8 * (v & 15)) : kRgOob;
    const u32x4 val = *reinterpret_cast<const u32x4*>(buf + (h < T.H ? (h * kTileTokens + t) * kRgKRow : 0) +
                                                      16 * (v & 15));
    __builtin_amdgcn_raw_buffer_store_b128(val, T.rout, (int)off, 0, 2);
  }
}

// W rows of one staging item: head h (of the workgroup), ranks k0..k0+3,
// columns colb..colb+7
__device__ __forceinline__ void rg_load_w(const RgTask& T, int h, int k0, int colb, uint32_t (&w)[4][4]) {
  const PlaneParams& Q = *T.Q;
  const uint16_t* wbase =
      Q.W + (int64_t)T.c * Q.w_s[0] + (int64_t)T.l * Q.w_s[1] + (int64_t)(T.h0 + h) * Q.w_s[2];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    w[r][0] = w[r][1] = w[r][2] = w[r][3] = 0u;
    const int k = k0 + r;
    if (h < T.H && k < T.m) {
      const uint16_t* p = wbase + (int64_t)k * Q.w_s[3] + colb;
      if (Q.w_vec) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(p);
        w[r][0] = v.x; w[r][1] = v.y; w[r][2] = v.z; w[r][3] = v.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) w[r][e >> 1] |= (e & 1) ? ((uint32_t)p[e] << 16) : (uint32_t)p[e];
      }
    }
  }
}

// transpose of one staging item into the W^T area: [head % 4][column][rank]
template <int MS>
__device__ __forceinline__ void rg_put_w(int hq, int k0, int colb, const uint32_t (&w)[4][4], uint8_t* lds) {
  uint8_t* base = lds + hq * 128 * rg_wt_row(MS);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int sh = (e & 1) ? 16 : 0;
    const uint32_t r0 = (w[0][e >> 1] >> sh) & 0xffffu, r1 = (w[1][e >> 1] >> sh) & 0xffffu;
    const uint32_t r2 = (w[2][e >> 1] >> sh) & 0xffffu, r3 = (w[3][e >> 1] >> sh) & 0xffffu;
    uint2 v;
    v.x = r0 | (r1 << 16);
    v.y = r2 | (r3 << 16);
    *reinterpret_cast<uint2*>(base + (colb + e) * rg_wt_row(MS) + 2 * k0) = v;
  }
}

template <int MS, int ROT, int HW, bool RELOC>
__device__ __forceinline__ void rg_run(const RehydrateParams& P, const RgTask& T, int tid, int t_begin, int t_end,
                                       uint8_t* lds, const double* s_freq, const int* s_coord, const float* s_dcs) {
  constexpr int NT = 64 * HW;
  constexpr int kIpt = 1024 / NT;               // W staging items per thread and round of 4 heads
  const int h = tid >> 6;                       // wave = head
  const int lane = tid & 63;
  const bool active = h < T.H;
  const int n_tiles = (t_end - t_begin + kTileTokens - 1) / kTileTokens;
  int* s_page = reinterpret_cast<int*>(lds + rg_lds_bytes(MS, HW) - kRgMaxBlock * 4);

  // set-up loads, in flight together: the block's pool pages, the first
  // tiles and the W rows of the first four heads
  int page[kRgMaxBlock / NT];
#pragma unroll
  for (int k = 0; k < kRgMaxBlock / NT; ++k) {
    const int j = t_begin + tid + NT * k;
    page[k] = -1;
    if (P.place.paged && j < t_end) {
      page[k] = P.place.page_table[(int64_t)T.c * P.place.pt_stride + j / P.place.page_size];
      if (page[k] < 0 || page[k] >= P.place.n_pool_pages) {
        if (P.place.status != nullptr) atomicOr(P.place.status, KAMERA_STATUS_BAD_PAGE);
        page[k] = -1;
      }
    }
  }
  RgRegs<MS> R[kRgDepth];
#pragma unroll
  for (int d = 0; d < kRgDepth; ++d)
    if (d < n_tiles) rg_load<MS, HW>(T, tid, t_begin + d * kTileTokens, R[d]);
  // staging item = (head of the round, rank quad, column chunk); the thread's
  // items are tid + NT * j, i.e. heads (tid >> 8) + j * NT / 256 of the round
  const int k0 = 4 * ((tid >> 4) & 15), colb = 8 * (tid & 15), hr = tid >> 8;
  const bool w_item = MS > 0 && T.m_steps > 0 && k0 < 32 * T.m_steps;
  uint32_t w[kIpt][4][4];
  if (w_item) {
#pragma unroll
    for (int j = 0; j < kIpt; ++j) rg_load_w(T, hr + j * (NT / 256), k0, colb, w[j]);
  }
#pragma unroll
  for (int k = 0; k < kRgMaxBlock / NT; ++k)
    if (P.place.paged && t_begin + tid + NT * k < t_end) s_page[tid + NT * k] = page[k];

  // W^T into registers: A operand of M-tile mt, K-step k for lane (g, t):
  // column 8*(t/4) + t%4 + 32*(mt/2) + 4*(mt%2), ranks 32k + 8g .. +7.
  // Rounds of four heads through LDS: round r holds heads 4r .. 4r + 3.
  u32x4 wa[8][MS > 0 ? MS : 1];
  if constexpr (MS > 0) {
    const int g = lane >> 4, t = lane & 15;
#pragma unroll
    for (int round = 0; round < HW / 4; ++round) {
      if (round > 0 && w_item) {
#pragma unroll
        for (int j = 0; j < kIpt; ++j) rg_load_w(T, 4 * round + hr + j * (NT / 256), k0, colb, w[j]);
      }
      if (w_item) {
#pragma unroll
        for (int j = 0; j < kIpt; ++j) rg_put_w<MS>(hr + j * (NT / 256), k0, colb, w[j], lds);
      }
      __syncthreads();
      if ((h >> 2) == round) {
        const uint8_t* hb = lds + (h & 3) * 128 * rg_wt_row(MS);
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
          const int col = 8 * (t >> 2) + (t & 3) + 32 * (mt >> 1) + 4 * (mt & 1);
#pragma unroll
          for (int k = 0; k < MS; ++k)
            wa[mt][k] = (k < T.m_steps) ? *reinterpret_cast<const u32x4*>(hb + col * rg_wt_row(MS) + 64 * k + 16 * g)
                                        : u32x4{0, 0, 0, 0};
        }
      }
      __syncthreads();
    }
  }

  // kRgDepth register sets (tiles in flight) and two LDS buffers: tile tt
  // uses set tt % kRgDepth and buffer tt % 2; two barriers per tile
  auto step = [&](int tt, RgRegs<MS>& R) {
    const int i0 = t_begin + tt * kTileTokens;
    uint8_t* buf = lds + (tt & 1) * rg_buf_bytes(MS, HW);
    rg_to_lds<MS, HW>(T, tid, R, buf);
    if (tt + kRgDepth < n_tiles) rg_load<MS, HW>(T, tid, i0 + kRgDepth * kTileTokens, R);
    __syncthreads();
    if (active) rg_compute<MS, ROT, HW, RELOC>(P, T, tid, i0, h, wa, buf, s_freq, s_coord, s_dcs);
    __syncthreads();
    rg_store<HW>(P, T, tid, t_begin, i0, buf, s_page);
  };
  for (int tile = 0; tile < n_tiles; tile += kRgDepth) {
#pragma unroll
    for (int d = 0; d < kRgDepth; ++d)
      if (tile + d < n_tiles) step(tile + d, R[d]);
  }
}

// Start, in a lane's (chunk, layer, 16-token tile) space, of the r-th of g
// pieces of equal weight.  Without a per-layer rank every tile weighs the
// same; with one, a tile of layer l weighs the bytes it moves per token and
// head, scaled by the tokens n of a unit: (512 + 2 r_l) n + 256 r_l -- the row
// in and out, its U row and its share of the unit's W (r_l the layer's rank).
// One wave's lanes take contiguous blocks of layers; a scan over the wave and
// a ballot find the layer that holds the cut.
__device__ __forceinline__ int64_t rg_cut(const RehydrateParams& P, const PlaneParams& Q, int64_t r, int tid) {
  const int64_t T = P.unit_tiles;
  const int L = P.n_layers;
  if (Q.layer_rank == nullptr) return r * ((int64_t)P.n_chunks * L * T) / P.lane_wgs;
  const int64_t n = T * kTileTokens;
  auto weight = [&](int l) -> int64_t {
    const int rk = min(max(Q.layer_rank[l], 0), Q.m);
    return (512 + 2 * (int64_t)rk) * n + 256 * (int64_t)rk;
  };
  const int lane = tid & 63;
  const int per = (L + 63) / 64;
  const int lb = min(L, lane * per), le = min(L, lb + per);
  int64_t own = 0;
  for (int l = lb; l < le; ++l) own += weight(l);
  int64_t incl = own;
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(incl, d);
    if (lane >= d) incl += y;
  }
  const int64_t chunk_w = __shfl(incl, 63) * T;
  const int64_t target = r * ((int64_t)P.n_chunks * chunk_w) / P.lane_wgs;
  const int64_t c = target / chunk_w;
  int64_t rem = target - c * chunk_w;
  const uint64_t holds = __ballot(incl * T > rem);
  const int owner = holds ? __builtin_ctzll(holds) : 63;
  rem -= __shfl(incl - own, owner) * T;
  int l = __shfl(lb, owner);
  const int l_end = __shfl(le, owner);
  while (l < l_end - 1 && rem >= weight(l) * T) {
    rem -= weight(l) * T;
    ++l;
  }
  const int64_t tile = min(rem / weight(l), T);
  return (c * L + l) * T + tile;
}

// One segment: 16-token tiles [tile0, tile1) (at most kRgMaxBlock tokens) of
// unit cl = chunk * n_layers + layer, for lane (plane, head group) `lane`.
// dcs_chunk names the chunk whose (cos, sin) of delta s_dcs holds (-1: none);
// a relocating segment of another chunk refills it.  Returns the chunk s_dcs
// holds afterwards.
template <int MS, int HW, bool RELOC>
__device__ __forceinline__ int rg_segment(const RehydrateParams& P, int lane, int64_t cl, int tile0, int tile1,
                                          int tid, int dcs_chunk, uint8_t* lds, double* s_freq, int* s_coord,
                                          float* s_dcs) {
  const int pl = lane % P.n_planes;
  const int hg = lane / P.n_planes;
  const PlaneParams& Q = P.plane[pl];
  const int rot = (Q.blk[0].flags & kBlkRotate) ? (P.rope.pairing == 0 ? 1 : 2) : 0;
  RgTask T;
  T.Q = &Q;
  T.l = (int)(cl % P.n_layers);
  T.c = (int)(cl / P.n_layers);
  T.h0 = hg * HW;
  T.H = min(HW, P.n_heads - T.h0);
  T.n_c = chunk_len(P.place, T.c);
  const int t_begin = tile0 * kTileTokens;
  if (t_begin >= T.n_c) return dcs_chunk;       // uniform: the whole workgroup skips
  const int t_end = min(tile1 * kTileTokens, T.n_c);
  T.t_end = t_end;
  T.m = Q.m;
  if (Q.layer_rank != nullptr) {
    const int lr = Q.layer_rank[T.l];
    T.m = lr < 0 ? 0 : (lr < Q.m ? lr : Q.m);
  }
  T.m_steps = (T.m + 31) / 32;
  T.in_head_major = Q.in_s[3] > Q.in_s[2];
  T.out_head_major = Q.out_s[3] > Q.out_s[2];
  T.s_in2 = (int)Q.in_s[2];
  T.s_in3 = (int)Q.in_s[3];
  T.s_u2 = (int)Q.u_s[2];
  T.s_u3 = (int)Q.u_s[3];
  T.s_o2 = (int)Q.out_s[2];
  T.s_o3 = (int)Q.out_s[3];
  // the slabs start at the workgroup's first head
  T.rin = rg_rsrc(Q.in + (int64_t)T.c * Q.in_s[0] + (int64_t)T.l * Q.in_s[1] + (int64_t)T.h0 * Q.in_s[3],
                  Q.in_rec - 2 * (int64_t)T.h0 * Q.in_s[3]);
  T.ru = rg_rsrc(Q.U != nullptr ? Q.U + (int64_t)T.c * Q.u_s[0] + (int64_t)T.l * Q.u_s[1] + (int64_t)T.h0 * Q.u_s[2]
                                : Q.in,
                 Q.U != nullptr ? Q.u_rec - 2 * (int64_t)T.h0 * Q.u_s[2] : 0);
  // paged: the layer's pool; dense: the chunk's rows from its row base on
  const int64_t out_base = P.place.paged ? 0
                           : (int64_t)T.c * Q.out_s[0] +
                                 (int64_t)(P.place.row_base ? P.place.row_base[T.c] : 0) * Q.out_s[2];
  T.rout = rg_rsrc(Q.out + out_base + (int64_t)T.l * Q.out_s[1] + (int64_t)T.h0 * Q.out_s[3],
                   Q.out_rec - 2 * (int64_t)T.h0 * Q.out_s[3]);
  T.cp0 = T.cp1 = T.cp2 = 0.0;
  T.dt = T.dh = T.dw = 0.0;
  if (RELOC) {
    T.dt = (double)P.delta[3 * T.c];
    T.dh = (double)P.delta[3 * T.c + 1];
    T.dw = (double)P.delta[3 * T.c + 2];
    if (rot != 0 && T.c != dcs_chunk) {
      // read only after the next barrier; an earlier segment's reads ended
      // before the barrier that closed it
      const int half = P.rope.rope_dim / 2;
      for (int j = threadIdx.x; j < half; j += 64 * HW) {
        const int sc = P.rope.coord[j];
        float sn, cs;
        sincos_rev(sc == 0 ? T.dt : (sc == 1 ? T.dh : T.dw), P.rope.rev_freq[j], sn, cs);
        s_dcs[2 * j] = cs;
        s_dcs[2 * j + 1] = sn;
      }
      dcs_chunk = T.c;
    }
  }
  if (P.chunk_pos != nullptr) {
    T.cp0 = (double)P.chunk_pos[3 * T.c];
    T.cp1 = (double)P.chunk_pos[3 * T.c + 1];
    T.cp2 = (double)P.chunk_pos[3 * T.c + 2];
  }
  switch (rot) {
    case 0: rg_run<MS, 0, HW, RELOC>(P, T, tid, t_begin, t_end, lds, s_freq, s_coord, s_dcs); break;
    case 1: rg_run<MS, 1, HW, RELOC>(P, T, tid, t_begin, t_end, lds, s_freq, s_coord, s_dcs); break;
    default: rg_run<MS, 2, HW, RELOC>(P, T, tid, t_begin, t_end, lds, s_freq, s_coord, s_dcs); break;
  }
  return dcs_chunk;
}

// Workgroup w serves lane w % lanes -- one (plane, group of HW heads) -- and
// range w / lanes of that lane's (chunk, layer, 16-token tile) space.  The
// workgroups of one range index are adjacent in the grid and walk the same
// tiles at the same pace, so the planes and head groups of a pool page are
// written together.
//  * PERSIST = false (block schedule): range r is token block r % nb of unit
//    r / nb (nb blocks of block_tiles per unit), one segment; there are more
//    workgroups than fit at once and the hardware hands them out.
//  * PERSIST = true: one resident wave of workgroups, lane_wgs ranges of equal
//    weight per lane (so that all finish together), each walked in segments
//    of at most one unit's tiles (and kRgMaxBlock tokens); a unit's set-up
//    (W^T, page numbers) is paid once per segment.
// RELOC: the keys are already rotated and move by the chunk's delta.
template <int MS, int HW, bool RELOC, bool PERSIST>
__global__ __launch_bounds__(64 * HW, rg_min_waves(MS, HW)) void rehydrate_rows_kernel(const RehydrateParams /*by value, read in place*/) {
  const RehydrateParams& P = kernel_params<RehydrateParams>();
  extern __shared__ __align__(16) uint8_t lds_dyn[];
  __shared__ double s_freq[kMaxPairs];
  __shared__ int s_coord[kMaxPairs];
  __shared__ float s_dcs[2 * kMaxPairs];        // relocation: cos, sin of delta per pair

  const int half = P.rope.rope_dim / 2;          // 0 when no plane rotates
  for (int j = threadIdx.x; j < half; j += 64 * HW) {
    s_freq[j] = P.rope.rev_freq[j];
    s_coord[j] = P.rope.coord[j];
  }
  const int lanes = P.n_planes * P.n_hgroups;
  if constexpr (!PERSIST) {
    const int64_t r = blockIdx.x / (uint32_t)lanes;
    const int nb = (P.unit_tiles + P.block_tiles - 1) / P.block_tiles;
    const int64_t u = r / nb;
    const int tile0 = (int)(r - u * nb) * P.block_tiles;
    const int tile1 = min(tile0 + P.block_tiles, P.unit_tiles);
    rg_segment<MS, HW, RELOC>(P, (int)(blockIdx.x % (uint32_t)lanes), u, tile0, tile1, threadIdx.x, -1, lds_dyn,
                              s_freq, s_coord, s_dcs);
  } else {
    // The segment cursor and the chunk s_dcs holds live in VGPRs across a
    // segment (whose tile loop needs every scalar register); the uniform
    // state of a segment is derived again from them and the launch
    // parameters.
    int32_t cur_lo, cur_hi, end_lo, end_hi, dcs_chunk_v = -1;
    {
      const int64_t r = blockIdx.x / (uint32_t)lanes;
      const PlaneParams& Q = P.plane[(blockIdx.x % (uint32_t)lanes) % P.n_planes];
      const int64_t f0 = rg_cut(P, Q, r, threadIdx.x), f1 = rg_cut(P, Q, r + 1, threadIdx.x);
      cur_lo = (int32_t)(uint32_t)f0;
      cur_hi = (int32_t)(f0 >> 32);
      end_lo = (int32_t)(uint32_t)f1;
      end_hi = (int32_t)(f1 >> 32);
    }
    for (;;) {
      asm volatile("" : "+v"(cur_lo), "+v"(cur_hi), "+v"(end_lo), "+v"(end_hi), "+v"(dcs_chunk_v));
      const int64_t f = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(cur_hi) << 32) |
                                  (uint32_t)__builtin_amdgcn_readfirstlane(cur_lo));
      const int64_t f_end = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(end_hi) << 32) |
                                      (uint32_t)__builtin_amdgcn_readfirstlane(end_lo));
      const int dcs_chunk = __builtin_amdgcn_readfirstlane(dcs_chunk_v);
      if (f >= f_end) break;
      const int64_t cl = f / P.unit_tiles;
      const int tile0 = (int)(f - cl * P.unit_tiles);
      int64_t tile1 = min((int64_t)P.unit_tiles, (int64_t)tile0 + (f_end - f));
      tile1 = min(tile1, (int64_t)tile0 + kRgMaxBlock / kTileTokens);
      {
        const int64_t next = f + (tile1 - tile0);
        cur_lo = (int32_t)(uint32_t)next;
        cur_hi = (int32_t)(next >> 32);
      }
      // the thread index as a value the compiler cannot see through: what is
      // derived from it is derived again per segment instead of held in
      // registers across the segment loop
      int tid = threadIdx.x;
      asm volatile("" : "+v"(tid));
      dcs_chunk_v = rg_segment<MS, HW, RELOC>(P, (int)(blockIdx.x % (uint32_t)lanes), cl, tile0, (int)tile1, tid,
                                              dcs_chunk, lds_dyn, s_freq, s_coord, s_dcs);
      __syncthreads();                          // LDS (tiles, W^T, pages, s_dcs) free for the next segment
    }
  }
}

// Workgroups of the persistent instantiation that the device holds at once
// (all CUs), asked once per device.
template <int MS, int HW, bool RELOC>
hipError_t rows_resident(int dev, int& resident) {
  static std::atomic<int> cache[kMaxDevices];
  const bool cached = dev >= 0 && dev < kMaxDevices;
  if (cached && (resident = cache[dev].load(std::memory_order_acquire)) > 0) return hipSuccess;
  int per_cu = 0, cus = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, rehydrate_rows_kernel<MS, HW, RELOC, true>,
                                                              64 * HW, rg_lds_bytes(MS, HW));
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  resident = per_cu * cus > 0 ? per_cu * cus : 1;
  if (cached) cache[dev].store(resident, std::memory_order_release);
  return hipSuccess;
}

template <int MS, int HW, bool RELOC>
hipError_t launch_rows(const RehydrateParams& p, hipStream_t s) {
  const int lanes = p.n_planes * p.n_hgroups;
  RehydrateParams q = p;
  if (p.block_tiles > 0) {
    // block schedule: one workgroup per token block; the hardware hands them out
    static std::atomic<bool> lds_set[kMaxDevices];
    hipError_t e = ensure_lds_limit((const void*)rehydrate_rows_kernel<MS, HW, RELOC, false>, rg_lds_bytes(MS, HW),
                                    lds_set);
    if (e != hipSuccess) return e;
    const int64_t g = (int64_t)p.n_chunks * p.n_layers * ((p.unit_tiles + p.block_tiles - 1) / p.block_tiles);
    q.lane_wgs = (int32_t)g;
    const dim3 grid((uint32_t)(lanes * g)), block(64 * HW);
    hipLaunchKernelGGL((rehydrate_rows_kernel<MS, HW, RELOC, false>), grid, block, rg_lds_bytes(MS, HW), s, q);
    return hipGetLastError();
  }
  static std::atomic<bool> lds_set[kMaxDevices];
  hipError_t e = ensure_lds_limit((const void*)rehydrate_rows_kernel<MS, HW, RELOC, true>, rg_lds_bytes(MS, HW),
                                  lds_set);
  if (e != hipSuccess) return e;
  int dev = 0, resident = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = rows_resident<MS, HW, RELOC>(dev, resident);
  if (e != hipSuccess) return e;
  // one resident wave of workgroups (or the caller's cap), at least one tile each
  if (p.max_wgs > 0 && p.max_wgs < resident) resident = p.max_wgs;
  const int64_t per_lane = (int64_t)p.n_chunks * p.n_layers * p.unit_tiles;
  int64_t g = resident / lanes > 0 ? resident / lanes : 1;
  g = g < per_lane ? g : per_lane;
  q.lane_wgs = (int32_t)g;
  const dim3 grid((uint32_t)(lanes * g)), block(64 * HW);
  hipLaunchKernelGGL((rehydrate_rows_kernel<MS, HW, RELOC, true>), grid, block, rg_lds_bytes(MS, HW), s, q);
  return hipGetLastError();
}

template <bool RELOC>
hipError_t launch_rows_reloc(const RehydrateParams& p, hipStream_t s, int max_steps) {
  if (p.row_group == 4) {
    switch (max_steps) {
      case 0: return launch_rows<0, 4, RELOC>(p, s);
      case 1: return launch_rows<1, 4, RELOC>(p, s);
      default: return launch_rows<2, 4, RELOC>(p, s);
    }
  }
  switch (max_steps) {
    case 0: return launch_rows<0, 8, RELOC>(p, s);
    case 1: return launch_rows<1, 8, RELOC>(p, s);
    default: return launch_rows<2, 8, RELOC>(p, s);
  }
}

hipError_t launch_rehydrate_rows(const RehydrateParams& p, hipStream_t s) {
  int max_steps = 0;
  for (int k = 0; k < p.n_planes; ++k) max_steps = max_steps > p.plane[k].m_steps ? max_steps : p.plane[k].m_steps;
  return p.delta != nullptr ? launch_rows_reloc<true>(p, s, max_steps) : launch_rows_reloc<false>(p, s, max_steps);
}

}  // namespace kamera
