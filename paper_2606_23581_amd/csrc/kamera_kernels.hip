// gfx950 kernels of the Kamera chunk-reuse operator.
//
// rehydrate: K' = R(pos)(K + U W), V' = V + U_v W_v  (Eq. eq:operator, Sec. 3;
//            serve step of App. A).  One grouped launch over
//            (plane, chunk, layer, head, token block, column block).  With a
//            per-chunk delta the keys are already rotated and move by delta
//            with a (removal) patch added at the target (Sec. 5, Table evict).
//            (The row-group form for rows of <= 8 heads is kamera_rows.hip.)
// shift:     K' = R(delta) K in place (R(delta) R(p) = R(p + delta), Sec. 1).
// scatter:   bit copy of token rows into page-table slots and back (App. E,
//            Sec. 6).
//
// Register layout of a rehydrate tile.  A wave owns 16 tokens x one column
// block of 32*NQ columns (NQ <= 4).  The rank-m patch U W is computed as
// (W^T U^T) with v_mfma_f32_16x16x32_bf16: M = block columns, N = the 16
// tokens, K = rank.  The block's columns are permuted onto the MFMA rows so
// that the accumulator a lane ends up holding is exactly what it loaded with
// 16-byte loads:
//     lane = 16*g + t  (g = lane group 0..3, t = token 0..15)
//     acc[mt][i] = column 8*(g + 4*(mt/2)) + 4*(mt%2) + i of token t
// i.e. lane (g, t) holds the 16-byte column chunks g, g+4, g+8, g+12 of its
// token row.  The accumulators are seeded with K (fp32), the MFMAs add U W on
// top, and the rotation pairs are lane-local: NeoX partner of chunk q is
// chunk q + NQ/2, interleaved partners are adjacent accumulator elements.
// LDS holds W^T (transposed once per workgroup), the per-pair frequencies and
// one padded 16-row buffer per wave: tiles pass through it between the
// row-contiguous global loads/stores (4 rows x 256 B per instruction) and the
// MFMA register layout, and U rows take the same route.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kamera_device.h"

namespace kamera {

// ---------------------------------------------------------------------------
// rehydrate
// ---------------------------------------------------------------------------

struct TileCtx {
  const PlaneParams* Q;
  int c, l, h, n_c;
  int col0;           // first column of the block
  int ldw;            // LDS row stride of W^T in elements
  bool patched;       // block intersects the patch columns and m > 0
  bool u_vec;         // 16-byte U loads are legal at this layer's rank
  int m;              // rank at this layer (layer_rank may lower the plane's m)
  int m_steps;        // ceil(m / 32)
  int64_t in_base;    // element offset of (c, l, token 0, h, col0) in the input
  int64_t u_base;     // element offset of (c, l, h, token 0) in U
};

// position of token i of chunk c on each coordinate, as exact doubles
__device__ __forceinline__ void token_position(const RehydrateParams& P, int c, int i,
                                               double& pt, double& ph, double& pw) {
  if (P.pos_mode == 0) {                       // linear: p0 + i
    const double p = (double)P.chunk_pos[3 * c] + (double)i;
    pt = ph = pw = p;
  } else if (P.pos_mode == 1) {                // grid of patches, row-major
    pt = (double)P.chunk_pos[3 * c];
    ph = (double)P.chunk_pos[3 * c + 1] + (double)(i / P.grid_w);
    pw = (double)P.chunk_pos[3 * c + 2] + (double)(i % P.grid_w);
  } else {                                     // explicit (t, h, w) per token
    const int32_t* e = P.explicit_pos + (int64_t)c * P.explicit_cs + 3 * (int64_t)i;
    pt = (double)e[0];
    ph = (double)e[1];
    pw = (double)e[2];
  }
}

// ROT: 1 = NeoX pairs (chunk q <-> q + NQ/2), 2 = interleaved (adjacent elements)
template <int NQ, int ROT>
__device__ __forceinline__ void rotate_tile(f32x4 (&acc)[2 * NQ], int g, const double* s_freq,
                                            const int* s_coord, double pt, double ph, double pw) {
  if constexpr (ROT == 1 && NQ % 2 == 0) {
#pragma unroll
    for (int q = 0; q < NQ / 2; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = 8 * g + 32 * q + e;
        const int sc = s_coord[j];
        const double pos = sc == 0 ? pt : (sc == 1 ? ph : pw);
        float sn, cs;
        sincos_rev(pos, s_freq[j], sn, cs);
        const int ax = 2 * q + (e >> 2), ay = 2 * (q + NQ / 2) + (e >> 2), k = e & 3;
        const float x = acc[ax][k];
        const float y = acc[ay][k];
        acc[ax][k] = x * cs - y * sn;
        acc[ay][k] = x * sn + y * cs;
      }
    }
  } else if constexpr (ROT == 2) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int j = 4 * g + 16 * q + (e >> 1);
        const int sc = s_coord[j];
        const double pos = sc == 0 ? pt : (sc == 1 ? ph : pw);
        float sn, cs;
        sincos_rev(pos, s_freq[j], sn, cs);
        const int a = 2 * q + (e >> 2), k = e & 3;
        const float x = acc[a][k];
        const float y = acc[a][k + 1];
        acc[a][k] = x * cs - y * sn;
        acc[a][k + 1] = x * sn + y * cs;
      }
    }
  }
}

// relocation: acc += R(delta) K for the lane's K chunks kc, with the chunk's
// (cos, sin) of delta per pair from s_dcs; the element-to-pair layout is that
// of rotate_tile (no rotation where rotate_tile rotates nothing)
template <int NQ, int ROT>
__device__ __forceinline__ void add_turned_tile(f32x4 (&acc)[2 * NQ], int g, const u32x4 (&kc)[NQ],
                                                const float* s_dcs) {
  auto kv = [&](int mt, int k) -> float {
    const u32x4& w = kc[mt >> 1];
    const uint32_t u = (mt & 1) ? (k < 2 ? w.z : w.w) : (k < 2 ? w.x : w.y);
    return (k & 1) ? bf_hi(u) : bf_lo(u);
  };
  if constexpr (ROT == 1 && NQ % 2 == 0) {
#pragma unroll
    for (int q = 0; q < NQ / 2; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = 8 * g + 32 * q + e;
        const float cs = s_dcs[2 * j], sn = s_dcs[2 * j + 1];
        const int ax = 2 * q + (e >> 2), ay = 2 * (q + NQ / 2) + (e >> 2), k = e & 3;
        const float x = kv(ax, k), y = kv(ay, k);
        acc[ax][k] += x * cs - y * sn;
        acc[ay][k] += x * sn + y * cs;
      }
    }
  } else if constexpr (ROT == 2) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int j = 4 * g + 16 * q + (e >> 1);
        const float cs = s_dcs[2 * j], sn = s_dcs[2 * j + 1];
        const int a = 2 * q + (e >> 2), k = e & 3;
        const float x = kv(a, k), y = kv(a, k + 1);
        acc[a][k] += x * cs - y * sn;
        acc[a][k + 1] += x * sn + y * cs;
      }
    }
  } else {
#pragma unroll
    for (int mt = 0; mt < 2 * NQ; ++mt)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[mt][k] += kv(mt, k);
  }
}

// ---------------------------------------------------------------------------
// Tile I/O.  Global memory is accessed row-contiguously: one load or store
// instruction of a wave covers 64 consecutive 16-byte chunks, i.e. whole
// token rows (4 rows of a 128-column block).  The MFMA layout above wants 4
// lanes per row instead, so each wave passes its tile through a private LDS
// buffer (padded rows keep both access orders free of bank conflicts).  The
// direct path (MFMA layout straight from global memory) remains for blocks of
// 96 columns and for U rows that are not 16-byte aligned.
// ---------------------------------------------------------------------------


template <int NQ>
struct Staged {
  static constexpr bool value = NQ == 1 || NQ == 2 || NQ == 4;
};

// LDS bytes of one wave's staging buffer: a 16 x 128-column bf16 tile, or the
// tile's U rows (16 x up to 128 ranks); the phases of a tile use it in turn.
__host__ __device__ constexpr int tile_lds_bytes() { return kTileTokens * (64 * 4 + kRowPad); }

template <int NQ, int MS>
struct TileRegs {
  u32x4 k[NQ];                  // K (or V) chunks, in load order
  u32x4 u[MS > 0 ? MS : 1];     // U chunks, in load order (staged) or B-operand order (direct)
};

// Issue the global loads of one tile.
template <int NQ, int MS>
__device__ __forceinline__ void tile_load(const TileCtx& T, int i0, TileRegs<NQ, MS>& R) {
  const PlaneParams& Q = *T.Q;
  const int lane = threadIdx.x & 63;
  if constexpr (Staged<NQ>::value) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int cidx = 64 * q + lane;                // chunk of the tile, row-major
      const int row = cidx / (4 * NQ), c16 = cidx % (4 * NQ);
      const int i = i0 + row;
      R.k[q] = i < T.n_c ? ld16(Q.in + T.in_base + (int64_t)i * Q.in_s[2] + 8 * c16) : u32x4{0, 0, 0, 0};
    }
  } else {
    const int g = lane >> 4, i = i0 + (lane & 15);
    const uint16_t* src = Q.in + T.in_base + (int64_t)i * Q.in_s[2];
#pragma unroll
    for (int q = 0; q < NQ; ++q) R.k[q] = i < T.n_c ? ld16(src + 8 * (g + 4 * q)) : u32x4{0, 0, 0, 0};
  }
  if constexpr (MS > 0) {
    if (!T.patched) return;
    if (T.u_vec && Staged<NQ>::value) {
      // 16 rows x 4*m_steps chunks (rank padded to 32); chunks past m stay zero
      const int cpr = T.m >> 3, cpad = 4 * T.m_steps;
#pragma unroll
      for (int s = 0; s < MS; ++s) {
        const int cidx = 64 * s + lane;
        u32x4 v = u32x4{0, 0, 0, 0};
        if (cidx < kTileTokens * cpad) {
          const int row = cidx / cpad, c = cidx % cpad;
          const int i = i0 + row;
          if (c < cpr && i < T.n_c) v = ld16(Q.U + T.u_base + (int64_t)i * Q.u_s[3] + 8 * c);
        }
        R.u[s] = v;
      }
    } else {
      const int g = lane >> 4, i = i0 + (lane & 15);
      const uint16_t* urow = Q.U + T.u_base + (int64_t)i * Q.u_s[3];
#pragma unroll
      for (int s = 0; s < MS; ++s) {
        u32x4 v = u32x4{0, 0, 0, 0};
        const int k0 = 32 * s + 8 * g;
        if (s < T.m_steps && i < T.n_c) {
          if (T.u_vec) {
            if (k0 < T.m) v = ld16(urow + k0);
          } else {
            uint32_t w4[4] = {0, 0, 0, 0};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const uint32_t b = (k0 + e < T.m) ? urow[k0 + e] : 0u;
              w4[e >> 1] |= (e & 1) ? (b << 16) : b;
            }
            v = u32x4{w4[0], w4[1], w4[2], w4[3]};
          }
        }
        R.u[s] = v;
      }
    }
  }
}

// One 16-token tile at i0.  R holds its loads.  With EARLY the loads of the
// wave's next tile (next_i0 >= 0) go into R as soon as the tile has been
// copied into LDS (row-staged blocks with staged or no U); the return value
// says whether they did (else the caller issues them).
template <int NQ, int MS, int ROT, bool RELOC, bool EARLY>
__device__ __forceinline__ bool tile_compute(const RehydrateParams& P, const TileCtx& T, int i0, int next_i0,
                                             TileRegs<NQ, MS>& R, const uint16_t* __restrict__ Wt,
                                             uint8_t* tile_lds, const double* s_freq,
                                             const int* s_coord, const float* s_dcs) {
  // relocation up to rank 64 as R(delta) K + R(p) U W (one set of per-token
  // angles, K kept in registers across the patch); at rank 128, where those
  // registers would spill, as R(p) (R(delta - p) K + U W)
  constexpr bool kOneAngle = RELOC && MS <= 2;
  const PlaneParams& Q = *T.Q;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int t = lane & 15;
  constexpr int kRowB = 64 * NQ + kRowPad;          // LDS row stride of the tile buffer
  const bool u_staged = MS > 0 && T.patched && T.u_vec && Staged<NQ>::value;
  const int u_rowb = 64 * Q.m_steps + kRowPad;

  // ---- K chunks in MFMA order: lane (g, t) takes chunks g + 4q of row t ----
  u32x4 kc[NQ];
  if constexpr (Staged<NQ>::value) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int cidx = 64 * q + lane;
      *reinterpret_cast<u32x4*>(tile_lds + (cidx / (4 * NQ)) * kRowB + 16 * (cidx % (4 * NQ))) = R.k[q];
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) kc[q] = *reinterpret_cast<const u32x4*>(tile_lds + t * kRowB + 16 * (g + 4 * q));
  } else {
#pragma unroll
    for (int q = 0; q < NQ; ++q) kc[q] = R.k[q];
  }
  // the K chunks are in registers now: the buffer takes the U rows
  uint8_t* u_lds = tile_lds;
  if constexpr (MS > 0) {
    if (u_staged) {
      const int cpad = 4 * T.m_steps;
#pragma unroll
      for (int s = 0; s < MS; ++s) {
        const int cidx = 64 * s + lane;
        if (cidx < kTileTokens * cpad)
          *reinterpret_cast<u32x4*>(u_lds + (cidx / cpad) * u_rowb + 16 * (cidx % cpad)) = R.u[s];
      }
    }
  }
  const bool early = EARLY && Staged<NQ>::value && (MS == 0 || !T.patched || u_staged);
  if (early && next_i0 >= 0) tile_load<NQ, MS>(T, next_i0, R);

  f32x4 acc[2 * NQ];
  if constexpr (kOneAngle) {
#pragma unroll
    for (int mt = 0; mt < 2 * NQ; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
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
  const bool valid = i < T.n_c;
  double pt = 0.0, ph = 0.0, pw = 0.0;
  if constexpr (ROT != 0) {
    token_position(P, T.c, valid ? i : T.n_c - 1, pt, ph, pw);
    // Rotation applied before the patch:
    //   post-rope frame:            R(p) K          (+ U W after)
    //   relocation, post-rope:      R(delta) K      (+ U W after)
    //   relocation, pre-rope:       R(-(p - delta)) K, the stored frame
    //                               (+ U W, then R(p) below)
    if constexpr (RELOC && !kOneAngle) {
      const double dt = (double)P.delta[3 * T.c], dh = (double)P.delta[3 * T.c + 1],
                   dw = (double)P.delta[3 * T.c + 2];
      if (P.patch_post_rope)
        rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, dt, dh, dw);
      else
        rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, dt - pt, dh - ph, dw - pw);
    } else if (!RELOC && P.patch_post_rope) {
      rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
    }
  }

  if constexpr (MS > 0) {
    if (T.patched) {
      // A operand row r = t: block column 8*(r/4) + 32*(mt/2) + 4*(mt%2) + r%4
      const int rbase = 8 * (t >> 2) + (t & 3);
#pragma unroll
      for (int s = 0; s < MS; ++s) {
        if (s < T.m_steps) {
          const u32x4 ub = u_staged ? *reinterpret_cast<const u32x4*>(u_lds + t * u_rowb + 2 * (32 * s + 8 * g))
                                    : R.u[s];
          const bf16x8 b = __builtin_bit_cast(bf16x8, ub);
#pragma unroll
          for (int mt = 0; mt < 2 * NQ; ++mt) {
            const int prow = rbase + 32 * (mt >> 1) + 4 * (mt & 1);
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(Wt + prow * T.ldw + 32 * s + 8 * g);
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[mt], 0, 0, 0);
          }
        }
      }
    }
  }

  if constexpr (kOneAngle) {
    if constexpr (ROT != 0) {
      if (!P.patch_post_rope && MS > 0 && T.patched) rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
    }
    add_turned_tile<NQ, ROT>(acc, g, kc, s_dcs);
  } else if constexpr (ROT != 0) {
    if (!P.patch_post_rope) rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
  }

  // ---- round to bf16 (nearest even) ----
  u32x4 o[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    o[q].x = pack_bf16x2(acc[2 * q][0], acc[2 * q][1]);
    o[q].y = pack_bf16x2(acc[2 * q][2], acc[2 * q][3]);
    o[q].z = pack_bf16x2(acc[2 * q + 1][0], acc[2 * q + 1][1]);
    o[q].w = pack_bf16x2(acc[2 * q + 1][2], acc[2 * q + 1][3]);
  }

  // ---- store ----
  auto row_dst = [&](int ii, int64_t& dst) -> bool {
    if (ii >= T.n_c) return false;
    if (P.place.paged) {
      const int64_t slot = page_slot(P.place, T.c, ii);
      if (slot < 0) return false;
      dst = (int64_t)T.l * Q.out_s[1] + slot * Q.out_s[2] + (int64_t)T.h * Q.out_s[3] + T.col0;
    } else {
      const int rb = P.place.row_base ? P.place.row_base[T.c] : 0;
      dst = (int64_t)T.c * Q.out_s[0] + (int64_t)T.l * Q.out_s[1] + (int64_t)(rb + ii) * Q.out_s[2] +
            (int64_t)T.h * Q.out_s[3] + T.col0;
    }
    return true;
  };
  if constexpr (Staged<NQ>::value) {
    // back through LDS (same buffer: its K and U contents are consumed)
#pragma unroll
    for (int q = 0; q < NQ; ++q) *reinterpret_cast<u32x4*>(tile_lds + t * kRowB + 16 * (g + 4 * q)) = o[q];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int cidx = 64 * q + lane;
      const int row = cidx / (4 * NQ), c16 = cidx % (4 * NQ);
      const u32x4 v = *reinterpret_cast<const u32x4*>(tile_lds + row * kRowB + 16 * c16);
      int64_t dst;
      if (row_dst(i0 + row, dst)) st16(Q.out + dst + 8 * c16, v);
    }
  } else {
    int64_t dst;
    if (row_dst(i, dst)) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) st16(Q.out + dst + 8 * (g + 4 * q), o[q]);
    }
  }
  return early;
}

// Stage W^T of one column block into LDS: Wt[col][k], col in [0, 32*NQ),
// k in [0, 32*m_steps); columns outside the patch range and k >= m are zero.
// A thread takes 4 ranks x 8 columns: four 16-byte row loads, transposed in
// registers into eight 8-byte LDS writes (4 consecutive ranks of one column).
template <int NQ>
__device__ __forceinline__ void stage_w(const TileCtx& T, uint16_t* Wt) {
  const PlaneParams& Q = *T.Q;
  const int m_pad = 32 * T.m_steps;
  const int k4s = m_pad / 4;
  const int n_items = k4s * (4 * NQ);
  const uint16_t* wbase = Q.W + (int64_t)T.c * Q.w_s[0] + (int64_t)T.l * Q.w_s[1] +
                          (int64_t)T.h * Q.w_s[2];
  for (int item = threadIdx.x; item < n_items; item += kThreads) {
    const int k0 = 4 * (item % k4s);
    const int colb = 8 * (item / k4s);               // block column of the 8-chunk
    const int wcol = T.col0 + colb - Q.patch_lo;     // W column
    const bool in_patch = T.col0 + colb >= Q.patch_lo && T.col0 + colb + 8 <= Q.patch_hi;
    uint32_t w[4][4];                                 // [rank][column pair]
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      w[r][0] = w[r][1] = w[r][2] = w[r][3] = 0u;
      const int k = k0 + r;
      if (in_patch && k < T.m) {
        const uint16_t* p = wbase + (int64_t)k * Q.w_s[3] + wcol;
        if (Q.w_vec) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(p);
          w[r][0] = v.x; w[r][1] = v.y; w[r][2] = v.z; w[r][3] = v.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) w[r][e >> 1] |= (e & 1) ? ((uint32_t)p[e] << 16) : (uint32_t)p[e];
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // column e of the chunk, ranks k0..k0+3
      const int sh = (e & 1) ? 16 : 0;
      const uint32_t r0 = (w[0][e >> 1] >> sh) & 0xffffu, r1 = (w[1][e >> 1] >> sh) & 0xffffu;
      const uint32_t r2 = (w[2][e >> 1] >> sh) & 0xffffu, r3 = (w[3][e >> 1] >> sh) & 0xffffu;
      uint2 v;
      v.x = r0 | (r1 << 16);
      v.y = r2 | (r3 << 16);
      *reinterpret_cast<uint2*>(Wt + (colb + e) * T.ldw + k0) = v;
    }
  }
}

template <int NQ, int MS, int ROT, bool RELOC>
__device__ __forceinline__ void rehydrate_block(const RehydrateParams& P, const TileCtx& T, int t_begin, int t_end,
                                                uint8_t* lds, double* s_freq, int* s_coord, float* s_dcs) {
  uint16_t* Wt = reinterpret_cast<uint16_t*>(lds);
  const int wave = threadIdx.x >> 6;
  uint8_t* tile_lds = lds + 128 * (32 * MS + 8) * 2 + wave * tile_lds_bytes();
  constexpr int kWaves = kThreads / 64;
  const int n_tiles = (t_end - t_begin + kTileTokens - 1) / kTileTokens;
  // Up to rank 32 the wave's first tile is in flight while W^T is staged (one
  // memory round trip before the first MFMA instead of two), and each next
  // tile's loads are issued during the current tile -- as soon as it is in LDS
  // where the registers allow (no relocation), else after its stores.  At
  // higher ranks the registers of a tile in flight beside the MFMA operands
  // would spill: a tile's loads are issued when it starts.
  constexpr bool kAhead = MS <= 1;
  constexpr bool kEarly = MS == 0 || (MS == 1 && !RELOC);
  TileRegs<NQ, MS> R;
  if (kAhead && wave < n_tiles) tile_load<NQ, MS>(T, t_begin + wave * kTileTokens, R);
  if constexpr (MS > 0) {
    if (T.patched) stage_w<NQ>(T, Wt);
  }
  if constexpr (ROT != 0) {
    const int half = P.rope.rope_dim / 2;
    for (int j = threadIdx.x; j < half; j += kThreads) {
      s_freq[j] = P.rope.rev_freq[j];
      s_coord[j] = P.rope.coord[j];
      if constexpr (RELOC && MS <= 2) {
        const int sc = P.rope.coord[j];
        float sn, cs;
        sincos_rev((double)P.delta[3 * T.c + (sc == 0 ? 0 : (sc == 1 ? 1 : 2))], P.rope.rev_freq[j], sn, cs);
        s_dcs[2 * j] = cs;
        s_dcs[2 * j + 1] = sn;
      }
    }
  }
  __syncthreads();
  for (int tile = wave; tile < n_tiles; tile += kWaves) {
    if (!kAhead) tile_load<NQ, MS>(T, t_begin + tile * kTileTokens, R);
    const int next_i0 = kAhead && tile + kWaves < n_tiles ? t_begin + (tile + kWaves) * kTileTokens : -1;
    const bool issued = tile_compute<NQ, MS, ROT, RELOC, kEarly>(P, T, t_begin + tile * kTileTokens, next_i0, R, Wt,
                                                                 tile_lds, s_freq, s_coord, s_dcs);
    if (!issued && next_i0 >= 0) tile_load<NQ, MS>(T, next_i0, R);
  }
}

// RELOC: the keys are already rotated and move by the chunk's delta
template <int MS, bool RELOC>
__global__ __launch_bounds__(kThreads, MS == 4 || RELOC ? 3 : 4) void rehydrate_kernel(const RehydrateParams /*by value, read in place*/) {
  const RehydrateParams& P = kernel_params<RehydrateParams>();
  extern __shared__ __align__(16) uint8_t lds_dyn[];
  __shared__ double s_freq[kMaxPairs];
  __shared__ int s_coord[kMaxPairs];
  __shared__ float s_dcs[2 * kMaxPairs];        // relocation: cos, sin of delta per pair

  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  // tasks of one (chunk, layer, head, token block) are adjacent: the key
  // blocks (rotation, VALU-heavier) run next to the value blocks (pure streams);
  // task < 2^31, so the coordinates come from 32-bit invariant divisions
  const uint32_t tk = (uint32_t)task;
  uint32_t rem = fast_div(tk, P.fd_bpg);
  const int r = (int)(tk - rem * (uint32_t)P.blocks_per_group);
  const int pl = (P.n_planes == 2 && r >= P.plane[1].block_base) ? 1 : 0;
  const PlaneParams& Q = P.plane[pl];
  const int b = r - Q.block_base;
  uint32_t q = fast_div(rem, P.fd_tblk);
  const int tb = (int)(rem - q * (uint32_t)P.n_tblk);
  rem = q;
  TileCtx T;
  T.Q = &Q;
  q = fast_div(rem, P.fd_heads);
  T.h = (int)(rem - q * (uint32_t)P.n_heads);
  rem = q;
  q = fast_div(rem, P.fd_layers);
  T.l = (int)(rem - q * (uint32_t)P.n_layers);
  T.c = (int)q;
  T.n_c = chunk_len(P.place, T.c);
  const int t_begin = tb * P.token_block;
  if (t_begin >= T.n_c) return;                 // uniform: the whole workgroup leaves
  const int t_end = min(t_begin + P.token_block, T.n_c);
  const ColBlock B = Q.blk[b];
  T.col0 = 8 * (int)B.col0;
  T.ldw = 32 * Q.m_steps + 8;
  T.m = Q.m;
  if (Q.layer_rank != nullptr) {
    const int r = Q.layer_rank[T.l];
    T.m = r < 0 ? 0 : (r < Q.m ? r : Q.m);
  }
  T.m_steps = (T.m + 31) / 32;
  T.u_vec = Q.u_vec && (T.m % 8 == 0);
  T.patched = (B.flags & kBlkPatch) && T.m > 0;
  T.in_base = (int64_t)T.c * Q.in_s[0] + (int64_t)T.l * Q.in_s[1] + (int64_t)T.h * Q.in_s[3] + T.col0;
  T.u_base = (int64_t)T.c * Q.u_s[0] + (int64_t)T.l * Q.u_s[1] + (int64_t)T.h * Q.u_s[2];
  const int rot = (B.flags & kBlkRotate) ? (P.rope.pairing == 0 ? 1 : 2) : 0;
  switch (B.nq * 3 + rot) {
    case 1 * 3 + 0: rehydrate_block<1, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 1 * 3 + 2: rehydrate_block<1, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 2 * 3 + 0: rehydrate_block<2, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 2 * 3 + 1: rehydrate_block<2, MS, 1, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 2 * 3 + 2: rehydrate_block<2, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 3 * 3 + 0: rehydrate_block<3, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 3 * 3 + 2: rehydrate_block<3, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 4 * 3 + 0: rehydrate_block<4, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 4 * 3 + 1: rehydrate_block<4, MS, 1, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    case 4 * 3 + 2: rehydrate_block<4, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord, s_dcs); break;
    default: break;                              // rejected on the host (NeoX needs an even NQ)
  }
}

hipError_t launch_rehydrate(const RehydrateParams& p, hipStream_t s) {
  int max_steps = 0;
  for (int k = 0; k < p.n_planes; ++k) max_steps = max_steps > p.plane[k].m_steps ? max_steps : p.plane[k].m_steps;
  const int ms = max_steps == 0 ? 0 : (max_steps <= 2 ? max_steps : 4);   // template rank steps
  const size_t lds = (size_t)128 * (32 * ms + 8) * sizeof(uint16_t) +
                     (size_t)(kThreads / 64) * tile_lds_bytes();
  if (p.row_group) return launch_rehydrate_rows(p, s);
  const dim3 grid((uint32_t)((int64_t)p.per_xcd * 8)), block(kThreads);
  if (p.delta != nullptr) {
    switch (max_steps) {
      case 0: hipLaunchKernelGGL((rehydrate_kernel<0, true>), grid, block, lds, s, p); break;
      case 1: hipLaunchKernelGGL((rehydrate_kernel<1, true>), grid, block, lds, s, p); break;
      case 2: hipLaunchKernelGGL((rehydrate_kernel<2, true>), grid, block, lds, s, p); break;
      default: hipLaunchKernelGGL((rehydrate_kernel<4, true>), grid, block, lds, s, p); break;
    }
  } else {
    switch (max_steps) {
      case 0: hipLaunchKernelGGL((rehydrate_kernel<0, false>), grid, block, lds, s, p); break;
      case 1: hipLaunchKernelGGL((rehydrate_kernel<1, false>), grid, block, lds, s, p); break;
      case 2: hipLaunchKernelGGL((rehydrate_kernel<2, false>), grid, block, lds, s, p); break;
      default: hipLaunchKernelGGL((rehydrate_kernel<4, false>), grid, block, lds, s, p); break;
    }
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// shift: K' = R(delta) K on the rope band, in place
// ---------------------------------------------------------------------------

constexpr int kShiftUnroll = 4;

__global__ __launch_bounds__(kThreads) void shift_kernel(const ShiftParams /*by value, read in place*/) {
  const ShiftParams& P = kernel_params<ShiftParams>();
  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  const uint32_t tk = (uint32_t)task, q = fast_div(tk, P.fd_tblk), c32 = fast_div(q, P.fd_layers);
  const int tb = (int)(tk - q * (uint32_t)P.n_tblk);
  const int l = (int)(q - c32 * (uint32_t)P.n_layers);
  const int c = (int)c32;
  const int n_c = chunk_len(P.place, c);
  const int t_begin = tb * P.token_block;
  if (t_begin >= n_c) return;
  const int t_end = min(t_begin + P.token_block, n_c);

  const int vpr = P.vec_per_row;
  const int rpp = kThreads / vpr;                 // rows per pass
  if ((int)threadIdx.x >= rpp * vpr) return;       // no barrier in this kernel
  const int v = threadIdx.x % vpr;
  const int r0 = threadIdx.x / vpr;
  const bool neox = P.rope.pairing == 0;
  const int half = P.rope.rope_dim / 2;

  // the angles depend only on (chunk delta, pair): computed once per thread
  const double d3[3] = {(double)P.delta[3 * c], (double)P.delta[3 * c + 1], (double)P.delta[3 * c + 2]};
  float cs[8], sn[8];
  const int npair = neox ? 8 : 4;
  const int j0 = neox ? 8 * v : 4 * v;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (e < npair) {
      const int j = j0 + e;
      sincos_rev(d3[P.rope.coord[j]], P.rope.rev_freq[j], sn[e], cs[e]);
    } else {
      sn[e] = 0.f;
      cs[e] = 1.f;
    }
  }
  const int xcol = P.rope.rope_offset + 8 * v;
  const int ycol = xcol + half;                   // NeoX partner chunk

  const int H = P.n_heads;
  const int rows = (t_end - t_begin) * H;
  for (int base = r0; base < rows; base += kShiftUnroll * rpp) {
    u32x4 xv[kShiftUnroll], yv[kShiftUnroll];
    uint16_t* rp[kShiftUnroll];
#pragma unroll
    for (int u = 0; u < kShiftUnroll; ++u) {
      const int row = base + u * rpp;
      rp[u] = nullptr;
      if (row < rows) {
        const int i = t_begin + row / H;
        const int h = row % H;
        int64_t off;
        if (P.place.paged) {
          const int64_t slot = page_slot(P.place, c, i);
          off = slot < 0 ? -1 : (int64_t)l * P.k_s[1] + slot * P.k_s[2] + (int64_t)h * P.k_s[3];
        } else {
          const int rb = P.place.row_base ? P.place.row_base[c] : 0;
          off = (int64_t)c * P.k_s[0] + (int64_t)l * P.k_s[1] + (int64_t)(rb + i) * P.k_s[2] +
                (int64_t)h * P.k_s[3];
        }
        if (off >= 0) {
          rp[u] = P.k + off;
          xv[u] = ld16(rp[u] + xcol);
          if (neox) yv[u] = ld16(rp[u] + ycol);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kShiftUnroll; ++u) {
      if (rp[u] == nullptr) continue;
      if (neox) {
        u32x4 xo, yo;
        uint32_t xw[4], yw[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t a = u4_get(xv[u], k), b = u4_get(yv[u], k);
          const float x0 = bf_lo(a), x1 = bf_hi(a), y0 = bf_lo(b), y1 = bf_hi(b);
          const int e0 = 2 * k, e1 = 2 * k + 1;
          xw[k] = pack_bf16x2(x0 * cs[e0] - y0 * sn[e0], x1 * cs[e1] - y1 * sn[e1]);
          yw[k] = pack_bf16x2(x0 * sn[e0] + y0 * cs[e0], x1 * sn[e1] + y1 * cs[e1]);
        }
        xo = u32x4{xw[0], xw[1], xw[2], xw[3]};
        yo = u32x4{yw[0], yw[1], yw[2], yw[3]};
        st16(rp[u] + xcol, xo);
        st16(rp[u] + ycol, yo);
      } else {
        uint32_t ow[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t a = u4_get(xv[u], k);
          const float x = bf_lo(a), y = bf_hi(a);
          ow[k] = pack_bf16x2(x * cs[k] - y * sn[k], x * sn[k] + y * cs[k]);
        }
        st16(rp[u] + xcol, u32x4{ow[0], ow[1], ow[2], ow[3]});
      }
    }
  }
}

hipError_t launch_shift(const ShiftParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.per_xcd * 8;
  hipLaunchKernelGGL(shift_kernel, dim3((uint32_t)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// scatter / gather: dense rows <-> page-table slots, bit for bit
// ---------------------------------------------------------------------------

constexpr int kScatterUnroll = 4;

__global__ __launch_bounds__(kThreads) void scatter_kernel(const ScatterParams /*by value, read in place*/) {
  const ScatterParams& P = kernel_params<ScatterParams>();
  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  const uint32_t tk = (uint32_t)task, q = fast_div(tk, P.fd_tblk), c32 = fast_div(q, P.fd_layers);
  const int tb = (int)(tk - q * (uint32_t)P.n_tblk);
  const int l = (int)(q - c32 * (uint32_t)P.n_layers);
  const int c = (int)c32;
  const int n_c = chunk_len(P.place, c);
  const int t_begin = tb * P.token_block;
  if (t_begin >= n_c) return;
  const int t_end = min(t_begin + P.token_block, n_c);
  const int64_t vpr = P.row_vecs;
  const int64_t total = (int64_t)(t_end - t_begin) * vpr;
  uint8_t* rbase = P.rows + (int64_t)c * P.rows_s[0] + (int64_t)l * P.rows_s[1];
  uint8_t* pbase = P.pool + (int64_t)l * P.pool_s[0];
  const bool gather = P.gather != 0;
  for (int64_t base = threadIdx.x; base < total; base += kScatterUnroll * kThreads) {
    u32x4 v[kScatterUnroll];
    uint8_t* dp[kScatterUnroll];
#pragma unroll
    for (int u = 0; u < kScatterUnroll; ++u) {
      const int64_t idx = base + (int64_t)u * kThreads;
      dp[u] = nullptr;
      if (idx < total) {
        const int i = t_begin + (int)(idx / vpr);
        const int64_t vec = idx % vpr;
        const int64_t slot = page_slot(P.place, c, i);
        if (slot >= 0) {
          uint8_t* dense = rbase + (int64_t)i * P.rows_s[2] + 16 * vec;
          uint8_t* paged = pbase + slot * P.pool_s[1] + 16 * vec;
          const uint8_t* sp = gather ? paged : dense;
          dp[u] = gather ? dense : paged;
          v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(sp));
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kScatterUnroll; ++u)
      if (dp[u] != nullptr) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(dp[u]));
  }
}

hipError_t launch_scatter(const ScatterParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.per_xcd * 8;
  hipLaunchKernelGGL(scatter_kernel, dim3((uint32_t)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace kamera
