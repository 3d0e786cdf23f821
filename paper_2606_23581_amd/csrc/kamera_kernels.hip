// gfx950 kernels of the Kamera chunk-reuse operator.
//
// rehydrate: K' = R(pos)(K + U W), V' = V + U_v W_v  (Eq. eq:operator, Sec. 3;
//            serve step of App. A).  One grouped launch over
//            (plane, chunk, layer, head, token block, column block).  With a
//            per-chunk delta the keys are already rotated and move by delta
//            with a (removal) patch added at the target (Sec. 5, Table evict).
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

#include "kamera.h"
#include "kamera_launch.h"

namespace kamera {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st16(uint16_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// bf16 -> fp32 is exact: the 16 bits are the top half of the binary32 pattern
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 pair -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ uint32_t u4_get(const u32x4& v, int k) {
  return k == 0 ? v.x : (k == 1 ? v.y : (k == 2 ? v.z : v.w));
}

// cos/sin of 2*pi*(pos * rev_freq).  The product and its reduction to
// [-1/2, 1/2] revolution run in fp64 (positions up to 2^31 keep ~1e-9 rev of
// accuracy); the reduced angle goes to the hardware sin/cos, which take
// revolutions.
__device__ __forceinline__ void sincos_rev(double pos, double rev_freq, float& s, float& c) {
  const double rev = pos * rev_freq;
  const float r = static_cast<float>(rev - __builtin_rint(rev));
  s = __builtin_amdgcn_sinf(r);
  c = __builtin_amdgcn_cosf(r);
}

__device__ __forceinline__ int chunk_len(const Placement& pl, int c) {
  if (pl.chunk_tokens == nullptr) return pl.n_tokens;
  const int n = pl.chunk_tokens[c];
  return n < 0 ? 0 : (n > pl.n_tokens ? pl.n_tokens : n);
}

// Slot of token i of chunk c in a paged pool, or -1 for a page number outside
// the pool (flagged in the status word, never written).
__device__ __forceinline__ int64_t page_slot(const Placement& pl, int c, int i) {
  const int page = pl.page_table[(int64_t)c * pl.pt_stride + i / pl.page_size];
  if (page < 0 || page >= pl.n_pool_pages) {
    if (pl.status != nullptr) atomicOr(pl.status, KAMERA_STATUS_BAD_PAGE);
    return -1;
  }
  return (int64_t)page * pl.page_size + i % pl.page_size;
}

// The launch parameters are read in place from the kernel-argument segment.
// Taking the address of a by-value kernel parameter (its arrays are indexed
// with run-time values) would make the compiler copy the whole struct into
// scratch memory first.
template <typename T>
__device__ __forceinline__ const T& kernel_params() {
  return *static_cast<const T*>((const void*)__builtin_amdgcn_kernarg_segment_ptr());
}

// XCD-aware task index: workgroups are dealt round-robin to the 8 XCDs, so
// workgroup w runs on XCD w % 8.  Give each XCD a contiguous range of tasks so
// neighbouring tasks (same chunk/layer/head, same W factor) share its L2.
__device__ __forceinline__ int64_t xcd_task(int32_t per_xcd) {
  const int64_t w = blockIdx.x;
  return (w & 7) * (int64_t)per_xcd + (w >> 3);
}

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

// ---------------------------------------------------------------------------
// Tile I/O.  Global memory is accessed row-contiguously: one load or store
// instruction of a wave covers 64 consecutive 16-byte chunks, i.e. whole
// token rows (4 rows of a 128-column block).  The MFMA layout above wants 4
// lanes per row instead, so each wave passes its tile through a private LDS
// buffer (padded rows keep both access orders free of bank conflicts).  The
// direct path (MFMA layout straight from global memory) remains for blocks of
// 96 columns and for U rows that are not 16-byte aligned.
// ---------------------------------------------------------------------------

constexpr int kRowPad = 16;                          // LDS row padding, bytes

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

template <int NQ, int MS, int ROT, bool RELOC>
__device__ __forceinline__ void tile_compute(const RehydrateParams& P, const TileCtx& T, int i0,
                                             const TileRegs<NQ, MS>& R, const uint16_t* __restrict__ Wt,
                                             uint8_t* tile_lds, const double* s_freq,
                                             const int* s_coord) {
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

  f32x4 acc[2 * NQ];
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
    if constexpr (RELOC) {
      const double dt = (double)P.delta[3 * T.c], dh = (double)P.delta[3 * T.c + 1],
                   dw = (double)P.delta[3 * T.c + 2];
      if (P.patch_post_rope)
        rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, dt, dh, dw);
      else
        rotate_tile<NQ, ROT>(acc, g, s_freq, s_coord, dt - pt, dh - ph, dw - pw);
    } else if (P.patch_post_rope) {
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

  if constexpr (ROT != 0) {
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
                                                uint8_t* lds, double* s_freq, int* s_coord) {
  uint16_t* Wt = reinterpret_cast<uint16_t*>(lds);
  const int wave = threadIdx.x >> 6;
  uint8_t* tile_lds = lds + 128 * (32 * MS + 8) * 2 + wave * tile_lds_bytes();
  if constexpr (MS > 0) {
    if (T.patched) stage_w<NQ>(T, Wt);
  }
  if constexpr (ROT != 0) {
    const int half = P.rope.rope_dim / 2;
    for (int j = threadIdx.x; j < half; j += kThreads) {
      s_freq[j] = P.rope.rev_freq[j];
      s_coord[j] = P.rope.coord[j];
    }
  }
  __syncthreads();
  constexpr int kWaves = kThreads / 64;
  const int n_tiles = (t_end - t_begin + kTileTokens - 1) / kTileTokens;
  for (int tile = wave; tile < n_tiles; tile += kWaves) {
    TileRegs<NQ, MS> R;
    tile_load<NQ, MS>(T, t_begin + tile * kTileTokens, R);
    tile_compute<NQ, MS, ROT, RELOC>(P, T, t_begin + tile * kTileTokens, R, Wt, tile_lds, s_freq, s_coord);
  }
}

// RELOC: the keys are already rotated and move by the chunk's delta
template <int MS, bool RELOC>
__global__ __launch_bounds__(kThreads, MS == 4 || RELOC ? 3 : 4) void rehydrate_kernel(const RehydrateParams /*by value, read in place*/) {
  const RehydrateParams& P = kernel_params<RehydrateParams>();
  extern __shared__ __align__(16) uint8_t lds_dyn[];
  __shared__ double s_freq[kMaxPairs];
  __shared__ int s_coord[kMaxPairs];

  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  // tasks of one (chunk, layer, head, token block) are adjacent: the key
  // blocks (rotation, VALU-heavier) run next to the value blocks (pure streams)
  int64_t rem = task / P.blocks_per_group;
  const int r = (int)(task % P.blocks_per_group);
  const int pl = (P.n_planes == 2 && r >= P.plane[1].block_base) ? 1 : 0;
  const PlaneParams& Q = P.plane[pl];
  const int b = r - Q.block_base;
  const int tb = (int)(rem % P.n_tblk);
  rem /= P.n_tblk;
  TileCtx T;
  T.Q = &Q;
  T.h = (int)(rem % P.n_heads);
  rem /= P.n_heads;
  T.l = (int)(rem % P.n_layers);
  T.c = (int)(rem / P.n_layers);
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
    case 1 * 3 + 0: rehydrate_block<1, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 1 * 3 + 2: rehydrate_block<1, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 2 * 3 + 0: rehydrate_block<2, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 2 * 3 + 1: rehydrate_block<2, MS, 1, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 2 * 3 + 2: rehydrate_block<2, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 3 * 3 + 0: rehydrate_block<3, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 3 * 3 + 2: rehydrate_block<3, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 4 * 3 + 0: rehydrate_block<4, MS, 0, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 4 * 3 + 1: rehydrate_block<4, MS, 1, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 4 * 3 + 2: rehydrate_block<4, MS, 2, RELOC>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    default: break;                              // rejected on the host (NeoX needs an even NQ)
  }
}

// ---------------------------------------------------------------------------
// rehydrate, row-group form: rows of <= 8 heads of 128 columns with one
// 128-column block per head (the rope band, if any, is the whole head), rank
// <= 64, positions linear or on a grid, no relocation.  A workgroup of 8 waves owns (plane,
// chunk, layer, token block) for every head of the row; wave h computes head
// h in the register layout of the per-head kernel above (lane (g, t) holds
// chunks g, g+4, g+8, g+12 of token t).  Per 16-token tile all heads move
//   HBM -> registers (two tiles in flight) -> LDS -> MFMA layout -> LDS -> HBM
// and the store phase writes every token's whole row of heads: a pool page of
// 16 tokens is written as one contiguous run instead of one 256-byte piece
// per head.  W^T of every head sits in registers for the whole token block,
// and the block's page numbers in LDS.  Tile loads and stores are buffer
// instructions whose out-of-range lanes (ragged tails, missing heads, pages
// outside the pool) read zeros or write nothing, so the tile loop issues the
// same memory instructions on every path and a tile's loads are awaited
// without waiting for the tile issued after it.
// ---------------------------------------------------------------------------

constexpr int kRgDepth = 2;                                // tiles in flight per thread
constexpr int kRgThreads = 512;                            // one wave per head
constexpr int kRgHeads = kRgMaxHeads;
constexpr int kRgKRow = 256 + kRowPad;                     // LDS bytes per (head, token) K row
__host__ __device__ constexpr int rg_u_row(int ms) { return 64 * ms + kRowPad; }
__host__ __device__ constexpr int rg_buf_bytes(int ms) {
  return kRgHeads * kTileTokens * (kRgKRow + rg_u_row(ms));
}
constexpr int kRgWtRow = 64 * 2 + kRowPad;                 // W^T staging row: 64 ranks + pad
constexpr int kRgMaxBlock = 1024;                          // tokens per row-group task
__host__ __device__ constexpr int rg_lds_bytes(int ms) {
  return (2 * rg_buf_bytes(ms) > 4 * 128 * kRgWtRow ? 2 * rg_buf_bytes(ms) : 4 * 128 * kRgWtRow) +
         kRgMaxBlock * 4;
}

constexpr int kRgKVec = kRgHeads * kTileTokens * 16 / kRgThreads;   // K vectors per thread and tile
constexpr int kRgUVec = kRgHeads * kTileTokens * 8 / kRgThreads;    // U vectors (rank 64)

struct RgRegs {              // one tile's global loads, in flight until the LDS write
  u32x4 k[kRgKVec];
  u32x4 u[kRgUVec];
};

constexpr uint32_t kRgOob = 0x7ffffff0u;                    // byte offset past every buffer extent
constexpr int kRgBufWord3 = 0x00020000;                    // raw buffer, 32-bit data format

struct RgTask {
  const PlaneParams* Q;
  int c, l, n_c, H;
  int m, m_steps;            // rank at this layer
  int t_end;                 // end of the task's token block
  bool in_head_major;        // rows of one head lie closer together than the heads
  bool out_head_major;
  int s_in2, s_in3;          // input token / head strides (elements)
  int s_u3, s_u2;            // U token / head strides
  int s_o2, s_o3;            // output row (slot) / head strides
  double cp0, cp1, cp2;      // chunk position (t, h, w) of token 0
  __amdgpu_buffer_rsrc_t rin, ru, rout;   // (chunk, layer) slabs of input, U and output
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rg_rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kRgBufWord3);
}

// 16-byte vector v of a tile (16 tokens x H heads x 16 chunks) -> (head, token)
__device__ __forceinline__ void rg_vec(int v, int H, bool head_major, int& h, int& t) {
  if (head_major) {
    h = v >> 8;
    t = (v >> 4) & 15;
  } else {
    t = v / (16 * H);
    h = (v >> 4) % H;
  }
}

template <int MS>
__device__ __forceinline__ void rg_load(const RgTask& T, int i0, RgRegs& R) {
  const int tid = threadIdx.x;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + kRgThreads * k;
    int h, t;
    rg_vec(v, T.H, T.in_head_major, h, t);
    const int i = i0 + t;
    const uint32_t off = (v < nv && i < T.t_end) ? 2u * (uint32_t)(i * T.s_in2 + h * T.s_in3 + 8 * (v & 15)) : kRgOob;
    R.k[k] = __builtin_amdgcn_raw_buffer_load_b128(T.rin, (int)off, 0, 2);
  }
  if constexpr (MS > 0) {
    const int cpr = 4 * (T.m_steps > 0 ? T.m_steps : 1);   // 16-byte chunks per U row (rank padded to 32)
#pragma unroll
    for (int k = 0; k < kRgUVec; ++k) {
      const int v = tid + kRgThreads * k;
      const int h = v / (kTileTokens * cpr), t = (v / cpr) % kTileTokens, c = v % cpr;
      const int i = i0 + t;
      const uint32_t off = (h < T.H && 8 * c < T.m && i < T.t_end)
                               ? 2u * (uint32_t)(h * T.s_u2 + i * T.s_u3 + 8 * c) : kRgOob;
      R.u[k] = __builtin_amdgcn_raw_buffer_load_b128(T.ru, (int)off, 0, 2);
    }
  }
}

template <int MS>
__device__ __forceinline__ void rg_to_lds(const RgTask& T, const RgRegs& R, uint8_t* buf) {
  const int tid = threadIdx.x;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + kRgThreads * k;
    int h, t;
    rg_vec(v, T.H, T.in_head_major, h, t);
    if (v < nv) *reinterpret_cast<u32x4*>(buf + (h * kTileTokens + t) * kRgKRow + 16 * (v & 15)) = R.k[k];
  }
  if constexpr (MS > 0) {
    if (T.m_steps > 0) {
      const int cpr = 4 * T.m_steps;
#pragma unroll
      for (int k = 0; k < kRgUVec; ++k) {
        const int v = tid + kRgThreads * k;
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
          *reinterpret_cast<u32x4*>(buf + kRgHeads * kTileTokens * kRgKRow + (h * kTileTokens + t) * rg_u_row(MS) +
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

// one wave: head h of the tile in LDS, result written back in place
template <int MS, int ROT>
__device__ __forceinline__ void rg_compute(const RehydrateParams& P, const RgTask& T, int i0, int h,
                                           const u32x4 (&wa)[8][MS > 0 ? MS : 1], uint8_t* buf,
                                           const double* s_freq, const int* s_coord) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, t = lane & 15;
  uint8_t* krow = buf + (h * kTileTokens + t) * kRgKRow;
  u32x4 kc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) kc[q] = *reinterpret_cast<const u32x4*>(krow + 16 * (g + 4 * q));
  f32x4 acc[8];
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
    if (P.patch_post_rope) rg_rotate<ROT>(acc, g, s_freq, s_coord, pt, ph, pw);
  }
  if constexpr (MS > 0) {
    const uint8_t* urow = buf + kRgHeads * kTileTokens * kRgKRow + (h * kTileTokens + t) * rg_u_row(MS);
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
  if constexpr (ROT != 0) {
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
__device__ __forceinline__ void rg_store(const RehydrateParams& P, const RgTask& T, int t_begin, int i0,
                                         const uint8_t* buf, const int* s_page) {
  const int tid = threadIdx.x;
  const int nv = T.H * kTileTokens * 16;
#pragma unroll
  for (int k = 0; k < kRgKVec; ++k) {
    const int v = tid + kRgThreads * k;
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

// W rows of one staging item: head h, ranks k0..k0+3, columns colb..colb+7
__device__ __forceinline__ void rg_load_w(const RgTask& T, int h, int k0, int colb, uint32_t (&w)[4][4]) {
  const PlaneParams& Q = *T.Q;
  const uint16_t* wbase = Q.W + (int64_t)T.c * Q.w_s[0] + (int64_t)T.l * Q.w_s[1] + (int64_t)h * Q.w_s[2];
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
__device__ __forceinline__ void rg_put_w(int hq, int k0, int colb, const uint32_t (&w)[4][4], uint8_t* lds) {
  uint8_t* base = lds + hq * 128 * kRgWtRow;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int sh = (e & 1) ? 16 : 0;
    const uint32_t r0 = (w[0][e >> 1] >> sh) & 0xffffu, r1 = (w[1][e >> 1] >> sh) & 0xffffu;
    const uint32_t r2 = (w[2][e >> 1] >> sh) & 0xffffu, r3 = (w[3][e >> 1] >> sh) & 0xffffu;
    uint2 v;
    v.x = r0 | (r1 << 16);
    v.y = r2 | (r3 << 16);
    *reinterpret_cast<uint2*>(base + (colb + e) * kRgWtRow + 2 * k0) = v;
  }
}

template <int MS, int ROT>
__device__ __forceinline__ void rg_run(const RehydrateParams& P, const RgTask& T, int t_begin, int t_end,
                                       uint8_t* lds, const double* s_freq, const int* s_coord) {
  const int tid = threadIdx.x;
  const int h = tid >> 6;                       // wave = head
  const int lane = tid & 63;
  const bool active = h < T.H;
  const int n_tiles = (t_end - t_begin + kTileTokens - 1) / kTileTokens;
  int* s_page = reinterpret_cast<int*>(lds + rg_lds_bytes(MS) - kRgMaxBlock * 4);

  // set-up loads, in flight together: the block's pool pages, the first
  // tiles and the W rows of heads 0..3 (two staging items per thread)
  int page[kRgMaxBlock / kRgThreads];
#pragma unroll
  for (int k = 0; k < kRgMaxBlock / kRgThreads; ++k) {
    const int j = t_begin + tid + kRgThreads * k;
    page[k] = -1;
    if (P.place.paged && j < t_end) {
      page[k] = P.place.page_table[(int64_t)T.c * P.place.pt_stride + j / P.place.page_size];
      if (page[k] < 0 || page[k] >= P.place.n_pool_pages) {
        if (P.place.status != nullptr) atomicOr(P.place.status, KAMERA_STATUS_BAD_PAGE);
        page[k] = -1;
      }
    }
  }
  RgRegs R[kRgDepth];
#pragma unroll
  for (int d = 0; d < kRgDepth; ++d)
    if (d < n_tiles) rg_load<MS>(T, t_begin + d * kTileTokens, R[d]);
  // staging item = (head, rank quad, column chunk); item tid + 512 * r
  const int k0 = 4 * ((tid >> 4) & 15), colb = 8 * (tid & 15), hq = tid >> 8;   // hq in {0, 1}
  const bool w_item = MS > 0 && T.m_steps > 0 && k0 < 32 * T.m_steps;
  uint32_t w[2][4][4];
  if (w_item) {
    rg_load_w(T, hq, k0, colb, w[0]);
    rg_load_w(T, hq + 2, k0, colb, w[1]);
  }
#pragma unroll
  for (int k = 0; k < kRgMaxBlock / kRgThreads; ++k)
    if (P.place.paged && t_begin + tid + kRgThreads * k < t_end) s_page[tid + kRgThreads * k] = page[k];

  // W^T into registers: A operand of M-tile mt, K-step k for lane (g, t):
  // column 8*(t/4) + t%4 + 32*(mt/2) + 4*(mt%2), ranks 32k + 8g .. +7.
  // Two rounds of four heads through LDS: round r holds heads 4r + hq and
  // 4r + 2 + hq of the thread's items.
  u32x4 wa[8][MS > 0 ? MS : 1];
  if constexpr (MS > 0) {
    const int g = lane >> 4, t = lane & 15;
#pragma unroll
    for (int round = 0; round < 2; ++round) {
      if (round == 1 && w_item) {
        rg_load_w(T, hq + 4, k0, colb, w[0]);
        rg_load_w(T, hq + 6, k0, colb, w[1]);
      }
      if (w_item) {
        rg_put_w(hq, k0, colb, w[0], lds);
        rg_put_w(hq + 2, k0, colb, w[1], lds);
      }
      __syncthreads();
      if ((h >> 2) == round) {
        const uint8_t* hb = lds + (h & 3) * 128 * kRgWtRow;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) {
          const int col = 8 * (t >> 2) + (t & 3) + 32 * (mt >> 1) + 4 * (mt & 1);
#pragma unroll
          for (int k = 0; k < MS; ++k)
            wa[mt][k] = (k < T.m_steps) ? *reinterpret_cast<const u32x4*>(hb + col * kRgWtRow + 64 * k + 16 * g)
                                        : u32x4{0, 0, 0, 0};
        }
      }
      __syncthreads();
    }
  }

  // kRgDepth register sets (tiles in flight) and two LDS buffers: tile tt
  // uses set tt % kRgDepth and buffer tt % 2; two barriers per tile
  auto step = [&](int tt, RgRegs& R) {
    const int i0 = t_begin + tt * kTileTokens;
    uint8_t* buf = lds + (tt & 1) * rg_buf_bytes(MS);
    rg_to_lds<MS>(T, R, buf);
    if (tt + kRgDepth < n_tiles) rg_load<MS>(T, i0 + kRgDepth * kTileTokens, R);
    __syncthreads();
    if (active) rg_compute<MS, ROT>(P, T, i0, h, wa, buf, s_freq, s_coord);
    __syncthreads();
    rg_store(P, T, t_begin, i0, buf, s_page);
  };
  for (int tile = 0; tile < n_tiles; tile += kRgDepth) {
#pragma unroll
    for (int d = 0; d < kRgDepth; ++d)
      if (tile + d < n_tiles) step(tile + d, R[d]);
  }
}

template <int MS>
__global__ __launch_bounds__(kRgThreads, 1) void rehydrate_rows_kernel(const RehydrateParams /*by value, read in place*/) {
  const RehydrateParams& P = kernel_params<RehydrateParams>();
  extern __shared__ __align__(16) uint8_t lds_dyn[];
  __shared__ double s_freq[kMaxPairs];
  __shared__ int s_coord[kMaxPairs];

  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  // the planes (K, V) of one (chunk, layer, token block) are adjacent tasks
  const int pl = (int)(task % P.n_planes);
  int64_t rem = task / P.n_planes;
  const int tb = (int)(rem % P.n_tblk);
  rem /= P.n_tblk;
  RgTask T;
  T.Q = &P.plane[pl];
  const PlaneParams& Q = *T.Q;
  T.l = (int)(rem % P.n_layers);
  T.c = (int)(rem / P.n_layers);
  T.H = P.n_heads;
  T.n_c = chunk_len(P.place, T.c);
  const int t_begin = tb * P.token_block;
  if (t_begin >= T.n_c) return;                 // uniform: the whole workgroup leaves
  const int t_end = min(t_begin + P.token_block, T.n_c);
  T.t_end = t_end;
  T.m = Q.m;
  if (Q.layer_rank != nullptr) {
    const int r = Q.layer_rank[T.l];
    T.m = r < 0 ? 0 : (r < Q.m ? r : Q.m);
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
  T.rin = rg_rsrc(Q.in + (int64_t)T.c * Q.in_s[0] + (int64_t)T.l * Q.in_s[1], Q.in_rec);
  T.ru = rg_rsrc(Q.U != nullptr ? Q.U + (int64_t)T.c * Q.u_s[0] + (int64_t)T.l * Q.u_s[1] : Q.in, Q.U != nullptr ? Q.u_rec : 0);
  // paged: the layer's pool; dense: the chunk's rows from its row base on
  const int64_t out_base = P.place.paged ? 0
                           : (int64_t)T.c * Q.out_s[0] +
                                 (int64_t)(P.place.row_base ? P.place.row_base[T.c] : 0) * Q.out_s[2];
  T.rout = rg_rsrc(Q.out + out_base + (int64_t)T.l * Q.out_s[1], Q.out_rec);
  T.cp0 = T.cp1 = T.cp2 = 0.0;
  if (P.chunk_pos != nullptr) {
    T.cp0 = (double)P.chunk_pos[3 * T.c];
    T.cp1 = (double)P.chunk_pos[3 * T.c + 1];
    T.cp2 = (double)P.chunk_pos[3 * T.c + 2];
  }
  const int rot = (Q.blk[0].flags & kBlkRotate) ? (P.rope.pairing == 0 ? 1 : 2) : 0;
  if (rot != 0) {
    const int half = P.rope.rope_dim / 2;
    for (int j = threadIdx.x; j < half; j += kRgThreads) {
      s_freq[j] = P.rope.rev_freq[j];
      s_coord[j] = P.rope.coord[j];
    }
  }
  switch (rot) {
    case 0: rg_run<MS, 0>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    case 1: rg_run<MS, 1>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
    default: rg_run<MS, 2>(P, T, t_begin, t_end, lds_dyn, s_freq, s_coord); break;
  }
}

hipError_t launch_rehydrate(const RehydrateParams& p, hipStream_t s) {
  int max_steps = 0;
  for (int k = 0; k < p.n_planes; ++k) max_steps = max_steps > p.plane[k].m_steps ? max_steps : p.plane[k].m_steps;
  const int ms = max_steps == 0 ? 0 : (max_steps <= 2 ? max_steps : 4);   // template rank steps
  const size_t lds = (size_t)128 * (32 * ms + 8) * sizeof(uint16_t) +
                     (size_t)(kThreads / 64) * tile_lds_bytes();
  const dim3 grid((uint32_t)((int64_t)p.per_xcd * 8)), block(kThreads);
  if (p.row_group) {
    // the LDS limit is raised once per device (a race only repeats the calls)
    static bool attr_set[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || !attr_set[dev]) {
      e = hipFuncSetAttribute((const void*)rehydrate_rows_kernel<0>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              rg_lds_bytes(0));
      if (e == hipSuccess)
        e = hipFuncSetAttribute((const void*)rehydrate_rows_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                rg_lds_bytes(1));
      if (e == hipSuccess)
        e = hipFuncSetAttribute((const void*)rehydrate_rows_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                rg_lds_bytes(2));
      if (e != hipSuccess) return e;
      if (dev >= 0 && dev < 64) attr_set[dev] = true;
    }
    const dim3 rblock(kRgThreads);
    switch (max_steps) {
      case 0: hipLaunchKernelGGL((rehydrate_rows_kernel<0>), grid, rblock, rg_lds_bytes(0), s, p); break;
      case 1: hipLaunchKernelGGL((rehydrate_rows_kernel<1>), grid, rblock, rg_lds_bytes(1), s, p); break;
      default: hipLaunchKernelGGL((rehydrate_rows_kernel<2>), grid, rblock, rg_lds_bytes(2), s, p); break;
    }
    return hipGetLastError();
  }
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
  const int tb = (int)(task % P.n_tblk);
  const int l = (int)((task / P.n_tblk) % P.n_layers);
  const int c = (int)(task / ((int64_t)P.n_tblk * P.n_layers));
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
  const int tb = (int)(task % P.n_tblk);
  const int l = (int)((task / P.n_tblk) % P.n_layers);
  const int c = (int)(task / ((int64_t)P.n_tblk * P.n_layers));
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
