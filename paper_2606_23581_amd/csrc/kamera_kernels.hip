// gfx950 kernels of the Kamera chunk-reuse operator.
//
// rehydrate: K' = R(pos)(K + U W), V' = V + U_v W_v  (Eq. eq:operator, Sec. 3;
//            serve step of App. A).  One grouped launch over
//            (plane, chunk, layer, head, token block, column block).
// shift:     K' = R(delta) K in place (R(delta) R(p) = R(p + delta), Sec. 1).
// scatter:   bit copy of token rows into page-table slots (App. E, Sec. 6).
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
// Nothing goes through LDS except W (transposed once per workgroup) and the
// per-pair frequencies.

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
  int flags;
  int ldw;            // LDS row stride of W^T in elements
};

// position of token i of chunk c on each coordinate, as exact doubles
__device__ __forceinline__ void token_position(const RehydrateParams& P, int c, int i,
                                               double& pt, double& ph, double& pw) {
  if (P.pos_mode == 0) {                       // linear: p0 + i
    const double p = (double)P.chunk_pos[3 * c] + (double)i;
    pt = ph = pw = p;
  } else if (P.pos_mode == 1) {                // 32x32-style grid of patches
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

template <int NQ>
__device__ __forceinline__ void rotate_tile(f32x4 (&acc)[2 * NQ], int g, int pairing,
                                            const double* s_freq, const int* s_coord,
                                            double pt, double ph, double pw) {
  if (pairing == 0) {
    if constexpr (NQ % 2 == 0) {
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
    }
  } else {
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

template <int NQ>
__device__ void rehydrate_tile(const RehydrateParams& P, const TileCtx& T, int i0,
                               const uint16_t* __restrict__ Wt, const double* s_freq,
                               const int* s_coord) {
  const PlaneParams& Q = *T.Q;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int t = lane & 15;
  const int i = i0 + t;
  const bool valid = i < T.n_c;

  // ---- load the K (or V) tile straight into accumulator order ----
  u32x4 raw[NQ];
  const uint16_t* src = Q.in + (int64_t)T.c * Q.in_s[0] + (int64_t)T.l * Q.in_s[1] +
                        (int64_t)i * Q.in_s[2] + (int64_t)T.h * Q.in_s[3] + T.col0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) raw[q] = valid ? ld16(src + 8 * (g + 4 * q)) : u32x4{0, 0, 0, 0};

  const bool patched = (T.flags & kBlkPatch) && Q.m > 0;
  // ---- patch coefficients of this token (B operand) ----
  bf16x8 ub[4];
  if (patched) {
    const uint16_t* urow = Q.U + (int64_t)T.c * Q.u_s[0] + (int64_t)T.l * Q.u_s[1] +
                           (int64_t)T.h * Q.u_s[2] + (int64_t)i * Q.u_s[3];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      u32x4 v = u32x4{0, 0, 0, 0};
      if (s < Q.m_steps) {
        const int k0 = 32 * s + 8 * g;
        if (Q.u_vec) {
          if (valid && k0 < Q.m) v = ld16(urow + k0);
        } else if (valid) {
          uint32_t w4[4] = {0, 0, 0, 0};
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t b = (k0 + e < Q.m) ? urow[k0 + e] : 0u;
            w4[e >> 1] |= (e & 1) ? (b << 16) : b;
          }
          v = u32x4{w4[0], w4[1], w4[2], w4[3]};
        }
      }
      ub[s] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x4 acc[2 * NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    acc[2 * q][0] = bf_lo(raw[q].x);
    acc[2 * q][1] = bf_hi(raw[q].x);
    acc[2 * q][2] = bf_lo(raw[q].y);
    acc[2 * q][3] = bf_hi(raw[q].y);
    acc[2 * q + 1][0] = bf_lo(raw[q].z);
    acc[2 * q + 1][1] = bf_hi(raw[q].z);
    acc[2 * q + 1][2] = bf_lo(raw[q].w);
    acc[2 * q + 1][3] = bf_hi(raw[q].w);
  }

  const bool rotated = (T.flags & kBlkRotate) != 0;
  double pt = 0.0, ph = 0.0, pw = 0.0;
  if (rotated) token_position(P, T.c, i < T.n_c ? i : T.n_c - 1, pt, ph, pw);

  if (rotated && P.patch_post_rope)
    rotate_tile<NQ>(acc, g, P.rope.pairing, s_freq, s_coord, pt, ph, pw);

  if (patched) {
    // A operand row r = t: block column 8*(r/4) + 32*(mt/2) + 4*(mt%2) + r%4
    const int rbase = 8 * (t >> 2) + (t & 3);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s < Q.m_steps) {
#pragma unroll
        for (int mt = 0; mt < 2 * NQ; ++mt) {
          const int prow = rbase + 32 * (mt >> 1) + 4 * (mt & 1);
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(Wt + prow * T.ldw + 32 * s + 8 * g);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, ub[s], acc[mt], 0, 0, 0);
        }
      }
    }
  }

  if (rotated && !P.patch_post_rope)
    rotate_tile<NQ>(acc, g, P.rope.pairing, s_freq, s_coord, pt, ph, pw);

  // ---- round to bf16 and store ----
  if (!valid) return;
  int64_t dst;
  if (P.place.paged) {
    const int64_t slot = page_slot(P.place, T.c, i);
    if (slot < 0) return;
    dst = (int64_t)T.l * Q.out_s[1] + slot * Q.out_s[2] + (int64_t)T.h * Q.out_s[3];
  } else {
    const int rb = P.place.row_base ? P.place.row_base[T.c] : 0;
    dst = (int64_t)T.c * Q.out_s[0] + (int64_t)T.l * Q.out_s[1] + (int64_t)(rb + i) * Q.out_s[2] +
          (int64_t)T.h * Q.out_s[3];
  }
  uint16_t* drow = Q.out + dst + T.col0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    u32x4 o;
    o.x = pack_bf16x2(acc[2 * q][0], acc[2 * q][1]);
    o.y = pack_bf16x2(acc[2 * q][2], acc[2 * q][3]);
    o.z = pack_bf16x2(acc[2 * q + 1][0], acc[2 * q + 1][1]);
    o.w = pack_bf16x2(acc[2 * q + 1][2], acc[2 * q + 1][3]);
    st16(drow + 8 * (g + 4 * q), o);
  }
}

// Stage W^T of one column block into LDS: Wt[col][k], col in [0, 32*NQ),
// k in [0, 32*m_steps); columns outside the patch range and k >= m are zero.
template <int NQ>
__device__ void stage_w(const RehydrateParams& P, const TileCtx& T, uint16_t* Wt) {
  const PlaneParams& Q = *T.Q;
  const int m_pad = 32 * Q.m_steps;
  const int n_items = m_pad * (4 * NQ);
  const uint16_t* wbase = Q.W + (int64_t)T.c * Q.w_s[0] + (int64_t)T.l * Q.w_s[1] +
                          (int64_t)T.h * Q.w_s[2];
  for (int item = threadIdx.x; item < n_items; item += kThreads) {
    const int k = item % m_pad;
    const int cc = item / m_pad;
    const int colb = 8 * cc;                        // block column of the 8-chunk
    const int wcol = T.col0 + colb - Q.patch_lo;    // W column
    uint32_t w4[4] = {0, 0, 0, 0};
    if (k < Q.m && T.col0 + colb >= Q.patch_lo && T.col0 + colb + 8 <= Q.patch_hi) {
      const uint16_t* p = wbase + (int64_t)k * Q.w_s[3] + wcol;
      if (Q.w_vec) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(p);
        w4[0] = v.x; w4[1] = v.y; w4[2] = v.z; w4[3] = v.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) w4[e >> 1] |= (e & 1) ? ((uint32_t)p[e] << 16) : (uint32_t)p[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t wv = w4[e >> 1];
      Wt[(colb + e) * T.ldw + k] = (uint16_t)((e & 1) ? (wv >> 16) : (wv & 0xffffu));
    }
  }
}

template <int NQ>
__device__ void rehydrate_block(const RehydrateParams& P, TileCtx& T, int t_begin, int t_end,
                                uint16_t* Wt, double* s_freq, int* s_coord) {
  const PlaneParams& Q = *T.Q;
  const bool patched = (T.flags & kBlkPatch) && Q.m > 0;
  if (patched) stage_w<NQ>(P, T, Wt);
  if (T.flags & kBlkRotate) {
    const int half = P.rope.rope_dim / 2;
    for (int j = threadIdx.x; j < half; j += kThreads) {
      s_freq[j] = P.rope.rev_freq[j];
      s_coord[j] = P.rope.coord[j];
    }
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6;
  const int n_tiles = (t_end - t_begin + kTileTokens - 1) / kTileTokens;
  for (int tile = wave; tile < n_tiles; tile += kThreads / 64)
    rehydrate_tile<NQ>(P, T, t_begin + tile * kTileTokens, Wt, s_freq, s_coord);
}

__global__ __launch_bounds__(kThreads) void rehydrate_kernel(const RehydrateParams P) {
  extern __shared__ __align__(16) uint16_t lds_w[];
  __shared__ double s_freq[kMaxPairs];
  __shared__ int s_coord[kMaxPairs];

  const int64_t task = xcd_task(P.per_xcd);
  if (task >= P.n_tasks) return;
  const int pl = (P.n_planes == 2 && task >= P.plane[1].task_base) ? 1 : 0;
  const PlaneParams& Q = P.plane[pl];
  int64_t rem = task - Q.task_base;
  const int b = (int)(rem % Q.n_blocks);
  rem /= Q.n_blocks;
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
  T.flags = B.flags;
  T.ldw = 32 * Q.m_steps + 8;
  switch (B.nq) {
    case 1: rehydrate_block<1>(P, T, t_begin, t_end, lds_w, s_freq, s_coord); break;
    case 2: rehydrate_block<2>(P, T, t_begin, t_end, lds_w, s_freq, s_coord); break;
    case 3: rehydrate_block<3>(P, T, t_begin, t_end, lds_w, s_freq, s_coord); break;
    default: rehydrate_block<4>(P, T, t_begin, t_end, lds_w, s_freq, s_coord); break;
  }
}

hipError_t launch_rehydrate(const RehydrateParams& p, hipStream_t s) {
  int max_steps = 0;
  for (int k = 0; k < p.n_planes; ++k) max_steps = max_steps > p.plane[k].m_steps ? max_steps : p.plane[k].m_steps;
  const size_t lds = max_steps > 0 ? (size_t)128 * (32 * max_steps + 8) * sizeof(uint16_t) : 16;
  const int64_t grid = (int64_t)p.per_xcd * 8;
  hipLaunchKernelGGL(rehydrate_kernel, dim3((uint32_t)grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// shift: K' = R(delta) K on the rope band, in place
// ---------------------------------------------------------------------------

constexpr int kShiftUnroll = 4;

__global__ __launch_bounds__(kThreads) void shift_kernel(const ShiftParams P) {
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
// scatter: dense rows -> page-table slots, bit for bit
// ---------------------------------------------------------------------------

constexpr int kScatterUnroll = 4;

__global__ __launch_bounds__(kThreads) void scatter_kernel(const ScatterParams P) {
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
  const uint8_t* sbase = P.src + (int64_t)c * P.src_s[0] + (int64_t)l * P.src_s[1];
  uint8_t* pbase = P.pool + (int64_t)l * P.pool_s[0];
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
          v[u] = __builtin_nontemporal_load(
              reinterpret_cast<const u32x4*>(sbase + (int64_t)i * P.src_s[2] + 16 * vec));
          dp[u] = pbase + slot * P.pool_s[1] + 16 * vec;
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
