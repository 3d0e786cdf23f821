// gfx950 kernels of the compile-side patch forming (App. A compile step):
// the top-m singular triplets of each deficit Delta (n x d) as the stored
// patch, W = V_m^T and U = Delta V_m (the singular values folded in).
//
// form_patch_kernel: one 1024-thread workgroup per (chunk, layer, head) unit,
// everything in LDS (d is padded to dp, a multiple of 16, with zero rows and
// columns):
//   1. Gram matrix G = Delta^T Delta at fp32 accuracy on bf16 MFMA (16x16x32):
//      Delta split exactly into three bf16 parts, six products per tile,
//      streamed in 64-row tiles with the next tile's loads in flight during
//      the products;
//   2. the m largest eigenpairs of G, by default (sweeps == 0) from its
//      tridiagonal form: Householder reduction, multisection on Sturm counts,
//      twisted-factorisation vectors, back-transformation (tridiag_solve
//      below).  A unit whose vectors fail that solver's checks (exactly
//      multiple eigenvalues) forms G again and takes the other method:
//   2b. block Jacobi on G: the indices form dp/8 blocks of 8; each step pairs
//      the blocks round-robin (circle method) into dp/16 groups of 16
//      indices; one wave per group runs one cyclic Jacobi sweep on the
//      group's 16x16 principal submatrix, accumulating its rotation Q; then
//      G <- J^T G J and V <- V J with J = diag(Q_group) as 16x16 tile
//      products on fp32 MFMA.  Sweeps stop once the off-diagonal mass is
//      negligible against the diagonal;
//   3. (after Jacobi) rank the eigenvalues (diag G) of the real indices,
//      keep the m largest;
//   4. W[k] = V[:, order[k]]^T, rounded to bf16, and sigma.
// form_u_kernel then forms U = Delta W^T from the stored W (below).
// With an orbit (Sec. 5, reorder) Delta is the mean of the members' deficits,
// formed on the fly wherever Delta is read.
// The eigenvalues of G are the squared singular values of Delta and its
// eigenvectors the right singular vectors, so U W is the rank-m truncation.
// Padded indices keep zero rows and columns: every rotation that touches
// one is the identity, so they never mix with the real spectrum.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kamera.h"
#include "kamera_launch.h"

namespace kamera {

namespace {

typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int kFormThreads = 1024;
constexpr int kWaves = kFormThreads / 64;
constexpr int kGramRows = 64;          // Delta rows per staged tile of the Gram product
constexpr int kBlk = 8;                // block-Jacobi block width
constexpr int kGrp = 2 * kBlk;         // indices of one rotated group (two blocks)
constexpr int kLdQ = kGrp + 1;         // padded row stride of a group's 16x16 scratch
constexpr int kFormFallbackSweeps = 12; // Jacobi limit after a failed tridiagonal solve

__host__ __device__ inline int pad16(int d) { return (d + 15) & ~15; }
// bf16 offset of rows 8 j .. 8 j + 7 of column c in a staged Gram part:
// columns of kGramRows rows, their 16-byte pieces permuted by (c >> 1) & 7,
// so that the 32 lanes of a half wave reading 8-row pieces of 16 consecutive
// columns (two pieces each), and 16 lanes storing one piece of consecutive
// columns, touch distinct banks (16-byte reads are served per half wave over
// 512 bytes of banks, 16-byte stores per quarter wave over 256 bytes)
__device__ __forceinline__ int gram_slot(int c, int j) { return c * kGramRows + 8 * (j ^ ((c >> 1) & 7)); }
// row stride of G and V: == 2 (mod 32), so an MFMA operand load of 16 rows
// x 2 columns (half a wave) and a 16-row tile's row pieces fall on distinct banks
__host__ __device__ inline int gv_ld(int dp) { return dp + ((2 - dp) % 32 + 32) % 32; }

// circle method over `n` items at `step`: the (smaller, larger) members of pair k
__device__ __forceinline__ void circle_pair(int n, int step, int k, int& a, int& b) {
  const int pa = k == 0 ? 0 : 1 + (k - 1 + step) % (n - 1);
  const int pb = 1 + (n - 2 - k + step) % (n - 1);
  a = pa < pb ? pa : pb;
  b = pa < pb ? pb : pa;
}

// global index of local index r (0..15) of the group made of blocks (bi, bj)
__device__ __forceinline__ int group_index(int bi, int bj, int r) {
  return r < kBlk ? kBlk * bi + r : kBlk * bj + (r - kBlk);
}

__device__ __forceinline__ f32x4v mfma4(float a, float b, f32x4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t to_bf16_rne(float x) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  f32x2 v = {x, 0.0f};
  const bf16x2 r = __builtin_convertvector(v, bf16x2);
  return (uint16_t)(__builtin_bit_cast(uint32_t, r) & 0xffffu);
}

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

// eight bf16 (element 2q in the low half of word q) from fp32 values
__device__ __forceinline__ u32x4v pack_bf16x8(const float (&x)[8]) {
  u32x4v r;
#pragma unroll
  for (int q = 0; q < 4; ++q) r[q] = (uint32_t)to_bf16_rne(x[2 * q]) | ((uint32_t)to_bf16_rne(x[2 * q + 1]) << 16);
  return r;
}

// x = hi + mid + lo exactly, each part bf16 (RNE): bf16 keeps 8 significant
// bits, so x - hi and x - hi - mid are exact in fp32 and the last remainder
// has at most 8 significant bits left (outside the subnormal range)
__device__ __forceinline__ void split3_bf16x8(const float (&x)[8], u32x4v& hi, u32x4v& mid, u32x4v& lo) {
  float r[8], q[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = x[e] - __uint_as_float((uint32_t)to_bf16_rne(x[e]) << 16);
#pragma unroll
  for (int e = 0; e < 8; ++e) q[e] = r[e] - __uint_as_float((uint32_t)to_bf16_rne(r[e]) << 16);
  hi = pack_bf16x8(x);
  mid = pack_bf16x8(r);
  lo = pack_bf16x8(q);
}

__device__ __forceinline__ float block_sum(float v, float* red) {
  // wave reduction, then across the 16 waves through LDS
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < kFormThreads / 64; ++w) s += red[w];
  return s;
}

// The workgroup's dynamic LDS (one unit's working set).
extern __shared__ __align__(16) float form_lds[];

// Rotation (c, s) = (cos, sin) and t = tan that zero a[p][q] of the 2x2
// symmetric block [[app, apq], [apq, aqq]]: t is the smaller root of
// t^2 + 2 theta t - 1 = 0 with theta = (aqq - app) / (2 apq); no rotation
// when apq is negligible.  Hardware reciprocal and (reciprocal) square root:
// c^2 + s^2 = 1 to a few ulp, which is all the iteration needs.  Branch free.
__device__ __forceinline__ void rotation(float app, float aqq, float apq, float& c, float& s, float& t) {
  const bool act = fabsf(apq) > 1e-30f;
  const float theta = (aqq - app) * __builtin_amdgcn_rcpf(2.f * (act ? apq : 1.f));
  const float tt = (theta >= 0.f ? 1.f : -1.f) *
                   __builtin_amdgcn_rcpf(fabsf(theta) + __builtin_amdgcn_sqrtf(fmaf(theta, theta, 1.f)));
  t = act ? tt : 0.f;
  c = __builtin_amdgcn_rsqf(fmaf(t, t, 1.f));
  s = t * c;
}

// One cyclic Jacobi sweep, by one wave, on a group's 16x16 symmetric matrix S
// (at form_lds + so, row stride kLdQ); Q (at form_lds + qo, identity on entry)
// accumulates the rotations, so that on exit S = Q^T S_in Q.  Lane (kr, kc) =
// (lane / 8, lane % 8) owns the 2x2 block of S on the rows of pair kr and the
// columns of pair kc, and rows kr and kr + 8 of Q on the columns of pair kc;
// it derives both pairs' rotations itself from the values it reads, so a
// step is one round of reads followed by one round of writes.  The wave's LDS
// accesses are performed in program order, so no barrier is needed.
__device__ __forceinline__ void group_sweep(int so, int qo, int lane, float* G, int ld, int bi, int bj) {
  const int kr = lane >> 3, kc = lane & 7;
  // circle positions of both pairs at step 0; every step moves positions
  // 1..15 on by one (position 0 stays)
  int ra = kr, rb = 15 - kr;
  int ca = kc, cb = 15 - kc;
  int p = 0, q = 0, p2 = 0, q2 = 0;
  float na = 0.f, nb = 0.f, ne = 0.f, nf = 0.f;
#pragma unroll 3
  for (int st = 0; st < kGrp - 1; ++st) {
    p = min(ra, rb);
    q = max(ra, rb);
    p2 = min(ca, cb);
    q2 = max(ca, cb);
    const float rpp = form_lds[so + p * kLdQ + p], rqq = form_lds[so + q * kLdQ + q];
    const float rpq = form_lds[so + p * kLdQ + q];
    const float cpp = form_lds[so + p2 * kLdQ + p2], cqq = form_lds[so + q2 * kLdQ + q2];
    const float cpq = form_lds[so + p2 * kLdQ + q2];
    const float a0 = form_lds[so + p * kLdQ + p2], b0 = form_lds[so + p * kLdQ + q2];
    const float e0 = form_lds[so + q * kLdQ + p2], f0 = form_lds[so + q * kLdQ + q2];
    const float qp0 = form_lds[qo + kr * kLdQ + p2], qq0 = form_lds[qo + kr * kLdQ + q2];
    const float qp1 = form_lds[qo + (kr + 8) * kLdQ + p2], qq1 = form_lds[qo + (kr + 8) * kLdQ + q2];
    float c1, s1, t1, c2, s2, t2;
    rotation(rpp, rqq, rpq, c1, s1, t1);
    rotation(cpp, cqq, cpq, c2, s2, t2);
    const float a1 = c1 * a0 - s1 * e0, e1 = s1 * a0 + c1 * e0;
    const float b1 = c1 * b0 - s1 * f0, f1 = s1 * b0 + c1 * f0;
    na = c2 * a1 - s2 * b1;
    nb = s2 * a1 + c2 * b1;
    ne = c2 * e1 - s2 * f1;
    nf = s2 * e1 + c2 * f1;
    if (kr == kc) {
      // the pivot block (same four addresses): exact diagonal update,
      // off-diagonal zeroed
      na = a0 - t1 * b0;
      nf = f0 + t1 * b0;
      nb = 0.f;
      ne = 0.f;
    }
    form_lds[so + p * kLdQ + p2] = na;
    form_lds[so + p * kLdQ + q2] = nb;
    form_lds[so + q * kLdQ + p2] = ne;
    form_lds[so + q * kLdQ + q2] = nf;
    form_lds[qo + kr * kLdQ + p2] = c2 * qp0 - s2 * qq0;
    form_lds[qo + kr * kLdQ + q2] = s2 * qp0 + c2 * qq0;
    form_lds[qo + (kr + 8) * kLdQ + p2] = c2 * qp1 - s2 * qq1;
    form_lds[qo + (kr + 8) * kLdQ + q2] = s2 * qp1 + c2 * qq1;
    __builtin_amdgcn_wave_barrier();
    ra = ra == 0 ? 0 : (ra == 15 ? 1 : ra + 1);
    rb = rb == 15 ? 1 : rb + 1;
    ca = ca == 0 ? 0 : (ca == 15 ? 1 : ca + 1);
    cb = cb == 15 ? 1 : cb + 1;
  }
  // The last step wrote every entry of S = Q^T G_gg Q: the group's diagonal
  // tile of the rotated G.  Lanes on and above the pair diagonal store their
  // 2x2 block with its mirror, so G stays exactly symmetric.
  if (kr <= kc) {
    const int gp = group_index(bi, bj, p), gq = group_index(bi, bj, q);
    const int gp2 = group_index(bi, bj, p2), gq2 = group_index(bi, bj, q2);
    G[gp * ld + gp2] = na;
    G[gp * ld + gq2] = nb;
    G[gq * ld + gp2] = ne;
    G[gq * ld + gq2] = nf;
    G[gp2 * ld + gp] = na;
    G[gq2 * ld + gp] = nb;
    G[gp2 * ld + gq] = ne;
    G[gq2 * ld + gq] = nf;
  }
}

// Rows i0 .. i0 + 7 of column j of the (orbit-mean) deficit (zero past n
// rows or d columns); a wave's lanes take consecutive columns, so each row's
// loads are one contiguous piece.  Orbit members are read two at a time, all
// their loads issued before the sums, which keep the members' order.
__device__ __forceinline__ void load_col8(const FormParams& P, const float* delta, int i0, int j, int n, int d,
                                          float (&x)[8]) {
  const float* v = delta + (int64_t)i0 * P.delta_s[3] + j;
  bool ok[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    ok[e] = j < d && i0 + e < n;
    x[e] = ok[e] ? v[(int64_t)e * P.delta_s[3]] : 0.f;
  }
  if (P.n_orbit > 1) {
    for (int o = 1; o < P.n_orbit; o += 2) {
      const bool two = o + 1 < P.n_orbit;
      const float* v1 = v + (int64_t)o * P.orbit_s;
      const float* v2 = two ? v1 + P.orbit_s : v1;
      float y[8], z[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        y[e] = ok[e] ? v1[(int64_t)e * P.delta_s[3]] : 0.f;
        z[e] = ok[e] && two ? v2[(int64_t)e * P.delta_s[3]] : 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = (x[e] + y[e]) + z[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] *= P.inv_orbit;
  }
}

// V <- V J for one block-Jacobi step: the 16-row tile rt of group b's
// columns becomes V_tile Q_b (Q at form_lds + qo, group blocks in grp).  The
// (dp / 16) x ng tiles are spread over waves [w0, w0 + nw), four at a time
// with their MFMA chains interleaved; tiles are disjoint, so each is updated
// in place by its wave.
__device__ __forceinline__ void apply_v(float* V, int ld, int qo, const int* grp, const int* ident, int ng, int dp,
                                        int w0, int nw, int wave, int lj, int lr) {
  const int ntile = (dp / 16) * ng;
  const uint32_t ng_magic = (65536u + ng - 1) / ng;
  for (int t0 = wave - w0; t0 < ntile; t0 += 4 * nw) {
    bool ok[4];
    int rtile[4], gb[4], qb[4];
    float vv[4][4], qv[4][4];
    f32x4v vt[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t0 + u * nw;
      ok[u] = t < ntile;
      const int rt = ok[u] ? (int)(((uint32_t)t * ng_magic) >> 16) : 0, b = ok[u] ? t - rt * ng : 0;
      ok[u] = ok[u] && !ident[b];            // Q_b = I leaves the tile as it is
      rtile[u] = rt;
      gb[u] = grp[b];
      qb[u] = qo + b * kGrp * kLdQ;
      const int bi = gb[u] & 0xff, bj = gb[u] >> 8;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int k = 4 * kb + lj;
        vv[u][kb] = ok[u] ? V[(16 * rt + lr) * ld + group_index(bi, bj, k)] : 0.f;
        qv[u][kb] = form_lds[qb[u] + k * kLdQ + lr];
      }
      vt[u] = (f32x4v){0.f, 0.f, 0.f, 0.f};
    }
    if (!ok[0] && !ok[1] && !ok[2] && !ok[3]) continue;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int u = 0; u < 4; ++u) vt[u] = mfma4(vv[u][kb], qv[u][kb], vt[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (ok[u]) {
        const int bi = gb[u] & 0xff, bj = gb[u] >> 8;
        const int gcol = group_index(bi, bj, lr);
#pragma unroll
        for (int i = 0; i < 4; ++i) V[(16 * rtile[u] + 4 * lj + i) * ld + gcol] = vt[u][i];
      }
    }
  }
}

}  // namespace

// The Gram tiles (I, J), I <= J, of nt x nt blocks of 16 go in sets of at
// most three consecutive tiles of one block row (row I's nt - I tiles split
// evenly), so a set's products share their A operand.  The sets are dealt
// largest first, in row order, each to the SIMD (wave mod 4) with the least
// work so far that still has a wave free.  Returns this wave's tile count
// (0: none) with its block row I and first block column J0; nt <= 8 makes at
// most 15 sets.
__device__ __forceinline__ int gram_set(int nt, int wave, int& I0, int& J0) {
  int l0 = 0, l1 = 0, l2 = 0, l3 = 0, u0 = 0, u1 = 0, u2 = 0, u3 = 0;
  for (int sz = 3; sz >= 1; --sz) {
    for (int I = 0; I < nt; ++I) {
      const int k = nt - I, ns = (k + 2) / 3, base = k / ns, extra = k - base * ns;
      int J = I;
      for (int s = 0; s < ns; ++s) {
        const int z = base + (s < extra ? 1 : 0);
        if (z == sz) {
          int q = -1, bl = 1 << 30;
          if (u0 < 4 && l0 < bl) { q = 0; bl = l0; }
          if (u1 < 4 && l1 < bl) { q = 1; bl = l1; }
          if (u2 < 4 && l2 < bl) { q = 2; bl = l2; }
          if (u3 < 4 && l3 < bl) { q = 3; bl = l3; }
          const int used = q == 0 ? u0 : q == 1 ? u1 : q == 2 ? u2 : u3;
          if (q + 4 * used == wave) {
            I0 = I;
            J0 = J;
            return z;
          }
          if (q == 0) { ++u0; l0 += z; }
          else if (q == 1) { ++u1; l1 += z; }
          else if (q == 2) { ++u2; l2 += z; }
          else { ++u3; l3 += z; }
        }
        J += z;
      }
    }
  }
  I0 = J0 = 0;
  return 0;
}

// The NS tiles (I, J0 + u) of a set on the staged rows: lane (kg, t) reads
// 8 consecutive rows of one column from each bf16 part (parts at Tb, part
// stride `part`), and a tile takes the six products of the parts that are
// not below 2^-27 relative.  A's three parts are loaded first; then B's parts
// one at a time, each used at once by the products that need it (hi: mid hi,
// lo hi, hi hi; mid: mid mid, hi mid; lo: hi lo), round the tiles, so
// consecutive MFMAs update different accumulators and only one B part per
// tile is held.  A diagonal first tile takes A's parts as its B.
template <int NS, bool DIAG>
__device__ __forceinline__ void gram_steps(const uint16_t* Tb, int part, int I, int J0, int kg, int t,
                                           f32x4v (&acc)[3]) {
#pragma unroll
  for (int ks = 0; ks < kGramRows / 32; ++ks) {
    const int kj = 4 * ks + kg;                // this lane's 8-row piece
    bf16x8v a[3];
    const uint16_t* pa = Tb + gram_slot(16 * I + t, kj);
#pragma unroll
    for (int q = 0; q < 3; ++q) a[q] = *reinterpret_cast<const bf16x8v*>(pa + q * part);
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      bf16x8v b[NS];
#pragma unroll
      for (int u = 0; u < NS; ++u)
        b[u] = (DIAG && u == 0) ? a[q]
                                : *reinterpret_cast<const bf16x8v*>(Tb + gram_slot(16 * (J0 + u) + t, kj) + q * part);
      constexpr int kCount[3] = {3, 2, 1};   // A parts 1, 2, 0 | 1, 0 | 0
#pragma unroll
      for (int r = 0; r < kCount[q]; ++r) {
        const int ia = q == 0 ? (r == 0 ? 1 : r == 1 ? 2 : 0) : q == 1 ? (r == 0 ? 1 : 0) : 0;
#pragma unroll
        for (int u = 0; u < NS; ++u) acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ia], b[u], acc[u], 0, 0, 0);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Tridiagonal eigensolver for the m largest eigenpairs of G (d x d block at
// row stride ld), the default method:
//   A. Householder reduction T = Q^T G Q, Q = H_0 ... H_{d-3}, H_j = I - beta_j
//      v_j v_j^T.  Step j takes column j below the diagonal, x = A[j+1.., j]:
//      alpha = -sign(x_0) |x|, v = x - alpha e_0, beta = 2 / v^T v; then the
//      trailing block A[j+1.., j+1..] becomes A - v w^T - w v^T with
//      p = beta A v, w = p - (beta / 2)(p^T v) v.  alpha is T's subdiagonal
//      b_j and A[j][j] its diagonal a_j; v is kept in G's row j for D.
//   B. The m largest eigenvalues of T by multisection on Sturm counts (the
//      number of eigenvalues below s is the number of negative pivots of
//      T - s I), four points per round on four lanes.
//   C. Their eigenvectors z by twisted factorisation: forward pivots D+ and
//      backward pivots D- of T - lambda I, twist r where |D+_r + D-_r -
//      (a_r - lambda)| is least, z_r = 1, z_i = -(b_i / D+_i) z_{i+1} for
//      i < r and z_i = -(b_{i-1} / D-_i) z_{i-1} for i > r; eigenvalues within
//      1e-3 |T| of the previous one form a cluster, whose t-th member takes
//      the t-th least twist and is orthogonalised against the members before
//      it.
//   D. V_m = Q Z: the reflectors applied to Z from H_{d-3} down to H_0.
// In A the matrix stays in registers: thread (rb, cb) holds the 8 x 2 block
// at rows 8 rb, columns 2 cb (cb = 4 wave + lane / 16, rb = lane % 16), so
// that a column block's 16 row blocks form one DPP row and every reduction
// is DPP adds and lane reads; a step moves only the vectors v and p through
// LDS, and the row holding column j+1 forms the next reflector as soon as
// its own update is done, so a step takes two barriers.  Pivots in B and C divide with the hardware
// reciprocal (1 ulp), an error of the order of the rounding already in T.
// Lanes own the columns they write in C and D, so those phases need no
// workgroup barrier.
// Exactly multiple eigenvalues (a deficit of lower rank than m, repeated
// columns, equal singular values) can give twisted vectors that coincide;
// before D every vector is checked (finite, its residual on T, and for a
// cluster member what is left after the orthogonalisation), and the solver
// returns false when one fails, leaving G destroyed.
// sv: LDS workspace of 9 dp floats (16-byte aligned).  Output (on true): eigenvalues at
// sv + 4 dp in descending order, eigenvectors as the columns of Z [d][ldz].
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
// sum over each aligned group of 8 lanes: quad_perm [1,0,3,2], [2,3,0,1],
// then row_half_mirror (lane i <-> 7 - i: the other quad)
__device__ __forceinline__ float sum8(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  return v + dpp_f<0x141>(v);
}

// A compile-time integer as a function argument.
template <int V>
struct IntC {
  static constexpr int value = V;
};

// 16-byte LDS load of four consecutive floats.
__device__ __forceinline__ f32x4v ld4(const float* p) { return *reinterpret_cast<const f32x4v*>(p); }

// One eigenvector of T (diagonal a, subdiagonal b, b2[i] = b_i^2 and
// b2s[i] = b_{i-1}^2, both floored at FLT_MIN, 0 where b does not exist) for
// the eigenvalue lam by twisted factorisation, into z[i * ldz].  D- is kept
// in the column while D+ is recomputed where it is needed: the twist search
// runs D+ forward beside it, then D+ overwrites D- above the twist (where D-
// is no longer read) for the upward recurrence.  The pivot recurrences run in
// IEEE arithmetic as the Sturm counts do, from an infinite pivot beyond the
// first row; in the vector's recurrences a zero pivot is replaced by 1e-30.
// The twist is the rank-th least |gamma_i| (ties: lower index).  Every loop
// runs over aligned groups of four rows (d is a multiple of 4) with the
// shared operands read as 16-byte vectors, the next group loaded ahead.
__device__ __forceinline__ void twisted_vector(const float* __restrict__ a, const float* __restrict__ b,
                                               const float* __restrict__ b2, const float* __restrict__ b2s,
                                               float* __restrict__ z, int ldz, int d, float lam, int rank) {
  const float tiny = 1e-30f;
  const int ng = d >> 2;
  {                                            // backward pivots D-, bottom up
    float dmv = __builtin_inff();
    f32x4v an = ld4(a + d - 4), bn = ld4(b2 + d - 4);
    for (int g = ng - 1; g >= 0; --g) {
      const f32x4v ac = an, bc = bn;
      if (g > 0) {
        an = ld4(a + 4 * g - 4);
        bn = ld4(b2 + 4 * g - 4);
      }
#pragma unroll
      for (int u = 3; u >= 0; --u) {
        dmv = (ac[u] - lam) - bc[u] * __builtin_amdgcn_rcpf(dmv);
        z[(4 * g + u) * ldz] = dmv;
      }
    }
  }
  int r = 0;
  float prev = -1.f;
  int prev_i = -1;
  for (int s2 = 0; s2 <= rank; ++s2) {         // twist search, D+ top down beside D-
    float best = 3.4e38f, dpv = __builtin_inff();
    int bi = 0;
    f32x4v an = ld4(a), bn = ld4(b2s);
    float zn[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) zn[u] = z[u * ldz];
    for (int g = 0; g < ng; ++g) {
      const f32x4v ac = an, bc = bn;
      float zc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) zc[u] = zn[u];
      if (g + 1 < ng) {
        an = ld4(a + 4 * g + 4);
        bn = ld4(b2s + 4 * g + 4);
#pragma unroll
        for (int u = 0; u < 4; ++u) zn[u] = z[(4 * g + 4 + u) * ldz];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = 4 * g + u;
        const float al = ac[u] - lam;
        dpv = al - bc[u] * __builtin_amdgcn_rcpf(dpv);
        const float gm = fabsf(dpv + zc[u] - al);
        // (bitwise, so that the selection compiles to selects, not branches)
        const bool take = ((gm > prev) | ((gm == prev) & (i > prev_i))) & (gm < best);
        best = take ? gm : best;
        bi = take ? i : bi;
      }
    }
    prev = best;
    prev_i = bi;
    r = bi;
  }
  {                                            // D+ above the twist
    float dpv = __builtin_inff();
    for (int g = 0; 4 * g < r; ++g) {
      const f32x4v ac = ld4(a + 4 * g), bc = ld4(b2s + 4 * g);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        dpv = (ac[u] - lam) - bc[u] * __builtin_amdgcn_rcpf(dpv);
        if (4 * g + u < r) z[(4 * g + u) * ldz] = dpv;
      }
    }
  }
  // the vector from the twist outwards; the pivots of a group are read
  // before any of its rows is overwritten, the next group's during this one.
  // Every row of a visited group is stored: rows outside the pass get back
  // the value just read (D- below the twist, the vector above it), so the
  // steps are selects and not branches.
  float nrm2 = 1.f, x = 1.f;
  if (r > 0) {
    int g = (r - 1) >> 2;
    float qn[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) qn[u] = z[(4 * g + u) * ldz];
    f32x4v bn = ld4(b + 4 * g);
    for (; g >= 0; --g) {
      float q[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) q[u] = qn[u];
      const f32x4v bc = bn;
      if (g > 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) qn[u] = z[(4 * g - 4 + u) * ldz];
        bn = ld4(b + 4 * g - 4);
      }
#pragma unroll
      for (int u = 3; u >= 0; --u) {
        const int i = 4 * g + u;
        const bool in = i < r;
        const float xn = -bc[u] * __builtin_amdgcn_rcpf(q[u] != 0.f ? q[u] : tiny) * x;
        x = in ? xn : x;
        nrm2 += in ? xn * xn : 0.f;
        z[i * ldz] = in ? xn : q[u];
      }
    }
  }
  z[r * ldz] = 1.f;
  x = 1.f;
  {
    int g = (r + 1) >> 2;
    float qn[4], bbn[4];
    auto load_group = [&](int gg) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = 4 * gg + u;
        qn[u] = z[i * ldz];
        bbn[u] = i > 0 ? b[i - 1] : 0.f;
      }
    };
    if (4 * g < d) load_group(g);
    for (; 4 * g < d; ++g) {
      float q[4], bb[4];                       // pivots D- and b_{i-1} of the group
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        q[u] = qn[u];
        bb[u] = bbn[u];
      }
      if (4 * g + 4 < d) load_group(g + 1);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = 4 * g + u;
        const bool in = i > r;
        const float xn = -bb[u] * __builtin_amdgcn_rcpf(q[u] != 0.f ? q[u] : tiny) * x;
        x = in ? xn : x;
        nrm2 += in ? xn * xn : 0.f;
        z[i * ldz] = in ? xn : q[u];
      }
    }
  }
  const float inv = 1.f / sqrtf(nrm2);
  for (int g = 0; g < ng; ++g) {
#pragma unroll
    for (int u = 0; u < 4; ++u) z[(4 * g + u) * ldz] *= inv;
  }
}

// The same vector with two lanes per eigenvalue, on two waves, where Z has a
// spare column per eigenvalue (2 m <= ldz): the lane pair's pivots D- (into
// the vector's column zm) and D+ (into the spare column zp) run at once; the
// twist is then a scan over both stored columns; the vector above the twist
// (from D+, written into zm) and below it (from D-, in place) again run at
// once, each pass writing only its own rows.  Same recurrences, same
// arithmetic as twisted_vector.
__device__ __forceinline__ void tw_pivots(const float* __restrict__ a, const float* __restrict__ b2,
                                          const float* __restrict__ b2s, float* __restrict__ z, int ldz, int d,
                                          float lam, bool backward) {
  const int ng = d >> 2;
  float pv = __builtin_inff();
  if (backward) {                              // D-, bottom up
    f32x4v an = ld4(a + d - 4), bn = ld4(b2 + d - 4);
    for (int g = ng - 1; g >= 0; --g) {
      const f32x4v ac = an, bc = bn;
      if (g > 0) {
        an = ld4(a + 4 * g - 4);
        bn = ld4(b2 + 4 * g - 4);
      }
#pragma unroll
      for (int u = 3; u >= 0; --u) {
        pv = (ac[u] - lam) - bc[u] * __builtin_amdgcn_rcpf(pv);
        z[(4 * g + u) * ldz] = pv;
      }
    }
  } else {                                     // D+, top down
    f32x4v an = ld4(a), bn = ld4(b2s);
    for (int g = 0; g < ng; ++g) {
      const f32x4v ac = an, bc = bn;
      if (g + 1 < ng) {
        an = ld4(a + 4 * g + 4);
        bn = ld4(b2s + 4 * g + 4);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        pv = (ac[u] - lam) - bc[u] * __builtin_amdgcn_rcpf(pv);
        z[(4 * g + u) * ldz] = pv;
      }
    }
  }
}

// the twist from the stored pivots: the rank-th least |gamma_i|,
// gamma_i = D+_i + D-_i - (a_i - lam) (ties: lower index)
__device__ __forceinline__ int tw_twist(const float* __restrict__ a, const float* __restrict__ zm,
                                        const float* __restrict__ zp, int ldz, int d, float lam, int rank) {
  const int ng = d >> 2;
  float prev = -1.f;
  int prev_i = -1, r = 0;
  for (int s2 = 0; s2 <= rank; ++s2) {
    float best = 3.4e38f;
    int bi = 0;
    for (int g = 0; g < ng; ++g) {
      const f32x4v ac = ld4(a + 4 * g);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = 4 * g + u;
        const float al = ac[u] - lam;
        const float gm = fabsf(zp[i * ldz] + zm[i * ldz] - al);
        const bool take = ((gm > prev) | ((gm == prev) & (i > prev_i))) & (gm < best);
        best = take ? gm : best;
        bi = take ? i : bi;
      }
    }
    prev = best;
    prev_i = bi;
    r = bi;
  }
  return r;
}

// rows r-1 .. 0 of the vector (x_r = 1) from D+ (column zp) into column zm;
// returns their sum of squares
__device__ __forceinline__ float tw_up(const float* __restrict__ b, const float* __restrict__ zp,
                                       float* __restrict__ zm, int ldz, int r) {
  const float tiny = 1e-30f;
  float n2 = 0.f, x = 1.f;
  if (r > 0) {
    int g = (r - 1) >> 2;
    float qn[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) qn[u] = zp[(4 * g + u) * ldz];
    f32x4v bn = ld4(b + 4 * g);
    for (; g >= 0; --g) {
      float q[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) q[u] = qn[u];
      const f32x4v bc = bn;
      if (g > 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) qn[u] = zp[(4 * g - 4 + u) * ldz];
        bn = ld4(b + 4 * g - 4);
      }
#pragma unroll
      for (int u = 3; u >= 0; --u) {
        const int i = 4 * g + u;
        const bool in = i < r;
        const float xn = -bc[u] * __builtin_amdgcn_rcpf(q[u] != 0.f ? q[u] : tiny) * x;
        x = in ? xn : x;
        n2 += in ? xn * xn : 0.f;
        if (in) zm[i * ldz] = xn;
      }
    }
  }
  return n2;
}

// rows r+1 .. d-1 of the vector (x_r = 1) from D- (column zm, in place);
// returns their sum of squares
__device__ __forceinline__ float tw_down(const float* __restrict__ b, float* __restrict__ zm, int ldz, int d,
                                         int r) {
  const float tiny = 1e-30f;
  float n2 = 0.f, x = 1.f;
  int g = (r + 1) >> 2;
  float qn[4], bbn[4];
  auto load_group = [&](int gg) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = 4 * gg + u;
      qn[u] = zm[i * ldz];
      bbn[u] = i > 0 ? b[i - 1] : 0.f;
    }
  };
  if (4 * g < d) load_group(g);
  for (; 4 * g < d; ++g) {
    float q[4], bb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      q[u] = qn[u];
      bb[u] = bbn[u];
    }
    if (4 * g + 4 < d) load_group(g + 1);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = 4 * g + u;
      const bool in = i > r;
      const float xn = -bb[u] * __builtin_amdgcn_rcpf(q[u] != 0.f ? q[u] : tiny) * x;
      x = in ? xn : x;
      n2 += in ? xn * xn : 0.f;
      if (in) zm[i * ldz] = xn;
    }
  }
  return n2;
}

// V_m = Q Z for the m columns of Z: the reflectors (v_j in G's row j, zero
// outside rows j+1 .. d-1; scale beta_j) applied from H_{d-3} down to H_0
// with Z in registers: 16 lanes (one DPP row) per column, lane rb holding
// rows 32 h + 2 rb + e (h < 4, e < 2), the next reflector loaded while this
// one is applied.  With that row split each 8-byte read of a reflector
// covers 128 contiguous bytes and the Z accesses of a wave fall on distinct
// banks (8 consecutive rows per lane made both conflict: 2-way and 8-way).
__device__ __forceinline__ void back_transform(const float* __restrict__ G, int ld, float* __restrict__ Z, int ldz,
                                               const float* __restrict__ beta, int d, int dp, int m) {
  typedef float f32x2v __attribute__((ext_vector_type(2)));
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rb = lane & 15;
  // rows 32 h + 2 rb and + 1 are both inside the padded rows or both past them
  bool vin[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) vin[h] = 32 * h + 2 * rb < dp;
  // rows past the padded ones take v = 0 (and keep z = 0)
  auto load_v = [&](int j, float* v) {
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const f32x2v t = vin[h] ? *reinterpret_cast<const f32x2v*>(G + j * ld + 32 * h + 2 * rb) : f32x2v{0.f, 0.f};
      v[2 * h] = t[0];
      v[2 * h + 1] = t[1];
    }
  };
  for (int k0 = 0; k0 < m; k0 += 4 * kWaves) {
    const int k = k0 + 4 * wave + (lane >> 4);
    const bool own = k < m;
    float z[8], vn[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 32 * (i >> 1) + 2 * rb + (i & 1);
      z[i] = own && vin[i >> 1] ? Z[r * ldz + k] : 0.f;
    }
    float bn = 0.f;
    if (d >= 3) {
      load_v(d - 3, vn);
      bn = beta[d - 3];
    }
    for (int j = d - 3; j >= 0; --j) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = vn[i];
      const float bj = bn;
      if (j > 0) {
        load_v(j - 1, vn);
        bn = beta[j - 1];
      }
      float y = 0.f, y2 = 0.f;
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        y += v[i] * z[i];
        y2 += v[i + 1] * z[i + 1];
      }
      y = sum8(y + y2);
      y = (y + dpp_f<0x140>(y)) * bj;          // row_mirror: the other 8 lanes of the row
#pragma unroll
      for (int i = 0; i < 8; ++i) z[i] -= y * v[i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 32 * (i >> 1) + 2 * rb + (i & 1);
      if (own && r < d) Z[r * ldz + k] = z[i];
    }
  }
}

__device__ bool tridiag_solve(float* G, int ld, float* Z, int ldz, int d, int dp, int m, float* sv, int* s_cs,
                              int* s_fail) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  float* const s_a = sv;                       // T's diagonal
  float* const s_b = sv + dp;                  // T's subdiagonal
  float* const s_beta = sv + 2 * dp;           // reflector scales
  float* const s_p = sv + 3 * dp;              // p of the current step; b_i^2 from B on
  float* const s_lam = sv + 4 * dp;            // eigenvalues, descending
  float* const s_v = sv + 5 * dp;              // [2][dp] v of alternate steps
  float* const s_misc = sv + 7 * dp;           // Gershgorin lo, hi
  float* const s_kred = sv + 7 * dp + 8;       // [16] per-wave p^T v partials
  float* const s_b2s = sv + 8 * dp;            // b_{i-1}^2 (0 at i = 0), from B on
  if (tid == 0) *s_fail = 0;

  // ---- A. Householder reduction, the matrix in registers ----
  {
    typedef float f32x2v __attribute__((ext_vector_type(2)));
    const int row16 = lane >> 4, rb = lane & 15, cb = 4 * wave + row16;
    const bool rin = 8 * rb < dp, cin = 2 * cb < dp;
    const bool b3 = lane & 8;                  // which of the block's two columns this lane ends with
    float A[8][2];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int r = 8 * rb + i, cc = 2 * cb + c;
        A[i][c] = (r < d && cc < d) ? G[r * ld + cc] : 0.f;
      }
    auto rl = [](float x, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); };
    // the reflector of column j, by the DPP row holding it (cb == j / 2):
    // writes v (zero outside rows j+1 .. d-1) into s_v[j & 1] and G's row j,
    // a_j, b_j and beta_j
    // (JJ = j % 2 as a compile-time constant: the column is picked without
    // selects, and never by a run-time index, which would move A out of
    // registers)
    auto reflect = [&](int j, auto jjc) {
      constexpr int JJ = decltype(jjc)::value;
      float colv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) colv[i] = A[i][JJ];
      // x below its first entry (rows j+2 .. d-1): v there, and its squares
      // summed as a tree
      float vv[8], q[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = 8 * rb + i;
        vv[i] = (r > j + 1 && r < d) ? colv[i] : 0.f;
        q[i] = vv[i] * vv[i];
      }
      float sq = ((q[0] + q[1]) + (q[2] + q[3])) + ((q[4] + q[5]) + (q[6] + q[7]));
      sq = sum8(sq);
      sq += dpp_f<0x140>(sq);                  // row_mirror: the other 8 lanes of the row
      // x_0 (row j+1) and a_j (row j): entry i % 8 of every lane, picked by a
      // three-level select tree, then read from the lane holding that row
      auto pick = [&](int i) {
        const float p01 = (i & 1) ? colv[1] : colv[0], p23 = (i & 1) ? colv[3] : colv[2];
        const float p45 = (i & 1) ? colv[5] : colv[4], p67 = (i & 1) ? colv[7] : colv[6];
        const float p03 = (i & 2) ? p23 : p01, p47 = (i & 2) ? p67 : p45;
        return (i & 4) ? p47 : p03;
      };
      const int rrow = 16 * ((j >> 1) & 3);    // first lane of this DPP row, as a scalar
      const float x0 = rl(pick((j + 1) & 7), rrow + ((j + 1) >> 3));
      const float aj = rl(pick(j & 7), rrow + (j >> 3));
      // (hardware square root and reciprocal, 1 ulp each: beta is formed from
      // the v that is stored, so H stays orthogonal to rounding)
      float beta = 0.f, alpha = x0, v0 = 0.f;
      if (sq != 0.f) {                         // else already reduced: H_j = I (and v = 0 below x_0)
        const float nrm = __builtin_amdgcn_sqrtf(x0 * x0 + sq);
        alpha = x0 >= 0.f ? -nrm : nrm;
        v0 = x0 - alpha;
        beta = 2.f * __builtin_amdgcn_rcpf(v0 * v0 + sq);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (8 * rb + i == j + 1) vv[i] = v0;
      if (rin) {
        f32x4v* sv4 = reinterpret_cast<f32x4v*>(s_v + (j & 1) * dp + 8 * rb);
        sv4[0] = (f32x4v){vv[0], vv[1], vv[2], vv[3]};
        sv4[1] = (f32x4v){vv[4], vv[5], vv[6], vv[7]};
        f32x2v* grow = reinterpret_cast<f32x2v*>(G + j * ld + 8 * rb);   // row j, for the back-transformation
#pragma unroll
        for (int h = 0; h < 4; ++h) grow[h] = (f32x2v){vv[2 * h], vv[2 * h + 1]};
      }
      if (rb == 0) {
        s_a[j] = aj;
        s_b[j] = alpha;
        s_beta[j] = beta;
      }
    };
    __syncthreads();                           // G is read into registers before rows of it are overwritten
    if (d >= 3 && cb == 0) reflect(0, IntC<0>{});
    for (int j = 0; j < d - 2; ++j) {
      __syncthreads();
      const float beta = s_beta[j];
      const float* vb = s_v + (j & 1) * dp;
      // columns of this wave: 8 wave .. 8 wave + 7; none left in the trailing block?
      const bool active = 8 * wave + 7 > j && 8 * wave < d;
      float vr[8], vc[2];
      if (active) {
        const f32x4v z4 = {0.f, 0.f, 0.f, 0.f};
        const f32x4v v0 = rin ? ld4(vb + 8 * rb) : z4, v1 = rin ? ld4(vb + 8 * rb + 4) : z4;
        const f32x2v c2 = cin ? *reinterpret_cast<const f32x2v*>(vb + 2 * cb) : (f32x2v){0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          vr[i] = v0[i];
          vr[4 + i] = v1[i];
        }
        vc[0] = c2[0];
        vc[1] = c2[1];
        // p = beta A v over this thread's block, summed over the row's 16
        // row blocks: the two column sums are halved by an exchange across
        // the row's halves (row_mirror), the kept one summed over its 8 lanes
        float part[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          float s0 = 0.f, s1 = 0.f;
#pragma unroll
          for (int i = 0; i < 8; i += 2) {
            s0 += A[i][c] * vr[i];
            s1 += A[i + 1][c] * vr[i + 1];
          }
          part[c] = s0 + s1;
        }
        float keep = (b3 ? part[1] : part[0]) + dpp_f<0x140>(b3 ? part[0] : part[1]);
        keep = sum8(keep) * beta;
        const int col = 2 * cb + (b3 ? 1 : 0);
        const bool trail = col > j && col < d;
        if ((lane & 7) == 0 && cin) s_p[col] = trail ? keep : 0.f;
        // p^T v over the wave's 8 columns: each row's two column values met
        // by row_mirror, then the four rows read out
        // (the lane reads stay outside the lane-0 branch: inside it the other
        // lanes are inactive and their values undefined)
        float pv = trail ? keep * (b3 ? vc[1] : vc[0]) : 0.f;
        pv += dpp_f<0x140>(pv);
        const float pvw = (rl(pv, 0) + rl(pv, 16)) + (rl(pv, 32) + rl(pv, 48));
        if (lane == 0) s_kred[wave] = pvw;
      } else {
        if ((lane & 7) == 0 && cin) s_p[2 * cb + (b3 ? 1 : 0)] = 0.f;
        if (lane == 0) s_kred[wave] = 0.f;
      }
      __syncthreads();
      // the wave that forms the next reflector goes first on its SIMD, so
      // that the reflector is ready when the other waves finish their updates
      const bool owner = wave == ((j + 1) >> 3) && j + 1 < d - 2;
      if (owner) __builtin_amdgcn_s_setprio(2);
      if (active) {
        // A -= v w^T + w v^T, w = p - K v, K = (beta / 2) p^T v; p and v are
        // zero outside the trailing block, so the update is too
        float kd = 0.f;
#pragma unroll
        for (int w4 = 0; w4 < kWaves / 4; ++w4) {
          const f32x4v k4 = ld4(s_kred + 4 * w4);
          kd += (k4[0] + k4[1]) + (k4[2] + k4[3]);
        }
        const float K = 0.5f * beta * kd;
        const f32x4v z4 = {0.f, 0.f, 0.f, 0.f};
        const f32x4v p0 = rin ? ld4(s_p + 8 * rb) : z4, p1 = rin ? ld4(s_p + 8 * rb + 4) : z4;
        const f32x2v pc2 = cin ? *reinterpret_cast<const f32x2v*>(s_p + 2 * cb) : (f32x2v){0.f, 0.f};
        float wr[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          wr[i] = p0[i] - K * vr[i];
          wr[4 + i] = p1[i] - K * vr[4 + i];
        }
        const float wc0 = pc2[0] - K * vc[0], wc1 = pc2[1] - K * vc[1];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          A[i][0] = fmaf(-vr[i], wc0, fmaf(-wr[i], vc[0], A[i][0]));
          A[i][1] = fmaf(-vr[i], wc1, fmaf(-wr[i], vc[1], A[i][1]));
        }
      }
      if (j + 1 < d - 2 && cb == ((j + 1) >> 1)) {
        if ((j + 1) & 1) reflect(j + 1, IntC<1>{});
        else reflect(j + 1, IntC<0>{});
      }
      if (owner) __builtin_amdgcn_s_setprio(0);
    }
    // the last 2 x 2 block of T (the whole of T when d <= 2)
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int r = 8 * rb + i, cc = 2 * cb + c;
        if (d >= 2 && cc == d - 2 && r == d - 2) s_a[d - 2] = A[i][c];
        if (d >= 2 && cc == d - 2 && r == d - 1) s_b[d - 2] = A[i][c];
        if (cc == d - 1 && r == d - 1) s_a[d - 1] = A[i][c];
      }
  }
  __syncthreads();

  // ---- B. the m largest eigenvalues: 8 lanes per eigenvalue ----
  // Sturm counts in IEEE arithmetic: a zero pivot gives an infinite next one,
  // whose reciprocal is zero, so the sequence runs on without a test; b^2 is
  // floored at FLT_MIN so that no 0 * inf occurs, and a pivot counts as
  // negative by its sign bit (-0 included), which keeps the count the one of
  // a nearby perturbed matrix.  The recurrence starts from an infinite pivot
  // before row 0 (b_{-1}^2 = 0) and takes a and b^2 four rows at a time, the
  // next four loaded ahead.
  float* const s_b2 = s_p;
  if (wave == 0) {                             // Gershgorin interval and b^2
    float lo = 3.4e38f, hi = -3.4e38f;
    for (int i = lane; i < d; i += 64) {
      const float bl = i > 0 ? s_b[i - 1] : 0.f, br = i < d - 1 ? s_b[i] : 0.f;
      const float r = fabsf(bl) + fabsf(br);
      lo = fminf(lo, s_a[i] - r);
      hi = fmaxf(hi, s_a[i] + r);
      s_b2[i] = i < d - 1 ? fmaxf(br * br, 1.17549435e-38f) : 0.f;
      s_b2s[i] = i > 0 ? fmaxf(bl * bl, 1.17549435e-38f) : 0.f;
    }
    for (int o = 32; o > 0; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o, 64));
      hi = fmaxf(hi, __shfl_xor(hi, o, 64));
    }
    if (lane == 0) {
      s_misc[0] = lo;
      s_misc[1] = hi;
    }
  }
  __syncthreads();
  const float tnorm = fmaxf(fabsf(s_misc[0]), fabsf(s_misc[1]));   // |T| bound
  // 9-section: the group's 8 lanes evaluate the 8 inner points of the
  // interval, so 8 rounds narrow it to width / 9^8, below fp32 rounding of
  // |T| (two waves per SIMD at rank 64: the Sturm recurrences are a
  // dependent chain per lane, and 16 lanes per eigenvalue were slower,
  // four waves per SIMD contending for the vector ALU)
  if (tid < 8 * m) {
    const int k = tid >> 3, t = tid & 7;
    const int q = d - 1 - k;                   // ascending index of the k-th largest
    float lo = s_misc[0], hi = s_misc[1];
    for (int it = 0; it < 8; ++it) {
      const float w = hi - lo;
      const float x = lo + w * (float)(t + 1) * (1.f / 9.f);
      float qv = __builtin_inff();
      uint32_t cnt = 0;
      f32x4v an = ld4(s_a), bn = ld4(s_b2s);
      for (int i = 0; i < d; i += 4) {
        const f32x4v ac = an, bc = bn;
        if (i + 4 < d) {
          an = ld4(s_a + i + 4);
          bn = ld4(s_b2s + i + 4);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          qv = (ac[u] - x) - bc[u] * __builtin_amdgcn_rcpf(qv);
          cnt += __float_as_uint(qv) >> 31;
        }
      }
      // the points at or below the eigenvalue: a prefix of the group's lanes
      const uint64_t bal = __ballot((int)cnt <= q);
      const int nb = __popcll((bal >> (lane & ~7)) & 0xffull);
      const float nlo = nb > 0 ? lo + w * (float)nb * (1.f / 9.f) : lo;
      const float nhi = nb < 8 ? lo + w * (float)(nb + 1) * (1.f / 9.f) : hi;
      lo = nlo;
      hi = fmaxf(nhi, nlo);
    }
    if (t == 0) s_lam[k] = 0.5f * (lo + hi);
  }
  __syncthreads();
  // clusters: runs of eigenvalues within 1e-3 |T| of their predecessor
  // (equal ones always, also when T = 0): s_cs[j] is the last run start at or
  // before j, a running maximum over the starts (wave 0, 64 entries a pass)
  if (wave == 0) {
    int carry = 0;
    for (int base = 0; base < m; base += 64) {
      const int j = base + lane;
      int v = (j < m && (j == 0 || !(s_lam[j - 1] - s_lam[j] <= 1e-3f * tnorm))) ? j : 0;
      for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(v, o, 64);
        if (lane >= o) v = v > u ? v : u;
      }
      v = v > carry ? v : carry;
      if (j < m) s_cs[j] = v;
      carry = __shfl(v, 63, 64);
    }
  }
  __syncthreads();

  // ---- C. eigenvectors of T: one lane per eigenvalue, in its column of Z ----
  // The twist rank of an eigenvalue is its place in its run of numerically
  // equal ones (within 2^-20 |T|), so that the members of an exactly
  // multiple eigenvalue take different twists; every other one takes its
  // best twist, which gives the accurate vector.
  if (2 * m <= ldz && m <= 64) {
    // two lanes per eigenvalue k = lane: wave 0 holds the vector's column k,
    // wave 1 the spare column m + k (free until the back-transformation)
    float* const s_n2 = sv + 9 * dp;           // [2][64] partial sums of squares
    int* const s_tw = reinterpret_cast<int*>(sv + 9 * dp + 128);   // [64] twists
    const bool pair = wave < 2 && lane < m;
    if (pair) tw_pivots(s_a, s_b2, s_b2s, Z + lane + wave * m, ldz, d, s_lam[lane], wave == 0);
    __syncthreads();
    if (wave == 0 && lane < m) {
      int rank = 0;
      while (rank < lane && rank < d - 1 && s_lam[lane - rank - 1] - s_lam[lane - rank] <= 0x1p-20f * tnorm) ++rank;
      const int r = tw_twist(s_a, Z + lane, Z + m + lane, ldz, d, s_lam[lane], rank);
      s_tw[lane] = r;
      Z[r * ldz + lane] = 1.f;                 // (row r of the spare column is not read again)
    }
    __syncthreads();
    if (pair) {
      const int r = s_tw[lane];
      s_n2[wave * 64 + lane] = wave == 0 ? tw_up(s_b, Z + m + lane, Z + lane, ldz, r)
                                         : tw_down(s_b, Z + lane, ldz, d, r);
    }
    __syncthreads();
    if (pair) {                                // rows split between the two waves
      const float inv = 1.f / sqrtf(1.f + s_n2[lane] + s_n2[64 + lane]);
      const int h = ((d >> 2) + 1) >> 1;      // groups of the first wave
      const int g0 = wave == 0 ? 0 : h, g1 = wave == 0 ? h : (d >> 2);
      for (int g = g0; g < g1; ++g) {
#pragma unroll
        for (int u = 0; u < 4; ++u) Z[(4 * g + u) * ldz + lane] *= inv;
      }
    }
  } else if (tid < m) {
    int rank = 0;
    while (rank < tid && rank < d - 1 && s_lam[tid - rank - 1] - s_lam[tid - rank] <= 0x1p-20f * tnorm) ++rank;
    twisted_vector(s_a, s_b, s_b2, s_b2s, Z + tid, ldz, d, s_lam[tid], rank);
  }
  __syncthreads();
  // cluster members orthogonalised against the members before them (wave 0):
  // z_k stays in registers (rows lane and lane + 64) through its member's
  // pass, and a wave sum is three DPP adds per 8 lanes, one row_mirror and
  // four lane reads (the loop bounds are the same on every lane)
  if (wave == 0) {
    auto wsum = [](float x) {
      x = sum8(x);
      x += dpp_f<0x140>(x);
      const auto rd = [&](int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); };
      return (rd(0) + rd(16)) + (rd(32) + rd(48));
    };
    const bool r0 = lane < d, r1 = lane + 64 < d;
    for (int k = 1; k < m; ++k) {
      const int c0 = s_cs[k];
      if (c0 == k) continue;
      float zk0 = r0 ? Z[lane * ldz + k] : 0.f, zk1 = r1 ? Z[(lane + 64) * ldz + k] : 0.f;
      for (int i = c0; i < k; ++i) {
        const float zi0 = r0 ? Z[lane * ldz + i] : 0.f, zi1 = r1 ? Z[(lane + 64) * ldz + i] : 0.f;
        const float dt = wsum(zi0 * zk0 + zi1 * zk1);
        zk0 -= dt * zi0;
        zk1 -= dt * zi1;
      }
      const float n2 = wsum(zk0 * zk0 + zk1 * zk1);
      // a member that was mostly inside the span of the ones before it is
      // not trusted (twisted vectors of an exactly multiple eigenvalue)
      if (lane == 0 && !(n2 >= 0.25f)) *s_fail = 1;
      const float inv = n2 > 0.f ? 1.f / sqrtf(n2) : 0.f;
      if (r0) Z[lane * ldz + k] = zk0 * inv;
      if (r1) Z[(lane + 64) * ldz + k] = zk1 * inv;
    }
  }
  __syncthreads();
  // every vector must satisfy |T z - lambda z| <= 2^-16 |T| (good ones reach
  // ~d u |T|); a larger or non-finite residual sends the unit to Jacobi.
  // The rows of a vector are split over four waves (two at rank > 64), the
  // partial sums meeting in LDS (phase C's scratch)
  {
    float* const s_r2 = sv + 9 * dp;           // [4][128]
    const int mc = (m + 63) >> 6, parts = 4 / mc;
    if (wave < 4) {
      const int k = lane + 64 * (wave % mc), part = wave / mc;
      const int i0 = part * (d / parts), i1 = i0 + d / parts;
      if (k < m) {
        const float lam = s_lam[k], inv_tn = tnorm > 0.f ? 1.f / tnorm : 0.f;
        float r2 = 0.f;
#pragma unroll 8
        for (int i = i0; i < i1; ++i) {
          float t = (s_a[i] - lam) * Z[i * ldz + k];
          if (i > 0) t += s_b[i - 1] * Z[(i - 1) * ldz + k];
          if (i < d - 1) t += s_b[i] * Z[(i + 1) * ldz + k];
          t *= inv_tn;
          r2 += t * t;
        }
        s_r2[part * 128 + k] = r2;
      }
    }
    __syncthreads();
    if (tid < m) {
      float r2 = 0.f;
      for (int q = 0; q < parts; ++q) r2 += s_r2[q * 128 + tid];
      if (!(r2 <= 0x1p-32f)) *s_fail = 1;
    }
  }
  __syncthreads();
  if (*s_fail) return false;

  // ---- D. V_m = Q Z ----
  back_transform(G, ld, Z, ldz, s_beta, d, dp, m);
  __syncthreads();
  return true;
}

__global__ __launch_bounds__(kFormThreads) void form_patch_kernel(const FormParams /*by value, read in place*/) {
  const FormParams& P = *static_cast<const FormParams*>((const void*)__builtin_amdgcn_kernarg_segment_ptr());
  float* const lds_f = form_lds;
  __shared__ int s_order[128];
  __shared__ float s_red[kWaves];
  __shared__ int s_grp[2][kFormMaxDim / (2 * kBlk)];   // blocks (bi | bj << 8) of each group, this and last step
  __shared__ int s_ident[2][kFormMaxDim / (2 * kBlk)]; // group kept Q = I, this and last step

  const int unit = blockIdx.x;
  if (unit >= P.n_units) return;
  const int h = unit % P.n_heads;
  const int l = (unit / P.n_heads) % P.n_layers;
  const int c = unit / (P.n_heads * P.n_layers);
  const int d = P.dim, n = P.n_tokens, m = P.m;
  const int dp = pad16(d);                   // padded size (zero rows/columns beyond d)
  const int ld = gv_ld(dp);                  // padded LDS row stride of G and V
  const int nb = dp / kBlk;                  // Jacobi blocks (even)
  const int ng = nb / 2;                     // groups rotated per step
  float* G = lds_f;                          // [dp][ld]
  float* V = lds_f + dp * ld;                // [dp][ld]; holds Delta tiles in phase 1
  float* Ss = V + dp * ld;                   // [ng][16][kLdQ] group matrices
  float* Qs2 = Ss + ng * kGrp * kLdQ;        // [2][ng][16][kLdQ] group rotations of this and the last step
  const float* delta = P.delta + (int64_t)c * P.delta_s[0] + (int64_t)l * P.delta_s[1] + (int64_t)h * P.delta_s[2];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int lj = lane >> 4, lr = lane & 15;  // MFMA operand slot (k within a step) and row/column

  // With the tridiagonal solver (sweeps == 0) a unit whose vectors fail its
  // checks forms G again and runs block Jacobi instead.
  int sweeps = P.sweeps;
  bool tri_ok = false;
  __shared__ int s_fail;
  // ---- 1. G = Delta^T Delta on MFMA: a wave owns up to 3 tiles of one block row ----
  auto form_gram = [&]() {
    const int nt = dp / 16;
    uint16_t* Tb = reinterpret_cast<uint16_t*>(V);   // staged parts hi, mid, lo: [3][dp][kGramRows] bf16
    const int part = dp * kGramRows;
    // this wave's tiles (gI, gJ + u), u < my: the same on every lane
    int gI, gJ;
    const int my = __builtin_amdgcn_readfirstlane(gram_set(nt, wave, gI, gJ));
    gI = __builtin_amdgcn_readfirstlane(gI);
    gJ = __builtin_amdgcn_readfirstlane(gJ);
    const bool gdiag = gI == gJ;
    f32x4v acc[3];
#pragma unroll
    for (int u = 0; u < 3; ++u) acc[u] = (f32x4v){0.f, 0.f, 0.f, 0.f};
    // thread (sg, sc) stages rows 8 sg .. 8 sg + 7 of column sc of each
    // kGramRows-row tile, split into three bf16 parts, as one 16-byte piece
    // per part; the next tile's loads are in flight during the products on
    // the current one
    const bool stager = tid < (kGramRows / 8) * dp;
    const int sg = stager ? tid / dp : 0, sc = stager ? tid - sg * dp : 0;
    float x[8];
    load_col8(P, delta, 8 * sg, stager ? sc : d, n, d, x);
    for (int t0 = 0; t0 < n; t0 += kGramRows) {
      __syncthreads();
      if (stager) {
        u32x4v hi, mid, lo;
        split3_bf16x8(x, hi, mid, lo);
        uint16_t* q = Tb + gram_slot(sc, sg);
        *reinterpret_cast<u32x4v*>(q) = hi;
        *reinterpret_cast<u32x4v*>(q + part) = mid;
        *reinterpret_cast<u32x4v*>(q + 2 * part) = lo;
      }
      __syncthreads();
      if (t0 + kGramRows < n) load_col8(P, delta, t0 + kGramRows + 8 * sg, stager ? sc : d, n, d, x);
      // the set is the same on every lane: one scalar branch picks a loop
      // without branches; rows past n are staged as zeros, so every tile
      // takes all k-steps
      if (gdiag) {
        if (my == 3) gram_steps<3, true>(Tb, part, gI, gJ, lj, lr, acc);
        else if (my == 2) gram_steps<2, true>(Tb, part, gI, gJ, lj, lr, acc);
        else if (my == 1) gram_steps<1, true>(Tb, part, gI, gJ, lj, lr, acc);
      } else {
        if (my == 3) gram_steps<3, false>(Tb, part, gI, gJ, lj, lr, acc);
        else if (my == 2) gram_steps<2, false>(Tb, part, gI, gJ, lj, lr, acc);
        else if (my == 1) gram_steps<1, false>(Tb, part, gI, gJ, lj, lr, acc);
      }
    }
    // lane (lj, lr) holds G[16 gI + 4 lj + i][16 (gJ + u) + lr]; store it and its mirror
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      if (u < my) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * gI + 4 * lj + i, col = 16 * (gJ + u) + lr;
          if (gI < gJ + u || row <= col) {
            G[row * ld + col] = acc[u][i];
            G[col * ld + row] = acc[u][i];
          }
        }
      }
    }
    __syncthreads();
    // V = I (the staged tile is no longer needed)
    for (int e = tid; e < dp * dp; e += kFormThreads) V[(e / dp) * ld + e % dp] = (e / dp == e % dp) ? 1.f : 0.f;
    __syncthreads();
  };
  form_gram();
  if (sweeps == 0) {
    // ---- 2'. tridiagonal eigensolver: eigenpairs in order, eigenvalues onto
    // G's diagonal and vectors into V's first m columns ----
    float* sv = Ss;                            // 9 dp + 512 floats of the 51 dp here
    tri_ok = tridiag_solve(G, ld, V, ld, d, dp, m, sv, s_order, &s_fail);
    if (tri_ok) {
      if (tid < m) {
        G[tid * ld + tid] = sv[4 * dp + tid];
        s_order[tid] = tid;
      }
      if (P.sweeps_done != nullptr && tid == 0) P.sweeps_done[unit] = 0;
      __syncthreads();
    } else {
      sweeps = kFormFallbackSweeps;
      form_gram();
    }
  }

  // ---- 2. block Jacobi ----
  // Each step's V <- V J is deferred to the next step's first phase, where the
  // waves without a group to solve apply it while the others run their inner
  // sweeps; the Q buffers and group lists alternate between steps.
  int sweeps_run = 0;
  int cur = 0;                                 // buffer of the step being formed
  bool pending = false;                        // V still owes the previous step's rotation
  for (int sweep = 0; sweep < (tri_ok ? 0 : sweeps); ++sweep) {
    // stop once the off-diagonal mass is negligible against the diagonal
    float off = 0.f, dia = 0.f;
    for (int e = tid; e < d * d; e += kFormThreads) {
      const int i = e / d, j = e % d;
      const float g = G[i * ld + j];
      if (i == j) dia += g * g; else off += g * g;
    }
    off = block_sum(off, s_red);
    dia = block_sum(dia, s_red);
    if (off <= 1e-9f * dia) break;             // ~(d * 4 eps)^2: the fp32 floor
    ++sweeps_run;
    for (int step = 0; step < nb - 1; ++step) {
      float* Qs = Qs2 + cur * ng * kGrp * kLdQ;
      const int* grp = s_grp[cur];
      // (a) one wave per group: a Jacobi sweep on the group's principal
      // submatrix; the remaining waves apply the previous step to V
      if (wave < ng) {
        int bi, bj;
        circle_pair(nb, step, wave, bi, bj);
        if (lane == 0) s_grp[cur][wave] = bi | (bj << 8);
        const int so = (int)(Ss - lds_f) + wave * kGrp * kLdQ;
        const int qo = (int)(Qs - lds_f) + wave * kGrp * kLdQ;
        float goff = 0.f;
#pragma unroll
        for (int u = 0; u < kGrp * kGrp / 64; ++u) {
          const int e = lane + 64 * u, r = e >> 4, cc = e & 15;
          const float g = G[group_index(bi, bj, r) * ld + group_index(bi, bj, cc)];
          lds_f[so + r * kLdQ + cc] = g;
          lds_f[qo + r * kLdQ + cc] = r == cc ? 1.f : 0.f;
          if (r != cc) goff += g * g;
        }
        for (int o = 32; o > 0; o >>= 1) goff += __shfl_xor(goff, o, 64);
        // a group whose block is already diagonal to well below the
        // convergence test (at most 120 such groups per sweep stay under it)
        // keeps Q = I, and the tile products it would leave unchanged are skipped
        const bool skip = goff <= 1e-12f * dia;
        if (lane == 0) s_ident[cur][wave] = skip ? 1 : 0;
        __builtin_amdgcn_wave_barrier();
        if (!skip) group_sweep(so, qo, lane, G, ld, bi, bj);
      } else if (pending) {
        apply_v(V, ld, (int)(Qs2 - lds_f) + (cur ^ 1) * ng * kGrp * kLdQ, s_grp[cur ^ 1], s_ident[cur ^ 1], ng, dp,
                ng, kWaves - ng, wave, lj, lr);
      }
      __syncthreads();
      // (b) G <- J^T G J.  The diagonal tiles (a, a) are the groups' rotated
      // blocks Q_a^T G_aa Q_a, written by their inner sweeps.  An off-diagonal
      // tile (a < b) becomes Q_a^T G_ab Q_b on MFMA and is stored with its
      // mirror, so G stays exactly symmetric: at most ng (ng - 1) / 2 = 28 of
      // them, two per wave, their loads issued together and their MFMA chains
      // interleaved.
      {
        const int ntile = ng * (ng - 1) / 2;
        bool ok[2];
        int rowa[2], ga[2], gb[2];
        float gv[2][4], qv[2][4];
        f32x4v mt[2], tt[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          int t = wave + u * kWaves, a = 0;
          ok[u] = t < ntile;
          if (ok[u]) {
            while (t >= ng - 1 - a) {        // row a of the strict upper triangle holds ng - 1 - a tiles
              t -= ng - 1 - a;
              ++a;
            }
          }
          const int b = ok[u] ? a + 1 + t : 0;
          ok[u] = ok[u] && !(s_ident[cur][a] && s_ident[cur][b]);   // both sides kept Q = I
          ga[u] = grp[a];
          gb[u] = grp[b];
          rowa[u] = a;
          const int ai = ga[u] & 0xff, aj = ga[u] >> 8, bi = gb[u] & 0xff, bj = gb[u] >> 8;
          const float* Qb = Qs + b * kGrp * kLdQ;
          const int grow = group_index(ai, aj, lr);
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) {
            const int k = 4 * kb + lj;
            gv[u][kb] = G[grow * ld + group_index(bi, bj, k)];
            qv[u][kb] = Qb[k * kLdQ + lr];
          }
          mt[u] = (f32x4v){0.f, 0.f, 0.f, 0.f};
          tt[u] = (f32x4v){0.f, 0.f, 0.f, 0.f};
        }
        if (ok[0] || ok[1]) {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int u = 0; u < 2; ++u) mt[u] = mfma4(gv[u][kb], qv[u][kb], mt[u]);
          // T = Q_a^T M: step i sums k = 4 lj + i, whose M row this lane already holds
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const float* Qa = Qs + rowa[u] * kGrp * kLdQ;
#pragma unroll
            for (int i = 0; i < 4; ++i) qv[u][i] = Qa[(4 * lj + i) * kLdQ + lr];
          }
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int u = 0; u < 2; ++u) tt[u] = mfma4(qv[u][i], mt[u][i], tt[u]);
          // lane (lj, lr) holds T[4 lj + i][lr]: row of group a, column of group b
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            if (ok[u]) {
              const int ai = ga[u] & 0xff, aj = ga[u] >> 8, bi = gb[u] & 0xff, bj = gb[u] >> 8;
              const int gcol = group_index(bi, bj, lr);
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int grw = group_index(ai, aj, 4 * lj + i);
                G[grw * ld + gcol] = tt[u][i];
                G[gcol * ld + grw] = tt[u][i];
              }
            }
          }
        }
      }
      __syncthreads();
      pending = true;
      cur ^= 1;
    }
  }
  if (pending) {
    // the last step's rotation of V
    apply_v(V, ld, (int)(Qs2 - lds_f) + (cur ^ 1) * ng * kGrp * kLdQ, s_grp[cur ^ 1], s_ident[cur ^ 1], ng, dp, 0,
            kWaves, wave, lj, lr);
    __syncthreads();
  }
  if (P.sweeps_done != nullptr && tid == 0 && !tri_ok) P.sweeps_done[unit] = sweeps_run;

  // ---- 3. the m largest eigenvalues (ties by index), after Jacobi ----
  if (!tri_ok && tid < d) {
    const float li = G[tid * ld + tid];
    int rank = 0;
    for (int j = 0; j < d; ++j) {
      const float lk = G[j * ld + j];
      rank += (lk > li) || (lk == li && j < tid);
    }
    if (rank < m) s_order[rank] = tid;
  }
  __syncthreads();

  // ---- 4. W = V_m^T and sigma (U = Delta W^T follows in form_u_kernel) ----
  uint16_t* Wout = P.W + (int64_t)c * P.w_s[0] + (int64_t)l * P.w_s[1] + (int64_t)h * P.w_s[2];
  for (int e = tid; e < m * d; e += kFormThreads) {
    const int k = e / d, j = e % d;
    Wout[(int64_t)k * P.w_s[3] + j] = to_bf16_rne(V[j * ld + s_order[k]]);
  }
  if (P.sigma != nullptr && tid < m) {
    const float lam = G[s_order[tid] * ld + s_order[tid]];
    P.sigma[(int64_t)c * P.sigma_s[0] + (int64_t)l * P.sigma_s[1] + (int64_t)h * P.sigma_s[2] + tid] =
        sqrtf(lam > 0.f ? lam : 0.f);
  }
}

// LDS floats: phase 1 G [dp][gv_ld] and the staged parts [3][dp][kGramRows] bf16;
// phase 2 G and V [dp][gv_ld] each, the groups' S [16][17] and two sets of
// their Q [16][17] (the tridiagonal solver's vectors live in that last area)
size_t form_lds_bytes(int dim, int /*m*/) {
  const size_t dp = (size_t)pad16(dim), ld = (size_t)gv_ld((int)dp), ng = dp / (2 * kBlk);
  const size_t f1 = dp * ld + 3 * dp * kGramRows / 2;
  const size_t f2 = 2 * dp * ld + 3 * ng * kGrp * kLdQ;
  return (f1 > f2 ? f1 : f2) * sizeof(float);
}

// ---------------------------------------------------------------------------
// U = Delta W^T, the factor's token side, from the W form_patch_kernel has
// stored (so U W is formed from exactly the kept W).  A wave takes kURows
// token rows of one unit, as 16-row tiles, and the ranks 64 at a time (the
// workgroup's four waves share those 64 W rows, staged once in LDS); the
// products are 16x16x32 bf16 MFMAs with fp32 accumulation.  Delta is read in
// fp32 and split into hi = bf16(Delta) and lo = bf16(Delta - hi), and both
// parts are multiplied, so Delta enters to ~2^-16 relative.  Lane (kg, t)
// holds row t of a tile on k-slots 8 kg .. 8 kg + 7 (A operand), rank t on
// the same slots (B operand), and rows 4 kg .. 4 kg + 3 of rank t of the
// product.  With an orbit the members' rows are averaged in fp32 first.
// ---------------------------------------------------------------------------
constexpr int kURows = 64;            // token rows per wave
constexpr int kUThreads = 256;
constexpr int kURowsPerBlock = kURows * (kUThreads / 64);
constexpr int kUWLd = 144;            // bf16 per staged W row: 288 bytes, so the B-operand reads
                                      // of a half wave (16 rows x 2 pieces) fall on distinct banks

__global__ __launch_bounds__(kUThreads) void form_u_kernel(const FormParams /*by value, read in place*/) {
  const FormParams& P = *static_cast<const FormParams*>((const void*)__builtin_amdgcn_kernarg_segment_ptr());
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = lane & 15, kg = lane >> 4;
  const int n = P.n_tokens, d = P.dim, m = P.m;
  const uint32_t bpu = (uint32_t)((n + kURowsPerBlock - 1) / kURowsPerBlock);   // blocks per unit
  // workgroups go to the 8 XCDs in turn: block b takes the place
  // (b mod 8) * (grid / 8) + b / 8, so that the blocks of one unit share an
  // XCD and read its W from that XCD's L2 (the grid is a multiple of 8)
  const uint32_t place = (blockIdx.x & 7u) * (gridDim.x >> 3) + (blockIdx.x >> 3);
  const uint32_t unit = place / bpu;
  if ((int)unit >= P.n_units) return;
  const int h = (int)(unit % (uint32_t)P.n_heads);
  const int l = (int)((unit / (uint32_t)P.n_heads) % (uint32_t)P.n_layers);
  const int c = (int)(unit / ((uint32_t)P.n_heads * (uint32_t)P.n_layers));
  const int row0 = (int)(place - unit * bpu) * kURowsPerBlock + wave * kURows;
  // (a wave past the unit's rows still takes part in the W staging)
  __shared__ __align__(16) uint16_t s_w[64 * kUWLd];
  const float* delta = P.delta + (int64_t)c * P.delta_s[0] + (int64_t)l * P.delta_s[1] + (int64_t)h * P.delta_s[2];
  const uint16_t* Wu = P.W + (int64_t)c * P.w_s[0] + (int64_t)l * P.w_s[1] + (int64_t)h * P.w_s[2];
  uint16_t* Uu = P.U + (int64_t)c * P.u_s[0] + (int64_t)l * P.u_s[1] + (int64_t)h * P.u_s[2];
  const int ks = (d + 31) / 32;                // k-steps of 32 dims (<= 4)
  // Delta row i, dims [8 kg + 32 s, +8) as fp32 (zero past n or d; d is a multiple of 4)
  auto load_rows = [&](int i, float (&x)[4][8]) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int j = 32 * s + 8 * kg + 4 * hf;
        f32x4v v = {0.f, 0.f, 0.f, 0.f};
        if (s < ks && i < n && j < d) {
          const float* row = delta + (int64_t)i * P.delta_s[3] + j;
          v = *reinterpret_cast<const f32x4v*>(row);
          if (P.n_orbit > 1) {
            for (int o = 1; o < P.n_orbit; ++o) v += *reinterpret_cast<const f32x4v*>(row + (int64_t)o * P.orbit_s);
            v *= P.inv_orbit;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) x[s][4 * hf + e] = v[e];
      }
  };
  for (int r0 = 0; r0 < m; r0 += 64) {
    // W rows r0 .. r0 + 63 into LDS, 16-byte pieces (zero past m or d), once
    // for the workgroup's four waves
    __syncthreads();                           // the previous ranks' W is consumed
#pragma unroll
    for (int q = 0; q < 64 * 16 / kUThreads; ++q) {
      const int e = threadIdx.x + q * kUThreads, rr = e >> 4, j0 = 8 * (e & 15);
      const int r = r0 + rr;
      u32x4v v = {0u, 0u, 0u, 0u};
      if (r < m && j0 < d) {
        const uint16_t* wr = Wu + (int64_t)r * P.w_s[3] + j0;
        if (P.w_vec && j0 + 8 <= d) {
          v = *reinterpret_cast<const u32x4v*>(wr);
        } else {
#pragma unroll
          for (int e2 = 0; e2 < 8; ++e2)
            if (j0 + e2 < d) v[e2 >> 1] |= (uint32_t)wr[e2] << (16 * (e2 & 1));
        }
      }
      *reinterpret_cast<u32x4v*>(s_w + rr * kUWLd + j0) = v;
    }
    __syncthreads();
    // B operands: W rows r0 + 16 ct + t, dims [8 kg + 32 s, +8)
    auto wb = [&](int ct, int s) {
      return *reinterpret_cast<const u32x4v*>(s_w + (16 * ct + t) * kUWLd + 32 * s + 8 * kg);
    };
    for (int rt = 0; rt < kURows / 16; ++rt) {
      const int i0 = row0 + 16 * rt;
      if (i0 >= n) break;                      // uniform in the wave (no barrier inside)
      float x[4][8];
      load_rows(i0 + t, x);
      f32x4v acc[4];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) acc[ct] = (f32x4v){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s < ks) {
          float lo[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) lo[e] = x[s][e] - __uint_as_float((uint32_t)to_bf16_rne(x[s][e]) << 16);
          const bf16x8v ahi = __builtin_bit_cast(bf16x8v, pack_bf16x8(x[s]));
          const bf16x8v alo = __builtin_bit_cast(bf16x8v, pack_bf16x8(lo));
#pragma unroll
          for (int ct = 0; ct < 4; ++ct) {
            const bf16x8v b = __builtin_bit_cast(bf16x8v, wb(ct, s));
            acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, b, acc[ct], 0, 0, 0);
            acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, b, acc[ct], 0, 0, 0);
          }
        }
      }
      if (P.u_pair) {
        // ranks t and t ^ 1 meet by a DPP swap; the even lane stores both
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const int r = r0 + 16 * ct + t;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float nb = dpp_f<0xB1>(acc[ct][q]);
            const int i = i0 + 4 * kg + q;
            if ((t & 1) == 0 && r < m && i < n) {
              uint16_t* dst = Uu + (int64_t)i * P.u_s[3] + r;
              if (r + 1 < m)
                *reinterpret_cast<uint32_t*>(dst) = (uint32_t)to_bf16_rne(acc[ct][q]) | ((uint32_t)to_bf16_rne(nb) << 16);
              else
                *dst = to_bf16_rne(acc[ct][q]);
            }
          }
        }
      } else {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const int r = r0 + 16 * ct + t;
          if (r < m) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int i = i0 + 4 * kg + q;
              if (i < n) Uu[(int64_t)i * P.u_s[3] + r] = to_bf16_rne(acc[ct][q]);
            }
          }
        }
      }
    }
  }
}

hipError_t launch_form_patch(const FormParams& p, hipStream_t s) {
  const size_t lds = form_lds_bytes(p.dim, p.m);
  static std::atomic<bool> lds_set[kMaxDevices];
  const hipError_t e =
      ensure_lds_limit((const void*)form_patch_kernel, (int)form_lds_bytes(kFormMaxDim, kFormMaxDim), lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(form_patch_kernel, dim3((uint32_t)p.n_units), dim3(kFormThreads), lds, s, p);
  const hipError_t e1 = hipGetLastError();
  if (e1 != hipSuccess) return e1;
  // U from the stored W, on the same stream: after the W of every unit
  const int64_t bpu = (p.n_tokens + kURowsPerBlock - 1) / kURowsPerBlock;
  const int64_t blocks = (bpu * p.n_units + 7) / 8 * 8;   // the places past the units return at once
  hipLaunchKernelGGL(form_u_kernel, dim3((uint32_t)blocks), dim3(kUThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace kamera
