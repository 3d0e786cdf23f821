// gfx950 kernel of the compile-side patch forming (App. A compile step):
// the top-m singular triplets of each deficit Delta (n x d) as the stored
// patch, U = Delta V_m (the singular values folded in) and W = V_m^T.
//
// One 1024-thread workgroup per (chunk, layer, head) unit, everything in LDS:
//   1. Gram matrix G = Delta^T Delta (fp32), Delta streamed in 32-row tiles;
//   2. cyclic Jacobi on G with the round-robin ordering: every step rotates
//      d/2 disjoint (p, q) pairs at once (G <- J^T G J as independent 2x2
//      blocks, V <- V J), sweeps until the off-diagonal mass is negligible;
//   3. rank the eigenvalues (diag G), keep the m largest;
//   4. W[k] = V[:, order[k]]^T and U = Delta V_m, rounded to bf16.
// With an orbit (Sec. 5, reorder) Delta is the mean of the members' deficits,
// formed on the fly wherever a Delta tile is staged.
// The eigenvalues of G are the squared singular values of Delta and its
// eigenvectors the right singular vectors, so U W is the rank-m truncation.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "kamera.h"
#include "kamera_launch.h"

namespace kamera {

namespace {

typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int kFormThreads = 1024;
constexpr int kFormTile = 32;          // Delta rows per staged tile

__device__ __forceinline__ uint16_t to_bf16_rne(float x) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  f32x2 v = {x, 0.0f};
  const bf16x2 r = __builtin_convertvector(v, bf16x2);
  return (uint16_t)(__builtin_bit_cast(uint32_t, r) & 0xffffu);
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

// Row i, columns [4 v4, 4 v4 + 4) of the (orbit-mean) deficit.
__device__ __forceinline__ f32x4v load_delta4(const FormParams& P, const float* delta, int64_t i, int v4) {
  const float* row = delta + i * P.delta_s[3] + 4 * v4;
  f32x4v x = *reinterpret_cast<const f32x4v*>(row);
  if (P.n_orbit > 1) {
    for (int o = 1; o < P.n_orbit; ++o) x += *reinterpret_cast<const f32x4v*>(row + (int64_t)o * P.orbit_s);
    x *= P.inv_orbit;
  }
  return x;
}

}  // namespace

__global__ __launch_bounds__(kFormThreads) void form_patch_kernel(const FormParams /*by value, read in place*/) {
  const FormParams& P = *static_cast<const FormParams*>((const void*)__builtin_amdgcn_kernarg_segment_ptr());
  extern __shared__ __align__(16) float lds_f[];
  __shared__ f32x4v s_pair[64];           // per pair: c, s, t, p | q << 8
  __shared__ int s_order[128];
  __shared__ float s_red[kFormThreads / 64];

  const int unit = blockIdx.x;
  if (unit >= P.n_units) return;
  const int h = unit % P.n_heads;
  const int l = (unit / P.n_heads) % P.n_layers;
  const int c = unit / (P.n_heads * P.n_layers);
  const int d = P.dim, n = P.n_tokens, m = P.m;
  const int ld = d + 1;                      // padded LDS row stride
  float* G = lds_f;                          // [d][d+1]
  float* V = lds_f + d * ld;                 // [d][d+1]; holds Delta tiles in phase 1
  const float* delta = P.delta + (int64_t)c * P.delta_s[0] + (int64_t)l * P.delta_s[1] + (int64_t)h * P.delta_s[2];
  const int tid = threadIdx.x;

  // ---- 1. G = Delta^T Delta: thread owns a 4x4 block (32x32 threads) ----
  {
    const int bi = 4 * (tid >> 5), bj = 4 * (tid & 31);
    const bool own = bi < d && bj < d;
    float acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = 0.f;
    float* T = V;                            // staged tile [kFormTile][d]
    const int vec_per_row = d / 4;
    for (int t0 = 0; t0 < n; t0 += kFormTile) {
      __syncthreads();
      for (int e = tid; e < kFormTile * vec_per_row; e += kFormThreads) {
        const int r = e / vec_per_row, v4 = e % vec_per_row;
        f32x4v x = {0.f, 0.f, 0.f, 0.f};
        if (t0 + r < n) x = load_delta4(P, delta, t0 + r, v4);
        *reinterpret_cast<f32x4v*>(T + r * d + 4 * v4) = x;
      }
      __syncthreads();
      if (own) {
        for (int r = 0; r < kFormTile; ++r) {
          const f32x4v a = *reinterpret_cast<const f32x4v*>(T + r * d + bi);
          const f32x4v b = *reinterpret_cast<const f32x4v*>(T + r * d + bj);
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) acc[x][y] = fmaf(a[x], b[y], acc[x][y]);
        }
      }
    }
    __syncthreads();
    if (own) {
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) G[(bi + x) * ld + bj + y] = acc[x][y];
    }
    // V = I
    for (int e = tid; e < d * d; e += kFormThreads) V[(e / d) * ld + e % d] = (e / d == e % d) ? 1.f : 0.f;
    __syncthreads();
  }

  // ---- 2. cyclic Jacobi, round-robin pair ordering ----
  const int half = d / 2;
  int sweeps_run = 0;
  for (int sweep = 0; sweep < P.sweeps; ++sweep) {
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
    for (int step = 0; step < d - 1; ++step) {
      if (tid < half) {
        // circle method: position 0 fixed, positions 1..d-1 rotate by `step`
        const int k = tid;
        const int pa = k == 0 ? 0 : 1 + (k - 1 + step) % (d - 1);
        const int pb = 1 + (d - 2 - k + step) % (d - 1);
        const int p = pa < pb ? pa : pb, q = pa < pb ? pb : pa;
        const float app = G[p * ld + p], aqq = G[q * ld + q], apq = G[p * ld + q];
        float cc = 1.f, ss = 0.f, t = 0.f;
        if (fabsf(apq) > 1e-30f) {
          // the smaller root of t^2 + 2 theta t - 1 = 0 zeroes G[p][q]
          const float theta = (aqq - app) / (2.f * apq);
          t = (theta >= 0.f ? 1.f : -1.f) / (fabsf(theta) + sqrtf(theta * theta + 1.f));
          cc = 1.f / sqrtf(t * t + 1.f);
          ss = t * cc;
        }
        const f32x4v pr = {cc, ss, t, __int_as_float(p | (q << 8))};
        s_pair[k] = pr;
      }
      __syncthreads();
      // G <- J^T G J in one pass: the pairs partition the indices, so each
      // 2x2 block (rows of pair k, columns of pair k2) is owned by one thread
      // (G, then V: a thread issues all its loads before its stores; the
      // blocks and the V column pairs are disjoint, so no store is read again)
      {
        constexpr int kG = (kFormMaxDim / 2) * (kFormMaxDim / 2) / kFormThreads;
        constexpr int kGb = kG / 2;                // G blocks in two batches (register budget)
#pragma unroll
        for (int u0 = 0; u0 < kG; u0 += kGb) {
          float g[kGb][4];
          f32x4v rr[kGb], rc[kGb];
#pragma unroll
          for (int u = 0; u < kGb; ++u) {
            const int e = tid + (u0 + u) * kFormThreads;
            if (e < half * half) {
              const int k = e / half, k2 = e - k * half;
              rr[u] = s_pair[k];
              rc[u] = s_pair[k2];
              const int p = __float_as_int(rr[u].w) & 0xff, q = __float_as_int(rr[u].w) >> 8;
              const int p2 = __float_as_int(rc[u].w) & 0xff, q2 = __float_as_int(rc[u].w) >> 8;
              g[u][0] = G[p * ld + p2];
              g[u][1] = G[p * ld + q2];
              g[u][2] = G[q * ld + p2];
              g[u][3] = G[q * ld + q2];
            }
          }
#pragma unroll
          for (int u = 0; u < kGb; ++u) {
            const int e = tid + (u0 + u) * kFormThreads;
            if (e < half * half) {
              const f32x4v r = rr[u], r2 = rc[u];
              const int p = __float_as_int(r.w) & 0xff, q = __float_as_int(r.w) >> 8;
              const int p2 = __float_as_int(r2.w) & 0xff, q2 = __float_as_int(r2.w) >> 8;
              if (p == p2) {
                // the pivot block: exact diagonal update, off-diagonal zeroed
                const float apq = g[u][1];
                G[p * ld + p] = g[u][0] - r.z * apq;
                G[q * ld + q] = g[u][3] + r.z * apq;
                G[p * ld + q] = 0.f;
                G[q * ld + p] = 0.f;
              } else {
                const float a1 = r.x * g[u][0] - r.y * g[u][2], e1 = r.y * g[u][0] + r.x * g[u][2];
                const float b1 = r.x * g[u][1] - r.y * g[u][3], f1 = r.y * g[u][1] + r.x * g[u][3];
                G[p * ld + p2] = r2.x * a1 - r2.y * b1;
                G[p * ld + q2] = r2.y * a1 + r2.x * b1;
                G[q * ld + p2] = r2.x * e1 - r2.y * f1;
                G[q * ld + q2] = r2.y * e1 + r2.x * f1;
              }
            }
          }
        }
        constexpr int kV = (kFormMaxDim / 2) * kFormMaxDim / kFormThreads;
        constexpr int kVb = kV / 2;                // V in two batches (register budget)
#pragma unroll
        for (int u0 = 0; u0 < kV; u0 += kVb) {
          float v[kVb][2];
          float vc[kVb], vs[kVb];
          int vp[kVb], vq[kVb];
#pragma unroll
          for (int u = 0; u < kVb; ++u) {
            const int e = tid + (u0 + u) * kFormThreads;
            if (e < half * d) {
              const int k = e / d, i = e - k * d;
              const f32x4v r = s_pair[k];
              vc[u] = r.x;
              vs[u] = r.y;
              vp[u] = i * ld + (__float_as_int(r.w) & 0xff);
              vq[u] = i * ld + (__float_as_int(r.w) >> 8);
              v[u][0] = V[vp[u]];
              v[u][1] = V[vq[u]];
            }
          }
#pragma unroll
          for (int u = 0; u < kVb; ++u) {
            const int e = tid + (u0 + u) * kFormThreads;
            if (e < half * d) {
              V[vp[u]] = vc[u] * v[u][0] - vs[u] * v[u][1];
              V[vq[u]] = vs[u] * v[u][0] + vc[u] * v[u][1];
            }
          }
        }
      }
      __syncthreads();
    }
  }

  if (P.sweeps_done != nullptr && tid == 0) P.sweeps_done[unit] = sweeps_run;

  // ---- 3. the m largest eigenvalues (ties by index) ----
  if (tid < d) {
    const float li = G[tid * ld + tid];
    int rank = 0;
    for (int j = 0; j < d; ++j) {
      const float lj = G[j * ld + j];
      rank += (lj > li) || (lj == li && j < tid);
    }
    if (rank < m) s_order[rank] = tid;
  }
  __syncthreads();

  // ---- 4. W = V_m^T, sigma, and U = Delta V_m ----
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
  // compact V_m [d][m] into G's space, then stream Delta tiles after it
  float* Vm = G;                             // [d][m]
  float* T = G + d * m;                      // [kFormTile][d]
  __syncthreads();
  for (int e = tid; e < d * m; e += kFormThreads) {
    const int j = e / m, k = e % m;
    Vm[j * m + k] = V[j * ld + s_order[k]];
  }
  uint16_t* Uout = P.U + (int64_t)c * P.u_s[0] + (int64_t)l * P.u_s[1] + (int64_t)h * P.u_s[2];
  const int vec_per_row = d / 4;
  for (int t0 = 0; t0 < n; t0 += kFormTile) {
    __syncthreads();
    for (int e = tid; e < kFormTile * vec_per_row; e += kFormThreads) {
      const int r = e / vec_per_row, v4 = e % vec_per_row;
      f32x4v x = {0.f, 0.f, 0.f, 0.f};
      if (t0 + r < n) x = load_delta4(P, delta, t0 + r, v4);
      *reinterpret_cast<f32x4v*>(T + r * d + 4 * v4) = x;
    }
    __syncthreads();
    for (int e = tid; e < kFormTile * m; e += kFormThreads) {
      const int r = e / m, k = e % m;
      if (t0 + r >= n) continue;
      float s = 0.f;
      for (int j = 0; j < d; ++j) s = fmaf(T[r * d + j], Vm[j * m + k], s);
      Uout[(int64_t)(t0 + r) * P.u_s[3] + k] = to_bf16_rne(s);
    }
  }
}

// LDS floats: phase 1 needs G [d][d+1] then the Delta tile after it, phases
// 2-3 G and V [d][d+1] each, phase 4 V_m [d][m] then the Delta tile
size_t form_lds_bytes(int dim, int m) {
  const size_t d = (size_t)dim;
  size_t f = 2 * d * (d + 1);
  f = f > d * (d + 1) + kFormTile * d ? f : d * (d + 1) + kFormTile * d;
  f = f > d * (size_t)m + kFormTile * d ? f : d * (size_t)m + kFormTile * d;
  return f * sizeof(float);
}

hipError_t launch_form_patch(const FormParams& p, hipStream_t s) {
  const size_t lds = form_lds_bytes(p.dim, p.m);
  // the LDS limit is raised once per device (a race only repeats the call)
  static bool attr_set[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64 || !attr_set[dev]) {
    e = hipFuncSetAttribute((const void*)form_patch_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)form_lds_bytes(kFormMaxDim, kFormMaxDim));
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) attr_set[dev] = true;
  }
  hipLaunchKernelGGL(form_patch_kernel, dim3((uint32_t)p.n_units), dim3(kFormThreads), lds, s, p);
  return hipGetLastError();
}

}  // namespace kamera
