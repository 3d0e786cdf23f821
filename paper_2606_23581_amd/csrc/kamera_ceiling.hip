// Measurement kernel, not part of the operator: a copy with the memory traffic
// of a paged rehydrate and none of its arithmetic.  It reads every input row
// (K and V), every U row and every W basis of the call and writes the input
// rows' bits into the pool slots of the same page table, with the work split
// the row-group rehydrate kernel uses (workgroups of 4 heads x one plane, and
// either equal contiguous ranges of 16-token tiles on one resident wave of
// workgroups, or one workgroup per token block handed out by the hardware),
// with 2 or 4 tiles of loads in flight and 2 or 4 workgroups per CU.  Run on
// the same buffers, the best of those variants is the practical ceiling of
// that read:write mix and page pattern on the device.  U and W are folded into one
// XOR word per workgroup so that their loads are not removed.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kHeads = 4;                 // heads per workgroup
constexpr int kThreads = 64 * kHeads;
constexpr int kTile = 16;                 // tokens per tile
constexpr int kKVec = kHeads * kTile * 16 / kThreads;   // 16-byte K vectors per thread and tile (4)
constexpr int kMaxUVec = kHeads * kTile * 8 / kThreads; // U vectors per thread and tile at rank 64 (2)

struct CeilParams {
  const uint16_t* in[2];                  // K, V rows: [c][l][token][head][128] strides in_s
  const uint16_t* U[2];                   // [c][l][head][token][m] strides u_s
  const uint16_t* W[2];                   // [c][l][head][m][128] strides w_s
  uint16_t* pool[2];                      // [l][slot][head][128] strides pool_s
  int64_t in_s[4];
  int64_t u_s[4];
  int64_t w_s[4];
  int64_t pool_s[3];
  const int32_t* page_table;
  uint32_t* sink;
  int32_t pt_stride, page_size;
  int32_t n_chunks, n_layers, n_heads, n_tokens, m;
  int32_t unit_tiles, lane_wgs, n_planes, n_hgroups;
  int32_t block_tiles;                    // > 0: one workgroup per token block of this many tiles
};

struct Regs {
  u32x4 k[kKVec];
  u32x4 u[kMaxUVec];
};

__device__ __forceinline__ u32x4 ld(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void ceiling_paged_copy_kernel(const CeilParams P) {
  const int lanes = P.n_planes * P.n_hgroups;
  const int lane = (int)(blockIdx.x % (uint32_t)lanes);
  const int64_t r = blockIdx.x / (uint32_t)lanes;
  const int64_t per_lane = (int64_t)P.n_chunks * P.n_layers * P.unit_tiles;
  int64_t f_begin = r * per_lane / P.lane_wgs, f_end = (r + 1) * per_lane / P.lane_wgs;
  if (P.block_tiles > 0) {
    const int nb = (P.unit_tiles + P.block_tiles - 1) / P.block_tiles;
    const int64_t u = r / nb;
    const int b = (int)(r - u * nb);
    f_begin = u * P.unit_tiles + (int64_t)b * P.block_tiles;
    f_end = u * P.unit_tiles + min((b + 1) * P.block_tiles, P.unit_tiles);
  }
  const int pl = lane % P.n_planes, h0 = (lane / P.n_planes) * kHeads;
  const int H = min(kHeads, P.n_heads - h0);
  const int tid = threadIdx.x;
  const int cpr = P.m / 8;                // U 16-byte chunks per token row
  uint32_t acc = 0;
  for (int64_t f = f_begin; f < f_end;) {
    const int64_t cl = f / P.unit_tiles;
    const int tile0 = (int)(f - cl * P.unit_tiles);
    const int tile1 = (int)min((int64_t)P.unit_tiles, tile0 + (f_end - f));
    f += tile1 - tile0;
    const int c = (int)(cl / P.n_layers), l = (int)(cl % P.n_layers);
    const uint16_t* in = P.in[pl] + c * P.in_s[0] + l * P.in_s[1] + h0 * P.in_s[3];
    const uint16_t* U = P.U[pl] + c * P.u_s[0] + l * P.u_s[1] + h0 * P.u_s[2];
    const uint16_t* W = P.W[pl] + c * P.w_s[0] + l * P.w_s[1] + h0 * P.w_s[2];
    uint16_t* pool = P.pool[pl] + l * P.pool_s[0] + h0 * P.pool_s[2];
    const int32_t* pt = P.page_table + (int64_t)c * P.pt_stride;
    // the segment's bases: H heads x m ranks x 128 columns
    for (int v = tid; v < H * P.m * 16; v += kThreads) {
      const int h = v / (P.m * 16), k = (v / 16) % P.m, q = v % 16;
      const u32x4 w = ld(W + h * P.w_s[2] + k * P.w_s[3] + 8 * q);
      acc ^= w.x ^ w.y ^ w.z ^ w.w;
    }
    auto load = [&](int tile, Regs& R) {
      const int i0 = tile * kTile;
#pragma unroll
      for (int j = 0; j < kKVec; ++j) {
        const int v = tid + kThreads * j;             // (token, head, chunk): a token's heads are adjacent
        const int t = v / (kHeads * 16), h = (v / 16) % kHeads, q = v % 16;
        R.k[j] = (h < H && i0 + t < P.n_tokens) ? ld(in + (i0 + t) * P.in_s[2] + h * P.in_s[3] + 8 * q)
                                                 : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int j = 0; j < kMaxUVec; ++j) {
        const int v = tid + kThreads * j;             // (head, token, chunk)
        const int h = v / (kTile * 8), t = (v / 8) % kTile, q = v % 8;
        R.u[j] = (h < H && q < cpr && i0 + t < P.n_tokens) ? ld(U + h * P.u_s[2] + (i0 + t) * P.u_s[3] + 8 * q)
                                                         : u32x4{0, 0, 0, 0};
      }
    };
    auto store = [&](int tile, const Regs& R) {
      const int i0 = tile * kTile;
#pragma unroll
      for (int j = 0; j < kKVec; ++j) {
        const int v = tid + kThreads * j;
        const int t = v / (kHeads * 16), h = (v / 16) % kHeads, q = v % 16;
        const int i = i0 + t;
        if (h < H && i < P.n_tokens) {
          const int64_t slot = (int64_t)pt[i / P.page_size] * P.page_size + i % P.page_size;
          __builtin_nontemporal_store(R.k[j], reinterpret_cast<u32x4*>(pool + slot * P.pool_s[1] + h * P.pool_s[2] + 8 * q));
        }
      }
#pragma unroll
      for (int j = 0; j < kMaxUVec; ++j) acc ^= R.u[j].x ^ R.u[j].y ^ R.u[j].z ^ R.u[j].w;
    };
    Regs R[D];                            // D tiles of loads in flight
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (tile0 + d < tile1) load(tile0 + d, R[d]);
    for (int tile = tile0; tile < tile1; tile += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        if (tile + d < tile1) {
          store(tile + d, R[d]);
          if (tile + d + D < tile1) load(tile + d + D, R[d]);
        }
      }
    }
  }
  // one word per workgroup: the loads feed a visible result
  for (int d = 32; d > 0; d >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, d);
  if ((tid & 63) == 0) atomicXor(P.sink + blockIdx.x, acc);
}

}  // namespace

// Copies the K and V rows of a paged rehydrate call (128-column heads, rank m
// a multiple of 8 up to 64, inputs [c][l][token][head][dim] by strides) into
// their pool slots, reading U and W as the rehydrate does, with `depth` (2
// or 4) tiles in flight and at most `wgs_per_cu` (2 or 4) workgroups per CU
// (an LDS reservation caps them).  blocks = 0: one resident wave of
// workgroups with equal ranges; 1: one workgroup per token block (up to 1024
// tokens, shrunk to >= 64 until there are 4096 blocks).  sink: device uint32
// [grid] (see the return value).  Returns the number of workgroups launched,
// or a negative value on a bad argument or a HIP error.
extern "C" int kamera_ceiling_paged_copy(const void* k_in, const void* v_in, const int64_t* in_stride,
                                         const void* u_k, const void* u_v, const int64_t* u_stride,
                                         const void* w_k, const void* w_v, const int64_t* w_stride, int32_t m,
                                         void* k_pool, void* v_pool, const int64_t* pool_stride,
                                         const int32_t* page_table, int32_t pt_stride, int32_t page_size,
                                         int32_t n_chunks, int32_t n_layers, int32_t n_heads, int32_t n_tokens,
                                         int32_t depth, int32_t wgs_per_cu, int32_t blocks, uint32_t* sink,
                                         int32_t sink_len, void* stream) {
  if ((depth != 2 && depth != 4) || (wgs_per_cu != 2 && wgs_per_cu != 4) || (blocks != 0 && blocks != 1) || m <= 0 ||
      m > 64 || m % 8 != 0 || n_heads <= 0 || n_tokens <= 0 || n_chunks <= 0 || n_layers <= 0 ||
      page_size <= 0 || k_in == nullptr || k_pool == nullptr || u_k == nullptr || w_k == nullptr ||
      page_table == nullptr || sink == nullptr ||
      (v_in != nullptr && (u_v == nullptr || w_v == nullptr || v_pool == nullptr)))
    return -1;
  CeilParams P = {};
  P.in[0] = static_cast<const uint16_t*>(k_in);
  P.in[1] = static_cast<const uint16_t*>(v_in);
  P.U[0] = static_cast<const uint16_t*>(u_k);
  P.U[1] = static_cast<const uint16_t*>(u_v);
  P.W[0] = static_cast<const uint16_t*>(w_k);
  P.W[1] = static_cast<const uint16_t*>(w_v);
  P.pool[0] = static_cast<uint16_t*>(k_pool);
  P.pool[1] = static_cast<uint16_t*>(v_pool);
  for (int k = 0; k < 4; ++k) {
    P.in_s[k] = in_stride[k];
    P.u_s[k] = u_stride[k];
    P.w_s[k] = w_stride[k];
  }
  for (int k = 0; k < 3; ++k) P.pool_s[k] = pool_stride[k];
  P.page_table = page_table;
  P.sink = sink;
  P.pt_stride = pt_stride;
  P.page_size = page_size;
  P.n_chunks = n_chunks;
  P.n_layers = n_layers;
  P.n_heads = n_heads;
  P.n_tokens = n_tokens;
  P.m = m;
  P.unit_tiles = (n_tokens + kTile - 1) / kTile;
  P.n_planes = v_in != nullptr ? 2 : 1;
  P.n_hgroups = (n_heads + kHeads - 1) / kHeads;
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -2;
  const void* fn = depth == 2 ? (const void*)ceiling_paged_copy_kernel<2> : (const void*)ceiling_paged_copy_kernel<4>;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, 0) != hipSuccess) return -2;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -2;
  const int resident = (per_cu < wgs_per_cu ? per_cu : wgs_per_cu) * cus;
  const int lanes = P.n_planes * P.n_hgroups;
  const int64_t per_lane = (int64_t)n_chunks * n_layers * P.unit_tiles;
  int64_t g;
  if (blocks) {
    const int64_t units = (int64_t)lanes * n_chunks * n_layers;
    int bt = 1024 / kTile;
    while (bt > 4 && units * ((P.unit_tiles + bt - 1) / bt) < 4096) bt /= 2;
    P.block_tiles = bt;
    g = (int64_t)n_chunks * n_layers * ((P.unit_tiles + bt - 1) / bt);
  } else {
    g = resident / lanes > 0 ? resident / lanes : 1;
    g = g < per_lane ? g : per_lane;
  }
  P.lane_wgs = (int32_t)g;
  if ((int64_t)lanes * g > sink_len) return -1;
  const int grid = (int)(lanes * g);
  // at most wgs_per_cu workgroups per CU: each reserves 1/wgs_per_cu of the
  // 160 KiB of LDS (less a little)
  const int lds = (160 * 1024) / wgs_per_cu - 1024;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) return -2;
  if (depth == 2)
    hipLaunchKernelGGL(ceiling_paged_copy_kernel<2>, dim3(grid), dim3(kThreads), lds, static_cast<hipStream_t>(stream), P);
  else
    hipLaunchKernelGGL(ceiling_paged_copy_kernel<4>, dim3(grid), dim3(kThreads), lds, static_cast<hipStream_t>(stream), P);
  return hipGetLastError() == hipSuccess ? grid : -2;
}
