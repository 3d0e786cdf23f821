// Launch parameters passed by value to the gfx950 kernels (kernel arguments),
// built and validated by the host layer in kamera_abi.cpp.
#pragma once

#include <stdint.h>

#include <atomic>

#include <hip/hip_runtime_api.h>

namespace kamera {

constexpr int kThreads = 256;        // 4 wave64 per workgroup
constexpr int kTileTokens = 16;      // tokens per wave tile (MFMA N dimension)
constexpr int kMaxBlocks = 36;       // column blocks per row (head_dim <= 4096)
constexpr int kMaxPairs = 64;        // rotated pairs (rope_dim <= 128)
constexpr int kRgMaxHeads = 8;       // heads of a row taken by one row-group workgroup

enum BlockFlags : int { kBlkPatch = 1, kBlkRotate = 2 };

// Division of n < 2^32 by an invariant divisor d >= 1 as a multiply-high, a
// subtraction, an add and two shifts (Granlund and Montgomery, "Division by
// invariant integers using multiplication", 1994, the unsigned method): with
// l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1 (< 2^32),
// floor(n / d) = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0), t = mulhi(m, n).
// The kernels take their task coordinates this way: the divisors are set on
// the host, and a run-time division costs a long instruction sequence.
struct FastDiv {
  uint32_t m;
  uint32_t s1, s2;
  uint32_t pad_;
};

inline FastDiv make_fast_div(uint32_t d) {       // d >= 1
  uint32_t l = 0;
  while (l < 32 && (uint64_t(1) << l) < d) ++l;
  FastDiv f;
  f.m = (uint32_t)((((uint64_t(1) << l) - d) << 32) / d + 1);
  f.s1 = l > 0 ? 1u : 0u;
  f.s2 = l > 0 ? l - 1 : 0u;
  f.pad_ = 0;
  return f;
}

// (constexpr: callable from device code too)
constexpr uint32_t fast_div(uint32_t n, const FastDiv& f) {
  const uint32_t t = (uint32_t)(((uint64_t)n * f.m) >> 32);
  return (t + ((n - t) >> f.s1)) >> f.s2;
}

// One rotated band: per-pair frequency in revolutions per position unit,
// theta^(-2j/rope_dim) / (2 pi), in fp64, and the coordinate (t, h, w) it uses.
struct RopeParams {
  double rev_freq[kMaxPairs];
  int8_t coord[kMaxPairs];
  int32_t rope_offset;
  int32_t rope_dim;
  int32_t pairing;                   // 0 NeoX, 1 interleaved
  int32_t pad_;
};

struct ColBlock {
  int16_t col0;                      // first column / 8  (column = 8 * col0)
  int8_t nq;                         // width = 32 * nq columns (1..4)
  int8_t flags;                      // kBlkPatch | kBlkRotate
};

struct PlaneParams {
  const uint16_t* in;
  uint16_t* out;
  const uint16_t* U;
  const uint16_t* W;
  int64_t in_s[4];
  int64_t out_s[4];
  int64_t u_s[4];
  int64_t w_s[4];
  int32_t m;
  int32_t m_steps;                   // ceil(m / 32): K-steps of the 16x16x32 MFMA
  int32_t patch_lo;
  int32_t patch_hi;
  int32_t u_vec;                     // 16-byte U loads are legal
  int32_t w_vec;                     // 16-byte W loads are legal
  int32_t n_blocks;
  int32_t block_base;                // index of this plane's first block within a task group
  const int32_t* layer_rank;         // optional per-layer rank (<= m)
  int32_t in_rec, u_rec, out_rec;    // row-group form: bytes of one (chunk, layer) input / U slab and
  int32_t pad_;                      // of one output slab (a layer's pool when paged)
  ColBlock blk[kMaxBlocks];
};

struct Placement {                   // where token i of chunk c lands / sits
  int32_t n_tokens;
  int32_t paged;
  const int32_t* chunk_tokens;
  const int32_t* row_base;
  const int32_t* page_table;
  int32_t pt_stride;
  int32_t page_size;
  int32_t n_pool_pages;
  int32_t pad_;
  uint32_t* status;
};

struct RehydrateParams {
  RopeParams rope;
  PlaneParams plane[2];
  Placement place;
  const int32_t* chunk_pos;
  const int32_t* explicit_pos;
  const int32_t* delta;              // relocation of already-rotated keys, or null
  int64_t explicit_cs;
  int32_t pos_mode;
  int32_t grid_w;
  int32_t patch_post_rope;
  int32_t n_planes;
  int32_t n_chunks, n_layers, n_heads;
  int32_t token_block;               // tokens per workgroup task (multiple of 64)
  int32_t n_tblk;                    // token blocks per chunk
  int32_t per_xcd;                   // tasks per XCD slice of the grid
  int32_t blocks_per_group;          // column blocks of all planes for one (chunk, layer, head, token block)
  int32_t row_group;                 // 0: per-head kernel; 4 or 8: heads per row-group workgroup
  int32_t n_hgroups;                 // row-group: head groups per row
  int32_t unit_tiles;                // row-group: 16-token tiles per (chunk, layer) unit (n_tokens / 16, rounded up)
  int32_t lane_wgs;                  // row-group: workgroups per (plane, head group) lane, set at launch
  int32_t max_wgs;                   // caller's cap on the workgroups of a launch (0: none)
  int32_t block_tiles;               // row-group: > 0 = one workgroup per token block of this many
                                     // tiles (hardware dispatch); 0 = persistent, equal ranges
  int64_t n_tasks;
  // per-head task decode: blocks_per_group, n_tblk, n_heads, n_layers
  FastDiv fd_bpg, fd_tblk, fd_heads, fd_layers;
};

struct ShiftParams {
  RopeParams rope;
  Placement place;
  const int32_t* delta;
  uint16_t* k;
  int64_t k_s[4];
  int32_t n_chunks, n_layers, n_heads;
  int32_t vec_per_row;               // 16-byte vectors of the band per row
  int32_t token_block;
  int32_t n_tblk;
  int32_t per_xcd;
  int32_t pad_;
  int64_t n_tasks;
  FastDiv fd_tblk, fd_layers;        // task decode
};

struct ScatterParams {
  Placement place;
  uint8_t* rows;
  uint8_t* pool;
  int64_t rows_s[3];
  int64_t pool_s[2];
  int64_t row_vecs;                  // 16-byte vectors per row
  int32_t n_chunks, n_layers;
  int32_t token_block;
  int32_t n_tblk;
  int32_t per_xcd;
  int32_t gather;                    // 1: pool -> dense rows
  int64_t n_tasks;
  FastDiv fd_tblk, fd_layers;        // task decode
};

constexpr int kFormMaxDim = 128;     // patch forming: columns of Delta

struct FormParams {
  const float* delta;
  uint16_t* U;
  uint16_t* W;
  float* sigma;
  int32_t* sweeps_done;             // optional, dense per unit
  int64_t delta_s[4];
  int64_t u_s[4];
  int64_t w_s[4];
  int64_t sigma_s[3];
  int64_t orbit_s;                  // elements between orbit members of delta
  int32_t n_chunks, n_layers, n_heads;
  int32_t n_tokens;
  int32_t dim;
  int32_t m;
  int32_t sweeps;
  int32_t n_units;
  int32_t n_orbit;                  // >= 1 deficits averaged per unit
  float inv_orbit;                  // 1 / n_orbit
  int32_t w_vec;                    // W rows 16-byte aligned: 8 entries per load
  int32_t u_pair;                   // U rows 4-byte aligned: 2 ranks per store
};

size_t form_lds_bytes(int dim, int m);

// Raises a kernel's dynamic-LDS limit on the current device the first time it
// is launched there.  `done` is the caller's per-device flag array (one per
// kernel instantiation); two threads that race on a first launch both make
// the same idempotent attribute call.
constexpr int kMaxDevices = 64;
inline hipError_t ensure_lds_limit(const void* fn, int bytes, std::atomic<bool> (&done)[kMaxDevices]) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const bool cached = dev >= 0 && dev < kMaxDevices;
  if (cached && done[dev].load(std::memory_order_acquire)) return hipSuccess;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && cached) done[dev].store(true, std::memory_order_release);
  return e;
}

hipError_t launch_rehydrate(const RehydrateParams& p, hipStream_t s);
hipError_t launch_rehydrate_rows(const RehydrateParams& p, hipStream_t s);
hipError_t launch_form_patch(const FormParams& p, hipStream_t s);
hipError_t launch_shift(const ShiftParams& p, hipStream_t s);
hipError_t launch_scatter(const ScatterParams& p, hipStream_t s);

}  // namespace kamera
