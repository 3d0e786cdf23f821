// Device helpers shared by the gfx950 kernels of the Kamera operator:
// vector types, nontemporal 16-byte accesses, bf16 conversions, angle
// evaluation, page-slot lookup, kernel-argument access and the XCD-aware
// task index.
#pragma once

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

constexpr int kRowPad = 16;                          // LDS row padding, bytes

}  // namespace kamera
