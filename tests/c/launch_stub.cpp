// Stand-in for the GPU side of libkamera, for CPU-only builds of the host
// layer (kamera_abi.cpp) under the address, undefined-behaviour and thread
// sanitizers.  Each launch function records the parameters it was handed and
// returns the error the test asked for; nothing touches a GPU.

#include <atomic>
#include <cstring>

#include "kamera_launch.h"
#include "launch_stub.h"

namespace {
std::atomic<int> g_fail{0};           // hipError_t the next launches return
std::atomic<long> g_launches{0};
thread_local kamera::RehydrateParams t_last_rehydrate;
}  // namespace

extern "C" void stub_set_launch_error(int e) { g_fail.store(e); }
extern "C" long stub_launches(void) { return g_launches.load(); }
extern "C" int stub_last_rehydrate_row_group(void) { return t_last_rehydrate.row_group; }
extern "C" long long stub_last_rehydrate_tasks(void) { return (long long)t_last_rehydrate.n_tasks; }
extern "C" int stub_last_rehydrate_block_tiles(void) { return t_last_rehydrate.block_tiles; }

extern "C" const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stub launch error"; }

namespace kamera {

hipError_t launch_rehydrate(const RehydrateParams& p, hipStream_t) {
  // read every byte of the parameters the host layer built
  std::memcpy(&t_last_rehydrate, &p, sizeof(p));
  g_launches.fetch_add(1);
  return static_cast<hipError_t>(g_fail.load());
}

hipError_t launch_shift(const ShiftParams& p, hipStream_t) {
  volatile long sink = 0;
  for (size_t k = 0; k < sizeof(p); ++k) sink += reinterpret_cast<const unsigned char*>(&p)[k];
  g_launches.fetch_add(1);
  return static_cast<hipError_t>(g_fail.load());
}

hipError_t launch_scatter(const ScatterParams& p, hipStream_t) {
  volatile long sink = 0;
  for (size_t k = 0; k < sizeof(p); ++k) sink += reinterpret_cast<const unsigned char*>(&p)[k];
  g_launches.fetch_add(1);
  return static_cast<hipError_t>(g_fail.load());
}

hipError_t launch_form_patch(const FormParams& p, hipStream_t) {
  volatile long sink = 0;
  for (size_t k = 0; k < sizeof(p); ++k) sink += reinterpret_cast<const unsigned char*>(&p)[k];
  g_launches.fetch_add(1);
  return static_cast<hipError_t>(g_fail.load());
}

}  // namespace kamera
