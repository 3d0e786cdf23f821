// The host layer of libkamera (argument validation and launch set-up,
// kamera_abi.cpp) under the CPU sanitizers, linked against stand-in launches
// (launch_stub.cpp) instead of the GPU kernels:
//   - every entry point's struct, valid and with random 4- and 8-byte words
//     overwritten by boundary values, through kamera_validate and through the
//     entry point itself: only documented codes come back, the error text is
//     set exactly on failure, and validation and the call agree;
//   - a launch that the runtime refuses turns into KAMERA_ERR_HIP;
//   - many threads calling at once, each seeing its own error text.
// Built with -fsanitize=address,undefined and with -fsanitize=thread by
// tests/test_sanitizers.py.  Prints "ok" and exits 0 on success.

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <thread>
#include <vector>

#include "kamera.h"
#include "kamera_launch.h"
#include "launch_stub.h"

namespace {

std::atomic<int> g_failures{0};

#define CHECK(cond)                                                                                        \
  do {                                                                                                     \
    if (!(cond)) {                                                                                         \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, kamera_last_error());    \
      g_failures.fetch_add(1);                                                                             \
    }                                                                                                      \
  } while (0)

// device addresses that are never dereferenced: validation only
constexpr uintptr_t kBase = 0x7E0000000000ull;
constexpr uintptr_t kGB = 1ull << 36;
template <typename T>
T* dev(uintptr_t off) {
  return reinterpret_cast<T*>(kBase + off);
}

kamera_rehydrate_args valid_rehydrate() {
  kamera_rehydrate_args a;
  std::memset(&a, 0, sizeof(a));
  a.n_chunks = 2, a.n_layers = 3, a.n_heads = 4, a.head_dim = 128, a.n_tokens = 64;
  a.rope.theta = 1e6, a.rope.rope_dim = 128, a.rope.pairing = KAMERA_PAIR_NEOX, a.rope.n_sections = 1;
  a.pos_mode = KAMERA_POS_LINEAR;
  a.chunk_pos = dev<const int32_t>(0);
  a.n_planes = 2;
  const int64_t st[4] = {3 * 64 * 4 * 128, 64 * 4 * 128, 4 * 128, 128};
  const int64_t us[4] = {3 * 4 * 64 * 16, 4 * 64 * 16, 64 * 16, 16};
  const int64_t ws[4] = {3 * 4 * 16 * 128, 4 * 16 * 128, 16 * 128, 128};
  for (int p = 0; p < 2; ++p) {
    kamera_plane& q = a.plane[p];
    q.in = dev<const void>((1 + p) * kGB);
    q.out = dev<void>((3 + p) * kGB);
    q.U = dev<const void>((5 + p) * kGB);
    q.W = dev<const void>((7 + p) * kGB);
    std::memcpy(q.in_stride, st, sizeof(st));
    std::memcpy(q.out_stride, st, sizeof(st));
    std::memcpy(q.u_stride, us, sizeof(us));
    std::memcpy(q.w_stride, ws, sizeof(ws));
    q.m = 16, q.rotate = 1 - p, q.patch_offset = 0, q.patch_dim = 128;
  }
  return a;
}

kamera_shift_args valid_shift() {
  kamera_shift_args a;
  std::memset(&a, 0, sizeof(a));
  a.n_chunks = 3, a.n_layers = 2, a.n_heads = 4, a.head_dim = 128, a.n_tokens = 50;
  a.rope.theta = 1e4, a.rope.rope_dim = 128, a.rope.pairing = KAMERA_PAIR_INTERLEAVED, a.rope.n_sections = 1;
  a.delta = dev<const int32_t>(0);
  a.k = dev<void>(kGB);
  const int64_t st[4] = {2 * 50 * 4 * 128, 50 * 4 * 128, 4 * 128, 128};
  std::memcpy(a.k_stride, st, sizeof(st));
  return a;
}

kamera_scatter_args valid_scatter() {
  kamera_scatter_args a;
  std::memset(&a, 0, sizeof(a));
  a.n_chunks = 2, a.n_layers = 2, a.n_tokens = 40;
  a.row_bytes = 1024;
  a.rows = dev<void>(kGB);
  a.rows_stride_bytes[0] = 2 * 40 * 1024, a.rows_stride_bytes[1] = 40 * 1024, a.rows_stride_bytes[2] = 1024;
  a.pool = dev<void>(3 * kGB);
  a.pool_stride_bytes[0] = 16 * 16 * 1024, a.pool_stride_bytes[1] = 1024;
  a.page_table = dev<const int32_t>(0);
  a.pt_stride = 3, a.page_size = 16, a.n_pool_pages = 16;
  return a;
}

kamera_form_args valid_form() {
  kamera_form_args a;
  std::memset(&a, 0, sizeof(a));
  a.n_chunks = 2, a.n_layers = 2, a.n_heads = 3, a.n_tokens = 100, a.dim = 128, a.m = 16;
  a.delta = dev<const float>(kGB);
  const int64_t ds[4] = {2 * 3 * 100 * 128, 3 * 100 * 128, 100 * 128, 128};
  std::memcpy(a.delta_stride, ds, sizeof(ds));
  a.U = dev<void>(3 * kGB);
  const int64_t us[4] = {2 * 3 * 100 * 16, 3 * 100 * 16, 100 * 16, 16};
  std::memcpy(a.u_stride, us, sizeof(us));
  a.W = dev<void>(5 * kGB);
  const int64_t ws[4] = {2 * 3 * 16 * 128, 3 * 16 * 128, 16 * 128, 128};
  std::memcpy(a.w_stride, ws, sizeof(ws));
  return a;
}

bool documented(int rc) {
  return rc == KAMERA_OK || rc == KAMERA_ERR_NULL || rc == KAMERA_ERR_SHAPE || rc == KAMERA_ERR_ALIGN ||
         rc == KAMERA_ERR_RANGE || rc == KAMERA_ERR_ALIAS || rc == KAMERA_ERR_UNSUPPORTED;
}

const int32_t kInts[] = {0, 1, -1, 2, 3, 5, 7, 8, 15, 16, 31, 32, 33, 63, 64, 65, 96, 100, 127, 128, 129, 256,
                         512, 576, 1023, 1024, 4096, 4097, 65536, 1 << 20, -(1 << 20), 0x7fffffff,
                         static_cast<int32_t>(0x80000000u)};
const uint64_t kWords[] = {0ull, 1ull, 2ull, 8ull, 16ull, 0xffffffffffffffffull, kBase, kBase + 2, kBase + kGB,
                           kBase + 5 * kGB + 16, 1ull << 40, 0x8000000000000000ull, 0x7fffffffffffffffull,
                           0x3ff0000000000000ull /* 1.0 */, 0x7ff0000000000000ull /* inf */,
                           0x7ff8000000000000ull /* nan */};

// overwrite up to three aligned words of the struct with boundary values
template <typename A>
A mutate(const A& valid, std::mt19937_64& rng) {
  A a = valid;
  unsigned char* b = reinterpret_cast<unsigned char*>(&a);
  const int n_mut = 1 + static_cast<int>(rng() % 3);
  for (int k = 0; k < n_mut; ++k) {
    if (rng() & 1) {
      const size_t off = 4 * (rng() % (sizeof(A) / 4));
      const int32_t v = kInts[rng() % (sizeof(kInts) / sizeof(kInts[0]))];
      std::memcpy(b + off, &v, 4);
    } else {
      const size_t off = 8 * (rng() % (sizeof(A) / 8));
      const uint64_t v = kWords[rng() % (sizeof(kWords) / sizeof(kWords[0]))];
      std::memcpy(b + off, &v, 8);
    }
  }
  return a;
}

int call(int which, const void* a) {
  switch (which) {
    case 0: return kamera_rehydrate(static_cast<const kamera_rehydrate_args*>(a), nullptr);
    case 1: return kamera_shift(static_cast<const kamera_shift_args*>(a), nullptr);
    case 2: return kamera_scatter_paged(static_cast<const kamera_scatter_args*>(a), nullptr);
    case 3: return kamera_gather_paged(static_cast<const kamera_scatter_args*>(a), nullptr);
    default: return kamera_form_patch(static_cast<const kamera_form_args*>(a), nullptr);
  }
}

// validation and the entry point agree on a (mutated) struct
void check_one(int which, const void* a) {
  const int rc = kamera_validate(which, a);
  CHECK(documented(rc));
  CHECK((rc == KAMERA_OK) == (kamera_last_error()[0] == '\0'));
  const int rc2 = call(which, a);
  CHECK(rc2 == rc);
  CHECK((rc2 == KAMERA_OK) == (kamera_last_error()[0] == '\0'));
  if (which == 0 && rc == KAMERA_OK) {
    const int plan = kamera_rehydrate_plan(static_cast<const kamera_rehydrate_args*>(a));
    CHECK(plan >= KAMERA_PLAN_NONE && plan <= KAMERA_PLAN_ROW_GROUP4);
    const int sched = kamera_rehydrate_schedule(static_cast<const kamera_rehydrate_args*>(a));
    CHECK((sched == 0) == (plan == KAMERA_PLAN_NONE || plan == KAMERA_PLAN_PER_HEAD));
    CHECK(sched >= 0 && sched <= KAMERA_SCHEDULE_BLOCKS);
  }
}

void fuzz(uint64_t seed, int iters) {
  std::mt19937_64 rng(seed);
  const kamera_rehydrate_args r = valid_rehydrate();
  const kamera_shift_args s = valid_shift();
  const kamera_scatter_args c = valid_scatter();
  const kamera_form_args f = valid_form();
  for (int it = 0; it < iters; ++it) {
    switch (it % 5) {
      case 0: { const kamera_rehydrate_args a = mutate(r, rng); check_one(0, &a); break; }
      case 1: { const kamera_shift_args a = mutate(s, rng); check_one(1, &a); break; }
      case 2: { const kamera_scatter_args a = mutate(c, rng); check_one(2, &a); break; }
      case 3: { const kamera_scatter_args a = mutate(c, rng); check_one(3, &a); break; }
      default: { const kamera_form_args a = mutate(f, rng); check_one(4, &a); break; }
    }
  }
}

}  // namespace

int main() {
  // the kernels' invariant-divisor division: exact for every dividend below
  // 2^32 (edge values around multiples of d, the extremes, random ones)
  {
    std::mt19937_64 rng(7);
    auto check_d = [&](uint32_t d) {
      const kamera::FastDiv f = kamera::make_fast_div(d);
      const uint32_t edges[] = {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x00FFFFFFu, 0x7FFFFFFFu, 0xFFFFFFFEu,
                                0xFFFFFFFFu, (0xFFFFFFFFu / d) * d, (0xFFFFFFFFu / d) * d - 1};
      for (uint32_t n : edges) CHECK(kamera::fast_div(n, f) == n / d);
      for (int k = 0; k < 64; ++k) {
        const uint32_t n = (uint32_t)rng();
        CHECK(kamera::fast_div(n, f) == n / d);
      }
    };
    for (uint32_t d = 1; d <= 4096; ++d) check_d(d);
    for (int k = 0; k < 4096; ++k) check_d(1u + (uint32_t)(rng() % 0x7FFFFFFFu));
    check_d(0x80000000u);
    check_d(0xFFFFFFFFu);
  }
  // the valid calls pass and launch once each
  {
    const kamera_rehydrate_args r = valid_rehydrate();
    const kamera_shift_args s = valid_shift();
    const kamera_scatter_args c = valid_scatter();
    const kamera_form_args f = valid_form();
    const long before = stub_launches();
    CHECK(kamera_rehydrate(&r, nullptr) == KAMERA_OK);
    CHECK(kamera_shift(&s, nullptr) == KAMERA_OK);
    CHECK(kamera_scatter_paged(&c, nullptr) == KAMERA_OK);
    CHECK(kamera_gather_paged(&c, nullptr) == KAMERA_OK);
    CHECK(kamera_form_patch(&f, nullptr) == KAMERA_OK);
    CHECK(stub_launches() - before == 5);
    CHECK(stub_last_rehydrate_tasks() > 0);
    // the row-group kernel's two schedules reach the launch: token blocks of
    // 64 tokens (this grid is small), or persistent ranges
    kamera_rehydrate_args rb = r;
    rb.kernel = KAMERA_KERNEL_ROW_GROUP4;
    rb.schedule = KAMERA_SCHEDULE_BLOCKS;
    CHECK(kamera_rehydrate(&rb, nullptr) == KAMERA_OK);
    CHECK(stub_last_rehydrate_row_group() == 4 && stub_last_rehydrate_block_tiles() == 4);
    rb.schedule = KAMERA_SCHEDULE_AUTO;
    CHECK(kamera_rehydrate(&rb, nullptr) == KAMERA_OK);
    CHECK(stub_last_rehydrate_row_group() == 4 && stub_last_rehydrate_block_tiles() == 0);
    // a launch the runtime refuses
    stub_set_launch_error(98);
    CHECK(kamera_rehydrate(&r, nullptr) == KAMERA_ERR_HIP);
    CHECK(std::strstr(kamera_last_error(), "launch failed") != nullptr);
    CHECK(kamera_form_patch(&f, nullptr) == KAMERA_ERR_HIP);
    stub_set_launch_error(0);
    // NULL structs
    CHECK(kamera_rehydrate(nullptr, nullptr) == KAMERA_ERR_NULL);
    CHECK(kamera_validate(9, &r) == KAMERA_ERR_SHAPE);
  }
  // the page-table check reads a host copy
  {
    std::vector<int32_t> pt = {3, 1, 2, 0, 7, 5};
    CHECK(kamera_check_page_table(pt.data(), 2, 3, 48, 16, 8) == KAMERA_OK);
    pt[4] = 1;
    CHECK(kamera_check_page_table(pt.data(), 2, 3, 48, 16, 8) == KAMERA_ERR_ALIAS);
    pt[4] = 8;
    CHECK(kamera_check_page_table(pt.data(), 2, 3, 48, 16, 8) == KAMERA_ERR_RANGE);
  }
  // randomised structs on one thread, then on many at once
  fuzz(12345, 20000);
  {
    std::vector<std::thread> ts;
    for (int t = 0; t < 8; ++t) ts.emplace_back([t] {
      fuzz(1000 + t, 4000);
      // each thread sees its own error text
      const kamera_rehydrate_args r = valid_rehydrate();
      kamera_rehydrate_args bad = r;
      bad.n_planes = 3 + t;
      for (int k = 0; k < 200; ++k) {
        CHECK(kamera_validate(0, &bad) == KAMERA_ERR_SHAPE);
        CHECK(std::strstr(kamera_last_error(), "n_planes") != nullptr);
        CHECK(kamera_validate(0, &r) == KAMERA_OK);
        CHECK(kamera_last_error()[0] == '\0');
      }
    });
    for (auto& th : ts) th.join();
  }
  if (g_failures.load() != 0) {
    std::fprintf(stderr, "%d checks failed\n", g_failures.load());
    return 1;
  }
  std::printf("ok\n");
  return 0;
}
