// Calls the C ABI's host-side paths -- shape planning, workspace sizing and
// the argument validation of every entry point -- with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code.  No call here reaches a
// kernel launch (each one fails validation first, or only sizes), so it runs
// without a GPU.  Test infrastructure only: tests/test_abi_sanitizers.py
// builds it together with the library source (sanitizers on the host side
// only) and runs it.  Exit status 0 when every status matches the
// documented one.
#include <climits>
#include <cstdint>
#include <cstdio>

#include "decode_attn.h"

static int failures = 0;

static void expect(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAILED: %s\n", what);
    ++failures;
  }
}

int main() {
  // Aligned stand-ins for device pointers: validation never dereferences them.
  alignas(256) static float buf[64];
  float* P = buf;
  int32_t* L = reinterpret_cast<int32_t*>(buf);
  float* mis = buf + 1;  // 4-byte aligned only

  // Planning and sizing over a spread of shapes, including the extremes.
  const int shapes[][6] = {{1, 1, 1, 1, 64, 64},         {1, 1, 1, 128, 64, 64},
                           {4, 64, 8, 131072, 128, 128}, {32, 32, 1, 16384, 128, 128},
                           {3, 40, 5, 77, 64, 128},      {2, 64, 2, 5000, 256, 256},
                           {300, 4, 2, 1000, 64, 64},    {4097, 1, 1, 769, 64, 64},
                           {1, 4, 1, 1 << 21, 64, 64},   {1 << 20, 1, 1, 1, 64, 64}};
  for (const auto& s : shapes) {
    const int c = da_decode_chunk_rows(s[0], s[1], s[2], s[3], s[4], s[5]);
    expect(c > 0 && c % 768 == 0, "chunk rows");
    const size_t w = da_decode_workspace_bytes(s[0], s[1], s[2], s[3], s[4], s[5]);
    const size_t n = da_decode_workspace_counter_bytes(s[0], s[1], s[2], s[3], s[4], s[5]);
    expect(w > 0 && n > 0 && n <= w, "workspace bytes");
    expect(da_decode_workspace_bytes_ex(s[0], s[1], s[2], s[3], s[4], s[5], 0) == w,
           "workspace bytes, library's chunk");
    expect(da_decode_workspace_bytes_ex(s[0], s[1], s[2], s[3], s[4], s[5], 1536) > 0,
           "workspace bytes, explicit chunk");
  }
  // invalid shapes and chunk sizes size to zero
  expect(da_decode_workspace_bytes(1, 3, 2, 10, 64, 64) == 0, "h_kv divides h_q");
  expect(da_decode_workspace_bytes(1, 1, 1, 10, 96, 64) == 0, "d_k supported");
  expect(da_decode_workspace_bytes_ex(1, 1, 1, 10, 64, 64, 384) == 0, "chunk multiple of 768");
  expect(da_decode_workspace_bytes(0, 1, 1, 10, 64, 64) == 0, "B >= 1");
  expect(da_decode_workspace_bytes(INT_MAX, INT_MAX, 1, INT_MAX, 256, 256) == 0,
         "overflowing shapes");
  expect(da_decode_chunk_rows(1, 1, 1, 0, 64, 64) == 0, "n_max >= 1");

  // da_decode_attn validation, in the documented order
  const size_t big = size_t(1) << 40;
  expect(da_decode_attn(nullptr, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_NULL, "null q");
  expect(da_decode_attn(P, P, P, L, 0.125f, nullptr, 1, 1, 1, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_NULL, "null out");
  expect(da_decode_attn(P, P, P, L, 0.125f, P, 1, 3, 2, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_SHAPE, "h_q % h_kv");
  expect(da_decode_attn(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 96, 64, P, big, nullptr) ==
             DA_ERR_UNSUPPORTED, "d_k 96");
  expect(da_decode_attn(mis, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_ALIGN, "misaligned q");
  expect(da_decode_attn(P, P, P, L, 1.f / 0.f, P, 1, 1, 1, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_SCALE, "infinite scale");
  expect(da_decode_attn(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, P, 16, nullptr) ==
             DA_ERR_WORKSPACE, "workspace too small");
  expect(da_decode_attn(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, nullptr, big, nullptr) ==
             DA_ERR_WORKSPACE, "null workspace");

  // the other entry points reject bad arguments the same way
  expect(da_decode_step(P, P, P, nullptr, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, P, big,
                        nullptr) == DA_ERR_NULL, "step: null k_new");
  expect(da_decode_partial(P, P, P, P, nullptr, L, 0.125f, 1, 1, 1, 128, 64, 64, P, big,
                           nullptr) == DA_ERR_NULL, "partial: one of k_new/v_new");
  expect(da_decode_merge(nullptr, nullptr, 1, 1, 1, 128, 64, 64, P, big, nullptr) ==
             DA_ERR_NULL, "merge: null out");
  expect(da_decode_multi(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, 0, P, big, nullptr) ==
             DA_ERR_SHAPE, "multi: T = 0");
  expect(da_decode_multi(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, 1 << 20, P, big,
                         nullptr) == DA_ERR_SHAPE, "multi: T too large");
  expect(da_decode_multi_step(P, P, P, P, P, L, 0.125f, P, 1, 2, 1, 128, 64, 64, 2, P, 16,
                              nullptr) == DA_ERR_WORKSPACE, "multi step: workspace");
  expect(da_decode_multi_ex(P, P, P, L, 0.125f, P, 1, 1, 1, 128, 64, 64, 1, 384, P, big,
                            nullptr) == DA_ERR_SHAPE, "multi ex: chunk rows");
  expect(da_decode_partial_ex(P, P, P, nullptr, nullptr, L, 0.125f, 1, 1, 1, 128, 64, 64, 2, 0,
                              P, 16, nullptr) == DA_ERR_WORKSPACE, "partial ex: workspace");
  expect(da_decode_merge_ex(P, nullptr, 1, 1, 1, 128, 64, 64, 0, 0, P, big, nullptr) ==
             DA_ERR_SHAPE, "merge ex: T = 0");
  expect(da_decode_workspace_reset(nullptr, big, 1, 1, 1, 128, 64, 64, nullptr) == DA_ERR_NULL,
         "reset: null workspace");
  expect(da_decode_workspace_reset(P, 16, 1, 1, 1, 128, 64, 64, nullptr) == DA_ERR_WORKSPACE,
         "reset: workspace below the counter region");
  expect(da_kv_append(P, P, P, P, nullptr, 1, 1, 128, 64, 64, nullptr) == DA_ERR_NULL,
         "append: null len");
  expect(da_kv_append(P, P, P, P, L, 1, 1, 128, 6, 64, nullptr) == DA_ERR_UNSUPPORTED,
         "append: d_k not a multiple of 4");
  expect(da_kv_append(P, P, P, P, L, 0, 1, 128, 64, 64, nullptr) == DA_ERR_SHAPE,
         "append: B = 0");
  expect(da_kv_append_rows(P, P, P, P, L, 1, 1, 128, 64, 64, 0, nullptr) == DA_ERR_SHAPE,
         "append rows: T = 0");

  // Every enumerator (C++ callers cannot form other values; C callers pass
  // plain ints, whose unknown codes the Python suite covers).
  for (int s = DA_OK; s <= DA_ERR_HIP; ++s)
    expect(da_status_string(static_cast<da_status>(s)) != nullptr, "status string");

  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("abi sanitizer driver: all checks passed\n");
  return 0;
}
