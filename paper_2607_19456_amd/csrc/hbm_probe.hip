// hbm_probe.hip -- practical HBM read ceiling of the machine, measured on the
// caller's own buffers: a plain streaming read of two device buffers (the K
// and V caches a decode reads), for the benchmark to report the decode's
// bandwidth as a fraction of what a read-only stream reaches.  Not part of
// the decode; it computes nothing the decode needs.
//
// Pattern: one workgroup of 256 threads per CU, each thread keeping eight
// independent 16-byte non-temporal loads in flight, grid-stride over the two
// buffers taken back to back.  Of the patterns tried on the MI355X (per-
// workgroup contiguous slices or grid-stride; 4, 8, 16 or 32 loads in
// flight; 256 to 4096 workgroups; default or non-temporal cache policy)
// this one read fastest; the default policy was 10-20 % slower.  Each thread
// writes the sum of what it read, so the read cannot be optimised away and
// can be checked.
#include <hip/hip_runtime.h>

#include <cstdint>

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kThreads = 256;
constexpr int kInFlight = 8;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const f4* __restrict__ a,
                                                               size_t na,
                                                               const f4* __restrict__ b,
                                                               size_t nb, float* partial) {
  const size_t total = na + nb;
  const size_t stride = (size_t)gridDim.x * kThreads;
  f4 acc = f4{0.f, 0.f, 0.f, 0.f};
  for (size_t base = (size_t)blockIdx.x * kThreads + threadIdx.x; base < total;
       base += stride * kInFlight) {
    f4 v[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const size_t i = base + (size_t)u * stride;
      v[u] = f4{0.f, 0.f, 0.f, 0.f};
      if (i < total) v[u] = __builtin_nontemporal_load(i < na ? a + i : b + (i - na));
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) acc += v[u];
  }
  partial[(size_t)blockIdx.x * kThreads + threadIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
}

}  // namespace

extern "C" {

// Threads per workgroup: `partial` holds grid * hbm_probe_threads() floats.
int hbm_probe_threads(void) { return kThreads; }

// Reads a_bytes at a and b_bytes at b (device pointers, 16-byte aligned,
// sizes multiples of 16; either size may be 0) with `grid` workgroups on
// `stream` (NULL: the default stream), asynchronously.  partial[w*256 + t]
// receives the sum of the floats thread t of workgroup w read.  Returns 0, or
// 1 for a NULL pointer or misaligned argument, 2 for bad sizes or grid, 3 if
// the launch failed.
int hbm_read_probe(const void* a, size_t a_bytes, const void* b, size_t b_bytes, float* partial,
                   int grid, void* stream) {
  if (!partial || (a_bytes && !a) || (b_bytes && !b)) return 1;
  const auto misaligned = [](const void* p, uintptr_t n) {
    return reinterpret_cast<uintptr_t>(p) % n != 0;
  };
  if ((a_bytes && misaligned(a, 16)) || (b_bytes && misaligned(b, 16)) ||
      misaligned(partial, 4))
    return 1;
  if (a_bytes % 16 || b_bytes % 16 || grid < 1 || grid > 65536) return 2;
  (void)hipGetLastError();
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)grid), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const f4*>(a), a_bytes / 16,
                     static_cast<const f4*>(b), b_bytes / 16, partial);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
