// HBM read-bandwidth probe: the achievable streaming-read ceiling that the
// decode kernels are measured against, beside the 8 TB/s HBM3E figure.
//
// Each lane keeps four independent 16-byte non-temporal loads in flight and
// folds the data into an XOR that is stored only if it equals a value no
// buffer of this probe's inputs produces, so the loads cannot be removed.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gva_probe.h"

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr unsigned kNever = 0x9E3779B9u;

__global__ void __launch_bounds__(kThreads) stream_read_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                               unsigned* sink) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  unsigned acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(src + i);
    const u32x4 b = __builtin_nontemporal_load(src + i + stride);
    const u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride);
    const u32x4 d = __builtin_nontemporal_load(src + i + 3 * stride);
    acc ^= a[0] ^ a[3] ^ b[1] ^ b[2] ^ c[0] ^ c[3] ^ d[1] ^ d[2];
  }
  for (; i < n16; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(src + i);
    acc ^= a[0] ^ a[3];
  }
  if (acc == kNever) sink[0] = acc;
}

}  // namespace

extern "C" int gva_probe_read(const void* buf, int64_t bytes, int32_t workgroups, unsigned* sink,
                              void* stream) {
  if (buf == nullptr || sink == nullptr || bytes < 16 || workgroups < 1) return -1;
  if ((reinterpret_cast<uintptr_t>(buf) & 15) != 0 || (reinterpret_cast<uintptr_t>(sink) & 3) != 0) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(workgroups), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
