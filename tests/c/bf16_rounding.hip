// Test infrastructure: the per-step kernels store bfloat16 through
// gc::f2_to_bf16x2_bits (the hardware's pair conversion plus the canonical-NaN
// rule).  This program checks it against the library's scalar rule
// gc::f_to_bf16_bits (round to nearest even, NaN -> 0x7fc0) on every float
// bit pattern: pairs (u, u + 1) for even u, 2^31 pairs in 256 launches.
// Prints the mismatch count and exits 0 only when it is zero.
#include <cstdio>

#include "gc_common.h"

namespace {

constexpr int kThreads = 256;
constexpr unsigned kBlocks = 1u << 15;   // kBlocks * kThreads = 2^23 pairs per launch

__global__ __launch_bounds__(kThreads) void k_check(uint32_t hi, unsigned long long* bad) {
  const uint32_t i = blockIdx.x * kThreads + threadIdx.x;   // < 2^23
  const uint32_t u = (hi << 24) | (i << 1);
  const float a = __uint_as_float(u), b = __uint_as_float(u | 1u);
  const uint32_t got = gc::f2_to_bf16x2_bits(a, b);
  const uint32_t want = gc::f_to_bf16_bits(a) | (gc::f_to_bf16_bits(b) << 16);
  if (got != want) atomicAdd(bad, 1ull);
}

}  // namespace

int main() {
  unsigned long long* bad = nullptr;
  if (hipMalloc(&bad, sizeof(*bad)) != hipSuccess || hipMemset(bad, 0, sizeof(*bad)) != hipSuccess) {
    std::printf("allocation failed\n");
    return 2;
  }
  for (uint32_t hi = 0; hi < 256; ++hi) hipLaunchKernelGGL(k_check, dim3(kBlocks), dim3(kThreads), 0, 0, hi, bad);
  unsigned long long n = 0;
  const hipError_t e = hipMemcpy(&n, bad, sizeof(n), hipMemcpyDeviceToHost);
  (void)hipFree(bad);
  if (e != hipSuccess) {
    std::printf("hip error: %s\n", hipGetErrorString(e));
    return 2;
  }
  std::printf("bf16 pair conversion: %llu mismatches over 2^32 float bit patterns\n", n);
  return n == 0 ? 0 : 1;
}
