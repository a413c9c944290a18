// Practical HBM ceiling of the GPU, measured by bench.py beside the per-step
// kernels: plain streaming kernels with the per-step kernels' access shape
// (one 16-byte vector per lane, 256-lane blocks, one block per 4 KiB).
// Benchmark infrastructure only; the transport library does not use it.
//
//   ceil_copy   read n16 vectors from src, write them to dst
//   ceil_read   read n16 vectors (a lane whose vector's words XOR to
//               0x9e3779b9 writes it to sink[block], so that the loads are
//               not removed; fill the buffer with anything else)
//   ceil_write  write n16 vectors of a constant
// nontemporal != 0 issues the loads and stores with the nontemporal hint
// (as the per-step kernels stream their data).  Calls are asynchronous on
// the given stream and return the launch status (0 = hipSuccess).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kBlock = 256;
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ v4u ld(const v4u* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  return *p;
}

template <bool NT>
__device__ __forceinline__ void st(v4u* p, v4u v) {
  if constexpr (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

template <bool NT>
__global__ __launch_bounds__(kBlock) void k_copy(const v4u* __restrict__ src, v4u* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n) st<NT>(dst + i, ld<NT>(src + i));
}

template <bool NT>
__global__ __launch_bounds__(kBlock) void k_read(const v4u* __restrict__ src, v4u* __restrict__ sink, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const v4u v = ld<NT>(src + i);
  // a store taken only for a value the compiler cannot rule out keeps the
  // load alive without a reduction (the benchmark's buffers never hold it)
  if ((v.x ^ v.y ^ v.z ^ v.w) == 0x9e3779b9u) sink[blockIdx.x] = v;
}

template <bool NT>
__global__ __launch_bounds__(kBlock) void k_write(v4u* __restrict__ dst, int64_t n, uint32_t value) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n) st<NT>(dst + i, v4u{value, value, value, (uint32_t)i});
}

unsigned blocks_of(int64_t n16) { return (unsigned)((n16 + kBlock - 1) / kBlock); }

}  // namespace

extern "C" int ceil_copy(const void* src, void* dst, int64_t n16, int nontemporal, hipStream_t stream) {
  if (n16 <= 0 || n16 > (int64_t)kBlock * 0x7fffffff) return (int)hipErrorInvalidValue;
  const v4u* s = static_cast<const v4u*>(src);
  v4u* d = static_cast<v4u*>(dst);
  if (nontemporal)
    hipLaunchKernelGGL(k_copy<true>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, s, d, n16);
  else
    hipLaunchKernelGGL(k_copy<false>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, s, d, n16);
  return (int)hipGetLastError();
}

// sink: at least ceil(n16 / 256) vectors
extern "C" int ceil_read(const void* src, int64_t n16, void* sink, int nontemporal, hipStream_t stream) {
  if (n16 <= 0 || n16 > (int64_t)kBlock * 0x7fffffff) return (int)hipErrorInvalidValue;
  const v4u* s = static_cast<const v4u*>(src);
  v4u* k = static_cast<v4u*>(sink);
  if (nontemporal)
    hipLaunchKernelGGL(k_read<true>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, s, k, n16);
  else
    hipLaunchKernelGGL(k_read<false>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, s, k, n16);
  return (int)hipGetLastError();
}

extern "C" int ceil_write(void* dst, int64_t n16, uint32_t value, int nontemporal, hipStream_t stream) {
  if (n16 <= 0 || n16 > (int64_t)kBlock * 0x7fffffff) return (int)hipErrorInvalidValue;
  v4u* d = static_cast<v4u*>(dst);
  if (nontemporal)
    hipLaunchKernelGGL(k_write<true>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, d, n16, value);
  else
    hipLaunchKernelGGL(k_write<false>, dim3(blocks_of(n16)), dim3(kBlock), 0, stream, d, n16, value);
  return (int)hipGetLastError();
}
