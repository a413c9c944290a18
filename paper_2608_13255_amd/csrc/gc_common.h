// Internal helpers shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include "geocache.h"

namespace gc {

// ---------------------------------------------------------------------------
// error reporting (host)
// ---------------------------------------------------------------------------
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();
// Map the launch status (hipGetLastError) and, with GC_SYNC_CHECK=1, the
// stream's completion status to GC_OK / GC_ERR_HIP.
int after_launch(hipStream_t stream, const char* what);
// Work items (target tokens x channel vectors) from which a per-step call
// given a visible-token index takes the split launch; smaller steps take the
// dense launch, whose per-token chain has one dependent load fewer (the same
// result bit for bit).  GC_SPLIT_MIN_ITEMS overrides the default 2^18.
int64_t split_min_items();

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return na && nb && a0 < b0 + nb && b0 < a0 + na;
}

inline int dtype_bytes(int dtype) { return dtype == GC_F32 ? 4 : (dtype == GC_BF16 ? 2 : 0); }

// Sampler coefficients, computed on the host in double and rounded once.
struct Recon {
  int32_t kind;     // GC_DDIM / GC_FLOW_EULER
  int32_t pred;     // GC_PRED_*
  float a_t, s_t, inv_s_t, a_n, s_n;   // DDIM: sqrt(abar), sqrt(1-abar), 1/sqrt(1-abar)
  float inv_sigma, dsigma;             // flow: 1/sigma_t, sigma_n - sigma_t
};

// Validate a sampler description and step and fill the coefficients.
int make_recon(const gc_sampler* smp, double t, double t_next, Recon* out);

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool finite_f(float x) {
  return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u;
}

__device__ __forceinline__ float bf16_bits_to_f(uint32_t h) { return __uint_as_float(h << 16); }

// float -> bfloat16 bits, round to nearest even; NaN -> canonical quiet NaN.
__device__ __forceinline__ uint32_t f_to_bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Two floats to a pair of bfloat16 (lo in the low half) with the hardware's
// conversion, which rounds to nearest even exactly as f_to_bf16_bits does
// for every non-NaN float; a NaN becomes the quiet NaN 0x7fc0, as there.
__device__ __forceinline__ uint32_t f2_to_bf16x2_bits(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v.x = (__bf16)lo;
  v.y = (__bf16)hi;
  uint32_t r;
  __builtin_memcpy(&r, &v, 4);
  if (lo != lo) r = (r & 0xffff0000u) | 0x7fc0u;
  if (hi != hi) r = (r & 0x0000ffffu) | 0x7fc00000u;
  return r;
}

}  // namespace gc
