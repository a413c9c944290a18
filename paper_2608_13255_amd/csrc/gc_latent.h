// Device helpers of the per-step kernels: the latent storage codec
// (float32 / bfloat16 vectors, cached or nontemporal access), the sampler
// step from x_t and x0 (Sec. 3.2, the paragraph after Eq. 1), the UniPC
// update on the x0 history, and the XCD-aware block order.
#pragma once

#include "gc_common.h"

namespace gc {

constexpr int kXcds = 8;   // MI355X: 8 XCDs, workgroups dealt round-robin

// Elements per channel vector: 16 bytes (4 float32 or 8 bfloat16), or 8
// bfloat16 bytes when the channel count is not a multiple of 8.
inline int pick_vec(int dtype, int64_t c) { return dtype == GC_F32 ? 4 : (c % 8 == 0 ? 8 : 4); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int BYTES> struct RawT;
template <> struct RawT<16> { using type = uint4; using nt = u32x4; };
template <> struct RawT<8> { using type = uint2; using nt = u32x2; };

// Storage codec for VEC elements of dtype DT packed in one raw vector.
template <int DT, int VEC> struct Codec {
  static constexpr int kBytes = VEC * (DT == GC_F32 ? 4 : 2);
  using Raw = typename RawT<kBytes>::type;
  using NT = typename RawT<kBytes>::nt;

  // cached load: anchor tiles gathered by several target tokens
  __device__ __forceinline__ static Raw load(const void* base, int64_t elem) {
    return *reinterpret_cast<const Raw*>(static_cast<const char*>(base) + elem * (DT == GC_F32 ? 4 : 2));
  }
  // streamed load / store: data touched exactly once per step.  The
  // nontemporal hint keeps it from displacing the gathered anchor tiles in L2.
  __device__ __forceinline__ static Raw load_stream(const void* base, int64_t elem) {
    const NT* p = reinterpret_cast<const NT*>(static_cast<const char*>(base) + elem * (DT == GC_F32 ? 4 : 2));
    const NT v = __builtin_nontemporal_load(p);
    Raw r;
    __builtin_memcpy(&r, &v, sizeof(Raw));
    return r;
  }
  __device__ __forceinline__ static void store_stream(void* base, int64_t elem, const Raw& r) {
    NT v;
    __builtin_memcpy(&v, &r, sizeof(Raw));
    __builtin_nontemporal_store(v, reinterpret_cast<NT*>(static_cast<char*>(base) + elem * (DT == GC_F32 ? 4 : 2)));
  }
  __device__ __forceinline__ static void unpack(const Raw& r, float (&f)[VEC]) {
    const uint32_t* w = reinterpret_cast<const uint32_t*>(&r);
    if constexpr (DT == GC_F32) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) f[e] = __uint_as_float(w[e]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC / 2; ++e) {
        f[2 * e] = bf16_bits_to_f(w[e] & 0xffffu);
        f[2 * e + 1] = bf16_bits_to_f(w[e] >> 16);
      }
    }
  }
  __device__ __forceinline__ static Raw pack(const float (&f)[VEC]) {
    Raw r;
    uint32_t* w = reinterpret_cast<uint32_t*>(&r);
    if constexpr (DT == GC_F32) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) w[e] = __float_as_uint(f[e]);
    } else {
#pragma unroll
      for (int e = 0; e < VEC / 2; ++e) w[e] = f2_to_bf16x2_bits(f[2 * e], f[2 * e + 1]);
    }
    return r;
  }
};

__device__ __forceinline__ int logical_block(int i, int n_blocks, int remap) {
  if (!remap) return i;
  const int per = (n_blocks + kXcds - 1) / kXcds;   // grid is padded to kXcds * per
  return (i % kXcds) * per + i / kXcds;
}

template <int VEC>
__device__ __forceinline__ void reconstruct_vec(const Recon& r, const float (&xt)[VEC], const float (&x0)[VEC],
                                                float (&xn)[VEC], float (&mo)[VEC]) {
  if (r.kind == GC_DDIM) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float eps = (xt[e] - r.a_t * x0[e]) * r.inv_s_t;
      xn[e] = r.a_n * x0[e] + r.s_n * eps;
      mo[e] = r.pred == GC_PRED_V ? r.a_t * eps - r.s_t * x0[e] : eps;
    }
  } else {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float vel = (xt[e] - x0[e]) * r.inv_sigma;
      xn[e] = xt[e] + r.dsigma * vel;
      mo[e] = vel;
    }
  }
}

// UniPC coefficients of one step (gc_unipc_coeffs, computed in double),
// rounded once to float, and which of the history inputs they read.
struct UniCoef {
  int32_t corr, need_m1, need_m2;
  float c_xprev, c_mk2, c_mk1, c_mk, p_xc, p_mk1, p_mk;
};

inline UniCoef make_unicoef(const gc_unipc_step& st) {
  UniCoef u;
  u.corr = st.use_corrector ? 1 : 0;
  u.need_m2 = (u.corr && st.c_mk2 != 0.0) ? 1 : 0;
  u.need_m1 = ((u.corr && st.c_mk1 != 0.0) || st.p_mk1 != 0.0) ? 1 : 0;
  u.c_xprev = (float)st.c_xprev;
  u.c_mk2 = (float)st.c_mk2;
  u.c_mk1 = (float)st.c_mk1;
  u.c_mk = (float)st.c_mk;
  u.p_xc = (float)st.p_xc;
  u.p_mk1 = (float)st.p_mk1;
  u.p_mk = (float)st.p_mk;
  return u;
}

// UniPC corrector (or the start sample) and predictor, fixed float order:
//   x_c = ((c_xprev x_prev + c_mk2 m_{k-2}) + c_mk1 m_{k-1}) + c_mk m_k   (corrector)
//   x_next = (p_xc x_c + p_mk1 m_{k-1}) + p_mk m_k
template <int VEC>
__device__ __forceinline__ void unipc_vec(const UniCoef& u, const float (&xin)[VEC], const float (&m2)[VEC],
                                          const float (&m1)[VEC], const float (&mk)[VEC], float (&xc)[VEC],
                                          float (&xn)[VEC]) {
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    xc[e] = u.corr ? ((u.c_xprev * xin[e] + u.c_mk2 * m2[e]) + u.c_mk1 * m1[e]) + u.c_mk * mk[e] : xin[e];
    xn[e] = (u.p_xc * xc[e] + u.p_mk1 * m1[e]) + u.p_mk * mk[e];
  }
}

}  // namespace gc
