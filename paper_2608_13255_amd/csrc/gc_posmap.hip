// Once-per-asset position-map kernels: area downsample to the latent grid and
// the per-asset bounding box / squared match tolerance.
//
// Both are HBM-streaming reductions (no contraction): each render sample is
// read once.  The downsample sums each block in double in the order of a
// plain row-major loop (rows of the block, then samples in a row), whichever
// kernel runs, so its float result does not depend on the launch shape.
#include "gc_common.h"

namespace gc {
namespace {

constexpr int kBlock = 256;
typedef float f32x4 __attribute__((ext_vector_type(4)));

// One thread per latent pixel, reading its f x f block directly (any f).
__global__ __launch_bounds__(kBlock) void k_downsample(const float* __restrict__ hi, int64_t n_pix,
                                                       int Hr, int Wr, int f, int H, int W,
                                                       float* __restrict__ lo) {
  const int64_t gid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (gid >= n_pix) return;
  const int i = (int)(gid % W);
  const int64_t mj = gid / W;
  const int j = (int)(mj % H);
  const int64_t m = mj / H;
  int n_fg = 0;
  double sx = 0.0, sy = 0.0, sz = 0.0;
  for (int dy = 0; dy < f; ++dy) {
    const float* row = hi + ((m * Hr + (int64_t)j * f + dy) * Wr + (int64_t)i * f) * 3;
    for (int dx = 0; dx < f; ++dx) {
      const float x = row[3 * dx], y = row[3 * dx + 1], z = row[3 * dx + 2];
      if (finite_f(x) && finite_f(y) && finite_f(z)) {
        n_fg += 1;
        sx += (double)x;
        sy += (double)y;
        sz += (double)z;
      }
    }
  }
  float* o = lo + gid * 3;
  if (2 * n_fg < f * f) {
    const float qnan = __uint_as_float(0x7fc00000u);
    o[0] = qnan;
    o[1] = qnan;
    o[2] = qnan;
  } else {
    const double n = (double)n_fg;
    o[0] = (float)(sx / n);
    o[1] = (float)(sy / n);
    o[2] = (float)(sz / n);
  }
}

// Vector variant for f = 4 and 8: one thread per latent pixel, each of its F
// render rows read as 3F/4 aligned 16-byte vectors (the pixel's segment of a
// render row is 3F contiguous floats at a multiple of 48 bytes), kRows rows
// in flight per step.  The strided vectors of one wave tile a contiguous run
// of the render row, so L2 serves the lines neighbouring lanes share (plain
// loads: a nontemporal hint makes those lines miss and halves the rate);
// no LDS and no barrier, and each thread folds its samples in the same
// row-major order as the direct kernel.
template <int F>
__global__ __launch_bounds__(kBlock) void k_downsample_vec(const float* __restrict__ hi, int64_t n_pix, int Hr,
                                                           int Wr, int H, int W, float* __restrict__ lo) {
  constexpr int kRow4 = 3 * F / 4;          // vectors per render-row segment
  constexpr int kRows = 4;                  // rows loaded together
  static_assert(F % 4 == 0, "F must be a multiple of 4");
  const int64_t gid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (gid >= n_pix) return;
  const int i = (int)(gid % W);
  const int64_t mj = gid / W;
  const int j = (int)(mj % H);
  const int64_t m = mj / H;
  const f32x4* src = reinterpret_cast<const f32x4*>(hi + ((m * Hr + (int64_t)j * F) * Wr + (int64_t)i * F) * 3);
  const int64_t rs = (int64_t)Wr * 3 / 4;   // vectors per render row
  int n_fg = 0;
  double sx = 0.0, sy = 0.0, sz = 0.0;
  for (int dy0 = 0; dy0 < F; dy0 += kRows) {
    float buf[kRows][3 * F];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int c = 0; c < kRow4; ++c) {
        const f32x4 q = src[(int64_t)(dy0 + r) * rs + c];
        buf[r][4 * c] = q.x;
        buf[r][4 * c + 1] = q.y;
        buf[r][4 * c + 2] = q.z;
        buf[r][4 * c + 3] = q.w;
      }
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int dx = 0; dx < F; ++dx) {
        const float x = buf[r][3 * dx], y = buf[r][3 * dx + 1], z = buf[r][3 * dx + 2];
        if (finite_f(x) && finite_f(y) && finite_f(z)) {
          n_fg += 1;
          sx += (double)x;
          sy += (double)y;
          sz += (double)z;
        }
      }
  }
  float* o = lo + gid * 3;
  if (2 * n_fg < F * F) {
    const float qnan = __uint_as_float(0x7fc00000u);
    o[0] = qnan;
    o[1] = qnan;
    o[2] = qnan;
  } else {
    const double n = (double)n_fg;
    o[0] = (float)(sx / n);
    o[1] = (float)(sy / n);
    o[2] = (float)(sz / n);
  }
}

// Order-preserving float <-> uint32 encoding for integer atomics.
__device__ __forceinline__ uint32_t enc_ord(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float dec_ord(uint32_t e) {
  return __uint_as_float((e & 0x80000000u) ? (e & 0x7fffffffu) : ~e);
}

// bbox[b] is used as the accumulator while the reduction runs:
// words 0..2 encoded min, 3..5 encoded max, 7 = 1 once a foreground sample is seen.
__global__ void k_bbox_init(uint32_t* __restrict__ acc, int B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  uint32_t* a = acc + (int64_t)b * 8;
  const uint32_t pinf = 0xFF800000u, ninf = 0x007FFFFFu;  // enc(+inf), enc(-inf)
  a[0] = pinf; a[1] = pinf; a[2] = pinf;
  a[3] = ninf; a[4] = ninf; a[5] = ninf;
  a[6] = 0u; a[7] = 0u;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}

// grid (chunks, B): every thread folds a strided slice of asset b's samples;
// waves reduce with cross-lane shuffles, the block through LDS, and one
// thread per block issues the atomics.
__global__ __launch_bounds__(kBlock) void k_bbox_accum(const float* __restrict__ pos, int64_t per_asset,
                                                       uint32_t* __restrict__ acc) {
  __shared__ uint32_t part[kBlock / 64][7];
  const int b = blockIdx.y;
  const float* p = pos + (int64_t)b * per_asset * 3;
  uint32_t mn[3] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  uint32_t mx[3] = {0u, 0u, 0u};
  bool any = false;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < per_asset; q += stride) {
    const float x = p[3 * q], y = p[3 * q + 1], z = p[3 * q + 2];
    if (!(finite_f(x) && finite_f(y) && finite_f(z))) continue;
    any = true;
    const uint32_t e[3] = {enc_ord(x), enc_ord(y), enc_ord(z)};
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      mn[c] = min(mn[c], e[c]);
      mx[c] = max(mx[c], e[c]);
    }
  }
  const uint32_t seen = __ballot(any) ? 1u : 0u;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    mn[c] = wave_min_u32(mn[c]);
    mx[c] = wave_max_u32(mx[c]);
  }
  const int wv = threadIdx.x / 64;
  if (__lane_id() == 0) {
    for (int c = 0; c < 3; ++c) {
      part[wv][c] = mn[c];
      part[wv][3 + c] = mx[c];
    }
    part[wv][6] = seen;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t bmn[3] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu}, bmx[3] = {0u, 0u, 0u}, bseen = 0u;
    for (int w = 0; w < kBlock / 64; ++w) {
      for (int c = 0; c < 3; ++c) {
        bmn[c] = min(bmn[c], part[w][c]);
        bmx[c] = max(bmx[c], part[w][3 + c]);
      }
      bseen |= part[w][6];
    }
    if (bseen) {
      uint32_t* a = acc + (int64_t)b * 8;
      for (int c = 0; c < 3; ++c) {
        atomicMin(a + c, bmn[c]);
        atomicMax(a + 3 + c, bmx[c]);
      }
      atomicOr(a + 7, 1u);
    }
  }
}

__global__ void k_bbox_final(uint32_t* __restrict__ acc, int B, float tol_frac) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  uint32_t* a = acc + (int64_t)b * 8;
  float* o = reinterpret_cast<float*>(a);
  if (a[7] == 0u) {
    for (int c = 0; c < 8; ++c) o[c] = 0.0f;
    return;
  }
  float mn[3], mx[3];
  for (int c = 0; c < 3; ++c) {
    mn[c] = dec_ord(a[c]);
    mx[c] = dec_ord(a[3 + c]);
  }
  const float ex = mx[0] - mn[0], ey = mx[1] - mn[1], ez = mx[2] - mn[2];
  const float d2 = (ex * ex + ey * ey) + ez * ez;
  const float tf2 = tol_frac * tol_frac;
  for (int c = 0; c < 3; ++c) {
    o[c] = mn[c];
    o[3 + c] = mx[c];
  }
  o[6] = tf2 * d2;
  o[7] = 0.0f;
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" int gc_posmap_downsample(const float* pos_hi, int64_t n_maps, int Hr, int Wr, int f,
                                    float* pos_lat, hipStream_t stream) {
  clear_error();
  if (!pos_hi || !pos_lat) return fail(GC_ERR_ARG, "downsample: null pointer");
  if (n_maps < 0 || Hr < 1 || Wr < 1) return fail(GC_ERR_SHAPE, "downsample: bad shape n_maps=%lld Hr=%d Wr=%d",
                                                 (long long)n_maps, Hr, Wr);
  if (f < 1 || f > 64 || Hr % f || Wr % f)
    return fail(GC_ERR_SHAPE, "downsample: factor %d must be in [1, 64] and divide Hr=%d, Wr=%d", f, Hr, Wr);
  const int H = Hr / f, W = Wr / f;
  if (H > GC_MAX_GRID || W > GC_MAX_GRID)
    return fail(GC_ERR_CAPACITY, "downsample: latent grid %dx%d exceeds %d", H, W, GC_MAX_GRID);
  if (!aligned16(pos_hi) || !aligned16(pos_lat)) return fail(GC_ERR_ALIGN, "downsample: pointers must be 16-byte aligned");
  const size_t nin = (size_t)n_maps * Hr * Wr * 3 * 4, nout = (size_t)n_maps * H * W * 3 * 4;
  if (overlaps(pos_hi, nin, pos_lat, nout)) return fail(GC_ERR_ALIAS, "downsample: output overlaps input");
  const int64_t n_pix = n_maps * (int64_t)H * W;
  if (n_pix == 0) return GC_OK;
  const int64_t blocks = (n_pix + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return fail(GC_ERR_CAPACITY, "downsample: too many latent pixels");
  if (f == 8) {
    hipLaunchKernelGGL(k_downsample_vec<8>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, pos_hi, n_pix, Hr, Wr, H,
                       W, pos_lat);
  } else if (f == 4) {
    hipLaunchKernelGGL(k_downsample_vec<4>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, pos_hi, n_pix, Hr, Wr, H,
                       W, pos_lat);
  } else {
    hipLaunchKernelGGL(k_downsample, dim3((unsigned)blocks), dim3(kBlock), 0, stream, pos_hi, n_pix, Hr, Wr, f, H,
                       W, pos_lat);
  }
  return after_launch(stream, "gc_posmap_downsample");
}

extern "C" int gc_posmap_bbox(const float* pos, int B, int N, int H, int W, float tol_frac, float* bbox,
                              hipStream_t stream) {
  clear_error();
  if (!pos || !bbox) return fail(GC_ERR_ARG, "bbox: null pointer");
  if (B < 1 || N < 1 || H < 1 || W < 1) return fail(GC_ERR_SHAPE, "bbox: bad shape B=%d N=%d H=%d W=%d", B, N, H, W);
  if (B > 65535) return fail(GC_ERR_CAPACITY, "bbox: B=%d exceeds 65535", B);
  if (!(tol_frac > 0.0f && tol_frac <= 1.0f)) return fail(GC_ERR_ARG, "bbox: tol_frac %g outside (0, 1]", tol_frac);
  if (!aligned16(pos) || !aligned16(bbox)) return fail(GC_ERR_ALIGN, "bbox: pointers must be 16-byte aligned");
  const int64_t per = (int64_t)N * H * W;
  if (overlaps(pos, (size_t)B * per * 12, bbox, (size_t)B * 32)) return fail(GC_ERR_ALIAS, "bbox: output overlaps input");
  uint32_t* acc = reinterpret_cast<uint32_t*>(bbox);
  hipLaunchKernelGGL(k_bbox_init, dim3((B + 63) / 64), dim3(64), 0, stream, acc, B);
  // enough blocks to stream the maps, few enough that the per-block atomics
  // on the asset's eight words stay cheap
  int64_t chunks = (per + 16 * kBlock - 1) / (16 * kBlock);
  if (chunks > 256) chunks = 256;
  if (chunks < 1) chunks = 1;
  hipLaunchKernelGGL(k_bbox_accum, dim3((unsigned)chunks, B), dim3(kBlock), 0, stream, pos, per, acc);
  hipLaunchKernelGGL(k_bbox_final, dim3((B + 63) / 64), dim3(64), 0, stream, acc, B, tol_frac);
  return after_launch(stream, "gc_posmap_bbox");
}
