// Correspondence builder: G_{A->v} for every non-anchor view of every asset,
// for one anchor set (once per asset and anchor set; the rotation has only a
// few distinct sets, so the host caches one build per set).
//
// One thread per target token.  For each anchor the thread projects the
// token's 3D point, tests the 2x2 footprint taps against the tolerance,
// keeps the K nearest, forms the area weights and finally divides by the
// number of anchors that see the token.  Every float operation is written in
// a fixed order and the library is compiled without contraction, so the
// tap choice (an integer decision taken in float) is reproducible exactly.
//
// Coverage statistics are reduced with wavefront ballots: each wave counts
// its visible pairs / pixels / taps with a ballot + popcount and one lane
// adds them to the asset's counters.
#include "gc_common.h"

namespace gc {
namespace {

constexpr int kBlock = 256;

struct BuildArgs {
  const float* pos;
  const gc_camera* cams;
  const float* bbox;
  int32_t* corr;
  float* weights;
  uint32_t* stats;
  int N, H, W, a, K, NT;
  int32_t anchor_view[GC_MAX_ANCHORS];
  int32_t target_view[GC_MAX_VIEWS];
};

__global__ void k_zero_u32(uint32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

__device__ __forceinline__ uint32_t wave_count(bool pred) {
  return (uint32_t)__popcll(__ballot(pred));
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v += (uint32_t)__shfl_xor((int)v, o);
  return v;
}

// grid: x = pixel blocks, y = b * NT + target slot.
__global__ __launch_bounds__(kBlock) void k_build(BuildArgs g) {
  const int HW = g.H * g.W;
  const int p = blockIdx.x * kBlock + threadIdx.x;
  const int bt = blockIdx.y;
  const int b = bt / g.NT;
  const int ti = bt - b * g.NT;
  const int v = g.target_view[ti];
  const bool live = p < HW;
  const float tol2 = g.bbox[(int64_t)b * 8 + 6];

  float P[3] = {0.f, 0.f, 0.f};
  bool fg = false;
  if (live) {
    const float* pp = g.pos + (((int64_t)b * g.N + v) * HW + p) * 3;
    P[0] = pp[0];
    P[1] = pp[1];
    P[2] = pp[2];
    fg = finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2]);
  }

  int32_t words[GC_MAX_ANCHORS];
  float wts[GC_MAX_ANCHORS][4];   // per-anchor normalised weights by tap k
  int n_vis = 0;
  int n_taps = 0;
  for (int s = 0; s < g.a; ++s) {
    words[s] = 0;
    for (int k = 0; k < 4; ++k) wts[s][k] = 0.0f;
    if (!fg) continue;
    const int u = g.anchor_view[s];
    const gc_camera cam = g.cams[(int64_t)b * g.N + u];
    const float* R = cam.R;
    const float xc = ((R[0] * P[0] + R[1] * P[1]) + R[2] * P[2]) + cam.t[0];
    const float yc = ((R[3] * P[0] + R[4] * P[1]) + R[5] * P[2]) + cam.t[1];
    const float zc = ((R[6] * P[0] + R[7] * P[1]) + R[8] * P[2]) + cam.t[2];
    float px, py;
    if (cam.model == 0) {
      if (!(zc > 0.0f)) continue;
      px = cam.fx * (xc / zc) + cam.cx;
      py = cam.fy * (yc / zc) + cam.cy;
    } else if (cam.model == 1) {
      px = cam.fx * xc + cam.cx;
      py = cam.fy * yc + cam.cy;
    } else {
      continue;
    }
    if (!(finite_f(px) && finite_f(py))) continue;
    if (px < -2.0f || px > (float)g.W + 2.0f || py < -2.0f || py > (float)g.H + 2.0f) continue;
    const float gx = px - 0.5f, gy = py - 0.5f;
    const float fx0 = floorf(gx), fy0 = floorf(gy);
    const float ax = gx - fx0, ay = gy - fy0;
    const int x0 = (int)fx0, y0 = (int)fy0;
    const float* src = g.pos + ((int64_t)b * g.N + u) * HW * 3;
    bool valid[4];
    float d2[4];
    int nvalid = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int x = x0 + (k & 1), y = y0 + (k >> 1);
      valid[k] = false;
      d2[k] = 0.0f;
      if (x < 0 || x >= g.W || y < 0 || y >= g.H) continue;
      const float* Q = src + ((int64_t)y * g.W + x) * 3;
      const float qx = Q[0], qy = Q[1], qz = Q[2];
      if (!(finite_f(qx) && finite_f(qy) && finite_f(qz))) continue;
      const float dx = qx - P[0], dy = qy - P[1], dz = qz - P[2];
      const float dd = (dx * dx + dy * dy) + dz * dz;
      if (!(dd <= tol2)) continue;
      valid[k] = true;
      d2[k] = dd;
      ++nvalid;
    }
    if (nvalid == 0) continue;
    bool sel[4] = {false, false, false, false};
    if (nvalid <= g.K) {
#pragma unroll
      for (int k = 0; k < 4; ++k) sel[k] = valid[k];
    } else {
      for (int r = 0; r < g.K; ++r) {
        int best = -1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (!valid[k] || sel[k]) continue;
          if (best < 0 || d2[k] < d2[best]) best = k;
        }
        sel[best] = true;
      }
    }
    const float wx[2] = {1.0f - ax, ax};
    const float wy[2] = {1.0f - ay, ay};
    float area[4];
    float S = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      area[k] = sel[k] ? wx[k & 1] * wy[k >> 1] : 0.0f;
      S = S + area[k];
    }
    int mask = 0;
    if (S > 0.0f) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (sel[k] && area[k] > 0.0f) {
          wts[s][k] = area[k] / S;
          mask |= 1 << k;
        }
      }
    } else {
      int best = -1;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (sel[k] && (best < 0 || d2[k] < d2[best])) best = k;
      wts[s][best] = 1.0f;
      mask = 1 << best;
    }
    ++n_vis;
    n_taps += __popc(mask);
    words[s] = (int32_t)((uint32_t)(x0 + 1) | ((uint32_t)(y0 + 1) << 12) | ((uint32_t)mask << 24));
  }

  if (live) {
    const int64_t row = ((int64_t)b * g.NT + ti) * HW + p;
    int32_t* cw = g.corr + row * g.a;
    float* ww = g.weights + row * g.a * g.K;
    const float inv = n_vis > 0 ? (float)n_vis : 1.0f;
    for (int s = 0; s < g.a; ++s) {
      cw[s] = words[s];
      const int mask = (int)(((uint32_t)words[s] >> 24) & 0xFu);
      int j = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (mask & (1 << k)) {
          ww[s * g.K + j] = wts[s][k] / inv;
          ++j;
        }
      }
      for (; j < g.K; ++j) ww[s * g.K + j] = 0.0f;
    }
  }

  if (g.stats) {
    // blocks never straddle assets (grid y is per asset and target), so every
    // lane of a wave adds to the same counters
    const uint32_t c_pairs = wave_sum((uint32_t)n_vis);
    const uint32_t c_pix = wave_count(live && n_vis > 0);
    const uint32_t c_fg = wave_count(live && fg);
    const uint32_t c_taps = wave_sum((uint32_t)n_taps);
    if (__lane_id() == 0 && (c_pairs | c_pix | c_fg | c_taps)) {
      uint32_t* st = g.stats + (int64_t)b * 4;
      atomicAdd(st + 0, c_pairs);
      atomicAdd(st + 1, c_pix);
      atomicAdd(st + 2, c_fg);
      atomicAdd(st + 3, c_taps);
    }
  }
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" int gc_build_correspondence(const float* pos, const gc_camera* cams, int B, int N, int H, int W,
                                       const int32_t* anchors, int a, int K, const float* bbox, int32_t* corr,
                                       float* weights, uint32_t* stats, hipStream_t stream) {
  clear_error();
  if (!pos || !cams || !anchors || !bbox) return fail(GC_ERR_ARG, "build: null input pointer");
  if (B < 1 || N < 1 || H < 1 || W < 1) return fail(GC_ERR_SHAPE, "build: bad shape B=%d N=%d H=%d W=%d", B, N, H, W);
  if (N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "build: N=%d exceeds %d", N, GC_MAX_VIEWS);
  if (H > GC_MAX_GRID || W > GC_MAX_GRID) return fail(GC_ERR_CAPACITY, "build: grid %dx%d exceeds %d", H, W, GC_MAX_GRID);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "build: a=%d outside [1, N=%d]", a, N);
  if (a > GC_MAX_ANCHORS) return fail(GC_ERR_CAPACITY, "build: a=%d exceeds %d", a, GC_MAX_ANCHORS);
  if (K < 1 || K > 4) return fail(GC_ERR_ARG, "build: K=%d outside [1, 4]", K);
  if ((int64_t)B * (N - a) > 65535) return fail(GC_ERR_CAPACITY, "build: B*(N-a) exceeds 65535");
  BuildArgs g{};
  bool is_anchor[GC_MAX_VIEWS] = {};
  for (int s = 0; s < a; ++s) {
    const int u = anchors[s];
    if (u < 0 || u >= N) return fail(GC_ERR_ARG, "build: anchor %d outside [0, %d)", u, N);
    if (is_anchor[u]) return fail(GC_ERR_ARG, "build: anchor %d listed twice", u);
    is_anchor[u] = true;
    g.anchor_view[s] = u;
  }
  const int NT = N - a;
  if (NT > 0 && (!corr || !weights)) return fail(GC_ERR_ARG, "build: null output pointer");
  if (!aligned16(pos) || (corr && !aligned16(corr)) || (weights && !aligned16(weights)))
    return fail(GC_ERR_ALIGN, "build: pos, corr and weights must be 16-byte aligned");
  const size_t HW = (size_t)H * W;
  const size_t n_corr = (size_t)B * NT * HW * a * 4, n_w = (size_t)B * NT * HW * a * K * 4;
  const size_t n_pos = (size_t)B * N * HW * 12;
  if (overlaps(corr, n_corr, pos, n_pos) || overlaps(weights, n_w, pos, n_pos) || overlaps(corr, n_corr, weights, n_w) ||
      overlaps(stats, (size_t)B * 16, corr, n_corr) || overlaps(stats, (size_t)B * 16, weights, n_w))
    return fail(GC_ERR_ALIAS, "build: outputs overlap each other or the position maps");
  int t = 0;
  for (int v = 0; v < N; ++v)
    if (!is_anchor[v]) g.target_view[t++] = v;
  g.pos = pos;
  g.cams = cams;
  g.bbox = bbox;
  g.corr = corr;
  g.weights = weights;
  g.stats = stats;
  g.N = N;
  g.H = H;
  g.W = W;
  g.a = a;
  g.K = K;
  g.NT = NT;
  if (stats) hipLaunchKernelGGL(k_zero_u32, dim3((4 * B + 255) / 256), dim3(256), 0, stream, stats, 4 * B);
  if (NT > 0) {
    const unsigned bx = (unsigned)((HW + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(k_build, dim3(bx, B * NT), dim3(kBlock), 0, stream, g);
  }
  return after_launch(stream, "gc_build_correspondence");
}
