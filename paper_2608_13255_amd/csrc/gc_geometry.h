// Device code of the correspondence operator G_{A->v} for one (target token,
// anchor) pair (Sec. 3.2, correspondence operator): projection into the
// anchor camera, the 2x2 footprint around the projection, the per-tap
// tolerance test, the K nearest in-tolerance taps and their normalised area
// weights.  Shared by the builder (which stores the result) and the fused
// on-the-fly transport (which uses it at once), so both take every decision
// with the same float operations in the same order.
#pragma once

#include "gc_common.h"

namespace gc {

struct AnchorTaps {
  int32_t word;   // (x0+1) | (y0+1) << 12 | mask << 24, or 0 when the anchor contributes nothing
  int mask;       // kept taps, bit k for tap (x0 + (k & 1), y0 + (k >> 1))
  float wk[4];    // this anchor's normalised weight of tap k (before the division by n_vis)
};

// P: the target token's 3D point (finite); cam: the anchor's camera;
// src: the anchor view's position map [H][W][3]; tol2: squared tolerance.
__device__ __forceinline__ AnchorTaps anchor_taps(const float (&P)[3], const gc_camera& cam, const float* src, int H,
                                                  int W, int K, float tol2) {
  AnchorTaps o;
  o.word = 0;
  o.mask = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) o.wk[k] = 0.0f;
  const float* R = cam.R;
  const float xc = ((R[0] * P[0] + R[1] * P[1]) + R[2] * P[2]) + cam.t[0];
  const float yc = ((R[3] * P[0] + R[4] * P[1]) + R[5] * P[2]) + cam.t[1];
  const float zc = ((R[6] * P[0] + R[7] * P[1]) + R[8] * P[2]) + cam.t[2];
  float px = 0.f, py = 0.f;
  bool ok = true;
  if (cam.model == 0) {
    ok = zc > 0.0f;
    if (ok) {
      px = cam.fx * (xc / zc) + cam.cx;
      py = cam.fy * (yc / zc) + cam.cy;
    }
  } else if (cam.model == 1) {
    px = cam.fx * xc + cam.cx;
    py = cam.fy * yc + cam.cy;
  } else {
    ok = false;
  }
  ok = ok && finite_f(px) && finite_f(py) &&
       !(px < -2.0f || px > (float)W + 2.0f || py < -2.0f || py > (float)H + 2.0f);
  if (!ok) return o;
  const float gx = px - 0.5f, gy = py - 0.5f;
  const float fx0 = floorf(gx), fy0 = floorf(gy);
  const float ax = gx - fx0, ay = gy - fy0;
  const int x0 = (int)fx0, y0 = (int)fy0;
  bool valid[4];
  float d2[4];
  int nvalid = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int x = x0 + (k & 1), y = y0 + (k >> 1);
    valid[k] = false;
    d2[k] = 0.0f;
    if (x < 0 || x >= W || y < 0 || y >= H) continue;
    const float* Q = src + ((int64_t)y * W + x) * 3;
    const float qx = Q[0], qy = Q[1], qz = Q[2];
    if (!(finite_f(qx) && finite_f(qy) && finite_f(qz))) continue;
    const float dx = qx - P[0], dy = qy - P[1], dz = qz - P[2];
    const float dd = (dx * dx + dy * dy) + dz * dz;
    if (!(dd <= tol2)) continue;
    valid[k] = true;
    d2[k] = dd;
    ++nvalid;
  }
  if (nvalid == 0) return o;
  bool sel[4] = {false, false, false, false};
  if (nvalid <= K) {
#pragma unroll
    for (int k = 0; k < 4; ++k) sel[k] = valid[k];
  } else {
    for (int r = 0; r < K; ++r) {
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
  if (S > 0.0f) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (sel[k] && area[k] > 0.0f) {
        o.wk[k] = area[k] / S;
        o.mask |= 1 << k;
      }
    }
  } else {
    int best = -1;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (sel[k] && (best < 0 || d2[k] < d2[best])) best = k;
#pragma unroll
    for (int k = 0; k < 4; ++k) o.wk[k] = k == best ? 1.0f : 0.0f;
    o.mask = 1 << best;
  }
  o.word = (int32_t)((uint32_t)(x0 + 1) | ((uint32_t)(y0 + 1) << 12) | ((uint32_t)o.mask << 24));
  return o;
}

}  // namespace gc
