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

// The operator for one pair runs in three steps so that callers can keep
// several anchors' tap loads in flight: anchor_project (arithmetic only),
// anchor_tap_positions (the four loads, all issued together) and
// anchor_select (the tests, the selection and the weights).  anchor_taps
// composes them for one anchor.

struct AnchorProj {
  bool ok;          // the projection lands within two pixels of the grid
  int x0, y0;       // the footprint's top-left tap
  float ax, ay;     // bilinear fractions
};

// P: the target token's 3D point (finite); cam: the anchor's camera.
__device__ __forceinline__ AnchorProj anchor_project(const float (&P)[3], const gc_camera& cam, int H, int W) {
  AnchorProj o;
  o.ok = false;
  o.x0 = 0;
  o.y0 = 0;
  o.ax = 0.0f;
  o.ay = 0.0f;
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
  o.ok = true;
  o.ax = gx - fx0;
  o.ay = gy - fy0;
  o.x0 = (int)fx0;
  o.y0 = (int)fy0;
  return o;
}

// Positions of the four taps (x0 + (k & 1), y0 + (k >> 1)) of the anchor
// view's map src [H][W][3].  Every load reads a pixel clamped onto the grid,
// so all four are issued without a branch; anchor_select ignores the taps
// that are off the grid (and all of them when the projection failed).
struct TapPos {
  float q[4][3];
};

__device__ __forceinline__ TapPos anchor_tap_positions(const AnchorProj& pj, const float* src, int H, int W) {
  // a view has fewer than 2^24 pixels, so the offsets within it are 32-bit
  const uint32_t xa = (uint32_t)min(max(pj.x0, 0), W - 1), xb = (uint32_t)min(max(pj.x0 + 1, 0), W - 1);
  const uint32_t ra = (uint32_t)min(max(pj.y0, 0), H - 1) * (uint32_t)W;
  const uint32_t rb = (uint32_t)min(max(pj.y0 + 1, 0), H - 1) * (uint32_t)W;
  const uint32_t px[4] = {ra + xa, ra + xb, rb + xa, rb + xb};
  TapPos t;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float* Q = src + px[k] * 3u;
    t.q[k][0] = Q[0];
    t.q[k][1] = Q[1];
    t.q[k][2] = Q[2];
  }
  return t;
}

// The per-tap tolerance test, the K nearest valid taps and their normalised
// area weights; tol2: squared tolerance.
__device__ __forceinline__ AnchorTaps anchor_select(const float (&P)[3], const AnchorProj& pj, const TapPos& tp, int H,
                                                    int W, int K, float tol2) {
  AnchorTaps o;
  o.word = 0;
  o.mask = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) o.wk[k] = 0.0f;
  if (!pj.ok) return o;
  const int x0 = pj.x0, y0 = pj.y0;
  const float ax = pj.ax, ay = pj.ay;
  bool valid[4];
  float d2[4];
  int nvalid = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int x = x0 + (k & 1), y = y0 + (k >> 1);
    valid[k] = false;
    d2[k] = 0.0f;
    if (x < 0 || x >= W || y < 0 || y >= H) continue;
    const float qx = tp.q[k][0], qy = tp.q[k][1], qz = tp.q[k][2];
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

// P: the target token's 3D point (finite); cam: the anchor's camera;
// src: the anchor view's position map [H][W][3]; tol2: squared tolerance.
__device__ __forceinline__ AnchorTaps anchor_taps(const float (&P)[3], const gc_camera& cam, const float* src, int H,
                                                  int W, int K, float tol2) {
  const AnchorProj pj = anchor_project(P, cam, H, W);
  const TapPos tp = anchor_tap_positions(pj, src, H, W);
  return anchor_select(P, pj, tp, H, W, K, tol2);
}

}  // namespace gc
