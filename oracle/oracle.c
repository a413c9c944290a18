/*
 * Oracle for GeoCache's per-step cross-view transport.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
 * CPU statement of what the transport path computes.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark use it; the
 * product library never links, loads or calls it, and it shares no code with
 * the HIP path.
 *
 * Paper: "GeoCache: Training-Free Acceleration of Multi-View Texture Diffusion
 * via Geometric Delta Transport", Sec. 3.2 (Methodology): the correspondence
 * operator, delta transport (Eq. 1), multi-anchor aggregation, invalid
 * matches, loop order, sampler-consistent reconstruction, and the
 * drift-bounding schedule.
 *
 * Precision:
 *   - every continuous output (area-downsampled positions, tap weights,
 *     transported x0, sampler outputs) is computed in double;
 *   - every quantity that decides an integer (which taps are visible, which
 *     are nearest, which footprint a projection lands in, the tolerance
 *     test) is computed in IEEE float with a fixed left-to-right operation
 *     order, because the GPU takes those decisions in float as well;
 *   - build with -ffp-contract=off -fno-fast-math (no fused multiply-add).
 *
 * Layouts (row-major, C order):
 *   position maps  float [B][N][H][W][3], NaN (any component) = background
 *   latents        [B][N][H][W][C] (float32, or bfloat16 bit patterns)
 *   correspondence int32 [B][N-a][H][W][a]   (target views ascending)
 *   weights        double [B][N-a][H][W][a][K]
 *   cameras        model int32 [B][N], R float [B][N][9] (world->camera,
 *                  row-major), t float [B][N][3], k float [B][N][4]
 *                  = fx, fy, cx, cy in latent-pixel units; pixel i spans
 *                  [i, i+1).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_BF16 1

int orc_version(void) { return 1; }

/* ------------------------------------------------------------------ */
/* bf16 storage                                                         */
/* ------------------------------------------------------------------ */

static float bf16_to_float(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Round a double to the nearest bfloat16 (ties to even), directly. */
static uint16_t double_to_bf16(double x) {
  if (isnan(x)) return 0x7FC0;
  if (isinf(x)) return x > 0 ? 0x7F80 : 0xFF80;
  double ax = fabs(x);
  uint16_t sign = (x < 0 || (x == 0 && signbit(x))) ? 0x8000 : 0;
  if (ax == 0) return sign;
  /* candidate: truncate the float nearest below |x| to bf16, then pick the
   * closer of the two neighbouring bf16 values in exact double arithmetic. */
  float fl = (float)ax;           /* may round up; fix below */
  if ((double)fl > ax) fl = nextafterf(fl, 0.0f);
  uint32_t u;
  memcpy(&u, &fl, 4);
  uint32_t lo_bits = u & 0xFFFF0000u;
  uint32_t hi_bits = lo_bits + 0x00010000u;
  float lo, hi;
  memcpy(&lo, &lo_bits, 4);
  memcpy(&hi, &hi_bits, 4);
  double dlo = ax - (double)lo, dhi = (double)hi - ax;
  uint32_t pick;
  if (dlo < dhi) pick = lo_bits;
  else if (dhi < dlo) pick = hi_bits;
  else pick = ((lo_bits >> 16) & 1) ? hi_bits : lo_bits;
  return (uint16_t)(sign | (pick >> 16));
}

static double load_val(const void* base, int64_t i, int dtype) {
  if (dtype == ORC_F32) return (double)((const float*)base)[i];
  return (double)bf16_to_float(((const uint16_t*)base)[i]);
}

static void store_val(void* base, int64_t i, int dtype, double v) {
  if (dtype == ORC_F32) ((float*)base)[i] = (float)v;
  else ((uint16_t*)base)[i] = double_to_bf16(v);
}

static void copy_val(void* dst, int64_t di, const void* src, int64_t si, int dtype) {
  if (dtype == ORC_F32) ((float*)dst)[di] = ((const float*)src)[si];
  else ((uint16_t*)dst)[di] = ((const uint16_t*)src)[si];
}

/* Round n doubles into the storage dtype. */
int orc_store(const double* x, int64_t n, int dtype, void* out) {
  if (dtype != ORC_F32 && dtype != ORC_BF16) return -3;
  for (int64_t i = 0; i < n; ++i) store_val(out, i, dtype, x[i]);
  return 0;
}

/* ------------------------------------------------------------------ */
/* O1: area downsample of a position map to the latent grid            */
/* ------------------------------------------------------------------ */
/*
 * Position maps give each latent token its 3D surface point (Sec. 3.1, "the
 * rendered position maps provide the 3D coordinates").  A render-resolution
 * map is reduced to the latent grid by averaging each f x f block over its
 * foreground samples (a sample is foreground when all three components are
 * finite).  A block whose foreground covers less than half of it is
 * background.  The mean is taken in double and stored as float.
 */
int orc_downsample(const float* hi, int64_t M, int Hr, int Wr, int f, float* lo) {
  if (f <= 0 || Hr % f || Wr % f) return -2;
  const int H = Hr / f, W = Wr / f;
  for (int64_t m = 0; m < M; ++m) {
    for (int j = 0; j < H; ++j) {
      for (int i = 0; i < W; ++i) {
        int n_fg = 0;
        double s[3] = {0.0, 0.0, 0.0};
        for (int dy = 0; dy < f; ++dy) {
          for (int dx = 0; dx < f; ++dx) {
            const float* p = hi + (((m * Hr) + (int64_t)j * f + dy) * Wr + (int64_t)i * f + dx) * 3;
            if (isfinite(p[0]) && isfinite(p[1]) && isfinite(p[2])) {
              n_fg += 1;
              s[0] += p[0];
              s[1] += p[1];
              s[2] += p[2];
            }
          }
        }
        float* o = lo + ((m * H + j) * (int64_t)W + i) * 3;
        if (2 * n_fg < f * f) {
          o[0] = o[1] = o[2] = NAN;
        } else {
          for (int c = 0; c < 3; ++c) o[c] = (float)(s[c] / (double)n_fg);
        }
      }
    }
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* O2: per-asset bounding box and squared tolerance                    */
/* ------------------------------------------------------------------ */
/*
 * The tolerance is 1% of the bounding-box diagonal (Sec. 3.2, correspondence
 * operator).  The box is taken per asset over every foreground latent sample
 * of every view.  The tolerance is only ever compared against squared float
 * distances, so it is kept squared, in float:
 *   e = max - min per axis;  d2 = (ex*ex + ey*ey) + ez*ez;
 *   tol2 = (tol_frac*tol_frac) * d2.
 * out[b] = {min x,y,z, max x,y,z, tol2, 0}; an asset with no foreground
 * sample gets all zeros.
 */
int orc_bbox(const float* pos, int B, int N, int H, int W, float tol_frac, float* out) {
  const int64_t per = (int64_t)N * H * W;
  for (int b = 0; b < B; ++b) {
    float mn[3] = {INFINITY, INFINITY, INFINITY}, mx[3] = {-INFINITY, -INFINITY, -INFINITY};
    int64_t cnt = 0;
    for (int64_t q = 0; q < per; ++q) {
      const float* p = pos + ((int64_t)b * per + q) * 3;
      if (!(isfinite(p[0]) && isfinite(p[1]) && isfinite(p[2]))) continue;
      ++cnt;
      for (int c = 0; c < 3; ++c) {
        if (p[c] < mn[c]) mn[c] = p[c];
        if (p[c] > mx[c]) mx[c] = p[c];
      }
    }
    float* o = out + (int64_t)b * 8;
    if (cnt == 0) {
      for (int c = 0; c < 8; ++c) o[c] = 0.0f;
      continue;
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
  return 0;
}

/* ------------------------------------------------------------------ */
/* O3: correspondence operator G_{A->v}                                 */
/* ------------------------------------------------------------------ */
/*
 * For every target token p of a non-anchor view v and every anchor u
 * (Sec. 3.2, correspondence operator and multi-anchor aggregation):
 *   1. P = pos_v(p); background -> no source anywhere.
 *   2. Project P into anchor u's camera (float, fixed order).  A pinhole
 *      point with z <= 0, a non-finite projection, or one far off-screen
 *      ([-2, W+2] x [-2, H+2]) sees nothing.
 *   3. Candidate source taps are the 2x2 pixels whose centres surround the
 *      projection: g = proj - 0.5, (x0, y0) = floor(g), a = g - floor(g);
 *      taps k = 0..3 at (x0 + (k&1), y0 + (k>>1)).
 *   4. A tap is in tolerance if it is on the grid, its source point Q is
 *      foreground and |Q - P|^2 <= tol2 (float).  This per-tap test is the
 *      visibility/occlusion test.
 *   5. Keep the K in-tolerance taps nearest in 3D (ties: lower k).
 *   6. Area weights: the overlap of a unit pixel centred on the projection
 *      with each source pixel, i.e. the bilinear weights
 *      (1-ax)(1-ay), ax(1-ay), (1-ax)ay, ax*ay, renormalised over the kept
 *      taps so the anchor's row sums to 1.  If every kept tap has zero area
 *      the nearest kept tap takes weight 1.  Zero-weight taps are dropped.
 *   7. Several anchors: the normalised sum of their transports, i.e. each
 *      visible anchor's row divided by the number n_vis of anchors that see
 *      p.  Rows with no in-tolerance tap stay zero (disocclusion).
 * Output word per (pixel, anchor): bits 0-11 = x0+1, bits 12-23 = y0+1,
 * bits 24-27 = tap mask (bit k = tap k), 0 iff the anchor contributes
 * nothing.  weights[..][s][j] = final weight of the j-th tap set in the mask
 * (ascending k), 0 beyond.
 */
static int anchor_slot_of(const int32_t* anchors, int a, int v) {
  for (int s = 0; s < a; ++s)
    if (anchors[s] == v) return s;
  return -1;
}

int orc_build(const float* pos, const int32_t* cam_model, const float* cam_R, const float* cam_t,
              const float* cam_k, int B, int N, int H, int W, const int32_t* anchors, int a,
              int K, const float* bbox, int32_t* corr, double* weights, int32_t* nvis_out) {
  if (a < 1 || a > N || a > 8 || K < 1 || K > 4 || H < 1 || W < 1 || H > 4094 || W > 4094)
    return -1;
  for (int s = 0; s < a; ++s) {
    if (anchors[s] < 0 || anchors[s] >= N) return -1;
    for (int r = 0; r < s; ++r)
      if (anchors[r] == anchors[s]) return -1;
  }
  const int NT = N - a;
  const int64_t HW = (int64_t)H * W;
  int ti = 0;
  for (int v = 0; v < N; ++v) {
    if (anchor_slot_of(anchors, a, v) >= 0) continue;
    for (int b = 0; b < B; ++b) {
      const float tol2 = bbox[(int64_t)b * 8 + 6];
      for (int64_t p = 0; p < HW; ++p) {
        const int64_t row = ((int64_t)b * NT + ti) * HW + p;
        int32_t* words = corr + row * a;
        double* wrow = weights + row * a * K;
        for (int s = 0; s < a; ++s) words[s] = 0;
        for (int s = 0; s < a * K; ++s) wrow[s] = 0.0;
        const float* P = pos + (((int64_t)b * N + v) * HW + p) * 3;
        double wtap[8][4];
        int masks[8];
        int n_vis = 0;
        for (int s = 0; s < a; ++s) {
          masks[s] = 0;
          for (int k = 0; k < 4; ++k) wtap[s][k] = 0.0;
        }
        if (isfinite(P[0]) && isfinite(P[1]) && isfinite(P[2])) {
          for (int s = 0; s < a; ++s) {
            const int u = anchors[s];
            const int64_t ci = (int64_t)b * N + u;
            const float* R = cam_R + ci * 9;
            const float* t = cam_t + ci * 3;
            const float* kk = cam_k + ci * 4;
            const float xc = ((R[0] * P[0] + R[1] * P[1]) + R[2] * P[2]) + t[0];
            const float yc = ((R[3] * P[0] + R[4] * P[1]) + R[5] * P[2]) + t[1];
            const float zc = ((R[6] * P[0] + R[7] * P[1]) + R[8] * P[2]) + t[2];
            float px, py;
            if (cam_model[ci] == 0) {
              if (!(zc > 0.0f)) continue;
              px = kk[0] * (xc / zc) + kk[2];
              py = kk[1] * (yc / zc) + kk[3];
            } else {
              px = kk[0] * xc + kk[2];
              py = kk[1] * yc + kk[3];
            }
            if (!(isfinite(px) && isfinite(py))) continue;
            if (px < -2.0f || px > (float)W + 2.0f || py < -2.0f || py > (float)H + 2.0f) continue;
            const float gx = px - 0.5f, gy = py - 0.5f;
            const float fx0 = floorf(gx), fy0 = floorf(gy);
            const float ax = gx - fx0, ay = gy - fy0;
            const int x0 = (int)fx0, y0 = (int)fy0;
            int valid[4];
            float d2[4];
            int nvalid = 0;
            for (int k = 0; k < 4; ++k) {
              const int x = x0 + (k & 1), y = y0 + (k >> 1);
              valid[k] = 0;
              d2[k] = 0.0f;
              if (x < 0 || x >= W || y < 0 || y >= H) continue;
              const float* Q = pos + (ci * HW + (int64_t)y * W + x) * 3;
              if (!(isfinite(Q[0]) && isfinite(Q[1]) && isfinite(Q[2]))) continue;
              const float dx = Q[0] - P[0], dy = Q[1] - P[1], dz = Q[2] - P[2];
              const float dd = (dx * dx + dy * dy) + dz * dz;
              if (!(dd <= tol2)) continue;
              valid[k] = 1;
              d2[k] = dd;
              ++nvalid;
            }
            if (nvalid == 0) continue;
            int sel[4] = {0, 0, 0, 0};
            if (nvalid <= K) {
              for (int k = 0; k < 4; ++k) sel[k] = valid[k];
            } else {
              for (int r = 0; r < K; ++r) {
                int best = -1;
                for (int k = 0; k < 4; ++k) {
                  if (!valid[k] || sel[k]) continue;
                  if (best < 0 || d2[k] < d2[best]) best = k;
                }
                sel[best] = 1;
              }
            }
            /* one-dimensional overlap factors (float, as the decision of a
             * zero-area tap is taken in float) */
            const float wx[2] = {1.0f - ax, ax};
            const float wy[2] = {1.0f - ay, ay};
            double area[4];
            double S = 0.0;
            for (int k = 0; k < 4; ++k) {
              area[k] = sel[k] ? (double)wx[k & 1] * (double)wy[k >> 1] : 0.0;
              S += area[k];
            }
            int mask = 0;
            if (S > 0.0) {
              for (int k = 0; k < 4; ++k) {
                if (sel[k] && area[k] > 0.0) {
                  wtap[s][k] = area[k] / S;
                  mask |= 1 << k;
                }
              }
            } else {
              int best = -1;
              for (int k = 0; k < 4; ++k)
                if (sel[k] && (best < 0 || d2[k] < d2[best])) best = k;
              wtap[s][best] = 1.0;
              mask = 1 << best;
            }
            masks[s] = mask;
            ++n_vis;
            words[s] = (int32_t)((uint32_t)(x0 + 1) | ((uint32_t)(y0 + 1) << 12) |
                                 ((uint32_t)mask << 24));
          }
        }
        if (nvis_out) nvis_out[row] = n_vis;
        if (n_vis == 0) continue;
        for (int s = 0; s < a; ++s) {
          int j = 0;
          for (int k = 0; k < 4; ++k) {
            if (masks[s] & (1 << k)) {
              wrow[s * K + j] = wtap[s][k] / (double)n_vis;
              ++j;
            }
          }
        }
      }
    }
    ++ti;
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* O4: delta transport (Eq. 1)                                          */
/* ------------------------------------------------------------------ */
/*
 * One cached step (Sec. 3.2, delta transport and loop order):
 *   anchor view u = A[s]:   x0_out(u) = x0_anchor_new(s)         (the store
 *                           keeps x0(t) for all N views)
 *   target view v not in A: x0_out(v) = x0_prev(v) + G_{A->v}[x0_anchor_new - x0_prev(A)]
 *   tokens with no valid source keep x0_prev unchanged.
 * The sum is formed in double; x0_exact receives the unrounded value and
 * x0_state the value rounded into the storage dtype.
 */
int orc_transport(const void* x0_prev, const void* x0_anew, const int32_t* corr,
                  const double* weights, const int32_t* anchors, int a, int B, int N, int H,
                  int W, int C, int K, int dtype, double* x0_exact, void* x0_state) {
  if (a < 1 || a > N || K < 1 || K > 4 || C < 1) return -1;
  if (dtype != ORC_F32 && dtype != ORC_BF16) return -3;
  const int NT = N - a;
  const int64_t HW = (int64_t)H * W;
  int ti = 0;
  for (int v = 0; v < N; ++v) {
    const int sv = anchor_slot_of(anchors, a, v);
    for (int b = 0; b < B; ++b) {
      for (int64_t p = 0; p < HW; ++p) {
        const int64_t orow = (((int64_t)b * N + v) * HW + p) * C;
        if (sv >= 0) {
          const int64_t irow = (((int64_t)b * a + sv) * HW + p) * C;
          for (int c = 0; c < C; ++c) {
            x0_exact[orow + c] = load_val(x0_anew, irow + c, dtype);
            copy_val(x0_state, orow + c, x0_anew, irow + c, dtype);
          }
          continue;
        }
        const int64_t crow = ((int64_t)b * NT + ti) * HW + p;
        const int32_t* words = corr + crow * a;
        const double* wrow = weights + crow * a * K;
        int n_vis = 0;
        for (int s = 0; s < a; ++s) n_vis += words[s] != 0;
        for (int c = 0; c < C; ++c) {
          const double prev = load_val(x0_prev, orow + c, dtype);
          if (n_vis == 0) {
            x0_exact[orow + c] = prev;
            copy_val(x0_state, orow + c, x0_prev, orow + c, dtype);
            continue;
          }
          double acc = 0.0;
          for (int s = 0; s < a; ++s) {
            const uint32_t word = (uint32_t)words[s];
            if (!word) continue;
            const int x0 = (int)(word & 0xFFFu) - 1;
            const int y0 = (int)((word >> 12) & 0xFFFu) - 1;
            const int mask = (int)((word >> 24) & 0xFu);
            const int u = anchors[s];
            int j = 0;
            for (int k = 0; k < 4; ++k) {
              if (!(mask & (1 << k))) continue;
              const int64_t q = (int64_t)(y0 + (k >> 1)) * W + (x0 + (k & 1));
              const double dnew = load_val(x0_anew, (((int64_t)b * a + s) * HW + q) * C + c, dtype);
              const double dold = load_val(x0_prev, (((int64_t)b * N + u) * HW + q) * C + c, dtype);
              acc += wrow[s * K + j] * (dnew - dold);
              ++j;
            }
          }
          const double out = prev + acc;
          x0_exact[orow + c] = out;
          store_val(x0_state, orow + c, dtype, out);
        }
      }
    }
    if (sv < 0) ++ti;
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* O5: sampler-consistent reconstruction                                */
/* ------------------------------------------------------------------ */
/*
 * From the transported x0 the sampler's own quantities are recovered with
 * the closed forms at the step's noise level (Sec. 3.2, after Eq. 1):
 *   DDIM (eta = 0):  eps = (x_t - sqrt(abar_t) x0) / sqrt(1 - abar_t)
 *                    v   = sqrt(abar_t) eps - sqrt(1 - abar_t) x0
 *                    x_next = sqrt(abar_n) x0 + sqrt(1 - abar_n) eps
 *   flow matching:   x_sigma = (1 - sigma) x0 + sigma eps, velocity
 *                    vel = (x_t - x0) / sigma_t,
 *                    x_next = x_t + (sigma_n - sigma_t) vel   (Euler)
 * abar_t = prod_{i<=t} (1 - beta_i), beta linear from beta_start to
 * beta_end over T steps (0-based), abar_{-1} = 1.
 * pred: 0 none, 1 eps, 2 v (DDIM), 3 velocity (flow).
 */
double orc_alpha_bar(int T, double beta_start, double beta_end, int t) {
  if (t < 0) return 1.0;
  double ab = 1.0;
  for (int i = 0; i <= t; ++i) {
    const double beta = beta_start + (beta_end - beta_start) * (double)i / (double)(T - 1);
    ab *= 1.0 - beta;
  }
  return ab;
}

int orc_reconstruct(const void* x_t, const void* x0, int64_t n, int dtype, int kind, int pred,
                    int T, double beta_start, double beta_end, double t, double t_next,
                    double* x_next, double* model_out) {
  if (dtype != ORC_F32 && dtype != ORC_BF16) return -3;
  if (kind == 0) {
    if (T < 2 || t < 0 || t >= T || t_next >= t || t_next < -1) return -1;
    if (pred != 0 && pred != 1 && pred != 2) return -1;
    const double ab_t = orc_alpha_bar(T, beta_start, beta_end, (int)t);
    const double ab_n = orc_alpha_bar(T, beta_start, beta_end, (int)t_next);
    const double a_t = sqrt(ab_t), s_t = sqrt(1.0 - ab_t);
    const double a_n = sqrt(ab_n), s_n = sqrt(1.0 - ab_n);
    for (int64_t i = 0; i < n; ++i) {
      const double xt = load_val(x_t, i, dtype), z = load_val(x0, i, dtype);
      const double eps = (xt - a_t * z) / s_t;
      x_next[i] = a_n * z + s_n * eps;
      if (pred == 1 && model_out) model_out[i] = eps;
      if (pred == 2 && model_out) model_out[i] = a_t * eps - s_t * z;
    }
    return 0;
  }
  if (kind == 1) {
    if (!(t > 0.0) || t > 1.0 || t_next < 0.0 || t_next > t) return -1;
    if (pred != 0 && pred != 3) return -1;
    for (int64_t i = 0; i < n; ++i) {
      const double xt = load_val(x_t, i, dtype), z = load_val(x0, i, dtype);
      const double vel = (xt - z) / t;
      x_next[i] = xt + (t_next - t) * vel;
      if (pred == 3 && model_out) model_out[i] = vel;
    }
    return 0;
  }
  return -1;
}

/* ------------------------------------------------------------------ */
/* O6: host schedule                                                    */
/* ------------------------------------------------------------------ */
/*
 * Anchors rotate every cached step and every view returns to the anchor set
 * within ceil(N/a) cached steps (Sec. 3.2, batch-sliced anchor forward).
 * Rule: A_c = {(c + floor(j*N/a)) mod N : j < a}, slots in ascending view
 * order.
 */
int orc_anchors(int N, int a, int64_t c, int32_t* out) {
  if (a < 1 || a > N || c < 0) return -1;
  for (int j = 0; j < a; ++j) out[j] = (int32_t)((c + ((int64_t)j * N) / a) % N);
  for (int i = 1; i < a; ++i) {
    int32_t x = out[i];
    int k = i - 1;
    while (k >= 0 && out[k] > x) {
      out[k + 1] = out[k];
      --k;
    }
    out[k + 1] = x;
  }
  return 0;
}

/*
 * Full-view steps (Sec. 3.2, drift-bounding schedule; Sec. 4.1,
 * configurations).  rule 0: every E-th step (0, E, 2E, ...); rule 1:
 * two-step head, one mid refresh at floor(S/2), one tail step S-1.
 * Step 0 is always full.  out[k] = 1 for a full step.
 */
int orc_full_steps(int rule, int S, int E, uint8_t* out) {
  if (S < 1) return -1;
  for (int k = 0; k < S; ++k) out[k] = 0;
  if (rule == 0) {
    if (E < 1) return -1;
    for (int k = 0; k < S; k += E) out[k] = 1;
  } else if (rule == 1) {
    out[0] = 1;
    if (S > 1) out[1] = 1;
    out[S / 2] = 1;
    out[S - 1] = 1;
  } else if (rule == 2) {
    /* Sec. 4.1, configurations: E full-view refresh steps at the end of the
     * trajectory, after the two-step head of the drift-bounding schedule */
    if (E < 0 || E > S) return -1;
    out[0] = 1;
    if (S > 1) out[1] = 1;
    for (int k = S - E; k < S; ++k) out[k] = 1;
  } else {
    return -1;
  }
  out[0] = 1;
  return 0;
}

/* DDIM "trailing" timesteps: t_k = round((S - k) * T / S) - 1, t_S = -1. */
int orc_ddim_timesteps(int T, int S, int32_t* out) {
  if (S < 1 || T < S) return -1;
  for (int k = 0; k < S; ++k) out[k] = (int32_t)floor((double)(S - k) * T / S + 0.5) - 1;
  out[S] = -1;
  return 0;
}

/* ------------------------------------------------------------------ */
/* O8: multistep (UniPC) sampler-consistent update                      */
/* ------------------------------------------------------------------ */
/*
 * The reconstruction keeps the solver's history in the parameterisation it
 * expects (Sec. 3.2, after Eq. 1).  For a multistep solver in data
 * prediction, that history is the x0 of previous steps -- for a cached step,
 * the transported x0 of every view.  This is the UniPC predictor-corrector
 * (Zhao et al. 2023) with B(h) = expm1(h) ("bh2"), data prediction, on the
 * DDIM noise schedule: alpha_t = sqrt(abar_t), sigma_t = sqrt(1 - abar_t),
 * lambda_t = log(alpha_t / sigma_t).  At sampler step k (time s0 = t_k):
 *   corrector (k >= 1, order pc = predictor order of step k-1):
 *     x_c = (sigma_s0/sigma_p) x_prev - alpha_s0 (e^{-h} - 1) m_{k-1}
 *           - alpha_s0 B_h (sum_j rho_c[j] D_j + rho_c[pc-1] (m_k - m_{k-1}))
 *     with h = lambda_s0 - lambda_{t_{k-1}}, x_prev the corrected sample of
 *     step k-1, D_1 = (m_{k-2} - m_{k-1}) / r_1 (pc = 2),
 *     r_1 = (lambda_{t_{k-2}} - lambda_{t_{k-1}}) / h; rho_c = [1/2] for
 *     pc = 1, else the solution of R rho = b (below);
 *   predictor (order pp):
 *     x_next = (sigma_n/sigma_s0) x_c - alpha_n (e^{-h'} - 1) m_k
 *              - alpha_n B_h' rho_p D'_1
 *     with h' = lambda_n - lambda_s0, D'_1 = (m_{k-1} - m_k) / r'_1,
 *     r'_1 = (lambda_{t_{k-1}} - lambda_s0) / h', rho_p = 1/2 (pp = 2).
 *   R[i][j] = r_j^i (r_last = 1), b_i = h_phi_{i+1} (i+1)! / B_h with
 *   h_phi_1 = expm1(-h), h_phi_{i+1} = h_phi_i / (-h) - 1/(i+1)!.
 *   Orders: pp = min(order, steps taken + 1, S - k) (warm-up and a
 *   first-order last step).  The last step goes to sigma_n = 0, where the
 *   predictor reduces to x_next = m_k.
 * The whole update is linear in (x_prev, m_{k-2}, m_{k-1}, m_k) or, without a
 * corrector, (x_k, m_{k-1}, m_k); orc_unipc_coeffs returns those
 * coefficients in double, orc_unipc_apply applies them in double.
 * coef layout: [0] use corrector, [1] pc, [2] pp,
 *   corrector x_c = c[3] x_prev + c[4] m_{k-2} + c[5] m_{k-1} + c[6] m_k,
 *   predictor x_next = c[7] x_c + c[8] m_{k-1} + c[9] m_k.
 */
static double unipc_lambda(int T, double bs, double be, int t) {
  const double ab = orc_alpha_bar(T, bs, be, t);
  return log(sqrt(ab)) - log(sqrt(1.0 - ab));
}

int orc_unipc_coeffs(int T, double beta_start, double beta_end, const int32_t* ts, int S, int k, int order,
                     int corrector, double* c) {
  if (order < 1 || order > 2 || k < 0 || k >= S) return -1;
  for (int i = 0; i < 10; ++i) c[i] = 0.0;
  /* predictor order at step j: warm-up and first-order final step */
  int pp_k = order;
  if (k + 1 < pp_k) pp_k = k + 1;
  if (S - k < pp_k) pp_k = S - k;
  const int t0 = ts[k];
  const double ab0 = orc_alpha_bar(T, beta_start, beta_end, t0);
  const double a0 = sqrt(ab0), s0 = sqrt(1.0 - ab0), l0 = log(a0) - log(s0);
  /* corrector: back from step k-1 to step k */
  if (corrector && k >= 1) {
    int pc = order;
    if (k < pc) pc = k;                    /* predictor order used at step k-1 */
    if (S - (k - 1) < pc) pc = S - (k - 1);
    const int tp = ts[k - 1];
    const double abp = orc_alpha_bar(T, beta_start, beta_end, tp);
    const double ap = sqrt(abp), sp = sqrt(1.0 - abp), lp = log(ap) - log(sp);
    const double h = l0 - lp, hh = -h;
    const double h_phi_1 = expm1(hh), B_h = expm1(hh);
    double rho[2];
    double r1 = 0.0;
    if (pc == 1) {
      rho[0] = 0.5;
    } else {
      const double lpp = unipc_lambda(T, beta_start, beta_end, ts[k - 2]);
      r1 = (lpp - lp) / h;
      /* R = [[1, 1], [r1, 1]], b_i = h_phi_{i+1} (i+1)! / B_h */
      double h_phi_k = h_phi_1 / hh - 1.0;
      const double b0 = h_phi_k * 1.0 / B_h;
      h_phi_k = h_phi_k / hh - 1.0 / 2.0;
      const double b1 = h_phi_k * 2.0 / B_h;
      const double det = 1.0 * 1.0 - 1.0 * r1;
      rho[0] = (b0 * 1.0 - 1.0 * b1) / det;
      rho[1] = (1.0 * b1 - r1 * b0) / det;
    }
    c[0] = 1.0;
    c[1] = pc;
    c[3] = s0 / sp;
    /* - a0 h_phi_1 m_{k-1} - a0 B_h rho_last (m_k - m_{k-1}) - a0 B_h rho_0 (m_{k-2} - m_{k-1}) / r1 */
    const double rl = pc == 1 ? rho[0] : rho[1];
    c[5] = -a0 * h_phi_1 + a0 * B_h * rl;
    c[6] = -a0 * B_h * rl;
    if (pc == 2) {
      c[4] = -a0 * B_h * rho[0] / r1;
      c[5] += a0 * B_h * rho[0] / r1;
    }
  }
  if ((pp_k == 2 && k < 1) || (c[1] == 2 && k < 2)) return -1;   /* no history that far back */
  c[2] = pp_k;
  /* predictor: step k -> k+1 */
  const int tn = ts[k + 1];
  if (tn < 0) {              /* sigma_n = 0: x_next = m_k */
    c[9] = 1.0;
    return 0;
  }
  const double abn = orc_alpha_bar(T, beta_start, beta_end, tn);
  const double an = sqrt(abn), sn = sqrt(1.0 - abn), ln = log(an) - log(sn);
  const double h = ln - l0, hh = -h;
  const double h_phi_1 = expm1(hh), B_h = expm1(hh);
  c[7] = sn / s0;
  c[9] = -an * h_phi_1;
  if (pp_k == 2) {
    const double lm = unipc_lambda(T, beta_start, beta_end, ts[k - 1]);
    const double r1 = (lm - l0) / h;
    /* - an B_h (1/2) (m_{k-1} - m_k) / r1 */
    c[8] = -an * B_h * 0.5 / r1;
    c[9] += an * B_h * 0.5 / r1;
  }
  return 0;
}

/* One UniPC update, elementwise in double.  x_cur is the sample the step
 * starts from when there is no corrector; x_prev the previous corrected
 * sample otherwise.  Outputs: x_c (the corrected sample, next step's x_prev)
 * and x_next.  Any of m_km2 / x_prev may be null when its coefficient is 0. */
int orc_unipc_apply(const void* x_cur, const void* x_prev, const void* m_km2, const void* m_km1, const void* m_k,
                    int64_t n, int dtype, const double* c, double* x_c, double* x_next) {
  if (dtype != ORC_F32 && dtype != ORC_BF16) return -3;
  for (int64_t i = 0; i < n; ++i) {
    const double mk = load_val(m_k, i, dtype);
    const double mk1 = m_km1 ? load_val(m_km1, i, dtype) : 0.0;
    double xc;
    if (c[0] != 0.0) {
      const double mk2 = m_km2 ? load_val(m_km2, i, dtype) : 0.0;
      xc = c[3] * load_val(x_prev, i, dtype) + c[4] * mk2 + c[5] * mk1 + c[6] * mk;
    } else {
      xc = load_val(x_cur, i, dtype);
    }
    x_c[i] = xc;
    x_next[i] = c[7] * xc + c[8] * mk1 + c[9] * mk;
  }
  return 0;
}

/* ===================================================================== */
/* O9: token staleness and the coverage-driven schedule                   */
/* ===================================================================== */
/* Sec. 3.2 (invalid matches): a token no anchor sees keeps its state and
 * misses that step's denoising until the next full step.  The limitations
 * section names adaptive anchor selection and visibility-aware refresh as
 * the remedy for regions few anchors observe; the paper defines neither, so
 * the definitions below are this implementation's reading:
 *   - staleness of token (b, v, p): the number of consecutive steps in which
 *     it received neither a fresh prediction (v an anchor, or a full step)
 *     nor a transported increment (some anchor of the step sees it),
 *     saturating at 254; background tokens (non-finite position) hold 255
 *     and are never counted;
 *   - per-view statistics after an update: foreground tokens, tokens with
 *     staleness >= R, the sum and the maximum of the staleness;
 *   - anchor selection: greedy weighted maximum coverage.  A candidate view
 *     u covers (b, v, p) when v = u or u sees it; a token counts with weight
 *     1 + staleness while no chosen view covers it.  Forced views are
 *     chosen first, then the candidate with the largest gain (ties: the
 *     lower view) until a views are chosen; the result is sorted;
 *   - refresh: due when (tokens with staleness >= R) / (foreground tokens)
 *     over all assets and views exceeds tau.
 * seen[u][b][v][p] (0/1) is whether anchor u alone sees token p of view v:
 * a non-zero O3 word for the anchor set {u}; seen[u][b][u][.] = 0.  Whether
 * a set A sees a token is the OR over u in A, since O3 tests each anchor on
 * its own. */

#define ORC_BG 255u
#define ORC_STALE_MAX 254u

int orc_cov_init(const float* pos, int64_t n_tok, uint8_t* stale) {
  if (n_tok < 0) return -2;
  for (int64_t i = 0; i < n_tok; ++i) {
    const float* P = pos + i * 3;
    stale[i] = (isfinite(P[0]) && isfinite(P[1]) && isfinite(P[2])) ? 0u : (uint8_t)ORC_BG;
  }
  return 0;
}

static int covers(const uint8_t* seen, int B, int N, int64_t HW, int u, int b, int v, int64_t p) {
  if (u == v) return 1;
  return seen[(((int64_t)u * B + b) * N + v) * HW + p] != 0;
}

int orc_cov_update(const uint8_t* seen, int B, int N, int64_t HW, const int32_t* anchors, int a, int R,
                   uint8_t* stale, uint32_t* stats) {
  if (B < 1 || N < 1 || HW < 0 || a < 1 || a > N || R < 1) return -2;
  for (int b = 0; b < B; ++b) {
    for (int v = 0; v < N; ++v) {
      uint32_t n_fg = 0, n_ge = 0, sum = 0, mx = 0;
      for (int64_t p = 0; p < HW; ++p) {
        uint8_t* s = stale + ((int64_t)b * N + v) * HW + p;
        if (*s == ORC_BG) continue;
        int fresh = 0;
        for (int j = 0; j < a; ++j) fresh |= covers(seen, B, N, HW, anchors[j], b, v, p);
        if (fresh) *s = 0;
        else if (*s < ORC_STALE_MAX) *s = (uint8_t)(*s + 1);
        n_fg += 1;
        n_ge += *s >= (uint32_t)R;
        sum += *s;
        if (*s > mx) mx = *s;
      }
      uint32_t* o = stats + ((int64_t)b * N + v) * 4;
      o[0] = n_fg;
      o[1] = n_ge;
      o[2] = sum;
      o[3] = mx;
    }
  }
  return 0;
}

int orc_cov_gains(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, const uint8_t* chosen,
                  uint64_t* gains) {
  if (B < 1 || N < 1 || HW < 0) return -2;
  for (int u = 0; u < N; ++u) gains[u] = 0;
  for (int b = 0; b < B; ++b)
    for (int v = 0; v < N; ++v)
      for (int64_t p = 0; p < HW; ++p) {
        const uint8_t s = stale[((int64_t)b * N + v) * HW + p];
        if (s == ORC_BG) continue;
        int covered = 0;
        for (int u = 0; u < N; ++u) covered |= chosen[u] && covers(seen, B, N, HW, u, b, v, p);
        if (covered) continue;
        for (int u = 0; u < N; ++u)
          if (!chosen[u] && covers(seen, B, N, HW, u, b, v, p)) gains[u] += 1u + s;
      }
  return 0;
}

int orc_cov_select(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, int a,
                   const int32_t* forced, int n_forced, int32_t* out) {
  if (B < 1 || N < 1 || N > 64 || a < 1 || a > N || n_forced < 0 || n_forced > a) return -2;
  uint8_t chosen[64] = {0};
  uint64_t gains[64];
  int n = 0;
  for (int j = 0; j < n_forced; ++j) {
    if (forced[j] < 0 || forced[j] >= N || chosen[forced[j]]) return -1;
    chosen[forced[j]] = 1;
    ++n;
  }
  while (n < a) {
    orc_cov_gains(seen, stale, B, N, HW, chosen, gains);
    int best = -1;
    for (int u = 0; u < N; ++u)
      if (!chosen[u] && (best < 0 || gains[u] > gains[best])) best = u;
    chosen[best] = 1;
    ++n;
  }
  int j = 0;
  for (int u = 0; u < N; ++u)
    if (chosen[u]) out[j++] = u;
  return 0;
}

/* Weighted coverage of candidate sets: score[m] = sum over foreground tokens
 * covered by set m (sets[m][0..a-1]) of 1 + staleness.  Choosing, among the
 * rotation's own sets, the one that covers the most keeps the rotation's
 * evenly spread anchors while following where the stale tokens are. */
int orc_cov_score(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, const int32_t* sets, int M,
                  int a, uint64_t* score) {
  if (B < 1 || N < 1 || HW < 0 || M < 1 || a < 1 || a > N) return -2;
  for (int m = 0; m < M; ++m) {
    score[m] = 0;
    for (int j = 0; j < a; ++j)
      if (sets[m * a + j] < 0 || sets[m * a + j] >= N) return -1;
  }
  for (int b = 0; b < B; ++b)
    for (int v = 0; v < N; ++v)
      for (int64_t p = 0; p < HW; ++p) {
        const uint8_t s = stale[((int64_t)b * N + v) * HW + p];
        if (s == ORC_BG) continue;
        for (int m = 0; m < M; ++m) {
          int covered = 0;
          for (int j = 0; j < a; ++j) covered |= covers(seen, B, N, HW, sets[m * a + j], b, v, p);
          if (covered) score[m] += 1u + s;
        }
      }
  return 0;
}

int orc_refresh_due(const uint32_t* stats, int B, int N, double tau) {
  if (B < 1 || N < 1) return -2;
  uint64_t fg = 0, ge = 0;
  for (int64_t i = 0; i < (int64_t)B * N; ++i) {
    fg += stats[i * 4 + 0];
    ge += stats[i * 4 + 1];
  }
  return fg > 0 && (double)ge > tau * (double)fg;
}
