// Seeded input generation: position-map rendering for synthetic assets.
//
// This file produces *inputs* only (per-view position maps: the 3D surface
// point seen through each pixel centre, NaN for background).  It contains none
// of the cross-view transport arithmetic; it is shared by the oracle and the
// HIP path only through the arrays it writes.
//
// Camera convention (world->camera, x right, y down, z forward):
//   x_c = R * X + t
//   pinhole:      (u, v) = (fx * x_c / z_c + cx, fy * y_c / z_c + cy)
//   orthographic: (u, v) = (fx * x_c + cx,       fy * y_c + cy)
// Pixel i spans [i, i+1); a pixel's ray goes through its centre (i+0.5, j+0.5).
// All geometry is done in double; the stored point is the exact ray hit,
// rounded once to float.
//
// Built with g++ -O2 -fopenmp into libsynth.so and called through ctypes.

#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>
#include <algorithm>
#include <omp.h>

namespace {

struct Cam {
  int model;          // 0 pinhole, 1 orthographic
  double R[9];        // row-major world->camera rotation
  double t[3];
  double fx, fy, cx, cy;
};

// cams: [ncam][17] doubles = model, R[9], t[3], fx, fy, cx, cy
Cam load_cam(const double* c) {
  Cam k;
  k.model = (int)c[0];
  for (int i = 0; i < 9; ++i) k.R[i] = c[1 + i];
  for (int i = 0; i < 3; ++i) k.t[i] = c[10 + i];
  k.fx = c[13]; k.fy = c[14]; k.cx = c[15]; k.cy = c[16];
  return k;
}

// Ray through the centre of render pixel (px, py): origin o, direction d
// (pinhole: d has unit camera-z component so the ray parameter is depth).
void pixel_ray(const Cam& k, double u, double v, double o[3], double d[3]) {
  const double* R = k.R;
  const double* t = k.t;
  // camera centre C = -R^T t
  double C[3];
  for (int i = 0; i < 3; ++i) C[i] = -(R[0 * 3 + i] * t[0] + R[1 * 3 + i] * t[1] + R[2 * 3 + i] * t[2]);
  const double xc = (u - k.cx) / k.fx;
  const double yc = (v - k.cy) / k.fy;
  if (k.model == 0) {
    const double dc[3] = {xc, yc, 1.0};
    for (int i = 0; i < 3; ++i) {
      o[i] = C[i];
      d[i] = R[0 * 3 + i] * dc[0] + R[1 * 3 + i] * dc[1] + R[2 * 3 + i] * dc[2];
    }
  } else {
    // point on the z_c = 0 plane with the pixel's (x_c, y_c), looking along +z_c
    const double pc[3] = {xc - t[0], yc - t[1], -t[2]};
    for (int i = 0; i < 3; ++i) {
      o[i] = R[0 * 3 + i] * pc[0] + R[1 * 3 + i] * pc[1] + R[2 * 3 + i] * pc[2];
      d[i] = R[2 * 3 + i];
    }
  }
}

void project(const Cam& k, const double X[3], double& u, double& v, double& z) {
  const double* R = k.R;
  double xc = R[0] * X[0] + R[1] * X[1] + R[2] * X[2] + k.t[0];
  double yc = R[3] * X[0] + R[4] * X[1] + R[5] * X[2] + k.t[1];
  double zc = R[6] * X[0] + R[7] * X[1] + R[8] * X[2] + k.t[2];
  z = zc;
  if (k.model == 0) {
    u = k.fx * xc / zc + k.cx;
    v = k.fy * yc / zc + k.cy;
  } else {
    u = k.fx * xc + k.cx;
    v = k.fy * yc + k.cy;
  }
}

// Moller-Trumbore with a tiny edge slack so shared edges do not crack.
bool ray_tri(const double o[3], const double d[3], const double* a, const double* b,
             const double* c, double& thit) {
  const double e1[3] = {b[0] - a[0], b[1] - a[1], b[2] - a[2]};
  const double e2[3] = {c[0] - a[0], c[1] - a[1], c[2] - a[2]};
  const double p[3] = {d[1] * e2[2] - d[2] * e2[1], d[2] * e2[0] - d[0] * e2[2],
                       d[0] * e2[1] - d[1] * e2[0]};
  const double det = e1[0] * p[0] + e1[1] * p[1] + e1[2] * p[2];
  if (std::fabs(det) < 1e-300) return false;
  const double inv = 1.0 / det;
  const double s[3] = {o[0] - a[0], o[1] - a[1], o[2] - a[2]};
  const double uu = (s[0] * p[0] + s[1] * p[1] + s[2] * p[2]) * inv;
  const double eps = 1e-10;
  if (uu < -eps || uu > 1.0 + eps) return false;
  const double q[3] = {s[1] * e1[2] - s[2] * e1[1], s[2] * e1[0] - s[0] * e1[2],
                       s[0] * e1[1] - s[1] * e1[0]};
  const double vv = (d[0] * q[0] + d[1] * q[1] + d[2] * q[2]) * inv;
  if (vv < -eps || uu + vv > 1.0 + eps) return false;
  thit = (e2[0] * q[0] + e2[1] * q[1] + e2[2] * q[2]) * inv;
  return thit > 0.0;
}

// Radial displacement field D(w) = (1/n) * sum_j sin(f_j * (w . d_j) + phi_j).
// params: [n][5] = d_x, d_y, d_z, f, phi
double radial_field(const double w[3], const double* params, int n) {
  double s = 0.0;
  for (int j = 0; j < n; ++j) {
    const double* q = params + 5 * j;
    s += std::sin(q[3] * (w[0] * q[0] + w[1] * q[1] + w[2] * q[2]) + q[4]);
  }
  return n > 0 ? s / n : 0.0;
}

// Signed "outside" function of the star-shaped surface r(w) = 1 + amp * D(w).
double radial_sdf(const double x[3], double amp, const double* params, int n) {
  const double r = std::sqrt(x[0] * x[0] + x[1] * x[1] + x[2] * x[2]);
  if (r == 0.0) return -1.0;
  const double w[3] = {x[0] / r, x[1] / r, x[2] / r};
  return r - (1.0 + amp * radial_field(w, params, n));
}

}  // namespace

extern "C" {

int synth_abi_version(void) { return 1; }

// Rasterise a triangle mesh into per-view position maps.
//   verts  [nv][3] double, tris [nt][3] int32
//   cams   [ncam][17] double (render-pixel units)
//   out    [ncam][H][W][3] float; NaN where no surface is hit
int synth_render_mesh(const double* verts, int64_t nv, const int32_t* tris, int64_t nt,
                      const double* cams, int ncam, int H, int W, float* out, int nthreads) {
  if (!verts || !tris || !cams || !out || nv <= 0 || nt <= 0 || ncam <= 0 || H <= 0 || W <= 0)
    return -1;
  for (int64_t i = 0; i < nt * 3; ++i)
    if (tris[i] < 0 || tris[i] >= nv) return -2;
  if (nthreads > 0) omp_set_num_threads(nthreads);
  const float qnan = std::numeric_limits<float>::quiet_NaN();
#pragma omp parallel for schedule(dynamic, 1)
  for (int ci = 0; ci < ncam; ++ci) {
    const Cam k = load_cam(cams + 17 * ci);
    std::vector<double> zbuf((size_t)H * W, std::numeric_limits<double>::infinity());
    std::vector<double> hit((size_t)H * W * 3, 0.0);
    std::vector<double> pu(nv), pv(nv), pz(nv);
    for (int64_t i = 0; i < nv; ++i) project(k, verts + 3 * i, pu[i], pv[i], pz[i]);
    for (int64_t ti = 0; ti < nt; ++ti) {
      const int32_t ia = tris[3 * ti], ib = tris[3 * ti + 1], ic = tris[3 * ti + 2];
      if (k.model == 0 && (pz[ia] <= 1e-9 || pz[ib] <= 1e-9 || pz[ic] <= 1e-9)) continue;
      const double umin = std::min(pu[ia], std::min(pu[ib], pu[ic]));
      const double umax = std::max(pu[ia], std::max(pu[ib], pu[ic]));
      const double vmin = std::min(pv[ia], std::min(pv[ib], pv[ic]));
      const double vmax = std::max(pv[ia], std::max(pv[ib], pv[ic]));
      int x0 = (int)std::floor(umin - 1.0), x1 = (int)std::ceil(umax + 1.0);
      int y0 = (int)std::floor(vmin - 1.0), y1 = (int)std::ceil(vmax + 1.0);
      if (x1 < 0 || y1 < 0 || x0 >= W || y0 >= H) continue;
      x0 = std::max(x0, 0); y0 = std::max(y0, 0);
      x1 = std::min(x1, W - 1); y1 = std::min(y1, H - 1);
      const double* A = verts + 3 * ia;
      const double* Bv = verts + 3 * ib;
      const double* Cv = verts + 3 * ic;
      for (int y = y0; y <= y1; ++y) {
        for (int x = x0; x <= x1; ++x) {
          double o[3], d[3], th;
          pixel_ray(k, x + 0.5, y + 0.5, o, d);
          if (!ray_tri(o, d, A, Bv, Cv, th)) continue;
          const size_t pix = (size_t)y * W + x;
          if (th < zbuf[pix]) {
            zbuf[pix] = th;
            for (int c = 0; c < 3; ++c) hit[3 * pix + c] = o[c] + th * d[c];
          }
        }
      }
    }
    float* dst = out + (size_t)ci * H * W * 3;
    for (size_t pix = 0; pix < (size_t)H * W; ++pix) {
      if (std::isinf(zbuf[pix])) {
        dst[3 * pix] = dst[3 * pix + 1] = dst[3 * pix + 2] = qnan;
      } else {
        for (int c = 0; c < 3; ++c) dst[3 * pix + c] = (float)hit[3 * pix + c];
      }
    }
  }
  return 0;
}

// Ray-cast the star-shaped surface r(w) = 1 + amp * D(w) analytically
// (march + bisection in double).  params: [nparams][5] (see radial_field).
int synth_raycast_radial(double amp, const double* params, int nparams, const double* cams,
                         int ncam, int H, int W, float* out, int nthreads) {
  if (!cams || !out || ncam <= 0 || H <= 0 || W <= 0 || nparams < 0) return -1;
  if (nthreads > 0) omp_set_num_threads(nthreads);
  const float qnan = std::numeric_limits<float>::quiet_NaN();
  const double rb = 1.0 + std::fabs(amp) + 1e-3;   // bounding sphere
  const double step = 2e-3;
#pragma omp parallel for schedule(dynamic, 1)
  for (int ci = 0; ci < ncam; ++ci) {
    const Cam k = load_cam(cams + 17 * ci);
    float* dst = out + (size_t)ci * H * W * 3;
    for (int y = 0; y < H; ++y) {
      for (int x = 0; x < W; ++x) {
        double o[3], d[3];
        pixel_ray(k, x + 0.5, y + 0.5, o, d);
        const double dn = std::sqrt(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
        for (int c = 0; c < 3; ++c) d[c] /= dn;
        // entry/exit of the bounding sphere
        const double b = o[0] * d[0] + o[1] * d[1] + o[2] * d[2];
        const double cc = o[0] * o[0] + o[1] * o[1] + o[2] * o[2] - rb * rb;
        const double disc = b * b - cc;
        float* px = dst + 3 * ((size_t)y * W + x);
        px[0] = px[1] = px[2] = qnan;
        if (disc <= 0.0) continue;
        const double sq = std::sqrt(disc);
        double s0 = -b - sq, s1 = -b + sq;
        if (s1 <= 0.0) continue;
        if (s0 < 0.0) s0 = 0.0;
        double sa = s0, fa;
        {
          const double X[3] = {o[0] + sa * d[0], o[1] + sa * d[1], o[2] + sa * d[2]};
          fa = radial_sdf(X, amp, params, nparams);
        }
        bool found = false;
        double sb = sa;
        while (sa < s1) {
          sb = std::min(sa + step, s1);
          const double X[3] = {o[0] + sb * d[0], o[1] + sb * d[1], o[2] + sb * d[2]};
          const double fb = radial_sdf(X, amp, params, nparams);
          if (fa > 0.0 && fb <= 0.0) { found = true; break; }
          sa = sb; fa = fb;
        }
        if (!found) continue;
        for (int it = 0; it < 100; ++it) {
          const double sm = 0.5 * (sa + sb);
          if (sm <= sa || sm >= sb) break;
          const double X[3] = {o[0] + sm * d[0], o[1] + sm * d[1], o[2] + sm * d[2]};
          if (radial_sdf(X, amp, params, nparams) > 0.0) sa = sm; else sb = sm;
        }
        const double sh = 0.5 * (sa + sb);
        for (int c = 0; c < 3; ++c) px[c] = (float)(o[c] + sh * d[c]);
      }
    }
  }
  return 0;
}

}  // extern "C"
