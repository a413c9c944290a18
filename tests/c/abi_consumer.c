/*
 * A plain C consumer of the C ABI (no Python): device buffers from
 * hipMalloc, one cached step through the library, results checked against
 * closed forms.  Test infrastructure; exits 0 and prints "C ABI OK" on
 * success.
 *
 * Problem: two views of the plane z = 0 seen by the same orthographic
 * camera (view 1 duplicates view 0), view 0 the anchor.  Every token of
 * view 1 then maps to the same token of view 0 with one tap of weight 1
 * (Sec. 3.2: row-stochastic operator; the neighbouring taps lie a pixel
 * pitch away, far outside the tolerance), so Eq. 1 gives
 * x0_out(1) = x0_prev(1) + 1 * (x0_new(0) - x0_prev(0)) in float, bit for
 * bit, and x0_out(0) = x0_new(0).  The DDIM step is checked against
 * eps = (x_t - sqrt(abar_t) x0) / sqrt(1 - abar_t),
 * x_next = sqrt(abar_n) x0 + sqrt(1 - abar_n) eps in double.
 *
 * The same step then runs through the other launches, each bit-identical to
 * the first: the split launch over the visible-token index (built with a
 * workspace and without one), and the on-the-fly step over the foreground
 * index.  Last, the coverage schedule on the same scene: each view sees all
 * of the other's tokens, so a full step leaves no token stale and the greedy
 * choice of one anchor is view 0 (equal gains go to the lower view).
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "geocache.h"

#define H 16
#define W 16
#define C 8
#define NV 2

static int fails = 0;
#define CHECK(cond, ...)                 \
  do {                                   \
    if (!(cond)) {                       \
      fprintf(stderr, __VA_ARGS__);      \
      fputc('\n', stderr);               \
      ++fails;                           \
    }                                    \
  } while (0)

#define HIP_OK(call)                                                        \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
      exit(2);                                                              \
    }                                                                       \
  } while (0)

static double alpha_bar(int t) {
  double ab = 1.0;
  for (int i = 0; i <= t; ++i) ab *= 1.0 - (1e-4 + (0.02 - 1e-4) * (double)i / 999.0);
  return ab;
}

static float frand(unsigned* s) {
  *s = *s * 1664525u + 1013904223u;
  return (float)((*s >> 8) & 0xffff) / 65536.0f - 0.5f;
}

int main(void) {
  const size_t n_tok = (size_t)NV * H * W, n_lat = n_tok * C;
  float pos[NV * H * W * 3];
  gc_camera cams[NV];
  for (int v = 0; v < NV; ++v)
    for (int j = 0; j < H; ++j)
      for (int i = 0; i < W; ++i) {
        float* p = pos + (((size_t)v * H + j) * W + i) * 3;
        p[0] = (float)i + 0.5f;
        p[1] = (float)j + 0.5f;
        p[2] = 0.0f;
      }
  for (int v = 0; v < NV; ++v) {
    memset(&cams[v], 0, sizeof(gc_camera));
    cams[v].model = 1;
    cams[v].R[0] = cams[v].R[4] = cams[v].R[8] = 1.0f;
    cams[v].fx = cams[v].fy = 1.0f;
  }
  float *x0_prev = malloc(n_lat * 4), *x0_new = malloc(n_lat / NV * 4), *x_t = malloc(n_lat * 4);
  unsigned seed = 12345u;
  for (size_t i = 0; i < n_lat; ++i) x0_prev[i] = frand(&seed), x_t[i] = frand(&seed);
  for (size_t i = 0; i < n_lat / NV; ++i) x0_new[i] = frand(&seed);

  float *d_pos, *d_bbox, *d_w, *d_prev, *d_new, *d_xt, *d_out, *d_next, *d_eps;
  gc_camera* d_cams;
  int32_t* d_corr;
  HIP_OK(hipMalloc((void**)&d_pos, sizeof pos));
  HIP_OK(hipMalloc((void**)&d_cams, sizeof cams));
  HIP_OK(hipMalloc((void**)&d_bbox, 32));
  HIP_OK(hipMalloc((void**)&d_corr, (size_t)H * W * 4));
  HIP_OK(hipMalloc((void**)&d_w, (size_t)H * W * 4 * 4));
  HIP_OK(hipMalloc((void**)&d_prev, n_lat * 4));
  HIP_OK(hipMalloc((void**)&d_new, n_lat / NV * 4));
  HIP_OK(hipMalloc((void**)&d_xt, n_lat * 4));
  HIP_OK(hipMalloc((void**)&d_out, n_lat * 4));
  HIP_OK(hipMalloc((void**)&d_next, n_lat * 4));
  HIP_OK(hipMalloc((void**)&d_eps, n_lat * 4));
  HIP_OK(hipMemcpy(d_pos, pos, sizeof pos, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_cams, cams, sizeof cams, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_prev, x0_prev, n_lat * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_new, x0_new, n_lat / NV * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_xt, x_t, n_lat * 4, hipMemcpyHostToDevice));

  CHECK(gc_abi_version() == GC_ABI_VERSION, "abi version %d", gc_abi_version());
  const int32_t anchors[1] = {0};
  int rc = gc_posmap_bbox(d_pos, 1, NV, H, W, 0.01f, d_bbox, 0);
  CHECK(rc == GC_OK, "bbox rc=%d %s", rc, gc_last_error());
  rc = gc_build_correspondence(d_pos, d_cams, 1, NV, H, W, anchors, 1, 4, d_bbox, d_corr, d_w, NULL, 0);
  CHECK(rc == GC_OK, "build rc=%d %s", rc, gc_last_error());
  gc_sampler smp;
  memset(&smp, 0, sizeof smp);
  smp.kind = GC_DDIM;
  smp.pred_out = GC_PRED_EPS;
  smp.T = 1000;
  smp.beta_start = 1e-4;
  smp.beta_end = 0.02;
  const int t = 700, tn = 666;
  rc = gc_transport_reconstruct(d_prev, d_new, d_corr, d_w, NULL, NULL, 0, d_xt, 1, NV, H, W, C, anchors, 1, 4,
                                GC_F32, &smp, t, tn, d_out, d_next, d_eps, 0);
  CHECK(rc == GC_OK, "fused rc=%d %s", rc, gc_last_error());
  HIP_OK(hipDeviceSynchronize());

  int32_t corr[H * W];
  float wts[H * W * 4];
  float *out = malloc(n_lat * 4), *next = malloc(n_lat * 4);
  HIP_OK(hipMemcpy(corr, d_corr, sizeof corr, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(wts, d_w, sizeof wts, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(out, d_out, n_lat * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(next, d_next, n_lat * 4, hipMemcpyDeviceToHost));
  for (int p = 0; p < H * W; ++p) {
    const int i = p % W, j = p / W;
    const uint32_t want = (uint32_t)(i + 1) | ((uint32_t)(j + 1) << 12) | (1u << 24);
    CHECK((uint32_t)corr[p] == want, "word %d: %08x, expected %08x", p, (unsigned)corr[p], want);
    CHECK(wts[p * 4] == 1.0f && wts[p * 4 + 1] == 0.0f, "weights of token %d", p);
  }
  const double at = sqrt(alpha_bar(t)), st = sqrt(1.0 - alpha_bar(t));
  const double an = sqrt(alpha_bar(tn)), sn = sqrt(1.0 - alpha_bar(tn));
  double max_err = 0.0;
  for (size_t p = 0; p < (size_t)H * W; ++p)
    for (int c = 0; c < C; ++c) {
      const size_t e0 = p * C + c, e1 = ((size_t)H * W + p) * C + c;
      CHECK(out[e0] == x0_new[e0], "anchor row %zu not a copy", e0);
      const float acc = 0.0f + 1.0f * (x0_new[e0] - x0_prev[e0]);
      const float want = x0_prev[e1] + acc;
      CHECK(out[e1] == want, "transported x0 %zu: %.9g vs %.9g", e1, out[e1], want);
      for (int v = 0; v < NV; ++v) {
        const size_t e = v ? e1 : e0;
        const double eps = ((double)x_t[e] - at * (double)out[e]) / st;
        const double xn = an * (double)out[e] + sn * eps;
        const double d = fabs(xn - (double)next[e]);
        if (d > max_err) max_err = d;
      }
    }
  CHECK(max_err <= 1e-5, "x_next max error %g", max_err);

  /* the split launch over the visible-token index, with and without a workspace */
  uint32_t* d_bits;
  int32_t *d_list, *d_nvis, *d_nvis2;
  void* d_ws;
  float* d_out2;
  const size_t n_tgt = (size_t)H * W;   /* target tokens: one target view */
  const size_t wsb = gc_index_workspace_bytes((int64_t)n_tgt);
  HIP_OK(hipMalloc((void**)&d_bits, (n_tgt + 31) / 32 * 4));
  HIP_OK(hipMalloc((void**)&d_list, n_tgt * 4));
  HIP_OK(hipMalloc((void**)&d_nvis, 4));
  HIP_OK(hipMalloc((void**)&d_nvis2, 4));
  HIP_OK(hipMalloc(&d_ws, wsb));
  HIP_OK(hipMalloc((void**)&d_out2, n_lat * 4 * 2));
  float* d_next2 = d_out2 + n_lat;
  rc = gc_index_correspondence(d_corr, 1, H, W, 1, d_bits, d_list, d_nvis, d_ws, wsb, 0);
  CHECK(rc == GC_OK, "index rc=%d %s", rc, gc_last_error());
  int32_t nv = 0, nv2 = 0;
  HIP_OK(hipMemcpy(&nv, d_nvis, 4, hipMemcpyDeviceToHost));
  CHECK(nv == H * W, "visible tokens %d, expected %d", nv, H * W);
  rc = gc_transport_reconstruct(d_prev, d_new, d_corr, d_w, d_bits, d_list, nv, d_xt, 1, NV, H, W, C, anchors, 1, 4,
                                GC_F32, &smp, t, tn, d_out2, d_next2, d_eps, 0);
  CHECK(rc == GC_OK, "split launch rc=%d %s", rc, gc_last_error());
  float *out2 = malloc(n_lat * 4 * 2), *next2 = out2 + n_lat;
  HIP_OK(hipMemcpy(out2, d_out2, n_lat * 4 * 2, hipMemcpyDeviceToHost));
  CHECK(memcmp(out2, out, n_lat * 4) == 0 && memcmp(next2, next, n_lat * 4) == 0, "split launch differs");
  int32_t* list = malloc(n_tgt * 4);
  int32_t* list2 = malloc(n_tgt * 4);
  HIP_OK(hipMemcpy(list, d_list, n_tgt * 4, hipMemcpyDeviceToHost));
  rc = gc_index_correspondence_noalloc(d_corr, 1, H, W, 1, d_bits, d_list, d_nvis2, 0);
  CHECK(rc == GC_OK, "allocation-free index rc=%d %s", rc, gc_last_error());
  HIP_OK(hipMemcpy(&nv2, d_nvis2, 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(list2, d_list, n_tgt * 4, hipMemcpyDeviceToHost));
  CHECK(nv2 == nv && memcmp(list, list2, (size_t)nv * 4) == 0, "allocation-free index differs");

  /* the on-the-fly step over the foreground index of the position maps */
  uint32_t* d_fgb;
  int32_t *d_rec, *d_nfg;
  void* d_ws2;
  const size_t wsb2 = gc_index_workspace_bytes((int64_t)n_tok);
  HIP_OK(hipMalloc((void**)&d_fgb, (n_tok + 31) / 32 * 4));
  HIP_OK(hipMalloc((void**)&d_rec, n_tok * 16));
  HIP_OK(hipMalloc((void**)&d_nfg, 4));
  HIP_OK(hipMalloc(&d_ws2, wsb2));
  rc = gc_index_foreground(d_pos, NV, H, W, d_fgb, d_rec, d_nfg, d_ws2, wsb2, 0);
  CHECK(rc == GC_OK, "foreground index rc=%d %s", rc, gc_last_error());
  int32_t nfg = 0;
  HIP_OK(hipMemcpy(&nfg, d_nfg, 4, hipMemcpyDeviceToHost));
  CHECK(nfg == (int32_t)n_tok, "foreground tokens %d, expected %zu", nfg, n_tok);
  rc = gc_transport_reconstruct_geom(d_prev, d_new, d_pos, d_cams, d_bbox, d_fgb, d_rec, nfg, d_xt, 1, NV, H, W, C,
                                     anchors, 1, 4, GC_F32, &smp, t, tn, d_out2, d_next2, d_eps, 0);
  CHECK(rc == GC_OK, "on-the-fly step rc=%d %s", rc, gc_last_error());
  HIP_OK(hipMemcpy(out2, d_out2, n_lat * 4 * 2, hipMemcpyDeviceToHost));
  CHECK(memcmp(out2, out, n_lat * 4) == 0 && memcmp(next2, next, n_lat * 4) == 0, "on-the-fly step differs");

  /* the coverage schedule: pairs, staleness, a full step fused with the next choice */
  uint32_t *d_pairs, *d_stats;
  uint8_t* d_stale;
  int32_t* d_sel;
  void* d_cws;
  const size_t npw = (size_t)gc_coverage_pair_words(1, NV, H, W), cwsb = gc_coverage_workspace_bytes();
  HIP_OK(hipMalloc((void**)&d_pairs, npw * 4));
  HIP_OK(hipMalloc((void**)&d_stats, (size_t)NV * 16));
  HIP_OK(hipMalloc((void**)&d_stale, n_tok));
  HIP_OK(hipMalloc((void**)&d_sel, 4));
  HIP_OK(hipMalloc(&d_cws, cwsb));
  rc = gc_coverage_pairs(d_pos, d_cams, d_bbox, 1, NV, H, W, d_pairs, 0);
  CHECK(rc == GC_OK, "pairs rc=%d %s", rc, gc_last_error());
  rc = gc_coverage_init(d_pos, 1, NV, H, W, d_stale, 0);
  CHECK(rc == GC_OK, "staleness init rc=%d %s", rc, gc_last_error());
  const int32_t all_views[NV] = {0, 1};
  rc = gc_coverage_update_select(d_pairs, 1, NV, H, W, all_views, NV, 2, d_stale, d_stats, 1, NULL, 0, d_sel, d_cws,
                                 cwsb, 0);
  CHECK(rc == GC_OK, "update + select rc=%d %s", rc, gc_last_error());
  uint32_t stats[NV * 4];
  int32_t chosen = -1;
  HIP_OK(hipMemcpy(stats, d_stats, sizeof stats, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(&chosen, d_sel, 4, hipMemcpyDeviceToHost));
  for (int v = 0; v < NV; ++v)
    CHECK(stats[v * 4] == H * W && stats[v * 4 + 1] == 0 && stats[v * 4 + 2] == 0 && stats[v * 4 + 3] == 0,
          "statistics of view %d: %u %u %u %u", v, stats[v * 4], stats[v * 4 + 1], stats[v * 4 + 2], stats[v * 4 + 3]);
  CHECK(chosen == 0, "greedy anchor %d, expected 0", chosen);
  hipFree(d_bits); hipFree(d_list); hipFree(d_nvis); hipFree(d_nvis2); hipFree(d_ws); hipFree(d_out2);
  hipFree(d_fgb); hipFree(d_rec); hipFree(d_nfg); hipFree(d_ws2);
  hipFree(d_pairs); hipFree(d_stats); hipFree(d_stale); hipFree(d_sel); hipFree(d_cws);
  free(out2); free(list); free(list2);

  /* argument errors: negative code, a message, nothing launched */
  rc = gc_transport_step(d_prev, d_new, d_corr, d_w, NULL, NULL, 0, 1, NV, H, W, C, anchors, 1, 5, GC_F32, d_out, 0);
  CHECK(rc == GC_ERR_ARG && strlen(gc_last_error()) > 0, "K=5 accepted (rc=%d)", rc);
  rc = gc_transport_step(d_prev, d_new, d_corr, d_w, NULL, NULL, 0, 1, NV, H, W, C, anchors, 1, 4, GC_F32, d_prev, 0);
  CHECK(rc == GC_ERR_ALIAS, "aliased output accepted (rc=%d)", rc);

  hipFree(d_pos); hipFree(d_cams); hipFree(d_bbox); hipFree(d_corr); hipFree(d_w); hipFree(d_prev);
  hipFree(d_new); hipFree(d_xt); hipFree(d_out); hipFree(d_next); hipFree(d_eps);
  free(x0_prev); free(x0_new); free(x_t); free(out); free(next);
  if (fails) {
    fprintf(stderr, "%d check(s) failed\n", fails);
    return 1;
  }
  printf("C ABI OK (x_next max error %.3g)\n", max_err);
  return 0;
}
