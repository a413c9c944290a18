/*
 * Runs every entry point of the oracle on one small problem, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer (test infrastructure): an
 * out-of-bounds access, a use after free, a signed overflow, an invalid
 * shift or a misaligned access stops the run with a report.  Every call must
 * also return 0.
 *
 * argv: dir B N H W M Hr Wr.  dir holds the seeded inputs the test writes:
 *   pos.bin   float32 [B][N][H][W][3]  latent-grid position maps (NaN = background)
 *   model.bin int32   [B*N]            camera model
 *   R.bin     float32 [B*N][9]         rotation, row-major
 *   t.bin     float32 [B*N][3]         translation
 *   k.bin     float32 [B*N][4]         fx, fy, cx, cy
 *   hi.bin    float32 [M][Hr][Wr][3]   render-resolution maps for the downsample
 * Latents are drawn here from a fixed linear congruential sequence.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int orc_store(const double* x, int64_t n, int dtype, void* out);
int orc_downsample(const float* hi, int64_t M, int Hr, int Wr, int f, float* lo);
int orc_bbox(const float* pos, int B, int N, int H, int W, float tol_frac, float* out);
int orc_build(const float* pos, const int32_t* cam_model, const float* cam_R, const float* cam_t, const float* cam_k,
              int B, int N, int H, int W, const int32_t* anchors, int a, int K, const float* bbox, int32_t* corr,
              double* weights, int32_t* nvis_out);
int orc_transport(const void* x0_prev, const void* x0_anew, const int32_t* corr, const double* weights,
                  const int32_t* anchors, int a, int B, int N, int H, int W, int C, int K, int dtype, double* x0_exact,
                  void* x0_state);
int orc_reconstruct(const void* x_t, const void* x0, int64_t n, int dtype, int kind, int pred, int T, double beta_start,
                    double beta_end, double t, double t_next, double* x_next, double* model_out);
int orc_anchors(int N, int a, int64_t c, int32_t* out);
int orc_full_steps(int rule, int S, int E, uint8_t* out);
int orc_ddim_timesteps(int T, int S, int32_t* out);
int orc_unipc_coeffs(int T, double beta_start, double beta_end, const int32_t* ts, int S, int k, int order,
                     int corrector, double* c);
int orc_unipc_apply(const void* x_cur, const void* x_prev, const void* m_km2, const void* m_km1, const void* m_k,
                    int64_t n, int dtype, const double* c, double* x_c, double* x_next);
int orc_cov_init(const float* pos, int64_t n_tok, uint8_t* stale);
int orc_cov_update(const uint8_t* seen, int B, int N, int64_t HW, const int32_t* anchors, int a, int R, uint8_t* stale,
                   uint32_t* stats);
int orc_cov_gains(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, const uint8_t* chosen,
                  uint64_t* gains);
int orc_cov_select(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, int a, const int32_t* forced,
                   int n_forced, int32_t* out);
int orc_cov_score(const uint8_t* seen, const uint8_t* stale, int B, int N, int64_t HW, const int32_t* sets, int M,
                  int a, uint64_t* score);
int orc_refresh_due(const uint32_t* stats, int B, int N, double tau);

#define CHECK(call)                                                    \
  do {                                                                 \
    const int rc_ = (call);                                            \
    if (rc_ < 0) {                                                     \
      fprintf(stderr, "%s:%d: %s returned %d\n", __FILE__, __LINE__, #call, rc_); \
      exit(1);                                                         \
    }                                                                  \
  } while (0)

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) {
    fprintf(stderr, "cannot open %s\n", path);
    exit(1);
  }
  void* p = malloc(bytes);
  if (fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short read %s\n", path);
    exit(1);
  }
  fclose(f);
  return p;
}

static uint64_t lcg_state = 12345u;
static double uniform(void) {   /* [-1, 1) */
  lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(lcg_state >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}

/* n values in [-amp, amp) stored in dtype (0 float32, 1 bfloat16) */
static void* latents(int64_t n, int dtype, double amp) {
  double* x = malloc((size_t)n * sizeof(double));
  for (int64_t i = 0; i < n; ++i) x[i] = amp * uniform();
  void* out = malloc((size_t)n * (dtype == 0 ? 4 : 2));
  CHECK(orc_store(x, n, dtype, out));
  free(x);
  return out;
}

int main(int argc, char** argv) {
  if (argc != 9) {
    fprintf(stderr, "usage: %s dir B N H W M Hr Wr\n", argv[0]);
    return 2;
  }
  const char* dir = argv[1];
  const int B = atoi(argv[2]), N = atoi(argv[3]), H = atoi(argv[4]), W = atoi(argv[5]);
  const int M = atoi(argv[6]), Hr = atoi(argv[7]), Wr = atoi(argv[8]);
  const int64_t HW = (int64_t)H * W, n_tok = (int64_t)B * N * HW;
  float* pos = read_file(dir, "pos.bin", (size_t)n_tok * 12);
  int32_t* model = read_file(dir, "model.bin", (size_t)B * N * 4);
  float* R = read_file(dir, "R.bin", (size_t)B * N * 36);
  float* t = read_file(dir, "t.bin", (size_t)B * N * 12);
  float* k = read_file(dir, "k.bin", (size_t)B * N * 16);
  float* hi = read_file(dir, "hi.bin", (size_t)M * Hr * Wr * 12);

  /* O1 downsample, every factor that divides the render size */
  for (int f = 1; f <= 8; f *= 2) {
    if (Hr % f || Wr % f) continue;
    float* lo = malloc((size_t)M * (Hr / f) * (Wr / f) * 12);
    CHECK(orc_downsample(hi, M, Hr, Wr, f, lo));
    free(lo);
  }

  /* O2 bbox */
  float* bbox = malloc((size_t)B * 8 * sizeof(float));
  CHECK(orc_bbox(pos, B, N, H, W, 0.03f, bbox));

  /* O3 correspondence, O4 transport, O5 reconstruction over several anchor sets, K and dtypes */
  const int C = 4;
  const int32_t sets[4][4] = {{0, 0, 0, 0}, {0, 2, 0, 0}, {1, 2, 3, 0}, {0, 1, 2, 3}};
  const int set_a[4] = {1, 2, 3, 4};
  for (int si = 0; si < 4; ++si) {
    const int a = set_a[si];
    if (a > N) continue;
    const int NT = N - a;
    for (int K = 1; K <= 4; K += 3) {
      const int64_t n_rows = (int64_t)B * NT * HW;
      int32_t* corr = malloc((size_t)(n_rows * a + 1) * 4);
      double* wts = malloc((size_t)(n_rows * a * K + 1) * sizeof(double));
      int32_t* nvis = malloc((size_t)(n_rows + 1) * 4);
      CHECK(orc_build(pos, model, R, t, k, B, N, H, W, sets[si], a, K, bbox, corr, wts, nvis));
      for (int dtype = 0; dtype <= 1; ++dtype) {
        const int64_t n_all = n_tok * C;
        void* prev = latents(n_all, dtype, 2.0);
        void* anew = latents((int64_t)B * a * HW * C, dtype, 2.0);
        void* xt = latents(n_all, dtype, 2.0);
        double* exact = malloc((size_t)n_all * sizeof(double));
        void* state = malloc((size_t)n_all * (dtype == 0 ? 4 : 2));
        CHECK(orc_transport(prev, anew, corr, wts, sets[si], a, B, N, H, W, C, K, dtype, exact, state));
        double* xn = malloc((size_t)n_all * sizeof(double));
        double* mo = malloc((size_t)n_all * sizeof(double));
        CHECK(orc_reconstruct(xt, state, n_all, dtype, 0, 1, 1000, 1e-4, 0.02, 800.0, 760.0, xn, mo));
        CHECK(orc_reconstruct(xt, state, n_all, dtype, 0, 2, 1000, 1e-4, 0.02, 32.0, -1.0, xn, mo));
        CHECK(orc_reconstruct(xt, state, n_all, dtype, 1, 3, 1000, 1e-4, 0.02, 0.5, 0.48, xn, mo));
        free(prev), free(anew), free(xt), free(exact), free(state), free(xn), free(mo);
      }
      free(corr), free(wts), free(nvis);
    }
  }

  /* O6 host schedule, O8 UniPC */
  int32_t anc[8];
  for (int64_t c = 0; c < 3 * N; ++c) CHECK(orc_anchors(N, N < 2 ? 1 : 2, c, anc));
  uint8_t full[30];
  for (int rule = 0; rule <= 2; ++rule) CHECK(orc_full_steps(rule, 30, rule == 1 ? 0 : 5, full));
  const int S = 10;
  int32_t ts[11];
  CHECK(orc_ddim_timesteps(1000, S, ts));
  {
    const int64_t n = n_tok * C;
    void* xc0 = latents(n, 1, 2.0);
    void* xp0 = latents(n, 1, 2.0);
    void* m2 = latents(n, 1, 1.0);
    void* m1 = latents(n, 1, 1.0);
    void* mk = latents(n, 1, 1.0);
    double* xc = malloc((size_t)n * sizeof(double));
    double* xn = malloc((size_t)n * sizeof(double));
    double coef[10];
    for (int kk = 0; kk < S; ++kk)
      for (int order = 1; order <= 2; ++order) {
        CHECK(orc_unipc_coeffs(1000, 1e-4, 0.02, ts, S, kk, order, 1, coef));
        CHECK(orc_unipc_apply(xc0, xp0, m2, m1, mk, n, 1, coef, xc, xn));
      }
    free(xc0), free(xp0), free(m2), free(m1), free(mk), free(xc), free(xn);
  }

  /* O9 coverage: single-anchor visibility from one build per anchor */
  {
    uint8_t* seen = calloc((size_t)N * B * N * HW, 1);
    for (int u = 0; u < N; ++u) {
      const int32_t au[1] = {u};
      const int64_t n_rows = (int64_t)B * (N - 1) * HW;
      int32_t* corr = malloc((size_t)(n_rows + 1) * 4);
      double* wts = malloc((size_t)(n_rows * 4 + 1) * sizeof(double));
      int32_t* nvis = malloc((size_t)(n_rows + 1) * 4);
      CHECK(orc_build(pos, model, R, t, k, B, N, H, W, au, 1, 4, bbox, corr, wts, nvis));
      for (int b = 0; b < B; ++b) {
        int ti = 0;
        for (int v = 0; v < N; ++v) {
          if (v == u) continue;
          for (int64_t p = 0; p < HW; ++p)
            seen[(((int64_t)u * B + b) * N + v) * HW + p] = corr[((int64_t)b * (N - 1) + ti) * HW + p] != 0;
          ++ti;
        }
      }
      free(corr), free(wts), free(nvis);
    }
    uint8_t* stale = malloc((size_t)n_tok);
    uint32_t* stats = malloc((size_t)B * N * 16);
    CHECK(orc_cov_init(pos, n_tok, stale));
    const int a = N < 2 ? 1 : 2;
    for (int step = 0; step < 3 * N; ++step) {
      CHECK(orc_anchors(N, a, step, anc));
      CHECK(orc_cov_update(seen, B, N, HW, anc, a, 1 + step % 3, stale, stats));
      uint8_t chosen[64] = {0};
      uint64_t gains[64];
      chosen[step % N] = 1;
      CHECK(orc_cov_gains(seen, stale, B, N, HW, chosen, gains));
      const int32_t forced[1] = {step % N};
      CHECK(orc_cov_select(seen, stale, B, N, HW, a, forced, step % 2, anc));
      int32_t rot[2 * 8];
      CHECK(orc_anchors(N, a, 0, rot));
      CHECK(orc_anchors(N, a, 1, rot + a));
      uint64_t score[2];
      CHECK(orc_cov_score(seen, stale, B, N, HW, rot, 2, a, score));
      CHECK(orc_refresh_due(stats, B, N, 0.05));
    }
    free(seen), free(stale), free(stats);
  }

  free(pos), free(model), free(R), free(t), free(k), free(hi), free(bbox);
  printf("oracle under sanitizers: ok\n");
  return 0;
}
