// Host-side parts of the library: error state, launch checking, the host
// schedule (anchor rotation, full-view steps, sampler step times) and the
// sampler coefficients.  No device memory is touched here.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>

#include "gc_common.h"

namespace gc {

namespace {
thread_local char g_err[512] = "";

bool sync_check_enabled() {
  static const bool on = [] {
    const char* e = std::getenv("GC_SYNC_CHECK");
    return e && e[0] && e[0] != '0';
  }();
  return on;
}
}  // namespace

int64_t split_min_items() {
  static const int64_t n = [] {
    const char* e = std::getenv("GC_SPLIT_MIN_ITEMS");
    if (!e || !e[0]) return (int64_t)1 << 18;
    char* end = nullptr;
    const long long v = std::strtoll(e, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (int64_t)v : (int64_t)1 << 18;
  }();
  return n;
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_err[0] = '\0'; }

int after_launch(hipStream_t stream, const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GC_ERR_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  if (sync_check_enabled()) {
    e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(GC_ERR_HIP, "%s: execution failed: %s", what, hipGetErrorString(e));
  }
  return GC_OK;
}

// abar_t = prod_{i<=t} (1 - beta_i), beta_i = beta_start + (beta_end - beta_start) i / (T - 1)
static double alpha_bar(const gc_sampler* smp, int t) {
  if (t < 0) return 1.0;
  double ab = 1.0;
  for (int i = 0; i <= t; ++i) {
    const double beta = smp->beta_start + (smp->beta_end - smp->beta_start) * (double)i / (double)(smp->T - 1);
    ab *= 1.0 - beta;
  }
  return ab;
}

static int check_sampler(const gc_sampler* smp) {
  if (!smp) return fail(GC_ERR_ARG, "sampler is null");
  if (smp->kind == GC_DDIM) {
    if (smp->T < 2 || smp->T > 100000) return fail(GC_ERR_ARG, "DDIM T=%d out of range [2, 100000]", smp->T);
    if (!(smp->beta_start > 0.0 && smp->beta_end < 1.0 && smp->beta_start <= smp->beta_end))
      return fail(GC_ERR_ARG, "DDIM betas must satisfy 0 < beta_start <= beta_end < 1");
    if (smp->pred_out != GC_PRED_NONE && smp->pred_out != GC_PRED_EPS && smp->pred_out != GC_PRED_V)
      return fail(GC_ERR_ARG, "DDIM pred_out %d is not NONE, EPS or V", smp->pred_out);
  } else if (smp->kind == GC_FLOW_EULER) {
    if (smp->pred_out != GC_PRED_NONE && smp->pred_out != GC_PRED_VEL)
      return fail(GC_ERR_ARG, "flow pred_out %d is not NONE or VEL", smp->pred_out);
  } else {
    return fail(GC_ERR_ARG, "unknown sampler kind %d", smp->kind);
  }
  return GC_OK;
}

int make_recon(const gc_sampler* smp, double t, double t_next, Recon* r) {
  int rc = check_sampler(smp);
  if (rc) return rc;
  std::memset(r, 0, sizeof(*r));
  r->kind = smp->kind;
  r->pred = smp->pred_out;
  if (smp->kind == GC_DDIM) {
    if (t != std::floor(t) || t_next != std::floor(t_next))
      return fail(GC_ERR_ARG, "DDIM timesteps must be integers (t=%g, t_next=%g)", t, t_next);
    if (t < 0 || t >= smp->T || t_next >= t || t_next < -1)
      return fail(GC_ERR_ARG, "DDIM step %g -> %g outside 0 <= t < T, -1 <= t_next < t", t, t_next);
    const double ab_t = alpha_bar(smp, (int)t), ab_n = alpha_bar(smp, (int)t_next);
    const double s_t = std::sqrt(1.0 - ab_t);
    r->a_t = (float)std::sqrt(ab_t);
    r->s_t = (float)s_t;
    r->inv_s_t = (float)(1.0 / s_t);
    r->a_n = (float)std::sqrt(ab_n);
    r->s_n = (float)std::sqrt(1.0 - ab_n);
  } else {
    if (!(t > 0.0 && t <= 1.0) || !(t_next >= 0.0 && t_next <= t))
      return fail(GC_ERR_ARG, "flow step sigma %g -> %g outside 0 < sigma_t <= 1, 0 <= sigma_n <= sigma_t", t,
                  t_next);
    r->inv_sigma = (float)(1.0 / t);
    r->dsigma = (float)(t_next - t);
  }
  return GC_OK;
}

}  // namespace gc

using namespace gc;

extern "C" {

int gc_abi_version(void) { return GC_ABI_VERSION; }

const char* gc_last_error(void) { return g_err; }

int gc_schedule_anchors(int N, int a, int64_t c, int32_t* anchors_out) {
  clear_error();
  if (!anchors_out) return fail(GC_ERR_ARG, "anchors_out is null");
  if (N < 1 || N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "N=%d outside [1, %d]", N, GC_MAX_VIEWS);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "a=%d outside [1, N=%d]", a, N);
  if (c < 0) return fail(GC_ERR_ARG, "cached-step counter %lld is negative", (long long)c);
  // rotate the evenly spread set {floor(j*N/a)} by c, then order by view
  bool member[GC_MAX_VIEWS] = {};
  for (int j = 0; j < a; ++j) member[(int)((c + (int64_t)j * N / a) % N)] = true;
  int n = 0;
  for (int v = 0; v < N; ++v)
    if (member[v]) anchors_out[n++] = v;
  return GC_OK;
}

int gc_schedule_full_steps(int rule, int S, int E, uint8_t* is_full_out) {
  clear_error();
  if (!is_full_out) return fail(GC_ERR_ARG, "is_full_out is null");
  if (S < 1) return fail(GC_ERR_ARG, "S=%d must be positive", S);
  std::memset(is_full_out, 0, (size_t)S);
  if (rule == GC_FULL_PERIODIC) {
    if (E < 1) return fail(GC_ERR_ARG, "periodic full steps need E >= 1 (got %d)", E);
    for (int k = 0; k < S; k += E) is_full_out[k] = 1;
  } else if (rule == GC_FULL_HEAD_MID_TAIL) {
    is_full_out[0] = 1;
    if (S > 1) is_full_out[1] = 1;
    is_full_out[S / 2] = 1;
    is_full_out[S - 1] = 1;
  } else if (rule == GC_FULL_HEAD_TAIL_E) {
    if (E < 0 || E > S) return fail(GC_ERR_ARG, "head + tail full steps need 0 <= E <= S (got E=%d, S=%d)", E, S);
    is_full_out[0] = 1;
    if (S > 1) is_full_out[1] = 1;
    for (int k = S - E; k < S; ++k) is_full_out[k] = 1;
  } else {
    return fail(GC_ERR_ARG, "unknown full-step rule %d", rule);
  }
  is_full_out[0] = 1;
  return GC_OK;
}

int gc_sampler_step_times(const gc_sampler* smp, int S, int k, double* t, double* t_next) {
  clear_error();
  int rc = check_sampler(smp);
  if (rc) return rc;
  if (!t || !t_next) return fail(GC_ERR_ARG, "output pointer is null");
  if (S < 1 || k < 0 || k >= S) return fail(GC_ERR_ARG, "step %d outside [0, S=%d)", k, S);
  if (smp->kind == GC_DDIM) {
    if (S > smp->T) return fail(GC_ERR_ARG, "S=%d exceeds T=%d", S, smp->T);
    auto ts = [&](int j) { return j >= S ? -1.0 : std::floor((double)(S - j) * smp->T / S + 0.5) - 1.0; };
    *t = ts(k);
    *t_next = ts(k + 1);
  } else {
    *t = 1.0 - (double)k / S;
    *t_next = 1.0 - (double)(k + 1) / S;
  }
  return GC_OK;
}

int gc_schedule_refresh_due(const uint32_t* stats, int B, int N, double tau, int* due) {
  clear_error();
  if (!stats || !due) return fail(GC_ERR_ARG, "refresh: null pointer");
  if (B < 1 || N < 1) return fail(GC_ERR_SHAPE, "refresh: bad shape B=%d N=%d", B, N);
  if (!(tau >= 0.0 && tau <= 1.0)) return fail(GC_ERR_ARG, "refresh: tau outside [0, 1]");
  uint64_t fg = 0, stale = 0;
  for (int64_t i = 0; i < (int64_t)B * N; ++i) {
    fg += stats[i * 4 + 0];
    stale += stats[i * 4 + 1];
  }
  *due = fg > 0 && (double)stale > tau * (double)fg;
  return GC_OK;
}

int gc_schedule_forced_views(const int32_t* gap, int N, int a, int max_gap, int32_t* forced_out, int* n_forced) {
  clear_error();
  if (!gap || !forced_out || !n_forced) return fail(GC_ERR_ARG, "forced views: null pointer");
  if (N < 1 || N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "forced views: N=%d outside [1, %d]", N, GC_MAX_VIEWS);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "forced views: a=%d outside [1, N=%d]", a, N);
  if (max_gap < 0) return fail(GC_ERR_ARG, "forced views: max_gap=%d is negative", max_gap);
  for (int v = 0; v < N; ++v)
    if (gap[v] < 0) return fail(GC_ERR_ARG, "forced views: gap[%d]=%d is negative", v, gap[v]);
  *n_forced = 0;
  if (max_gap == 0) return GC_OK;
  // a rounds of "the due view with the longest gap, the lowest such view"
  bool taken[GC_MAX_VIEWS] = {};
  for (int r = 0; r < a; ++r) {
    int best = -1;
    for (int v = 0; v < N; ++v)
      if (!taken[v] && gap[v] >= max_gap && (best < 0 || gap[v] > gap[best])) best = v;
    if (best < 0) break;
    taken[best] = true;
    forced_out[(*n_forced)++] = best;
  }
  return GC_OK;
}

int gc_schedule_advance_gaps(int32_t* gap, int N, const int32_t* views, int n_views, int full) {
  clear_error();
  if (!gap || (n_views > 0 && !views)) return fail(GC_ERR_ARG, "advance gaps: null pointer");
  if (N < 1 || N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "advance gaps: N=%d outside [1, %d]", N, GC_MAX_VIEWS);
  if (n_views < 0 || n_views > N) return fail(GC_ERR_ARG, "advance gaps: n_views=%d outside [0, N=%d]", n_views, N);
  bool fresh[GC_MAX_VIEWS] = {};
  for (int i = 0; i < n_views; ++i) {
    if (views[i] < 0 || views[i] >= N) return fail(GC_ERR_ARG, "advance gaps: view %d outside [0, %d)", views[i], N);
    fresh[views[i]] = true;
  }
  for (int v = 0; v < N; ++v)
    if (gap[v] < 0) return fail(GC_ERR_ARG, "advance gaps: gap[%d]=%d is negative", v, gap[v]);
  for (int v = 0; v < N; ++v) gap[v] = (full || fresh[v]) ? 0 : (gap[v] == INT32_MAX ? INT32_MAX : gap[v] + 1);
  return GC_OK;
}

int gc_sampler_alpha_bar(const gc_sampler* smp, int t, double* abar) {
  clear_error();
  if (!smp || !abar) return fail(GC_ERR_ARG, "null argument");
  if (smp->kind != GC_DDIM) return fail(GC_ERR_ARG, "alpha_bar needs a DDIM sampler");
  int rc = check_sampler(smp);
  if (rc) return rc;
  if (t < -1 || t >= smp->T) return fail(GC_ERR_ARG, "t=%d outside [-1, T)", t);
  *abar = alpha_bar(smp, t);
  return GC_OK;
}

// UniPC (bh2, data prediction) coefficients of step k.  Times: trailing
// DDIM timesteps, the step after the last one at sigma = 0.
int gc_unipc_coeffs(const gc_sampler* smp, int S, int k, int order, int corrector, gc_unipc_step* out) {
  clear_error();
  if (!smp || !out) return fail(GC_ERR_ARG, "unipc: null argument");
  if (smp->kind != GC_DDIM) return fail(GC_ERR_ARG, "unipc: needs a GC_DDIM sampler for its noise schedule");
  int rc = check_sampler(smp);
  if (rc) return rc;
  if (order < 1 || order > 2) return fail(GC_ERR_ARG, "unipc: order %d outside [1, 2]", order);
  if (S < 1 || S > smp->T || k < 0 || k >= S) return fail(GC_ERR_ARG, "unipc: step %d outside [0, S=%d)", k, S);
  auto tstep = [&](int j) { return j >= S ? -1 : (int)(std::floor((double)(S - j) * smp->T / S + 0.5) - 1.0); };
  auto ab = [&](int t) { return alpha_bar(smp, t); };
  auto lam = [&](int t) {
    const double a = ab(t);
    return 0.5 * std::log(a / (1.0 - a));   // log(alpha / sigma)
  };
  auto pred_order = [&](int j) {
    int o = order;
    if (j + 1 < o) o = j + 1;   // warm-up: no older x0 yet
    if (S - j < o) o = S - j;   // first-order last step
    return o;
  };
  std::memset(out, 0, sizeof(*out));
  const int t0 = tstep(k);
  const double a0 = std::sqrt(ab(t0)), s0 = std::sqrt(1.0 - ab(t0)), l0 = lam(t0);
  if (corrector && k >= 1) {
    const int pc = pred_order(k - 1);
    const int tp = tstep(k - 1);
    const double sp = std::sqrt(1.0 - ab(tp)), lp = lam(tp);
    const double h = l0 - lp, hh = -h;
    const double phi1 = std::expm1(hh), Bh = std::expm1(hh);
    out->use_corrector = 1;
    out->corrector_order = pc;
    out->c_xprev = s0 / sp;
    if (pc == 1) {
      // x_c = s0/sp x_prev - a0 phi1 m_{k-1} - a0 Bh (1/2) (m_k - m_{k-1})
      out->c_mk1 = -a0 * phi1 + 0.5 * a0 * Bh;
      out->c_mk = -0.5 * a0 * Bh;
    } else {
      const double r1 = (lam(tstep(k - 2)) - lp) / h;
      // rho solves [[1, 1], [r1, 1]] rho = (g1, g2), g_i = hphi_i i! / Bh
      const double hphi2 = phi1 / hh - 1.0;
      const double hphi3 = hphi2 / hh - 0.5;
      const double g1 = hphi2 / Bh, g2 = 2.0 * hphi3 / Bh;
      const double rho0 = (g1 - g2) / (1.0 - r1);
      const double rho1 = g1 - rho0;
      // ... - a0 Bh (rho0 (m_{k-2} - m_{k-1}) / r1 + rho1 (m_k - m_{k-1}))
      out->c_mk2 = -a0 * Bh * rho0 / r1;
      out->c_mk1 = -a0 * phi1 + a0 * Bh * (rho0 / r1 + rho1);
      out->c_mk = -a0 * Bh * rho1;
    }
  }
  const int pp = pred_order(k);
  out->predictor_order = pp;
  const int tn = tstep(k + 1);
  if (tn < 0) {
    out->p_mk = 1.0;   // sigma = 0: the sample is the clean estimate
    return GC_OK;
  }
  const double an = std::sqrt(ab(tn)), sn = std::sqrt(1.0 - ab(tn)), ln = lam(tn);
  const double h = ln - l0, hh = -h;
  const double phi1 = std::expm1(hh), Bh = std::expm1(hh);
  out->p_xc = sn / s0;
  out->p_mk = -an * phi1;
  if (pp == 2) {
    const double r1 = (lam(tstep(k - 1)) - l0) / h;
    // ... - an Bh (1/2) (m_{k-1} - m_k) / r1
    out->p_mk1 = -0.5 * an * Bh / r1;
    out->p_mk += 0.5 * an * Bh / r1;
  }
  return GC_OK;
}

}  // extern "C"
