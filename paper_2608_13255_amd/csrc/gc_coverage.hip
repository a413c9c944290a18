// Token staleness and the coverage-driven schedule.
//
// A token no anchor sees keeps its state and misses that step's denoising
// until the next full step (Sec. 3.2, invalid matches); regions few anchors
// observe rely on the full steps, which adaptive anchor selection and
// visibility-aware refresh would relieve (the paper's limitations section).
// The library's reading of those two policies:
//   staleness    per token, the consecutive steps without a fresh prediction
//                (its view an anchor, or a full step) or a transported
//                increment (an anchor of the step sees it), saturating at
//                254; background tokens hold 255 and never count;
//   selection    greedy weighted maximum coverage: view u covers (b, v, p)
//                when v = u or u sees it, an uncovered foreground token
//                weighs 1 + staleness; forced views first, then the largest
//                gain (ties: lower view), a views in all, sorted;
//   refresh      due when the fraction of foreground tokens with staleness
//                >= R exceeds tau (host, gc_schedule_refresh_due).
// Visibility comes from single-anchor pairs: whether anchor u alone sees
// token p of view v, one bit each, from the correspondence operator's own
// tap test (gc_geometry.h).  A set sees a token iff one of its anchors does,
// because each anchor is tested on its own.
//
// All counters are integers, so the reductions (wave ballots and shuffles,
// block sums in LDS, one atomic per block and counter) are deterministic.
#include "gc_common.h"
#include "gc_geometry.h"

namespace gc {
namespace {

constexpr int kBlock = 256;
constexpr uint8_t kBackground = 255;
constexpr uint8_t kStaleMax = 254;

__device__ __forceinline__ uint32_t wave_add(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v += (uint32_t)__shfl_xor((int)v, o);
  return v;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}

__device__ __forceinline__ bool pair_bit(const uint32_t* bits, int B, int N, int wpr, int u, int b, int v, int p) {
  return (bits[(((int64_t)u * B + b) * N + v) * wpr + (p >> 5)] >> (p & 31)) & 1u;
}

// grid: x = token chunks of kBlock, y = (u * B + b) * N + v.  A wave's
// ballot gives two 32-token words of the row.
__global__ __launch_bounds__(kBlock) void k_cov_pairs(const float* __restrict__ pos, const gc_camera* __restrict__ cams,
                                                      const float* __restrict__ bbox, int B, int N, int H, int W,
                                                      int wpr, uint32_t* __restrict__ bits) {
  const int row = blockIdx.y;
  const int v = row % N;
  const int ub = row / N;
  const int b = ub % B;
  const int u = ub / B;
  const int HW = H * W;
  const int p = blockIdx.x * kBlock + (int)threadIdx.x;
  bool seen = false;
  if (p < HW && u != v) {
    const float* pp = pos + (((int64_t)b * N + v) * HW + p) * 3;
    const float P[3] = {pp[0], pp[1], pp[2]};
    if (finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2])) {
      const AnchorTaps at = anchor_taps(P, cams[(int64_t)b * N + u], pos + ((int64_t)b * N + u) * HW * 3, H, W, 4,
                                        bbox[(int64_t)b * 8 + 6]);
      seen = at.word != 0;
    }
  }
  const unsigned long long m = __ballot(seen);
  const int lane = __lane_id();
  const int w = p >> 5;
  if ((lane & 31) == 0 && w < wpr) bits[(int64_t)row * wpr + w] = (uint32_t)(m >> (lane & 32));
}

__global__ void k_cov_init(const float* __restrict__ pos, int64_t n_tok, uint8_t* __restrict__ stale) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n_tok) return;
  const float* P = pos + i * 3;
  stale[i] = (finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2])) ? 0 : kBackground;
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, int n, uint32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// grid: x = token chunks, y = b * N + v.  stats[b][v] = foreground tokens,
// tokens with staleness >= R, sum, max (after the update).
__global__ __launch_bounds__(kBlock) void k_cov_update(const uint32_t* __restrict__ bits, int B, int N, int HW,
                                                       int wpr, uint64_t anchor_mask, int R, uint8_t* __restrict__ stale,
                                                       uint32_t* __restrict__ stats) {
  const int bv = blockIdx.y;
  const int b = bv / N, v = bv % N;
  const int p = blockIdx.x * kBlock + (int)threadIdx.x;
  bool fg = false;
  uint32_t s = 0;
  if (p < HW) {
    uint8_t* sp = stale + (int64_t)bv * HW + p;
    s = *sp;
    fg = s != kBackground;
    if (fg) {
      bool fresh = (anchor_mask >> v) & 1ull;
      for (uint64_t m = anchor_mask; m && !fresh; m &= m - 1) fresh = pair_bit(bits, B, N, wpr, __ffsll((long long)m) - 1, b, v, p);
      s = fresh ? 0u : (s < kStaleMax ? s + 1u : (uint32_t)kStaleMax);
      *sp = (uint8_t)s;
    }
  }
  if (!fg) s = 0;
  __shared__ uint32_t part[kBlock / 64][4];
  const uint32_t c_fg = (uint32_t)__popcll(__ballot(fg));
  const uint32_t c_ge = (uint32_t)__popcll(__ballot(fg && s >= (uint32_t)R));
  const uint32_t c_sum = wave_add(s);
  const uint32_t c_max = wave_max(s);
  const int wv = threadIdx.x / 64;
  if (__lane_id() == 0) {
    part[wv][0] = c_fg;
    part[wv][1] = c_ge;
    part[wv][2] = c_sum;
    part[wv][3] = c_max;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    uint32_t acc = 0;
    for (int i = 0; i < kBlock / 64; ++i) acc = threadIdx.x == 3 ? max(acc, part[i][3]) : acc + part[i][threadIdx.x];
    uint32_t* o = stats + (int64_t)bv * 4 + threadIdx.x;
    if (threadIdx.x == 3)
      atomicMax(o, acc);
    else if (acc)
      atomicAdd(o, acc);
  }
}

// Selection state in the workspace.
struct SelState {
  unsigned long long gains[GC_MAX_VIEWS];
  unsigned long long chosen;   // bit u: view u chosen
};

__global__ void k_sel_begin(SelState* st, unsigned long long forced, int N) {
  const int u = threadIdx.x;
  if (u < N) st->gains[u] = 0ull;
  if (u == 0) st->chosen = forced;
}

// grid: x = token chunks, y = b * N + v.  Gains of every unchosen view.
__global__ __launch_bounds__(kBlock) void k_sel_gains(const uint32_t* __restrict__ bits,
                                                      const uint8_t* __restrict__ stale, int B, int N, int HW, int wpr,
                                                      SelState* st) {
  __shared__ uint32_t g_lds[GC_MAX_VIEWS];
  const int bv = blockIdx.y;
  const int b = bv / N, v = bv % N;
  const int p = blockIdx.x * kBlock + (int)threadIdx.x;
  const unsigned long long chosen = st->chosen;
  if ((int)threadIdx.x < N) g_lds[threadIdx.x] = 0u;
  __syncthreads();
  uint32_t w = 0;
  if (p < HW) {
    const uint8_t s = stale[(int64_t)bv * HW + p];
    if (s != kBackground) {
      bool covered = (chosen >> v) & 1ull;
      for (unsigned long long m = chosen; m && !covered; m &= m - 1)
        covered = pair_bit(bits, B, N, wpr, __ffsll((long long)m) - 1, b, v, p);
      w = covered ? 0u : 1u + s;
    }
  }
  for (int u = 0; u < N; ++u) {   // uniform loop: every lane reaches the shuffles
    if ((chosen >> u) & 1ull) continue;
    const bool hit = w && (u == v || (p < HW && pair_bit(bits, B, N, wpr, u, b, v, p)));
    const uint32_t sum = wave_add(hit ? w : 0u);
    if (__lane_id() == 0 && sum) atomicAdd(&g_lds[u], sum);
  }
  __syncthreads();
  if ((int)threadIdx.x < N && g_lds[threadIdx.x]) atomicAdd(&st->gains[threadIdx.x], (unsigned long long)g_lds[threadIdx.x]);
}

// one thread: take the unchosen view with the largest gain (ties: lower
// view), then clear the gains for the next round
__global__ void k_sel_pick(SelState* st, int N) {
  if (threadIdx.x != 0) return;
  int best = -1;
  for (int u = 0; u < N; ++u) {
    if ((st->chosen >> u) & 1ull) continue;
    if (best < 0 || st->gains[u] > st->gains[best]) best = u;
  }
  if (best >= 0) st->chosen |= 1ull << best;
  for (int u = 0; u < N; ++u) st->gains[u] = 0ull;
}

__global__ void k_sel_finish(const SelState* st, int N, int32_t* out) {
  if (threadIdx.x != 0) return;
  int j = 0;
  for (int u = 0; u < N; ++u)
    if ((st->chosen >> u) & 1ull) out[j++] = u;
}

// Candidate sets as view masks (at most kMaxSets per call).
constexpr int kMaxSets = 64;
struct SetMasks {
  unsigned long long m[kMaxSets];
};

__global__ void k_fill_u64(unsigned long long* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

// grid: x = token chunks, y = b * N + v.  score[m] += 1 + staleness over the
// foreground tokens set m covers.
__global__ __launch_bounds__(kBlock) void k_cov_score(const uint32_t* __restrict__ bits,
                                                      const uint8_t* __restrict__ stale, int B, int N, int HW, int wpr,
                                                      SetMasks sets, int M, unsigned long long* __restrict__ score) {
  __shared__ uint32_t s_lds[kMaxSets];
  const int bv = blockIdx.y;
  const int b = bv / N, v = bv % N;
  const int p = blockIdx.x * kBlock + (int)threadIdx.x;
  if ((int)threadIdx.x < M) s_lds[threadIdx.x] = 0u;
  __syncthreads();
  uint32_t w = 0;
  if (p < HW) {
    const uint8_t s = stale[(int64_t)bv * HW + p];
    w = s == kBackground ? 0u : 1u + s;
  }
  for (int m = 0; m < M; ++m) {   // uniform loop: every lane reaches the shuffles
    bool covered = false;
    if (w) {
      covered = (sets.m[m] >> v) & 1ull;
      for (unsigned long long q = sets.m[m]; q && !covered; q &= q - 1)
        covered = pair_bit(bits, B, N, wpr, __ffsll((long long)q) - 1, b, v, p);
    }
    const uint32_t sum = wave_add(covered ? w : 0u);
    if (__lane_id() == 0 && sum) atomicAdd(&s_lds[m], sum);
  }
  __syncthreads();
  if ((int)threadIdx.x < M && s_lds[threadIdx.x]) atomicAdd(&score[threadIdx.x], (unsigned long long)s_lds[threadIdx.x]);
}

int check_grid(int B, int N, int H, int W, const char* who) {
  if (B < 1 || N < 1 || H < 1 || W < 1) return fail(GC_ERR_SHAPE, "%s: bad shape B=%d N=%d H=%d W=%d", who, B, N, H, W);
  if (N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "%s: N=%d exceeds %d", who, N, GC_MAX_VIEWS);
  if (H > GC_MAX_GRID || W > GC_MAX_GRID) return fail(GC_ERR_CAPACITY, "%s: grid %dx%d exceeds %d", who, H, W, GC_MAX_GRID);
  if ((int64_t)B * N * N > 65535) return fail(GC_ERR_CAPACITY, "%s: B*N*N exceeds 65535", who);
  return GC_OK;
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" int64_t gc_coverage_pair_words(int B, int N, int H, int W) {
  if (B < 1 || N < 1 || H < 1 || W < 1) return 0;
  const int64_t wpr = ((int64_t)H * W + 31) / 32;
  return (int64_t)N * B * N * wpr;
}

extern "C" int gc_coverage_pairs(const float* pos, const gc_camera* cams, const float* bbox, int B, int N, int H,
                                 int W, uint32_t* pair_bits, hipStream_t stream) {
  clear_error();
  if (!pos || !cams || !bbox || !pair_bits) return fail(GC_ERR_ARG, "gc_coverage_pairs: null pointer");
  int rc = check_grid(B, N, H, W, "gc_coverage_pairs");
  if (rc) return rc;
  if (!aligned16(pos) || !aligned16(pair_bits)) return fail(GC_ERR_ALIGN, "gc_coverage_pairs: pos and pair_bits must be 16-byte aligned");
  const size_t HW = (size_t)H * W;
  const int wpr = (int)((HW + 31) / 32);
  const size_t nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  if (overlaps(pair_bits, nb, pos, (size_t)B * N * HW * 12) || overlaps(pair_bits, nb, cams, (size_t)B * N * sizeof(gc_camera)) ||
      overlaps(pair_bits, nb, bbox, (size_t)B * 32))
    return fail(GC_ERR_ALIAS, "gc_coverage_pairs: pair_bits overlaps an input");
  const dim3 grid((unsigned)((HW + kBlock - 1) / kBlock), (unsigned)(N * B * N));
  hipLaunchKernelGGL(k_cov_pairs, grid, dim3(kBlock), 0, stream, pos, cams, bbox, B, N, H, W, wpr, pair_bits);
  return after_launch(stream, "gc_coverage_pairs");
}

extern "C" int gc_coverage_init(const float* pos, int B, int N, int H, int W, uint8_t* stale, hipStream_t stream) {
  clear_error();
  if (!pos || !stale) return fail(GC_ERR_ARG, "gc_coverage_init: null pointer");
  int rc = check_grid(B, N, H, W, "gc_coverage_init");
  if (rc) return rc;
  const int64_t n_tok = (int64_t)B * N * H * W;
  if (overlaps(stale, (size_t)n_tok, pos, (size_t)n_tok * 12)) return fail(GC_ERR_ALIAS, "gc_coverage_init: stale overlaps pos");
  hipLaunchKernelGGL(k_cov_init, dim3((unsigned)((n_tok + kBlock - 1) / kBlock)), dim3(kBlock), 0, stream, pos, n_tok,
                     stale);
  return after_launch(stream, "gc_coverage_init");
}

extern "C" int gc_coverage_update(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a,
                                  int R, uint8_t* stale, uint32_t* stats, hipStream_t stream) {
  clear_error();
  if (!pair_bits || !anchors || !stale || !stats) return fail(GC_ERR_ARG, "gc_coverage_update: null pointer");
  int rc = check_grid(B, N, H, W, "gc_coverage_update");
  if (rc) return rc;
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "gc_coverage_update: a=%d outside [1, N=%d]", a, N);
  if (R < 1) return fail(GC_ERR_ARG, "gc_coverage_update: R=%d must be >= 1", R);
  unsigned long long mask = 0;
  for (int s = 0; s < a; ++s) {
    if (anchors[s] < 0 || anchors[s] >= N) return fail(GC_ERR_ARG, "gc_coverage_update: anchor %d outside [0, %d)", anchors[s], N);
    if ((mask >> anchors[s]) & 1ull) return fail(GC_ERR_ARG, "gc_coverage_update: anchor %d listed twice", anchors[s]);
    mask |= 1ull << anchors[s];
  }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  if (overlaps(stats, (size_t)B * N * 16, stale, n_tok) || overlaps(stats, (size_t)B * N * 16, pair_bits, nb) ||
      overlaps(stale, n_tok, pair_bits, nb))
    return fail(GC_ERR_ALIAS, "gc_coverage_update: stale, stats and pair_bits must not overlap");
  if (!aligned16(pair_bits) || !aligned16(stats)) return fail(GC_ERR_ALIGN, "gc_coverage_update: pair_bits and stats must be 16-byte aligned");
  const int wpr = (int)((HW + 31) / 32);
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((B * N * 4 + 255) / 256)), dim3(256), 0, stream, stats, B * N * 4, 0u);
  const dim3 grid((unsigned)((HW + kBlock - 1) / kBlock), (unsigned)(B * N));
  hipLaunchKernelGGL(k_cov_update, grid, dim3(kBlock), 0, stream, pair_bits, B, N, (int)HW, wpr, (uint64_t)mask, R, stale,
                     stats);
  return after_launch(stream, "gc_coverage_update");
}

extern "C" size_t gc_coverage_workspace_bytes(void) { return (sizeof(SelState) + 255) / 256 * 256; }

extern "C" int gc_coverage_select(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, int a,
                                  const int32_t* forced, int n_forced, int32_t* anchors_out, void* workspace,
                                  size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!pair_bits || !stale || !anchors_out || !workspace) return fail(GC_ERR_ARG, "gc_coverage_select: null pointer");
  int rc = check_grid(B, N, H, W, "gc_coverage_select");
  if (rc) return rc;
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "gc_coverage_select: a=%d outside [1, N=%d]", a, N);
  if (a > GC_MAX_ANCHORS) return fail(GC_ERR_CAPACITY, "gc_coverage_select: a=%d exceeds %d", a, GC_MAX_ANCHORS);
  if (n_forced < 0 || n_forced > a || (n_forced > 0 && !forced))
    return fail(GC_ERR_ARG, "gc_coverage_select: n_forced=%d outside [0, a=%d]", n_forced, a);
  if (ws_bytes < gc_coverage_workspace_bytes())
    return fail(GC_ERR_CAPACITY, "gc_coverage_select: workspace of %zu bytes, %zu needed", ws_bytes, gc_coverage_workspace_bytes());
  if (!aligned16(workspace) || !aligned16(pair_bits)) return fail(GC_ERR_ALIGN, "gc_coverage_select: workspace and pair_bits must be 16-byte aligned");
  unsigned long long mask = 0;
  for (int j = 0; j < n_forced; ++j) {
    if (forced[j] < 0 || forced[j] >= N) return fail(GC_ERR_ARG, "gc_coverage_select: forced view %d outside [0, %d)", forced[j], N);
    if ((mask >> forced[j]) & 1ull) return fail(GC_ERR_ARG, "gc_coverage_select: forced view %d listed twice", forced[j]);
    mask |= 1ull << forced[j];
  }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  const size_t ws = gc_coverage_workspace_bytes();
  if (overlaps(workspace, ws, pair_bits, nb) || overlaps(workspace, ws, stale, n_tok) ||
      overlaps(anchors_out, (size_t)a * 4, workspace, ws) || overlaps(anchors_out, (size_t)a * 4, pair_bits, nb) ||
      overlaps(anchors_out, (size_t)a * 4, stale, n_tok))
    return fail(GC_ERR_ALIAS, "gc_coverage_select: workspace / anchors_out overlap an input");
  SelState* st = static_cast<SelState*>(workspace);
  const int wpr = (int)((HW + 31) / 32);
  hipLaunchKernelGGL(k_sel_begin, dim3(1), dim3(64), 0, stream, st, mask, N);
  const dim3 grid((unsigned)((HW + kBlock - 1) / kBlock), (unsigned)(B * N));
  for (int r = n_forced; r < a; ++r) {
    hipLaunchKernelGGL(k_sel_gains, grid, dim3(kBlock), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, st);
    hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(64), 0, stream, st, N);
  }
  hipLaunchKernelGGL(k_sel_finish, dim3(1), dim3(64), 0, stream, st, N, anchors_out);
  return after_launch(stream, "gc_coverage_select");
}

extern "C" int gc_coverage_score(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W,
                                 const int32_t* sets, int M, int a, uint64_t* scores, hipStream_t stream) {
  clear_error();
  if (!pair_bits || !stale || !sets || !scores) return fail(GC_ERR_ARG, "gc_coverage_score: null pointer");
  int rc = check_grid(B, N, H, W, "gc_coverage_score");
  if (rc) return rc;
  if (M < 1 || M > kMaxSets) return fail(GC_ERR_CAPACITY, "gc_coverage_score: M=%d outside [1, %d]", M, kMaxSets);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "gc_coverage_score: a=%d outside [1, N=%d]", a, N);
  SetMasks masks;
  std::memset(&masks, 0, sizeof(masks));
  for (int m = 0; m < M; ++m)
    for (int j = 0; j < a; ++j) {
      const int u = sets[m * a + j];
      if (u < 0 || u >= N) return fail(GC_ERR_ARG, "gc_coverage_score: view %d of set %d outside [0, %d)", u, m, N);
      masks.m[m] |= 1ull << u;
    }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  if (overlaps(scores, (size_t)M * 8, pair_bits, nb) || overlaps(scores, (size_t)M * 8, stale, n_tok))
    return fail(GC_ERR_ALIAS, "gc_coverage_score: scores overlap an input");
  if (!aligned16(pair_bits) || ((uintptr_t)scores & 7u)) return fail(GC_ERR_ALIGN, "gc_coverage_score: pair_bits 16-byte, scores 8-byte aligned");
  const int wpr = (int)((HW + 31) / 32);
  hipLaunchKernelGGL(k_fill_u64, dim3(1), dim3(64), 0, stream, reinterpret_cast<unsigned long long*>(scores), M);
  const dim3 grid((unsigned)((HW + kBlock - 1) / kBlock), (unsigned)(B * N));
  hipLaunchKernelGGL(k_cov_score, grid, dim3(kBlock), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, masks, M,
                     reinterpret_cast<unsigned long long*>(scores));
  return after_launch(stream, "gc_coverage_score");
}
