// Correspondence builder: G_{A->v} for every non-anchor view of every asset,
// for one anchor set (once per asset and anchor set; the rotation has only a
// few distinct sets, so the host caches one build per set).
//
// Every float operation is written in a fixed order and the library is
// compiled without contraction, so the tap choice (an integer decision taken
// in float) is reproducible exactly.
//
// Visibility reductions use wavefront ballots: the anchors that see a token
// are counted by a ballot over its lane group, and each wave counts its
// visible pairs / tokens / taps with ballot + popcount before one lane adds
// them to the asset's counters.
#include "gc_common.h"
#include "gc_geometry.h"

namespace gc {
namespace {

constexpr int kBlock = 256;
// Launch size of the builder, in blocks per CU (256 CUs).  The coverage
// counters cost one device-scope atomic per block and counter, and atomics
// on one address serialise, so a build that counts uses fewer, longer
// blocks; one that does not uses enough blocks to hide its load latency.
constexpr int kBuildBlocksPerCU = 16;
constexpr int kBuildBlocksPerCUStats = 4;

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

// One lane per (target token, anchor slot): a group of G = 4 or 8 adjacent
// lanes serves one token (lanes with slot >= a idle).  Each lane projects the
// token into its own anchor, tests the four footprint taps, keeps the K
// nearest and forms that anchor's normalised area weights; the number of
// anchors that see the token (n_vis) is a ballot over the lane group.  Words
// and weights of one token are adjacent, so a group writes them coalesced.
// grid: y = b * NT + target slot; x = blocks that stride over the view's
// token chunks (kBlock / G tokens each).  A block counts its visible pairs /
// tokens / foreground tokens / taps over all its chunks and adds them to
// the asset's counters once: few blocks per asset keep the same-address
// atomics from serialising.  The block's anchor cameras are staged in LDS.
template <int G>
__global__ __launch_bounds__(kBlock) void k_build(BuildArgs g) {
  __shared__ gc_camera cam_lds[GC_MAX_ANCHORS];
  const int HW = g.H * g.W;
  const int bt = blockIdx.y;
  const int b = bt / g.NT;
  const int ti = bt - b * g.NT;
  const int v = g.target_view[ti];
  __shared__ int32_t view_lds[GC_MAX_ANCHORS];   // a lane's own slot: from LDS, not a per-lane kernel-argument load
  if (threadIdx.x < g.a) {
    view_lds[threadIdx.x] = g.anchor_view[threadIdx.x];
    cam_lds[threadIdx.x] = g.cams[(int64_t)b * g.N + g.anchor_view[threadIdx.x]];
  }
  __syncthreads();

  const int s = threadIdx.x & (G - 1);                   // anchor slot of this lane
  const float tol2 = g.bbox[(int64_t)b * 8 + 6];
  const int n_chunks = (HW + kBlock / G - 1) / (kBlock / G);
  uint32_t c_pairs = 0, c_pix = 0, c_fg = 0;   // wave totals (uniform across the wave)
  uint32_t taps_lane = 0;                       // this lane's kept taps, summed over the wave at the end
  for (int chunk = blockIdx.x; chunk < n_chunks; chunk += gridDim.x) {
    const int p = chunk * (kBlock / G) + threadIdx.x / G;
    const bool live = p < HW && s < g.a;

    float P[3] = {0.f, 0.f, 0.f};
    bool fg = false;
    if (p < HW) {
      const float* pp = g.pos + (((int64_t)b * g.N + v) * HW + p) * 3;
      P[0] = pp[0];
      P[1] = pp[1];
      P[2] = pp[2];
      fg = finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2]);
    }

    int32_t word = 0;
    float wk[4] = {0.f, 0.f, 0.f, 0.f};   // this anchor's normalised weight of tap k
    int mask = 0;
    if (live && fg) {
      const AnchorTaps at = anchor_taps(P, cam_lds[s], g.pos + ((int64_t)b * g.N + view_lds[s]) * HW * 3, g.H,
                                        g.W, g.K, tol2);
      word = at.word;
      mask = at.mask;
#pragma unroll
      for (int k = 0; k < 4; ++k) wk[k] = at.wk[k];
    }

    // n_vis: anchors of this token that see it -- a ballot over the lane group
    const unsigned long long seen = __ballot(word != 0);
    const int lane = __lane_id();
    const int gbase = lane & ~(G - 1);
    const int n_vis = __popcll((seen >> gbase) & ((G == 64) ? ~0ull : ((1ull << G) - 1)));

    if (live) {
      const int64_t row = ((int64_t)b * g.NT + ti) * HW + p;
      g.corr[row * g.a + s] = word;
    }
    // weights only for pairs the anchor sees: the transport reads a pair's
    // weights only when its word is non-zero (most pairs' words are zero)
    if (live && word != 0) {
      const int64_t row = ((int64_t)b * g.NT + ti) * HW + p;
      float out[4] = {0.f, 0.f, 0.f, 0.f};
      const float inv = n_vis > 0 ? (float)n_vis : 1.0f;
      int j = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (mask & (1 << k)) {
          // j-th kept tap -> slot j
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (q == j) out[q] = wk[k] / inv;
          ++j;
        }
      }
      float* ww = g.weights + (row * g.a + s) * g.K;
      if (g.K == 4) {   // 16-byte aligned: the weights base is, and each (token, slot) row is 16 bytes
        *reinterpret_cast<float4*>(ww) = make_float4(out[0], out[1], out[2], out[3]);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (q < g.K) ww[q] = out[q];
      }
    }

    if (g.stats) {
      const bool lead = (threadIdx.x & (G - 1)) == 0 && p < HW;
      c_pairs += (uint32_t)__popcll(seen);
      c_pix += wave_count(lead && n_vis > 0);
      c_fg += wave_count(lead && fg);
      taps_lane += live ? (uint32_t)__popc(mask) : 0u;
    }
  }

  if (g.stats) {
    // blocks never straddle assets (grid y is per asset and target): the
    // block sums its waves' totals in LDS, one thread per counter adds them
    // to the asset's counters
    __shared__ uint32_t part[kBlock / 64][4];
    const uint32_t c_taps = wave_sum(taps_lane);
    const int wv = threadIdx.x / 64;
    if (__lane_id() == 0) {
      part[wv][0] = c_pairs;
      part[wv][1] = c_pix;
      part[wv][2] = c_fg;
      part[wv][3] = c_taps;
    }
    __syncthreads();
    if (threadIdx.x < 4) {
      uint32_t sum = 0;
      for (int w = 0; w < kBlock / 64; ++w) sum += part[w][threadIdx.x];
      if (sum) atomicAdd(g.stats + (int64_t)b * 4 + threadIdx.x, sum);
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
    // x-blocks per (asset, target), from the launch size above
    const int tok = a <= 4 ? kBlock / 4 : kBlock / 8;
    const int64_t chunks = ((int64_t)HW + tok - 1) / tok;
    const int64_t per_cu = stats ? kBuildBlocksPerCUStats : kBuildBlocksPerCU;
    int64_t bx = (per_cu * 256 + (int64_t)B * NT - 1) / ((int64_t)B * NT);
    if (bx > chunks) bx = chunks;
    if (bx < 1) bx = 1;
    if (a <= 4)
      hipLaunchKernelGGL(k_build<4>, dim3((unsigned)bx, B * NT), dim3(kBlock), 0, stream, g);
    else
      hipLaunchKernelGGL(k_build<8>, dim3((unsigned)bx, B * NT), dim3(kBlock), 0, stream, g);
  }
  return after_launch(stream, "gc_build_correspondence");
}
