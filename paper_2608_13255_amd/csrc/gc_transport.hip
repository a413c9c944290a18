// Per-step kernels: delta transport (Eq. 1), sampler-consistent
// reconstruction, the two fused into one pass, and the multistep variant
// (Eq. 1 fused with the UniPC corrector + predictor on the x0 history).
//
// All of them are HBM-streaming: each latent element is read and written
// once; the only reuse is the gather of anchor taps, which neighbouring
// target tokens share and which stays in L2.  No MFMA: nothing here is a
// dense contraction.
//
// Work mapping: one thread per (asset, view, pixel, channel vector); a
// channel vector is 16 bytes (4 floats or 8 bfloat16; 4 bfloat16 when C is
// not a multiple of 8), so every latent access is one 16-byte (or 8-byte)
// load/store, consecutive lanes touch consecutive addresses, and the threads
// of one pixel share its correspondence words and weights through L1.
//
// Dense launch (no visible-token index): every block tiles (asset, view)
// rows and each target thread reads its token's words.  Split launch (with
// gc_index_correspondence's index): gather blocks over the compact list of
// visible tokens come first, in XCD-contiguous slices so that an XCD gathers
// from only its own assets' anchor views, which fit its L2; streaming blocks
// over all rows follow in the hardware's round-robin order and skip the
// visible tokens by their bit.  Data each thread touches once (its own
// x0_prev and x_t, every output) is read and written with nontemporal hints;
// the gathered anchor tiles, and an anchor row's own inputs that the gathers
// also read (its new prediction, its x0_prev for UniPC), go through L2
// normally.
#include "gc_common.h"
#include "gc_latent.h"

namespace gc {
namespace {

constexpr int kBlock = 256;

struct TArgs {
  const void* x0_prev;
  const void* x0_new;
  const int32_t* corr;
  const float* weights;
  const void* x_t;
  void* x0_out;
  void* x_next;
  void* model_out;
  int64_t n_threads;   // B * N * H * W * (C / VEC) chunks
  int N, H, W, HW, C, a, K, NT, CV;
  int cv_shift;        // log2(CV) when CV is a power of two, else -1
  int bpv;             // blocks per view: ceil(HW * CV / kBlock)
  int n_blocks;        // logical blocks = B * N * bpv (before XCD padding)
  int remap;           // 1: XCD-contiguous block order
  int32_t anchor_view[GC_MAX_ANCHORS];   // view of anchor slot s
  // optional visible-token index (gc_index_correspondence): split launch
  const uint32_t* vis_bits;
  const int32_t* vis_list;
  int64_t n_tokens;    // B * NT * HW
  int n_vis;
  int gblocks;         // gather blocks in front of the streaming blocks (multiple of kXcds)
  int32_t sorted_anchor[GC_MAX_ANCHORS];  // anchor views ascending, padded with INT_MAX
  Recon r;
  // UniPC mode: x_t is x_cur; x_prev / m_km2 inputs, x_c output; coefficients in float
  const void* x_prev;
  const void* m_km2;
  void* x_c;
  UniCoef u;
};

// What a step does after the transport: nothing, the sampler reconstruction
// (DDIM / flow Euler), or the UniPC corrector + predictor.
enum StepMode { kTransportOnly = 0, kReconstruct = 1, kUniPC = 2 };

// What the caller of token_step knows about a target token.
enum TokenMode { kAnchorRow = 0, kTargetCheck = 1, kTargetSeen = 2, kTargetUnseen = 3 };

// One cached step for one (token, channel vector): Eq. 1 for a target token
// (or the copy for an anchor row), then, when fused, the reconstruction.
template <int DT, int VEC, int MODE>
__device__ __forceinline__ void token_step(const TArgs& g, int b, int p, int cv, int s_self, int64_t crow,
                                           int64_t base, TokenMode mode) {
  using CD = Codec<DT, VEC>;
  using Raw = typename CD::Raw;
  // issue every load of data this thread owns before using any of it
  Raw xtr, m2r, m1r;
  if constexpr (MODE == kReconstruct) xtr = CD::load_stream(g.x_t, base);
  if constexpr (MODE == kUniPC) {
    xtr = CD::load_stream(g.u.corr ? g.x_prev : g.x_t, base);
    if (g.u.need_m2) m2r = CD::load_stream(g.m_km2, base);
    // an anchor row's own x0_prev is also gathered by the target tokens that
    // see it: a cached load (measured faster than a nontemporal one)
    if (g.u.need_m1 && mode == kAnchorRow) m1r = CD::load(g.x0_prev, base);
  }
  Raw x0r;
  float x0f[VEC];
  if (mode == kAnchorRow) {
    // anchor row: the store keeps this step's prediction
    x0r = CD::load(g.x0_new, (((int64_t)b * g.a + s_self) * g.HW + p) * g.C + (int64_t)cv * VEC);
    CD::unpack(x0r, x0f);
  } else if (mode == kTargetUnseen) {
    x0r = CD::load_stream(g.x0_prev, base);   // no anchor sees this token: it keeps its own state
    CD::unpack(x0r, x0f);
    if constexpr (MODE == kUniPC) m1r = x0r;
  } else {
    const Raw prevr = CD::load_stream(g.x0_prev, base);
    if constexpr (MODE == kUniPC) m1r = prevr;
    const int32_t* cw = g.corr + crow * g.a;
    int32_t words[GC_MAX_ANCHORS];
    if (g.a == 4) {   // the common layout: one 16-byte load (rows are 16-byte aligned)
      const int4 q = *reinterpret_cast<const int4*>(cw);
      words[0] = q.x;
      words[1] = q.y;
      words[2] = q.z;
      words[3] = q.w;
#pragma unroll
      for (int s = 4; s < GC_MAX_ANCHORS; ++s) words[s] = 0;
    } else {
#pragma unroll
      for (int s = 0; s < GC_MAX_ANCHORS; ++s) words[s] = s < g.a ? cw[s] : 0;
    }
    bool any = false;
#pragma unroll
    for (int s = 0; s < GC_MAX_ANCHORS; ++s) any |= words[s] != 0;
    if (!any) {
      x0r = prevr;
      CD::unpack(x0r, x0f);
    } else {
      float prevf[VEC], acc[VEC];
      CD::unpack(prevr, prevf);
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = 0.0f;
      const float* wr = g.weights + crow * g.a * g.K;
#pragma unroll
      for (int s = 0; s < GC_MAX_ANCHORS; ++s) {
        const uint32_t w = (uint32_t)words[s];
        if (!w) continue;
        const int x0 = (int)(w & 0xfffu) - 1;
        const int y0 = (int)((w >> 12) & 0xfffu) - 1;
        const uint32_t mask = (w >> 24) & 0xfu;
        const int64_t new_view = ((int64_t)b * g.a + s) * g.HW;
        const int64_t old_view = ((int64_t)b * g.N + g.anchor_view[s]) * g.HW;
        const float* ws = wr + s * g.K;
        int j = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          // words come from the caller: taps off the grid or beyond K are ignored
          const int x = x0 + (k & 1), y = y0 + (k >> 1);
          const bool on = (mask & (1u << k)) && j < g.K && x >= 0 && x < g.W && y >= 0 && y < g.H;
          if (!on) continue;
          const int q = y * g.W + x;
          const float wt = ws[j++];
          float nf[VEC], of[VEC];
          CD::unpack(CD::load(g.x0_new, (new_view + q) * g.C + (int64_t)cv * VEC), nf);
          CD::unpack(CD::load(g.x0_prev, (old_view + q) * g.C + (int64_t)cv * VEC), of);
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] = acc[e] + wt * (nf[e] - of[e]);
        }
      }
      float y[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) y[e] = prevf[e] + acc[e];
      x0r = CD::pack(y);
      CD::unpack(x0r, x0f);   // the reconstruction reads x0 as stored
    }
  }
  CD::store_stream(g.x0_out, base, x0r);
  if constexpr (MODE == kReconstruct) {
    float xtf[VEC], xn[VEC], mo[VEC];
    CD::unpack(xtr, xtf);
    reconstruct_vec<VEC>(g.r, xtf, x0f, xn, mo);
    CD::store_stream(g.x_next, base, CD::pack(xn));
    if (g.model_out) CD::store_stream(g.model_out, base, CD::pack(mo));
  }
  if constexpr (MODE == kUniPC) {
    float xin[VEC], m2[VEC], m1[VEC], xc[VEC], xn[VEC];
    CD::unpack(xtr, xin);
#pragma unroll
    for (int e = 0; e < VEC; ++e) m2[e] = m1[e] = 0.0f;
    if (g.u.need_m2) CD::unpack(m2r, m2);
    if (g.u.need_m1) CD::unpack(m1r, m1);
    unipc_vec<VEC>(g.u, xin, m2, m1, x0f, xc, xn);
    CD::store_stream(g.x_c, base, CD::pack(xc));
    CD::store_stream(g.x_next, base, CD::pack(xn));
  }
}

// Dense launch: blocks tile every (asset, view) in order.  Split launch (with
// a visible-token index): the first g.gblocks blocks each take a slice of the
// visible-token list and do all the gathering; the remaining blocks stream
// every other token, skipping the visible ones by their bit.  Gather blocks go
// first so that their dependent-load latency overlaps the streaming.
template <int DT, int VEC, int MODE, bool SPLIT>
__global__ __launch_bounds__(kBlock) void k_transport(TArgs g) {
  int i = blockIdx.x;
  if constexpr (SPLIT) {
    if (i < g.gblocks) {
      const int per = g.gblocks / kXcds;           // XCD-contiguous slices of the list
      const int lb = (i % kXcds) * per + i / kXcds;
      const int e = lb * kBlock + (int)threadIdx.x;
      if (e >= g.n_vis * g.CV) return;
      int le, cv;
      if (g.cv_shift >= 0) {
        le = e >> g.cv_shift;
        cv = e & (g.CV - 1);
      } else {
        le = e / g.CV;
        cv = e - le * g.CV;
      }
      const int tok = g.vis_list[le];
      if (tok < 0 || (int64_t)tok >= g.n_tokens) return;   // list entries come from the caller
      const int bt = tok / g.HW;
      const int p = tok - bt * g.HW;
      const int b = bt / g.NT;
      int v = bt - b * g.NT;                        // target slot -> view
#pragma unroll
      for (int s = 0; s < GC_MAX_ANCHORS; ++s) v += g.sorted_anchor[s] <= v ? 1 : 0;
      const int64_t base = (((int64_t)b * g.N + v) * g.HW + p) * g.C + (int64_t)cv * VEC;
      token_step<DT, VEC, MODE>(g, b, p, cv, -1, tok, base, kTargetSeen);
      return;
    }
    i -= g.gblocks;
  }
  // Blocks never straddle a view, so the (asset, view) split and the view's
  // role (anchor slot or target slot) are wave-uniform scalar values; only
  // the chunk -> (token, channel vector) split is per lane.
  // The split launch's streaming blocks gather nothing: they run in the
  // hardware's round-robin order over the XCDs (measured faster than one
  // contiguous slice per XCD); the dense launch keeps the slices.
  const int lb = logical_block(i, g.n_blocks, SPLIT ? 0 : g.remap);
  if (lb >= g.n_blocks) return;
  const int bv = __builtin_amdgcn_readfirstlane(lb / g.bpv);   // b * N + v
  const int t = (lb - bv * g.bpv) * kBlock + (int)threadIdx.x;
  if (t >= g.HW * g.CV) return;
  const int b = __builtin_amdgcn_readfirstlane(bv / g.N);
  const int v = bv - b * g.N;
  int s_self = -1, n_before = 0;
#pragma unroll
  for (int s = 0; s < GC_MAX_ANCHORS; ++s) {
    if (s < g.a) {
      const int u = g.anchor_view[s];
      s_self = u == v ? s : s_self;
      n_before += u < v;
    }
  }
  int p, cv;
  if (g.cv_shift >= 0) {
    p = t >> g.cv_shift;
    cv = t & (g.CV - 1);
  } else {
    p = t / g.CV;
    cv = t - p * g.CV;
  }
  const int64_t base = ((int64_t)bv * g.HW + p) * g.C + (int64_t)cv * VEC;
  if (s_self >= 0) {
    token_step<DT, VEC, MODE>(g, b, p, cv, s_self, 0, base, kAnchorRow);
    return;
  }
  const int64_t crow = ((int64_t)b * g.NT + (v - n_before)) * g.HW + p;
  if constexpr (SPLIT) {
    if ((g.vis_bits[crow >> 5] >> (crow & 31)) & 1u) return;   // a gather block owns this token
    token_step<DT, VEC, MODE>(g, b, p, cv, -1, crow, base, kTargetUnseen);
  } else {
    token_step<DT, VEC, MODE>(g, b, p, cv, -1, crow, base, kTargetCheck);
  }
}

template <int DT, int VEC>
__global__ __launch_bounds__(kBlock) void k_reconstruct(const void* __restrict__ x_t, const void* __restrict__ x0,
                                                        void* x_next, void* __restrict__ model_out, int64_t n_vec,
                                                        Recon r) {
  using CD = Codec<DT, VEC>;
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n_vec) return;
  float xtf[VEC], x0f[VEC], xn[VEC], mo[VEC];
  CD::unpack(CD::load_stream(x_t, i * VEC), xtf);
  CD::unpack(CD::load_stream(x0, i * VEC), x0f);
  reconstruct_vec<VEC>(r, xtf, x0f, xn, mo);
  CD::store_stream(x_next, i * VEC, CD::pack(xn));
  if (model_out) CD::store_stream(model_out, i * VEC, CD::pack(mo));
}

template <int DT, int VEC>
__global__ __launch_bounds__(kBlock) void k_unipc(TArgs g, const void* __restrict__ m_k, int64_t n_vec) {
  using CD = Codec<DT, VEC>;
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n_vec) return;
  float xin[VEC], m2[VEC], m1[VEC], mk[VEC], xc[VEC], xn[VEC];
  CD::unpack(CD::load_stream(g.u.corr ? g.x_prev : g.x_t, i * VEC), xin);
#pragma unroll
  for (int e = 0; e < VEC; ++e) m2[e] = m1[e] = 0.0f;
  if (g.u.need_m2) CD::unpack(CD::load_stream(g.m_km2, i * VEC), m2);
  if (g.u.need_m1) CD::unpack(CD::load_stream(g.x0_prev, i * VEC), m1);
  CD::unpack(CD::load_stream(m_k, i * VEC), mk);
  unipc_vec<VEC>(g.u, xin, m2, m1, mk, xc, xn);
  CD::store_stream(g.x_c, i * VEC, CD::pack(xc));
  CD::store_stream(g.x_next, i * VEC, CD::pack(xn));
}


// Validation shared by the transport entry points; fills g (except the
// reconstruction coefficients and the fused-only pointers).
int prepare_transport(const void* x0_prev, const void* x0_new, const int32_t* corr, const float* weights,
                      const uint32_t* vis_bits, const int32_t* vis_list, int64_t n_vis, int B, int N, int H, int W,
                      int C, const int32_t* anchors, int a, int K, int dtype, void* x0_out, const char* who,
                      TArgs* g) {
  if (!x0_prev || !x0_new || !anchors || !x0_out) return fail(GC_ERR_ARG, "%s: null pointer", who);
  if (dtype != GC_F32 && dtype != GC_BF16) return fail(GC_ERR_DTYPE, "%s: unknown dtype %d", who, dtype);
  if (B < 1 || N < 1 || H < 1 || W < 1 || C < 1)
    return fail(GC_ERR_SHAPE, "%s: bad shape B=%d N=%d H=%d W=%d C=%d", who, B, N, H, W, C);
  if (C % 4) return fail(GC_ERR_SHAPE, "%s: C=%d is not a multiple of 4", who, C);
  if (C > GC_MAX_CHANNELS) return fail(GC_ERR_CAPACITY, "%s: C=%d exceeds %d", who, C, GC_MAX_CHANNELS);
  if (N > GC_MAX_VIEWS) return fail(GC_ERR_CAPACITY, "%s: N=%d exceeds %d", who, N, GC_MAX_VIEWS);
  if (H > GC_MAX_GRID || W > GC_MAX_GRID) return fail(GC_ERR_CAPACITY, "%s: grid %dx%d exceeds %d", who, H, W, GC_MAX_GRID);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "%s: a=%d outside [1, N=%d]", who, a, N);
  if (a > GC_MAX_ANCHORS) return fail(GC_ERR_CAPACITY, "%s: a=%d exceeds %d", who, a, GC_MAX_ANCHORS);
  if (K < 1 || K > 4) return fail(GC_ERR_ARG, "%s: K=%d outside [1, 4]", who, K);
  const int NT = N - a;
  if (NT > 0 && (!corr || !weights)) return fail(GC_ERR_ARG, "%s: null correspondence", who);
  if (!aligned16(x0_prev) || !aligned16(x0_new) || !aligned16(x0_out) || (corr && !aligned16(corr)) ||
      (weights && !aligned16(weights)))
    return fail(GC_ERR_ALIGN, "%s: device pointers must be 16-byte aligned", who);
  std::memset(g, 0, sizeof(*g));
  bool is_anchor[GC_MAX_VIEWS] = {};
  for (int s = 0; s < a; ++s) {
    const int u = anchors[s];
    if (u < 0 || u >= N) return fail(GC_ERR_ARG, "%s: anchor %d outside [0, %d)", who, u, N);
    if (is_anchor[u]) return fail(GC_ERR_ARG, "%s: anchor %d listed twice", who, u);
    is_anchor[u] = true;
    g->anchor_view[s] = u;
  }
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t HW = (size_t)H * W;
  const size_t n_all = (size_t)B * N * HW * C * es, n_new = (size_t)B * a * HW * C * es;
  if (overlaps(x0_out, n_all, x0_prev, n_all) || overlaps(x0_out, n_all, x0_new, n_new))
    return fail(GC_ERR_ALIAS, "%s: x0_out overlaps x0_prev or x0_anchor_new", who);
  const int vec = pick_vec(dtype, C);
  g->x0_prev = x0_prev;
  g->x0_new = x0_new;
  g->corr = corr;
  g->weights = weights;
  g->x0_out = x0_out;
  g->N = N;
  g->H = H;
  g->HW = (int)HW;
  g->W = W;
  g->C = C;
  g->a = a;
  g->K = K;
  g->NT = NT;
  g->CV = C / vec;
  g->cv_shift = -1;
  for (int sh = 0; sh < 8; ++sh)
    if ((1 << sh) == g->CV) g->cv_shift = sh;
  g->n_threads = (int64_t)B * N * (int64_t)HW * g->CV;
  g->bpv = (int)(((int64_t)HW * g->CV + kBlock - 1) / kBlock);
  const int64_t nb = (int64_t)B * N * g->bpv;
  if (nb > (int64_t)0x7fffffff - kXcds) return fail(GC_ERR_CAPACITY, "%s: problem too large for one launch", who);
  g->n_blocks = (int)nb;
  g->remap = 1;
  // optional visible-token index
  if ((vis_bits == nullptr) != (vis_list == nullptr))
    return fail(GC_ERR_ARG, "%s: vis_bits and vis_list must both be given or both be null", who);
  g->n_tokens = (int64_t)B * NT * (int64_t)HW;
  if (vis_bits) {
    if (g->n_tokens > 0x7fffffffLL) return fail(GC_ERR_CAPACITY, "%s: too many target tokens for an index", who);
    if (n_vis < 0 || n_vis > g->n_tokens)
      return fail(GC_ERR_ARG, "%s: n_vis=%lld outside [0, %lld]", who, (long long)n_vis, (long long)g->n_tokens);
    if (!aligned16(vis_bits) || !aligned16(vis_list)) return fail(GC_ERR_ALIGN, "%s: index pointers must be 16-byte aligned", who);
    if (overlaps(x0_out, n_all, vis_bits, (size_t)(g->n_tokens + 31) / 32 * 4) ||
        overlaps(x0_out, n_all, vis_list, (size_t)n_vis * 4))
      return fail(GC_ERR_ALIAS, "%s: x0_out overlaps the index", who);
    g->vis_bits = vis_bits;
    g->vis_list = vis_list;
    g->n_vis = (int)n_vis;
    const int64_t gb = ((int64_t)n_vis * g->CV + kBlock - 1) / kBlock;
    const int64_t gblocks = (gb + kXcds - 1) / kXcds * kXcds;
    // a gather lane's item index (block * kBlock + lane) is a 32-bit int
    if (gblocks * kBlock > (int64_t)0x7fffffff)
      return fail(GC_ERR_CAPACITY, "%s: n_vis=%lld times %d channel vectors exceeds the gather part's 2^31 lanes", who,
                  (long long)n_vis, g->CV);
    g->gblocks = (int)gblocks;
    if ((int64_t)g->gblocks + nb > (int64_t)0x7fffffff - kXcds)
      return fail(GC_ERR_CAPACITY, "%s: problem too large for one launch", who);
    // a small step takes the dense launch: the list's extra dependent load
    // does not pay there (checked above all the same; same result bit for bit)
    if (g->n_tokens * g->CV < split_min_items()) {
      g->vis_bits = nullptr;
      g->vis_list = nullptr;
      g->n_vis = 0;
      g->gblocks = 0;
    }
  }
  int sorted[GC_MAX_ANCHORS];
  for (int s = 0; s < a; ++s) sorted[s] = anchors[s];
  for (int s = 1; s < a; ++s)
    for (int r = s; r > 0 && sorted[r - 1] > sorted[r]; --r) {
      const int tmp = sorted[r];
      sorted[r] = sorted[r - 1];
      sorted[r - 1] = tmp;
    }
  for (int s = 0; s < GC_MAX_ANCHORS; ++s) g->sorted_anchor[s] = s < a ? sorted[s] : 0x7fffffff;
  return GC_OK;
}

template <int MODE>
void launch_transport(const TArgs& g, int dtype, hipStream_t stream) {
  const int per = (g.n_blocks + kXcds - 1) / kXcds;
  const unsigned stream_blocks = g.remap ? (unsigned)(per * kXcds) : (unsigned)g.n_blocks;
  const bool split = g.vis_bits != nullptr;
  const dim3 grid(stream_blocks + (split ? (unsigned)g.gblocks : 0u));
  const int vec = g.C / g.CV;
#define GC_LAUNCH(DT_, VEC_)                                                                       \
  do {                                                                                             \
    if (split)                                                                                     \
      hipLaunchKernelGGL((k_transport<DT_, VEC_, MODE, true>), grid, dim3(kBlock), 0, stream, g);  \
    else                                                                                           \
      hipLaunchKernelGGL((k_transport<DT_, VEC_, MODE, false>), grid, dim3(kBlock), 0, stream, g); \
  } while (0)
  if (dtype == GC_F32)
    GC_LAUNCH(GC_F32, 4);
  else if (vec == 8)
    GC_LAUNCH(GC_BF16, 8);
  else
    GC_LAUNCH(GC_BF16, 4);
#undef GC_LAUNCH
}

// Validate UniPC coefficients / buffers and load them into g.
int prepare_unipc(const gc_unipc_step* st, const void* x_cur, const void* x_prev, const void* m_km2,
                  const void* m_km1, const char* who, TArgs* g) {
  if (!st) return fail(GC_ERR_ARG, "%s: null coefficients", who);
  g->u = make_unicoef(*st);
  if (g->u.corr && !x_prev) return fail(GC_ERR_ARG, "%s: the corrector needs x_prev", who);
  if (!g->u.corr && !x_cur) return fail(GC_ERR_ARG, "%s: without the corrector x_cur is needed", who);
  if (g->u.need_m2 && !m_km2) return fail(GC_ERR_ARG, "%s: the coefficients need m_{k-2}", who);
  if (g->u.need_m1 && !m_km1) return fail(GC_ERR_ARG, "%s: the coefficients need m_{k-1}", who);
  const void* ins[4] = {x_cur, x_prev, m_km2, m_km1};
  for (const void* q : ins)
    if (q && !aligned16(q)) return fail(GC_ERR_ALIGN, "%s: device pointers must be 16-byte aligned", who);
  g->x_t = x_cur;
  g->x_prev = x_prev;
  g->m_km2 = m_km2;
  return GC_OK;
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" int gc_transport_step(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr,
                                 const float* weights, const uint32_t* vis_bits, const int32_t* vis_list,
                                 int64_t n_vis, int B, int N, int H, int W, int C, const int32_t* anchors, int a,
                                 int K, int dtype, void* x0_out, hipStream_t stream) {
  clear_error();
  TArgs g;
  int rc = prepare_transport(x0_prev, x0_anchor_new, corr, weights, vis_bits, vis_list, n_vis, B, N, H, W, C,
                             anchors, a, K, dtype, x0_out, "gc_transport_step", &g);
  if (rc) return rc;
  if (g.n_threads == 0) return GC_OK;
  launch_transport<kTransportOnly>(g, dtype, stream);
  return after_launch(stream, "gc_transport_step");
}

extern "C" int gc_sampler_reconstruct(const void* x_t, const void* x0, void* x_next, void* model_out,
                                      int64_t n_elems, int dtype, const gc_sampler* smp, double t, double t_next,
                                      hipStream_t stream) {
  clear_error();
  if (!x_t || !x0 || !x_next) return fail(GC_ERR_ARG, "gc_sampler_reconstruct: null pointer");
  if (dtype != GC_F32 && dtype != GC_BF16) return fail(GC_ERR_DTYPE, "gc_sampler_reconstruct: unknown dtype %d", dtype);
  if (n_elems < 0 || n_elems % 4) return fail(GC_ERR_SHAPE, "gc_sampler_reconstruct: n_elems=%lld must be a non-negative multiple of 4",
                                              (long long)n_elems);
  Recon r;
  int rc = make_recon(smp, t, t_next, &r);
  if (rc) return rc;
  if ((r.pred != GC_PRED_NONE) != (model_out != nullptr))
    return fail(GC_ERR_ARG, "gc_sampler_reconstruct: model_out must be given iff pred_out != GC_PRED_NONE");
  if (!aligned16(x_t) || !aligned16(x0) || !aligned16(x_next) || (model_out && !aligned16(model_out)))
    return fail(GC_ERR_ALIGN, "gc_sampler_reconstruct: device pointers must be 16-byte aligned");
  const size_t nb = (size_t)n_elems * dtype_bytes(dtype);
  if ((x_next != x_t && overlaps(x_next, nb, x_t, nb)) || overlaps(x_next, nb, x0, nb) ||
      overlaps(model_out, nb, x_t, nb) || overlaps(model_out, nb, x0, nb) || overlaps(model_out, nb, x_next, nb))
    return fail(GC_ERR_ALIAS, "gc_sampler_reconstruct: outputs overlap inputs (only x_next == x_t is allowed)");
  if (n_elems == 0) return GC_OK;
  const int vec = pick_vec(dtype, n_elems);
  const int64_t n_vec = n_elems / vec;
  const int64_t blocks = (n_vec + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return fail(GC_ERR_CAPACITY, "gc_sampler_reconstruct: too many elements");
  if (dtype == GC_F32)
    hipLaunchKernelGGL((k_reconstruct<GC_F32, 4>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, x_t, x0, x_next,
                       model_out, n_vec, r);
  else if (vec == 8)
    hipLaunchKernelGGL((k_reconstruct<GC_BF16, 8>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, x_t, x0, x_next,
                       model_out, n_vec, r);
  else
    hipLaunchKernelGGL((k_reconstruct<GC_BF16, 4>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, x_t, x0, x_next,
                       model_out, n_vec, r);
  return after_launch(stream, "gc_sampler_reconstruct");
}

extern "C" int gc_transport_reconstruct(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr,
                                        const float* weights, const uint32_t* vis_bits, const int32_t* vis_list,
                                        int64_t n_vis, const void* x_t, int B, int N, int H, int W, int C,
                                        const int32_t* anchors, int a, int K, int dtype, const gc_sampler* smp,
                                        double t, double t_next, void* x0_out, void* x_next, void* model_out,
                                        hipStream_t stream) {
  clear_error();
  TArgs g;
  int rc = prepare_transport(x0_prev, x0_anchor_new, corr, weights, vis_bits, vis_list, n_vis, B, N, H, W, C,
                             anchors, a, K, dtype, x0_out, "gc_transport_reconstruct", &g);
  if (rc) return rc;
  if (!x_t || !x_next) return fail(GC_ERR_ARG, "gc_transport_reconstruct: null x_t or x_next");
  rc = make_recon(smp, t, t_next, &g.r);
  if (rc) return rc;
  if ((g.r.pred != GC_PRED_NONE) != (model_out != nullptr))
    return fail(GC_ERR_ARG, "gc_transport_reconstruct: model_out must be given iff pred_out != GC_PRED_NONE");
  if (!aligned16(x_t) || !aligned16(x_next) || (model_out && !aligned16(model_out)))
    return fail(GC_ERR_ALIGN, "gc_transport_reconstruct: device pointers must be 16-byte aligned");
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t n_all = (size_t)B * N * H * W * C * es, n_new = (size_t)B * a * H * W * C * es;
  const void* ins[3] = {x0_prev, x0_anchor_new, x0_out};
  const size_t lens[3] = {n_all, n_new, n_all};
  for (int i = 0; i < 3; ++i) {
    if (overlaps(x_next, n_all, ins[i], lens[i]) || overlaps(model_out, n_all, ins[i], lens[i]))
      return fail(GC_ERR_ALIAS, "gc_transport_reconstruct: x_next/model_out overlap x0_prev, x0_anchor_new or x0_out");
  }
  if (overlaps(x_t, n_all, x0_out, n_all) || (x_next != x_t && overlaps(x_next, n_all, x_t, n_all)) ||
      overlaps(model_out, n_all, x_t, n_all) || overlaps(model_out, n_all, x_next, n_all))
    return fail(GC_ERR_ALIAS, "gc_transport_reconstruct: outputs overlap x_t (only x_next == x_t is allowed)");
  g.x_t = x_t;
  g.x_next = x_next;
  g.model_out = model_out;
  if (g.n_threads == 0) return GC_OK;
  launch_transport<kReconstruct>(g, dtype, stream);
  return after_launch(stream, "gc_transport_reconstruct");
}

extern "C" int gc_unipc_update(const void* x_cur, const void* x_prev, const void* m_km2, const void* m_km1,
                               const void* m_k, int64_t n_elems, int dtype, const gc_unipc_step* st, void* x_c,
                               void* x_next, hipStream_t stream) {
  clear_error();
  if (!m_k || !x_c || !x_next) return fail(GC_ERR_ARG, "gc_unipc_update: null pointer");
  if (dtype != GC_F32 && dtype != GC_BF16) return fail(GC_ERR_DTYPE, "gc_unipc_update: unknown dtype %d", dtype);
  if (n_elems < 0 || n_elems % 4)
    return fail(GC_ERR_SHAPE, "gc_unipc_update: n_elems=%lld must be a non-negative multiple of 4", (long long)n_elems);
  TArgs g;
  std::memset(&g, 0, sizeof(g));
  const size_t nb = (size_t)n_elems * dtype_bytes(dtype);
  int rc = prepare_unipc(st, x_cur, x_prev, m_km2, m_km1, "gc_unipc_update", &g);
  if (rc) return rc;
  g.x0_prev = m_km1;
  g.x_c = x_c;
  g.x_next = x_next;
  if (!aligned16(m_k) || !aligned16(x_c) || !aligned16(x_next))
    return fail(GC_ERR_ALIGN, "gc_unipc_update: device pointers must be 16-byte aligned");
  const void* ins[5] = {x_cur, x_prev, m_km2, m_km1, m_k};
  for (int i = 0; i < 5; ++i) {
    if (!ins[i]) continue;
    if ((ins[i] != x_cur && overlaps(x_next, nb, ins[i], nb)) || (ins[i] != x_prev && overlaps(x_c, nb, ins[i], nb)))
      return fail(GC_ERR_ALIAS, "gc_unipc_update: outputs overlap inputs (only x_c == x_prev, x_next == x_cur)");
  }
  if (overlaps(x_c, nb, x_next, nb)) return fail(GC_ERR_ALIAS, "gc_unipc_update: x_c overlaps x_next");
  if (n_elems == 0) return GC_OK;
  const int vec = pick_vec(dtype, n_elems);
  const int64_t n_vec = n_elems / vec;
  const int64_t blocks = (n_vec + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return fail(GC_ERR_CAPACITY, "gc_unipc_update: too many elements");
  if (dtype == GC_F32)
    hipLaunchKernelGGL((k_unipc<GC_F32, 4>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, g, m_k, n_vec);
  else if (vec == 8)
    hipLaunchKernelGGL((k_unipc<GC_BF16, 8>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, g, m_k, n_vec);
  else
    hipLaunchKernelGGL((k_unipc<GC_BF16, 4>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, g, m_k, n_vec);
  return after_launch(stream, "gc_unipc_update");
}

extern "C" int gc_transport_unipc(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr,
                                  const float* weights, const uint32_t* vis_bits, const int32_t* vis_list,
                                  int64_t n_vis, const void* x_cur, const void* x_prev, const void* m_km2, int B,
                                  int N, int H, int W, int C, const int32_t* anchors, int a, int K, int dtype,
                                  const gc_unipc_step* st, void* x0_out, void* x_c, void* x_next,
                                  hipStream_t stream) {
  clear_error();
  TArgs g;
  int rc = prepare_transport(x0_prev, x0_anchor_new, corr, weights, vis_bits, vis_list, n_vis, B, N, H, W, C,
                             anchors, a, K, dtype, x0_out, "gc_transport_unipc", &g);
  if (rc) return rc;
  if (!x_c || !x_next) return fail(GC_ERR_ARG, "gc_transport_unipc: null x_c or x_next");
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t n_all = (size_t)B * N * H * W * C * es, n_new = (size_t)B * a * H * W * C * es;
  rc = prepare_unipc(st, x_cur, x_prev, m_km2, x0_prev, "gc_transport_unipc", &g);
  if (rc) return rc;
  if (!aligned16(x_c) || !aligned16(x_next)) return fail(GC_ERR_ALIGN, "gc_transport_unipc: outputs must be 16-byte aligned");
  const void* ins[5] = {x0_prev, x0_anchor_new, x_cur, x_prev, m_km2};
  const size_t lens[5] = {n_all, n_new, n_all, n_all, n_all};
  for (int i = 0; i < 5; ++i) {
    if (!ins[i]) continue;
    if ((ins[i] != x_cur && overlaps(x_next, n_all, ins[i], lens[i])) ||
        (ins[i] != x_prev && overlaps(x_c, n_all, ins[i], lens[i])) || overlaps(x0_out, n_all, ins[i], lens[i]))
      return fail(GC_ERR_ALIAS, "gc_transport_unipc: outputs overlap inputs (only x_c == x_prev, x_next == x_cur)");
  }
  if (overlaps(x_c, n_all, x_next, n_all) || overlaps(x_c, n_all, x0_out, n_all) || overlaps(x_next, n_all, x0_out, n_all))
    return fail(GC_ERR_ALIAS, "gc_transport_unipc: outputs overlap each other");
  g.x_c = x_c;
  g.x_next = x_next;
  if (g.n_threads == 0) return GC_OK;
  launch_transport<kUniPC>(g, dtype, stream);
  return after_launch(stream, "gc_transport_unipc");
}
