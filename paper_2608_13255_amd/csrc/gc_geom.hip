// Cached step with the correspondence computed on the fly: Eq. 1 (and then
// the sampler reconstruction or the UniPC update) reading the position maps
// and cameras directly instead of a stored G_{A->v}.  The operator is a function of the position
// maps and cameras only (Sec. 3.2, correspondence operator), so it can be
// rebuilt inside the step from 12 bytes of position per target token plus
// the anchors' position taps; nothing has to be built or stored per anchor
// set.  That pays when anchor sets do not repeat (e.g. chosen adaptively);
// with the rotation's few repeating sets the stored operator and its
// visible-token index are cheaper per step.
//
// Work mapping: in a target-view block a group of G adjacent lanes serves
// one target token, G the number of channel vectors rounded up to a power of
// two (at most 8).  Lane j of the group evaluates anchor slots j, j + G, ...
// exactly as the builder does (same device function, same float order), and
// n_vis is a ballot over the group.  The block then ranks its tokens, the
// visible ones (some anchor sees them) first and the others after them,
// keeps the visible tokens' words and weights in LDS, and hands out one
// (token, channel vector) item per lane in that order: the gathers fill
// whole waves while the other waves only stream, as in the stored-operator
// split launch.  A visible item blends its anchors in ascending slot order
// with the builder's stored weights (w_k / n_vis in float), so the result
// equals gc_build_correspondence followed by gc_transport_step (or the fused
// reconstruction / UniPC calls) bit for bit.
//
// Blocked launch (no foreground index): the target-view blocks, whose
// dependent loads (position, the anchors' position taps, then the latent
// taps) set the pace, come first; the anchor rows, which only copy the new
// prediction and stream the sampler step, follow as dense blocks of one lane
// per channel vector and fill the machine while the last target blocks
// finish.  Each part is dealt to the XCDs in contiguous slices, so an XCD
// gathers from few assets' anchor views, and blocks never straddle a view.
//
// Foreground launch (with gc_index_foreground's index of the position
// maps): only a token with a finite position can be seen by an anchor, so
// the geometry runs in blocks over the compact list of foreground tokens,
// whose records carry each token's position (one 16-byte load gives a lane
// both), while every other token -- the background of the target views and
// all of the anchor rows -- is streamed by blocks in the hardware's
// round-robin order that skip the listed target tokens by their bit.  The
// list covers all views; a record of an anchor view is skipped.  A block of
// the list may straddle views and assets, so it stages the cameras of every
// (asset, anchor slot) in LDS (B * a <= kMaxCamLds; beyond that the blocked
// launch runs, with the same result).  Its tokens are all foreground and
// mostly visible, so it does without the blocked launch's ranking: each lane
// serves its own token's channel vectors.
#include "gc_common.h"
#include "gc_geometry.h"
#include "gc_latent.h"

namespace gc {
namespace {

constexpr int kBlock = 256;
static_assert(GC_MAX_VIEWS <= 256 && GC_MAX_ANCHORS <= 8, "view_bytes holds one byte per anchor slot");

// What a step does after the transport: nothing, the sampler reconstruction,
// or the UniPC corrector + predictor on the x0 history.
enum GeomMode { kGeomTransport = 0, kGeomReconstruct = 1, kGeomUniPC = 2 };

struct GArgs {
  const void* x0_prev;
  const void* x0_new;
  const float* pos;
  const gc_camera* cams;
  const float* bbox;
  const void* x_t;
  void* x0_out;
  void* x_next;
  void* model_out;
  int N, H, W, HW, C, a, K, CV, NT;
  int G;            // lanes per target token (geom_group)
  int cv_shift;     // log2(CV) when CV is a power of two, else -1
  int bpv_t;        // target blocks per target view: ceil(HW / tokens per block)
  int n_tblocks;    // B * NT * bpv_t
  int tgrid;        // target part of the grid, padded to a multiple of kXcds
  int bpv_a;        // anchor-row blocks per anchor view: ceil(HW * CV / kBlock)
  int n_ablocks;    // B * a * bpv_a
  int32_t anchor_view[GC_MAX_ANCHORS];     // view of anchor slot s
  int32_t sorted_anchor[GC_MAX_ANCHORS];   // anchor views ascending, padded with INT_MAX
  uint64_t view_bytes;                     // byte s: view of anchor slot s
  Recon r;
  // UniPC mode: x_t is x_cur; x_prev / m_km2 inputs, x_c output
  const void* x_prev;
  const void* m_km2;
  void* x_c;
  UniCoef u;
  // foreground launch
  const uint32_t* fg_bits;   // bit per token of [B][N][H][W]: finite position
  const int4* fg_recs;       // [n_fg] {token, x, y, z}, in the index's tile order
  int n_fg;
  int B;
  int gblocks;               // list blocks in front of the streaming blocks (multiple of kXcds)
  int bpv_s;                 // streaming blocks per view: ceil(HW * CV / kBlock)
  int n_sblocks;             // B * N * bpv_s
};

constexpr int kMaxCamLds = 64;   // (asset, anchor slot) cameras a list block can stage

// An item's own inputs besides its x0_prev: x_t for the reconstruction; for
// UniPC x_prev (corrector) or x_cur, m_{k-2}, and m_{k-1} (an anchor row
// loads its x0_prev here; a target token's is the x0_prev it reads anyway).
template <int DT, int VEC> struct Side {
  typename Codec<DT, VEC>::Raw xin, m2, m1;
};

template <int DT, int VEC, int MODE>
__device__ __forceinline__ Side<DT, VEC> load_side(const GArgs& g, int64_t e, bool anchor_row) {
  using CD = Codec<DT, VEC>;
  Side<DT, VEC> sd{};
  if constexpr (MODE == kGeomReconstruct) sd.xin = CD::load_stream(g.x_t, e);
  if constexpr (MODE == kGeomUniPC) {
    sd.xin = CD::load_stream(g.u.corr ? g.x_prev : g.x_t, e);
    if (g.u.need_m2) sd.m2 = CD::load_stream(g.m_km2, e);
    // an anchor row's own x0_prev is also gathered by the target tokens that
    // see it: a cached load (measured faster than a nontemporal one)
    if (anchor_row && g.u.need_m1) sd.m1 = CD::load(g.x0_prev, e);
  }
  return sd;
}

// Stores a token's channel vector: x0 as given, then (reconstruction) the
// sampler step from x_t and that x0 as stored, or (UniPC) the corrector and
// predictor with m_k = that x0 as stored.
template <int DT, int VEC, int MODE>
__device__ __forceinline__ void finish_item(const GArgs& g, int64_t e, const typename Codec<DT, VEC>::Raw& x0r,
                                            const Side<DT, VEC>& sd) {
  using CD = Codec<DT, VEC>;
  CD::store_stream(g.x0_out, e, x0r);
  if constexpr (MODE == kGeomReconstruct) {
    float xtf[VEC], x0f[VEC], xn[VEC], mo[VEC];
    CD::unpack(x0r, x0f);   // the reconstruction reads x0 as stored
    CD::unpack(sd.xin, xtf);
    reconstruct_vec<VEC>(g.r, xtf, x0f, xn, mo);
    CD::store_stream(g.x_next, e, CD::pack(xn));
    if (g.model_out) CD::store_stream(g.model_out, e, CD::pack(mo));
  }
  if constexpr (MODE == kGeomUniPC) {
    float xin[VEC], m2[VEC], m1[VEC], mk[VEC], xc[VEC], xn[VEC];
    CD::unpack(sd.xin, xin);
    CD::unpack(x0r, mk);
#pragma unroll
    for (int q = 0; q < VEC; ++q) m2[q] = m1[q] = 0.0f;
    if (g.u.need_m2) CD::unpack(sd.m2, m2);
    if (g.u.need_m1) CD::unpack(sd.m1, m1);
    unipc_vec<VEC>(g.u, xin, m2, m1, mk, xc, xn);
    CD::store_stream(g.x_c, e, CD::pack(xc));
    CD::store_stream(g.x_next, e, CD::pack(xn));
  }
}

// Eq. 1's sum for one (token, channel vector c) of asset b: the anchors'
// (new - previous) x0 at the kept taps of each slot's word, in ascending slot
// and tap order, each weighted by the builder's stored weight w_k / n_vis
// (words and w_k as the selection left them in LDS).  A slot's taps lie 0,
// 1, W and W + 1 tokens from its footprint's top-left tap, so only that tap's
// address is computed per slot; dividing by a power-of-two n_vis is
// multiplying by its exact reciprocal.
template <int DT, int VEC>
__device__ __forceinline__ void gather_delta(const GArgs& g, int b, int c, const int32_t* words, const float* wk,
                                             int n_vis, float (&acc)[VEC]) {
  using CD = Codec<DT, VEC>;
  using Raw = typename CD::Raw;
  constexpr int kEs = DT == GC_F32 ? 4 : 2;
  const float inv = (float)n_vis;
  const bool pow2 = (n_vis & (n_vis - 1)) == 0;
  const float rcp = __builtin_ldexpf(1.0f, -__builtin_ctz((unsigned)n_vis));
  const int64_t tb = (int64_t)g.C * kEs;   // bytes per token
  const int64_t dk[4] = {0, tb, (int64_t)g.W * tb, (int64_t)(g.W + 1) * tb};
  const char* nb = static_cast<const char*>(g.x0_new) + (int64_t)c * VEC * kEs;
  const char* ob = static_cast<const char*>(g.x0_prev) + (int64_t)c * VEC * kEs;
#pragma unroll
  for (int q = 0; q < VEC; ++q) acc[q] = 0.0f;
  for (int s = 0; s < g.a; ++s) {
    const uint32_t w = (uint32_t)words[s];
    if (!w) continue;
    const int x0 = (int)(w & 0xfffu) - 1;
    const int y0 = (int)((w >> 12) & 0xfffu) - 1;
    const uint32_t mask = (w >> 24) & 0xfu;
    const int64_t pix = (int64_t)y0 * g.W + x0;   // may lie off the grid; only kept taps are read
    const char* pn = nb + (((int64_t)b * g.a + s) * g.HW + pix) * tb;
    const char* po = ob + (((int64_t)b * g.N + g.anchor_view[s]) * g.HW + pix) * tb;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (!(mask & (1u << k))) continue;
      const Raw nr = CD::load(pn + dk[k], 0);
      const Raw orr = CD::load(po + dk[k], 0);
      const float wt = pow2 ? wk[s * 4 + k] * rcp : wk[s * 4 + k] / inv;
      float nf[VEC], of[VEC];
      CD::unpack(nr, nf);
      CD::unpack(orr, of);
#pragma unroll
      for (int q = 0; q < VEC; ++q) acc[q] = acc[q] + wt * (nf[q] - of[q]);
    }
  }
}

// G lanes per target token; AMAX (4 or 8) bounds the anchor count, so each
// lane evaluates up to AMAX / G anchor slots.
template <int DT, int VEC, int MODE, int G, int AMAX>
__global__ __launch_bounds__(kBlock) void k_transport_geom(GArgs g) {
  using CD = Codec<DT, VEC>;
  using Raw = typename CD::Raw;
  constexpr int kTok = kBlock / G;   // target tokens per block
  constexpr int kApl = AMAX / G;     // anchor slots per lane
  static_assert(kApl >= 1 && kApl * G == AMAX, "G must divide AMAX");
  __shared__ gc_camera cam_lds[GC_MAX_ANCHORS];
  if ((int)blockIdx.x >= g.tgrid) {
    // anchor row: one lane per (token, channel vector); the store takes the
    // new prediction
    const int lb = logical_block((int)blockIdx.x - g.tgrid, g.n_ablocks, 1);
    if (lb >= g.n_ablocks) return;
    const int bs = __builtin_amdgcn_readfirstlane(lb / g.bpv_a);   // b * a + s
    const int b = __builtin_amdgcn_readfirstlane(bs / g.a);
    const int s = bs - b * g.a;
    const int t = (lb - bs * g.bpv_a) * kBlock + (int)threadIdx.x;
    if (t >= g.HW * g.CV) return;
    int p, c;
    if (g.cv_shift >= 0) {
      p = t >> g.cv_shift;
      c = t & (g.CV - 1);
    } else {
      p = t / g.CV;
      c = t - p * g.CV;
    }
    const int64_t e = (((int64_t)b * g.N + g.anchor_view[s]) * g.HW + p) * g.C + (int64_t)c * VEC;
    const Side<DT, VEC> sd = load_side<DT, VEC, MODE>(g, e, true);
    const Raw x0r = CD::load(g.x0_new, ((int64_t)bs * g.HW + p) * g.C + (int64_t)c * VEC);
    finish_item<DT, VEC, MODE>(g, e, x0r, sd);
    return;
  }
  const int lb = logical_block((int)blockIdx.x, g.n_tblocks, 1);
  if (lb >= g.n_tblocks) return;   // XCD padding: whole block
  const int bt = __builtin_amdgcn_readfirstlane(lb / g.bpv_t);   // b * NT + target slot
  const int b = __builtin_amdgcn_readfirstlane(bt / g.NT);
  int v = bt - b * g.NT;                                          // target slot -> view
#pragma unroll
  for (int s = 0; s < GC_MAX_ANCHORS; ++s) v += g.sorted_anchor[s] <= v ? 1 : 0;
  const int bv = b * g.N + v;
  const int lane_g = (int)threadIdx.x & (G - 1);
  const int p = (lb - bt * g.bpv_t) * kTok + (int)threadIdx.x / G;
  const bool tok_ok = p < g.HW;

  // the token's position is loaded first, so its latency overlaps the
  // camera setup and its barrier
  float P[3] = {0.f, 0.f, 0.f};
  if (tok_ok) {
    const float* pp = g.pos + ((int64_t)bv * g.HW + p) * 3;
    P[0] = pp[0];
    P[1] = pp[1];
    P[2] = pp[2];
  }
  // target token: lane j of the group evaluates anchor slots j, j + G, ...
  __shared__ int32_t view_lds[GC_MAX_ANCHORS];   // anchor views in LDS: a per-lane index into the kernel
                                                  // arguments would be a memory load ordered after the taps
  if (threadIdx.x < g.a) {
    // the slot's view by a shift of a scalar argument: indexing anchor_view
    // per lane would be a memory load in front of the camera load
    const int u = (int)((g.view_bytes >> (8 * threadIdx.x)) & 0xffu);
    view_lds[threadIdx.x] = u;
    cam_lds[threadIdx.x] = g.cams[(int64_t)b * g.N + u];
  }
  __syncthreads();
  const bool fg = tok_ok && finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2]);
  // all of the lane's slots are projected first and all their tap loads are
  // issued together (a lane without a slot, or a background token, loads the
  // grid's corner taps of slot 0's map and ignores them); a wave in which no
  // projection succeeded (all background, mostly) skips the loads
  AnchorProj pj[kApl];
  AnchorTaps at[kApl];
  bool any_ok = false;
  if (__ballot(fg)) {   // a wave of background tokens projects nothing
#pragma unroll
    for (int j = 0; j < kApl; ++j) {   // branch-free: a lane without the slot keeps the result unused
      const int s = j * G + lane_g;
      pj[j] = anchor_project(P, cam_lds[s < g.a ? s : 0], g.H, g.W);
      pj[j].ok = pj[j].ok && tok_ok && fg && s < g.a;
      any_ok = any_ok || pj[j].ok;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kApl; ++j) pj[j] = AnchorProj{false, 0, 0, 0.0f, 0.0f};
  }
  if (__ballot(any_ok)) {
    TapPos tp[kApl];
#pragma unroll
    for (int j = 0; j < kApl; ++j) {
      const int s = j * G + lane_g;
      const int sc = s < g.a ? s : 0;
      tp[j] = anchor_tap_positions(pj[j], g.pos + ((int64_t)b * g.N + view_lds[sc]) * g.HW * 3, g.H, g.W);
    }
    const float tol2 = g.bbox[(int64_t)b * 8 + 6];
#pragma unroll
    for (int j = 0; j < kApl; ++j) at[j] = anchor_select(P, pj[j], tp[j], g.H, g.W, g.K, tol2);
  } else {
#pragma unroll
    for (int j = 0; j < kApl; ++j) {
      at[j].word = 0;
      at[j].mask = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) at[j].wk[k] = 0.0f;
    }
  }
  // n_vis: a ballot over the group (every lane reaches the ballots)
  const int gbase = __lane_id() & ~(G - 1);
  int n_vis = 0;
#pragma unroll
  for (int j = 0; j < kApl; ++j) n_vis += __popcll((__ballot(at[j].word != 0) >> gbase) & ((1ull << G) - 1));

  // Compaction: the block's visible tokens first (ascending), then the other
  // tokens (ascending); the visible tokens' words and weights go to LDS.  The
  // latent phase gives each lane one (token, channel vector) item in that
  // order, so the gathering and the streaming fall into separate waves.
  __shared__ int32_t s_tok[kTok];
  __shared__ int32_t s_nvis[kTok];
  __shared__ int32_t s_word[kTok][AMAX + 1];       // +1: no bank conflicts between consecutive tokens
  __shared__ float s_wk[kTok][AMAX * 4 + 1];
  __shared__ int32_t s_count[kBlock / 64][2];      // per wave: visible tokens, live tokens
  const bool vis = tok_ok && n_vis > 0;
  const bool lead = lane_g == 0;
  const unsigned long long bvis = __ballot(lead && vis);
  const unsigned long long blive = __ballot(lead && tok_ok);
  const int wv = (int)threadIdx.x / 64;
  if (__lane_id() == 0) {
    s_count[wv][0] = __popcll(bvis);
    s_count[wv][1] = __popcll(blive);
  }
  __syncthreads();
  int off_v = 0, off_l = 0, nv = 0, nl = 0;
#pragma unroll
  for (int q = 0; q < kBlock / 64; ++q) {
    const int cv_ = s_count[q][0], cl_ = s_count[q][1];
    off_v += q < wv ? cv_ : 0;
    off_l += q < wv ? cl_ : 0;
    nv += cv_;
    nl += cl_;
  }
  if (tok_ok) {
    const unsigned long long below = (1ull << gbase) - 1;   // the groups before this one in the wave
    const int rv = off_v + __popcll(bvis & below);
    const int rl = off_l + __popcll(blive & below);
    if (lead) s_tok[vis ? rv : nv + (rl - rv)] = p;
    if (vis) {
#pragma unroll
      for (int j = 0; j < kApl; ++j) {
        const int s = j * G + lane_g;
        if (s < g.a) {
          s_word[rv][s] = at[j].word;
#pragma unroll
          for (int k = 0; k < 4; ++k) s_wk[rv][s * 4 + k] = at[j].wk[k];
        }
      }
      if (lead) s_nvis[rv] = n_vis;
    }
  }
  __syncthreads();

  const int n_items = nl * g.CV;
  for (int it = (int)threadIdx.x; it < n_items; it += kBlock) {
    int slot, c;
    if (g.cv_shift >= 0) {
      slot = it >> g.cv_shift;
      c = it & (g.CV - 1);
    } else {
      slot = it / g.CV;
      c = it - slot * g.CV;
    }
    const int64_t e = ((int64_t)bv * g.HW + s_tok[slot]) * g.C + (int64_t)c * VEC;
    Side<DT, VEC> sd = load_side<DT, VEC, MODE>(g, e, false);
    const Raw prevr = CD::load_stream(g.x0_prev, e);
    sd.m1 = prevr;   // m_{k-1}: the token's own stored x0
    Raw x0r;
    if (slot < nv) {
      float acc[VEC];
      gather_delta<DT, VEC>(g, b, c, s_word[slot], s_wk[slot], s_nvis[slot], acc);
      float prevf[VEC], y[VEC];
      CD::unpack(prevr, prevf);
#pragma unroll
      for (int q = 0; q < VEC; ++q) y[q] = prevf[q] + acc[q];
      x0r = CD::pack(y);
    } else {
      x0r = prevr;   // no anchor sees this token: it keeps its own state
    }
    finish_item<DT, VEC, MODE>(g, e, x0r, sd);
  }
}

// Foreground launch: g.gblocks list blocks (G lanes per listed token), then
// g.n_sblocks streaming blocks (one lane per token and channel vector).
template <int DT, int VEC, int MODE, int G, int AMAX>
__global__ __launch_bounds__(kBlock) void k_transport_geom_fg(GArgs g) {
  using CD = Codec<DT, VEC>;
  using Raw = typename CD::Raw;
  constexpr int kTok = kBlock / G;   // listed tokens per block
  constexpr int kApl = AMAX / G;     // anchor slots per lane
  static_assert(kApl >= 1 && kApl * G == AMAX, "G must divide AMAX");
  const int i = (int)blockIdx.x;
  if (i >= g.gblocks) {
    // streaming: anchor rows take the new prediction; a target token that is
    // listed belongs to a list block; any other keeps its own state
    const int lb = i - g.gblocks;
    if (lb >= g.n_sblocks) return;
    const int bv = __builtin_amdgcn_readfirstlane(lb / g.bpv_s);   // b * N + v
    const int t = (lb - bv * g.bpv_s) * kBlock + (int)threadIdx.x;
    if (t >= g.HW * g.CV) return;
    const int b = __builtin_amdgcn_readfirstlane(bv / g.N);
    const int v = bv - b * g.N;
    int s_self = -1;
#pragma unroll
    for (int s = 0; s < GC_MAX_ANCHORS; ++s) s_self = s < g.a && g.anchor_view[s] == v ? s : s_self;
    int p, c;
    if (g.cv_shift >= 0) {
      p = t >> g.cv_shift;
      c = t & (g.CV - 1);
    } else {
      p = t / g.CV;
      c = t - p * g.CV;
    }
    const int64_t e = ((int64_t)bv * g.HW + p) * g.C + (int64_t)c * VEC;
    if (s_self >= 0) {
      const Side<DT, VEC> sd = load_side<DT, VEC, MODE>(g, e, true);
      const Raw x0r = CD::load(g.x0_new, (((int64_t)b * g.a + s_self) * g.HW + p) * g.C + (int64_t)c * VEC);
      finish_item<DT, VEC, MODE>(g, e, x0r, sd);
      return;
    }
    const int64_t tk = (int64_t)bv * g.HW + p;
    if ((g.fg_bits[tk >> 5] >> (tk & 31)) & 1u) return;
    Side<DT, VEC> sd = load_side<DT, VEC, MODE>(g, e, false);
    const Raw prevr = CD::load_stream(g.x0_prev, e);
    sd.m1 = prevr;
    finish_item<DT, VEC, MODE>(g, e, prevr, sd);
    return;
  }

  // list block: an XCD-contiguous slice of the foreground list
  const int per = g.gblocks / kXcds;
  const int lb = (i % kXcds) * per + i / kXcds;
  const int lane_g = (int)threadIdx.x & (G - 1);
  const int r = lb * kTok + (int)threadIdx.x / G;
  const int64_t n_all = (int64_t)g.B * g.N * g.HW;
  int4 rec = make_int4(-1, 0, 0, 0);
  if (r < g.n_fg) rec = g.fg_recs[r];   // loaded first: its latency overlaps the camera setup
  __shared__ gc_camera cam_lds[kMaxCamLds];     // camera of (asset b, anchor slot s) at b * a + s
  __shared__ int32_t view_lds[GC_MAX_ANCHORS];  // anchor views (a per-lane index into the arguments is a load)
  for (int q = (int)threadIdx.x; q < g.B * g.a; q += kBlock) {
    const int bb = q / g.a, s = q - bb * g.a;
    cam_lds[q] = g.cams[(int64_t)bb * g.N + (int)((g.view_bytes >> (8 * s)) & 0xffu)];
  }
  if (threadIdx.x < g.a) view_lds[threadIdx.x] = (int)((g.view_bytes >> (8 * threadIdx.x)) & 0xffu);
  __syncthreads();
  // records come from the caller: a token outside the maps is ignored
  const int tokg = rec.x >= 0 && (int64_t)rec.x < n_all ? rec.x : -1;
  const int bv = tokg >= 0 ? tokg / g.HW : 0;
  const int b = bv / g.N;
  const int v = bv - b * g.N;
  bool anchor_row = false;
#pragma unroll
  for (int s = 0; s < GC_MAX_ANCHORS; ++s) anchor_row = anchor_row || (s < g.a && g.anchor_view[s] == v);
  const bool tok_ok = tokg >= 0 && !anchor_row;   // a target token of the list
  const float P[3] = {__int_as_float(rec.y), __int_as_float(rec.z), __int_as_float(rec.w)};
  const bool fg = tok_ok && finite_f(P[0]) && finite_f(P[1]) && finite_f(P[2]);

  // the operator, as in the blocked launch: lane j of the group evaluates
  // anchor slots j, j + G, ...; a wave in which no projection succeeded skips
  // the tap loads
  AnchorProj pj[kApl];
  AnchorTaps at[kApl];
  bool any_ok = false;
  if (__ballot(fg)) {   // a wave of anchor-view records projects nothing
#pragma unroll
    for (int j = 0; j < kApl; ++j) {   // branch-free: a lane without the slot keeps the result unused
      const int s = j * G + lane_g;
      pj[j] = anchor_project(P, cam_lds[b * g.a + (s < g.a ? s : 0)], g.H, g.W);
      pj[j].ok = pj[j].ok && fg && s < g.a;
      any_ok = any_ok || pj[j].ok;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kApl; ++j) pj[j] = AnchorProj{false, 0, 0, 0.0f, 0.0f};
  }
  const bool loaded = __ballot(any_ok) != 0ull;
  TapPos tp[kApl];
  if (loaded) {
#pragma unroll
    for (int j = 0; j < kApl; ++j) {
      const int s = j * G + lane_g;
      const int sc = s < g.a ? s : 0;
      tp[j] = anchor_tap_positions(pj[j], g.pos + ((int64_t)b * g.N + view_lds[sc]) * g.HW * 3, g.H, g.W);
    }
  }
  // The latent phase reads the token's own x0_prev and sampler input (and,
  // for UniPC, m_{k-2}) only after the tap tests; one dword of each, loaded now into
  // an LDS sink that nothing reads, brings their lines into L2 meanwhile
  // without holding a register (issued after the tap loads, so the tap
  // tests do not wait for them; the block's barriers wait on LDS only).
  if (tok_ok) {
    __shared__ float s_sink[64];
    const int64_t off = (int64_t)tokg * g.C * (DT == GC_F32 ? 4 : 2);
    const void* own = nullptr;
    if (lane_g == 0) own = g.x0_prev;
    if (lane_g == (G > 1 ? 1 : 0)) {
      const void* side = MODE == kGeomReconstruct ? g.x_t : MODE == kGeomUniPC ? (g.u.corr ? g.x_prev : g.x_t) : nullptr;
      if (G > 1) own = side;
      else if (side)
        __builtin_amdgcn_global_load_lds(static_cast<const char*>(side) + off,
                                         (__attribute__((address_space(3))) void*)s_sink, 4, 0, 0);
    }
    if (own)
      __builtin_amdgcn_global_load_lds(static_cast<const char*>(own) + off,
                                       (__attribute__((address_space(3))) void*)s_sink, 4, 0, 0);
    if constexpr (MODE == kGeomUniPC) {   // UniPC reads a third stream of its own
      if (lane_g == 0 && g.u.need_m2)
        __builtin_amdgcn_global_load_lds(static_cast<const char*>(g.m_km2) + off,
                                         (__attribute__((address_space(3))) void*)s_sink, 4, 0, 0);
    }
  }
  if (loaded) {
    const float tol2 = g.bbox[(int64_t)b * 8 + 6];
#pragma unroll
    for (int j = 0; j < kApl; ++j) at[j] = anchor_select(P, pj[j], tp[j], g.H, g.W, g.K, tol2);
  } else {
#pragma unroll
    for (int j = 0; j < kApl; ++j) {
      at[j].word = 0;
      at[j].mask = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) at[j].wk[k] = 0.0f;
    }
  }
  const int gbase = __lane_id() & ~(G - 1);
  int n_vis = 0;
#pragma unroll
  for (int j = 0; j < kApl; ++j) n_vis += __popcll((__ballot(at[j].word != 0) >> gbase) & ((1ull << G) - 1));

  // No ranking here: a list block's tokens are all foreground and mostly
  // visible (the blocked launch's blocks also hold background), so each lane
  // serves its own token's channel vectors lane_g, lane_g + G, ...  The
  // group's lanes put their anchor slots' words and weights in LDS and read
  // all of them back; the group is part of one wave, so a wave barrier
  // orders the writes before the reads (no block barrier).
  __shared__ int32_t s_word[kTok][AMAX + 1];       // +1: no bank conflicts between consecutive tokens
  __shared__ float s_wk[kTok][AMAX * 4 + 1];
  const int rl = (int)threadIdx.x / G;             // this token's place in the block
  if (tok_ok && n_vis > 0) {
#pragma unroll
    for (int j = 0; j < kApl; ++j) {
      const int s = j * G + lane_g;
      if (s < g.a) {
        s_word[rl][s] = at[j].word;
#pragma unroll
        for (int k = 0; k < 4; ++k) s_wk[rl][s * 4 + k] = at[j].wk[k];
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (!tok_ok) return;
  for (int c = lane_g; c < g.CV; c += G) {
    const int64_t e = (int64_t)tokg * g.C + (int64_t)c * VEC;   // latents are [B][N][H][W][C]
    Side<DT, VEC> sd = load_side<DT, VEC, MODE>(g, e, false);
    const Raw prevr = CD::load_stream(g.x0_prev, e);
    sd.m1 = prevr;   // m_{k-1}: the token's own stored x0
    Raw x0r;
    if (n_vis > 0) {
      float acc[VEC];
      gather_delta<DT, VEC>(g, b, c, s_word[rl], s_wk[rl], n_vis, acc);
      float prevf[VEC], y[VEC];
      CD::unpack(prevr, prevf);
#pragma unroll
      for (int q = 0; q < VEC; ++q) y[q] = prevf[q] + acc[q];
      x0r = CD::pack(y);
    } else {
      x0r = prevr;   // no anchor sees this token: it keeps its own state
    }
    finish_item<DT, VEC, MODE>(g, e, x0r, sd);
  }
}

// Lanes per target token: the channel vectors rounded up to a power of two,
// at most 8 (with more vectors a lane takes several items).
int geom_group(int CV) { return CV <= 1 ? 1 : CV <= 2 ? 2 : CV <= 4 ? 4 : 8; }

int prepare_geom(const void* x0_prev, const void* x0_new, const float* pos, const gc_camera* cams, const float* bbox,
                 const uint32_t* fg_bits, const int32_t* fg_recs, int64_t n_fg, int B, int N, int H, int W, int C,
                 const int32_t* anchors, int a, int K, int dtype, void* x0_out, const char* who, GArgs* g) {
  if (!x0_prev || !x0_new || !pos || !cams || !bbox || !anchors || !x0_out)
    return fail(GC_ERR_ARG, "%s: null pointer", who);
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
  if (!aligned16(x0_prev) || !aligned16(x0_new) || !aligned16(x0_out) || !aligned16(pos))
    return fail(GC_ERR_ALIGN, "%s: latents and position maps must be 16-byte aligned", who);
  // optional foreground index: both pointers null (and n_fg 0) for the blocked launch
  const int64_t n_tok_all = (int64_t)B * N * H * W;
  if (!fg_bits && (fg_recs || n_fg != 0))
    return fail(GC_ERR_ARG, "%s: fg_recs / n_fg given without fg_bits", who);
  if (fg_bits) {
    if (n_fg < 0 || n_fg > n_tok_all)
      return fail(GC_ERR_ARG, "%s: n_fg=%lld outside [0, B*N*H*W=%lld]", who, (long long)n_fg, (long long)n_tok_all);
    if (n_fg > 0 && !fg_recs) return fail(GC_ERR_ARG, "%s: null fg_recs with n_fg > 0", who);
    if (n_tok_all > 0x7fffffffLL)
      return fail(GC_ERR_CAPACITY, "%s: B*N*H*W=%lld exceeds 2^31-1 (foreground index)", who, (long long)n_tok_all);
    if (!aligned16(fg_bits) || (fg_recs && !aligned16(fg_recs)))
      return fail(GC_ERR_ALIGN, "%s: fg_bits and fg_recs must be 16-byte aligned", who);
  }
  std::memset(g, 0, sizeof(*g));
  bool is_anchor[GC_MAX_VIEWS] = {};
  for (int s = 0; s < a; ++s) {
    const int u = anchors[s];
    if (u < 0 || u >= N) return fail(GC_ERR_ARG, "%s: anchor %d outside [0, %d)", who, u, N);
    if (is_anchor[u]) return fail(GC_ERR_ARG, "%s: anchor %d listed twice", who, u);
    is_anchor[u] = true;
    g->anchor_view[s] = u;
    g->view_bytes |= (uint64_t)u << (8 * s);
  }
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t HW = (size_t)H * W;
  const size_t n_all = (size_t)B * N * HW * C * es, n_new = (size_t)B * a * HW * C * es;
  if (overlaps(x0_out, n_all, x0_prev, n_all) || overlaps(x0_out, n_all, x0_new, n_new) ||
      overlaps(x0_out, n_all, pos, (size_t)B * N * HW * 12) || overlaps(x0_out, n_all, cams, (size_t)B * N * sizeof(gc_camera)) ||
      overlaps(x0_out, n_all, bbox, (size_t)B * 32) ||
      overlaps(x0_out, n_all, fg_bits, (size_t)(n_tok_all + 31) / 32 * 4) ||
      overlaps(x0_out, n_all, fg_recs, (size_t)n_fg * 16))
    return fail(GC_ERR_ALIAS, "%s: x0_out overlaps an input", who);
  g->x0_prev = x0_prev;
  g->x0_new = x0_new;
  g->pos = pos;
  g->cams = cams;
  g->bbox = bbox;
  g->x0_out = x0_out;
  g->N = N;
  g->H = H;
  g->W = W;
  g->HW = (int)HW;
  g->C = C;
  g->a = a;
  g->K = K;
  g->CV = C / pick_vec(dtype, C);
  g->NT = N - a;
  g->cv_shift = (g->CV & (g->CV - 1)) == 0 ? __builtin_ctz((unsigned)g->CV) : -1;
  int n_sorted = 0;
  for (int u = 0; u < N; ++u)
    if (is_anchor[u]) g->sorted_anchor[n_sorted++] = u;
  for (int s = n_sorted; s < GC_MAX_ANCHORS; ++s) g->sorted_anchor[s] = INT32_MAX;
  g->G = geom_group(g->CV);
  const int tok = kBlock / g->G;
  g->bpv_t = (int)(((int64_t)HW + tok - 1) / tok);
  g->bpv_a = (int)(((int64_t)HW * g->CV + kBlock - 1) / kBlock);
  const int64_t nt = (int64_t)B * g->NT * g->bpv_t, na = (int64_t)B * a * g->bpv_a;
  const int64_t tgrid = (nt + kXcds - 1) / kXcds * kXcds, agrid = (na + kXcds - 1) / kXcds * kXcds;
  if (tgrid + agrid > (int64_t)0x7fffffff) return fail(GC_ERR_CAPACITY, "%s: problem too large for one launch", who);
  g->n_tblocks = (int)nt;
  g->tgrid = (int)tgrid;
  g->n_ablocks = (int)na;
  g->B = B;
  if (fg_bits && (int64_t)B * a <= kMaxCamLds) {   // the foreground launch
    const int64_t gb = (n_fg + tok - 1) / tok;
    const int64_t bpv_s = ((int64_t)HW * g->CV + kBlock - 1) / kBlock;
    const int64_t ns = (int64_t)B * N * bpv_s;
    const int64_t gblocks = (gb + kXcds - 1) / kXcds * kXcds;
    // a list lane's record index (block * tokens per block + lane / G) is a 32-bit int
    if (gblocks * tok > (int64_t)0x7fffffff)
      return fail(GC_ERR_CAPACITY, "%s: n_fg=%lld exceeds the list part's 2^31 records", who, (long long)n_fg);
    if (gblocks + ns > (int64_t)0x7fffffff) return fail(GC_ERR_CAPACITY, "%s: problem too large for one launch", who);
    g->fg_bits = fg_bits;
    g->fg_recs = reinterpret_cast<const int4*>(fg_recs);
    g->n_fg = (int)n_fg;
    g->gblocks = (int)gblocks;
    g->bpv_s = (int)bpv_s;
    g->n_sblocks = (int)ns;
  }
  return GC_OK;
}

template <int MODE>
void launch_geom(const GArgs& g, int dtype, hipStream_t stream) {
  const int agrid = (g.n_ablocks + kXcds - 1) / kXcds * kXcds;
  const bool fg = g.fg_bits != nullptr;
  const dim3 grid((unsigned)(fg ? g.gblocks + g.n_sblocks : g.tgrid + agrid));
  const int vec = g.C / g.CV;
#define GC_GEOM_K(DT_, VEC_, G_, AMAX_)                                                                       \
  do {                                                                                                      \
    if (fg)                                                                                                 \
      hipLaunchKernelGGL((k_transport_geom_fg<DT_, VEC_, MODE, G_, AMAX_>), grid, dim3(kBlock), 0, stream, g); \
    else                                                                                                    \
      hipLaunchKernelGGL((k_transport_geom<DT_, VEC_, MODE, G_, AMAX_>), grid, dim3(kBlock), 0, stream, g);    \
  } while (0)
#define GC_LAUNCH_GEOM(DT_, VEC_)                  \
  do {                                             \
    const bool small = g.a <= 4;                   \
    switch (g.G) {                                 \
      case 1:                                      \
        if (small)                                 \
          GC_GEOM_K(DT_, VEC_, 1, 4);              \
        else                                       \
          GC_GEOM_K(DT_, VEC_, 1, 8);              \
        break;                                     \
      case 2:                                      \
        if (small)                                 \
          GC_GEOM_K(DT_, VEC_, 2, 4);              \
        else                                       \
          GC_GEOM_K(DT_, VEC_, 2, 8);              \
        break;                                     \
      case 4:                                      \
        if (small)                                 \
          GC_GEOM_K(DT_, VEC_, 4, 4);              \
        else                                       \
          GC_GEOM_K(DT_, VEC_, 4, 8);              \
        break;                                     \
      default:                                     \
        GC_GEOM_K(DT_, VEC_, 8, 8);                \
    }                                              \
  } while (0)
  if (dtype == GC_F32)
    GC_LAUNCH_GEOM(GC_F32, 4);
  else if (vec == 8)
    GC_LAUNCH_GEOM(GC_BF16, 8);
  else
    GC_LAUNCH_GEOM(GC_BF16, 4);
#undef GC_LAUNCH_GEOM
#undef GC_GEOM_K
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" int gc_transport_step_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos,
                                      const gc_camera* cams, const float* bbox, const uint32_t* fg_bits,
                                      const int32_t* fg_recs, int64_t n_fg, int B, int N, int H, int W, int C,
                                      const int32_t* anchors, int a, int K, int dtype, void* x0_out,
                                      hipStream_t stream) {
  clear_error();
  GArgs g;
  int rc = prepare_geom(x0_prev, x0_anchor_new, pos, cams, bbox, fg_bits, fg_recs, n_fg, B, N, H, W, C, anchors, a,
                        K, dtype, x0_out, "gc_transport_step_geom", &g);
  if (rc) return rc;
  launch_geom<kGeomTransport>(g, dtype, stream);
  return after_launch(stream, "gc_transport_step_geom");
}

extern "C" int gc_transport_reconstruct_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos,
                                             const gc_camera* cams, const float* bbox, const uint32_t* fg_bits,
                                             const int32_t* fg_recs, int64_t n_fg, const void* x_t, int B, int N,
                                             int H, int W, int C, const int32_t* anchors, int a, int K, int dtype,
                                             const gc_sampler* smp, double t, double t_next, void* x0_out,
                                             void* x_next, void* model_out, hipStream_t stream) {
  clear_error();
  GArgs g;
  int rc = prepare_geom(x0_prev, x0_anchor_new, pos, cams, bbox, fg_bits, fg_recs, n_fg, B, N, H, W, C, anchors, a,
                        K, dtype, x0_out, "gc_transport_reconstruct_geom", &g);
  if (rc) return rc;
  if (!x_t || !x_next) return fail(GC_ERR_ARG, "gc_transport_reconstruct_geom: null x_t or x_next");
  rc = make_recon(smp, t, t_next, &g.r);
  if (rc) return rc;
  if ((g.r.pred != GC_PRED_NONE) != (model_out != nullptr))
    return fail(GC_ERR_ARG, "gc_transport_reconstruct_geom: model_out must be given iff pred_out != GC_PRED_NONE");
  if (!aligned16(x_t) || !aligned16(x_next) || (model_out && !aligned16(model_out)))
    return fail(GC_ERR_ALIGN, "gc_transport_reconstruct_geom: device pointers must be 16-byte aligned");
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t HW = (size_t)H * W;
  const size_t n_all = (size_t)B * N * HW * C * es, n_new = (size_t)B * a * HW * C * es;
  const void* ins[8] = {x0_prev, x0_anchor_new, x0_out, pos, cams, bbox, fg_bits, fg_recs};
  const size_t lens[8] = {n_all, n_new, n_all, (size_t)B * N * HW * 12, (size_t)B * N * sizeof(gc_camera),
                          (size_t)B * 32, ((size_t)B * N * HW + 31) / 32 * 4, (size_t)n_fg * 16};
  for (int i = 0; i < 8; ++i) {
    if (!ins[i]) continue;   // the optional index: a null pointer overlaps nothing (nor a null model_out)
    if (overlaps(x_next, n_all, ins[i], lens[i]) || overlaps(model_out, n_all, ins[i], lens[i]))
      return fail(GC_ERR_ALIAS, "gc_transport_reconstruct_geom: x_next/model_out overlap an input or x0_out");
  }
  if (overlaps(x_t, n_all, x0_out, n_all) || (x_next != x_t && overlaps(x_next, n_all, x_t, n_all)) ||
      overlaps(model_out, n_all, x_t, n_all) || overlaps(model_out, n_all, x_next, n_all))
    return fail(GC_ERR_ALIAS, "gc_transport_reconstruct_geom: outputs overlap x_t (only x_next == x_t is allowed)");
  g.x_t = x_t;
  g.x_next = x_next;
  g.model_out = model_out;
  launch_geom<kGeomReconstruct>(g, dtype, stream);
  return after_launch(stream, "gc_transport_reconstruct_geom");
}

extern "C" int gc_transport_unipc_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos,
                                       const gc_camera* cams, const float* bbox, const uint32_t* fg_bits,
                                       const int32_t* fg_recs, int64_t n_fg, const void* x_cur, const void* x_prev,
                                       const void* m_km2, int B, int N, int H, int W, int C, const int32_t* anchors,
                                       int a, int K, int dtype, const gc_unipc_step* st, void* x0_out, void* x_c,
                                       void* x_next, hipStream_t stream) {
  clear_error();
  GArgs g;
  int rc = prepare_geom(x0_prev, x0_anchor_new, pos, cams, bbox, fg_bits, fg_recs, n_fg, B, N, H, W, C, anchors, a,
                        K, dtype, x0_out, "gc_transport_unipc_geom", &g);
  if (rc) return rc;
  if (!st) return fail(GC_ERR_ARG, "gc_transport_unipc_geom: null coefficients");
  if (!x_c || !x_next) return fail(GC_ERR_ARG, "gc_transport_unipc_geom: null x_c or x_next");
  g.u = make_unicoef(*st);
  if (g.u.corr && !x_prev) return fail(GC_ERR_ARG, "gc_transport_unipc_geom: the corrector needs x_prev");
  if (!g.u.corr && !x_cur) return fail(GC_ERR_ARG, "gc_transport_unipc_geom: without the corrector x_cur is needed");
  if (g.u.need_m2 && !m_km2) return fail(GC_ERR_ARG, "gc_transport_unipc_geom: the coefficients need m_{k-2}");
  // m_{k-1} is x0_prev, the previous step's stored x0
  const void* al[5] = {x_cur, x_prev, m_km2, x_c, x_next};
  for (const void* q : al)
    if (q && !aligned16(q)) return fail(GC_ERR_ALIGN, "gc_transport_unipc_geom: device pointers must be 16-byte aligned");
  const size_t es = (size_t)dtype_bytes(dtype);
  const size_t HW = (size_t)H * W;
  const size_t n_all = (size_t)B * N * HW * C * es, n_new = (size_t)B * a * HW * C * es;
  const void* ins[10] = {x0_prev, x0_anchor_new, x_cur, x_prev, m_km2, pos, cams, bbox, fg_bits, fg_recs};
  const size_t lens[10] = {n_all, n_new, n_all, n_all, n_all, (size_t)B * N * HW * 12, (size_t)B * N * sizeof(gc_camera),
                           (size_t)B * 32, ((size_t)B * N * HW + 31) / 32 * 4, (size_t)n_fg * 16};
  for (int i = 0; i < 10; ++i) {
    if (!ins[i]) continue;
    if ((ins[i] != x_cur && overlaps(x_next, n_all, ins[i], lens[i])) ||
        (ins[i] != x_prev && overlaps(x_c, n_all, ins[i], lens[i])) || overlaps(x0_out, n_all, ins[i], lens[i]))
      return fail(GC_ERR_ALIAS,
                  "gc_transport_unipc_geom: outputs overlap inputs (only x_c == x_prev, x_next == x_cur)");
  }
  if (overlaps(x_c, n_all, x_next, n_all) || overlaps(x_c, n_all, x0_out, n_all) || overlaps(x_next, n_all, x0_out, n_all))
    return fail(GC_ERR_ALIAS, "gc_transport_unipc_geom: outputs overlap each other");
  g.x_t = x_cur;
  g.x_prev = x_prev;
  g.m_km2 = m_km2;
  g.x_c = x_c;
  g.x_next = x_next;
  launch_geom<kGeomUniPC>(g, dtype, stream);
  return after_launch(stream, "gc_transport_unipc_geom");
}
