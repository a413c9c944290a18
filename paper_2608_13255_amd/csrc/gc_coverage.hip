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

// Wave-wide sum and maximum, returned wave-uniform; every lane of the wave
// must be active.  Within each row of 16 lanes, DPP moves pair lane i with i
// xor 1, i xor 2, 7 - i (within 8) and 15 - i, so every lane ends with its
// row's total; the four row totals are then read into scalar registers.
constexpr int kDppXor1 = 0xb1;          // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4e;          // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;   // row_half_mirror
constexpr int kDppMirror = 0x140;       // row_mirror

__device__ __forceinline__ uint32_t wave_add(uint32_t v) {
  int x = (int)v;
  x += __builtin_amdgcn_mov_dpp(x, kDppXor1, 0xf, 0xf, false);
  x += __builtin_amdgcn_mov_dpp(x, kDppXor2, 0xf, 0xf, false);
  x += __builtin_amdgcn_mov_dpp(x, kDppHalfMirror, 0xf, 0xf, false);
  x += __builtin_amdgcn_mov_dpp(x, kDppMirror, 0xf, 0xf, false);
  return (uint32_t)__builtin_amdgcn_readlane(x, 0) + (uint32_t)__builtin_amdgcn_readlane(x, 16) +
         (uint32_t)__builtin_amdgcn_readlane(x, 32) + (uint32_t)__builtin_amdgcn_readlane(x, 48);
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, kDppXor1, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, kDppXor2, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, kDppHalfMirror, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, kDppMirror, 0xf, 0xf, false));
  return max(max((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16)),
             max((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48)));
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

// The token kernels give each lane one pair word: 32 consecutive tokens of
// a row, the staleness bytes of those tokens (two 16-byte loads, or bytewise
// when the rows are not 16-byte aligned) and, per view, one coalesced uint32
// of the pair bits.  A 64-lane wave covers 2048 tokens of one (asset, view)
// row: an item.  Per-item sums go through one wave sum each.

__device__ __forceinline__ uint32_t pair_word(const uint32_t* __restrict__ bits, int B, int N, int wpr, int u, int b,
                                              int v, int wi) {
  return bits[(((int64_t)u * B + b) * N + v) * wpr + wi];
}

// Tokens of word wi of view v that the views in mask cover: all of them when
// v is in the set, else those some view of the set sees.
__device__ __forceinline__ uint32_t set_covers(const uint32_t* __restrict__ bits, int B, int N, int wpr,
                                               unsigned long long mask, int b, int v, int wi) {
  if ((mask >> v) & 1ull) return ~0u;
  uint32_t acc = 0u;
  for (; mask; mask &= mask - 1) acc |= pair_word(bits, B, N, wpr, __ffsll((long long)mask) - 1, b, v, wi);
  return acc;
}

// Bits of word wi that are tokens of the row (the last word may be partial).
__device__ __forceinline__ uint32_t valid_bits(int HW, int wi) {
  const int n = HW - wi * 32;
  return n >= 32 ? ~0u : (n <= 0 ? 0u : (1u << n) - 1u);
}

// Staleness bytes of tokens t0 .. t0 + 31 of a row, four per register (token
// t0 + 4k + j in byte j of d[k]); tokens past the row read as background.
// VEC: the row starts 16-byte aligned and holds a multiple of 16 tokens.
template <bool VEC>
__device__ __forceinline__ void load_word_bytes(const uint8_t* __restrict__ row, int HW, int t0, uint32_t (&d)[8]) {
  if constexpr (VEC) {
    const uint4 bg = make_uint4(~0u, ~0u, ~0u, ~0u);
    const uint4 lo = t0 < HW ? *reinterpret_cast<const uint4*>(row + t0) : bg;
    const uint4 hi = t0 + 16 < HW ? *reinterpret_cast<const uint4*>(row + t0 + 16) : bg;
    d[0] = lo.x; d[1] = lo.y; d[2] = lo.z; d[3] = lo.w;
    d[4] = hi.x; d[5] = hi.y; d[6] = hi.z; d[7] = hi.w;
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      uint32_t x = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 4 * k + j;
        x |= (t < HW ? (uint32_t)row[t] : 0xffu) << (8 * j);
      }
      d[k] = x;
    }
  }
}

template <bool VEC>
__device__ __forceinline__ void store_word_bytes(uint8_t* __restrict__ row, int HW, int t0, const uint32_t (&d)[8]) {
  if constexpr (VEC) {
    if (t0 < HW) *reinterpret_cast<uint4*>(row + t0) = make_uint4(d[0], d[1], d[2], d[3]);
    if (t0 + 16 < HW) *reinterpret_cast<uint4*>(row + t0 + 16) = make_uint4(d[4], d[5], d[6], d[7]);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 4 * k + j;
        if (t < HW) row[t] = (uint8_t)(d[k] >> (8 * j));
      }
  }
}

// Bytewise (x + 1) mod 256: the token weight 1 + staleness, 0 for background.
__device__ __forceinline__ uint32_t bytes_plus_one(uint32_t x) {
  return ((x & 0x7f7f7f7fu) + 0x01010101u) ^ (x & 0x80808080u);
}

// 0x80 in each byte of x that is not zero, 0 elsewhere.
__device__ __forceinline__ uint32_t bytes_nonzero(uint32_t x) {
  return (((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x) & 0x80808080u;
}

// Bits 4k .. 4k + 3 of sel as bytes 0 / 1 (nibble bit j moves to bit 8 j:
// the product's partial terms land on distinct bits, so nothing carries).
__device__ __forceinline__ uint32_t nibble_bytes(uint32_t sel, int k) {
  return (((sel >> (4 * k)) & 0xfu) * 0x00204081u) & 0x01010101u;
}

// Sum of the weight bytes w of the tokens whose bit is set in sel.
__device__ __forceinline__ uint32_t weighted_count(const uint32_t (&w)[8], uint32_t sel) {
  uint32_t acc = 0u;
#pragma unroll
  for (int k = 0; k < 8; ++k) acc = __builtin_amdgcn_udot4(w[k], nibble_bytes(sel, k), acc, false);
  return acc;
}

// One block per (asset, view) row (blockIdx.x = b * N + v); its lanes
// stride over the row's pair words.  stats[b][v] = foreground tokens, tokens
// with staleness >= R, sum, max (after the update), reduced in the block and
// written once: no atomics, and no zeroing launch in front.
constexpr int kRowBlock = 512;

template <bool VEC>
__global__ __launch_bounds__(kRowBlock) void k_cov_update(const uint32_t* __restrict__ bits, int B, int N, int HW,
                                                          int wpr, unsigned long long anchor_mask, int R,
                                                          uint8_t* __restrict__ stale, uint32_t* __restrict__ stats) {
  __shared__ uint32_t part[kRowBlock / 64][4];
  const int bv = blockIdx.x;
  const int b = bv / N, v = bv % N;
  uint8_t* row = stale + (int64_t)bv * HW;
  uint32_t c_fg = 0, c_ge = 0, c_sum = 0, c_max = 0;   // this lane's totals
  for (int wi = (int)threadIdx.x; wi < wpr; wi += kRowBlock) {
    const uint32_t fresh = set_covers(bits, B, N, wpr, anchor_mask, b, v, wi) & valid_bits(HW, wi);
    uint32_t d[8];
    load_word_bytes<VEC>(row, HW, wi * 32, d);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint32_t s = d[k];
      const uint32_t fg = bytes_nonzero(~s);                       // s != 255
      const uint32_t inc = bytes_nonzero(~(s | 0x01010101u)) >> 7;   // s < 254
      const uint32_t fgm = (fg >> 7) * 0xffu;
      const uint32_t zero = nibble_bytes(fresh, k) * 0xffu & fgm;
      const uint32_t n = (s + inc) & ~zero;
      d[k] = n;
      const uint32_t nf = n & fgm;                                   // background reads 0
      c_fg += (uint32_t)__popc(fg);
      c_sum = __builtin_amdgcn_udot4(nf, 0x01010101u, c_sum, false);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t x = (nf >> (8 * j)) & 0xffu;
        c_ge += x >= (uint32_t)R ? 1u : 0u;
        c_max = max(c_max, x);
      }
    }
    store_word_bytes<VEC>(row, HW, wi * 32, d);
  }
  // every lane reaches the wave reductions (none returned early)
  c_fg = wave_add(c_fg);
  c_ge = wave_add(c_ge);
  c_sum = wave_add(c_sum);
  c_max = wave_max(c_max);
  const int wv = (int)threadIdx.x / 64;
  if (__lane_id() == 0) {
    part[wv][0] = c_fg;
    part[wv][1] = c_ge;
    part[wv][2] = c_sum;
    part[wv][3] = c_max;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    const int k = (int)threadIdx.x;
    uint32_t acc = 0u;
    for (int q = 0; q < kRowBlock / 64; ++q) acc = k == 3 ? max(acc, part[q][k]) : acc + part[q][k];
    stats[(int64_t)bv * 4 + k] = acc;
  }
}

// ---------------------------------------------------------------------------
// Selection and scores through the coverage histogram (N <= kHistViews).
// Every foreground token has a cover mask: bit v for its own view v and bit
// u for every view u that sees it.  H[m], the summed weight 1 + staleness of
// the tokens whose mask is m, decides both: with Y[X] the sum of H[m] over
// the masks m that are subsets of X (the subset sums of H) and U all views,
//   gain(u | S) = Y[U \ S] - Y[U \ (S + u)]   (the uncovered weight u covers)
//   score(S)    = Y[U] - Y[U \ S]             (the weight S covers)
// as exact integer sums.  Two launches: H and a block counter are cleared,
// then one kernel makes the pass over the tokens -- each block builds its
// histogram in LDS and adds its non-zero bins to H with integer atomics --
// and its last block to finish (the counter's ticket) takes the subset sums
// and runs every greedy round, or scores every set, with two lookups per
// candidate.  No block waits for another.
constexpr int kHistViews = 12;
constexpr int kHistBins = 1 << kHistViews;
constexpr int kHistThreads = 1024;                // 4 lanes per pair word, 8 tokens each
constexpr int kHistBlocks = 256;                  // blocks of the token pass (more for huge inputs)
constexpr int64_t kHistMaxWords = 1 << 16;        // words per block: 2^21 tokens * 255 < 2^32 per LDS bin

struct HistState {
  unsigned long long H[kHistBins];
  unsigned int ticket;                            // blocks of the token pass that have added their bins
};

// Clears H, the ticket and (the fused update) the statistics.
__global__ void k_hist_clear(HistState* __restrict__ hs, int nb, uint32_t* __restrict__ stats, int n_stats) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nb) hs->H[i] = 0ull;
  if (i < n_stats) stats[i] = 0u;
  if (i == 0) hs->ticket = 0u;
}

// Staleness bytes of tokens t0 .. t0 + 7 of a row, four per register;
// tokens past the row read as background.  VEC: 16-byte aligned rows of a
// multiple of 16 tokens (t0, a multiple of 8, then has all 8 in the row).
template <bool VEC>
__device__ __forceinline__ void load_8_bytes(const uint8_t* __restrict__ row, int HW, int t0, uint32_t (&d)[2]) {
  if constexpr (VEC) {
    const uint2 q = t0 < HW ? *reinterpret_cast<const uint2*>(row + t0) : make_uint2(~0u, ~0u);
    d[0] = q.x;
    d[1] = q.y;
  } else {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      uint32_t x = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 4 * k + j;
        x |= (t < HW ? (uint32_t)row[t] : 0xffu) << (8 * j);
      }
      d[k] = x;
    }
  }
}

// Y = the subset sums of H, left in y (LDS, indexed by mask).  The calling
// block has acquired the other blocks' additions to H (the ticket), so plain
// loads see them.  256 threads each hold 16 masks that differ in four bits
// and add along those bits in registers: bits 0-3 (masks 16t .. 16t + 15),
// then, after a transpose through y, bits 4-7, then bits 8-11; the passes
// over bits at or above N are skipped (their masks are never read).
__device__ __forceinline__ void subset_sums(const HistState* __restrict__ hs, int N, unsigned long long* y) {
  const int nb = 1 << N;
  const int t = (int)threadIdx.x;
  unsigned long long r[16];
  auto sum4 = [&r]() {
#pragma unroll
    for (int bit = 0; bit < 4; ++bit)
#pragma unroll
      for (int j = 0; j < 16; ++j)
        if ((j >> bit) & 1) r[j] += r[j ^ (1 << bit)];
  };
  if (t < kHistBins / 16) {
    const int m0 = 16 * t;
    if (m0 < nb) {   // nb >= 16 whenever N >= 4; a smaller nb fills one partial row
      const ulonglong2* src = reinterpret_cast<const ulonglong2*>(hs->H + m0);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const ulonglong2 q = 2 * j < nb - m0 ? src[j] : make_ulonglong2(0ull, 0ull);
        r[2 * j] = q.x;
        r[2 * j + 1] = 2 * j + 1 < nb - m0 ? q.y : 0ull;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 16; ++j) r[j] = 0ull;
    }
    sum4();
#pragma unroll
    for (int j = 0; j < 16; ++j) y[m0 + j] = r[j];
  }
  __syncthreads();
  for (int ph = 1; ph < 3 && 4 * ph < N; ++ph) {   // uniform
    const int sh = 4 * ph;                          // this pass's four bits: sh .. sh + 3
    const int low = t & ((1 << sh) - 1);            // bits below sh
    const int high = (t >> sh) << (sh + 4);         // bits above sh + 3
    if (t < kHistBins / 16) {
#pragma unroll
      for (int j = 0; j < 16; ++j) r[j] = y[high | (j << sh) | low];
      sum4();
#pragma unroll
      for (int j = 0; j < 16; ++j) y[high | (j << sh) | low] = r[j];
    }
    __syncthreads();
  }
}

// The views of mask in ascending order.
__device__ __forceinline__ void write_set(unsigned long long mask, int N, int32_t* out) {
  int j = 0;
  for (int u = 0; u < N; ++u)
    if ((mask >> u) & 1ull) out[j++] = u;
}

// Candidate sets as view masks.
constexpr int kMaxSets = 64;       // candidate sets per gc_coverage_score call
struct SetMasks {
  unsigned long long m[kMaxSets];
};

// Staleness bytes of a lane's 8 tokens written back (VEC as for load_8_bytes).
template <bool VEC>
__device__ __forceinline__ void store_8_bytes(uint8_t* __restrict__ row, int HW, int t0, const uint32_t (&d)[2]) {
  if constexpr (VEC) {
    if (t0 < HW) *reinterpret_cast<uint2*>(row + t0) = make_uint2(d[0], d[1]);
  } else {
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = t0 + 4 * k + j;
        if (t < HW) row[t] = (uint8_t)(d[k] >> (8 * j));
      }
  }
}

// The per-step staleness rule on four tokens' bytes s (token j in byte j):
// background (255) stays; a token whose byte of fresh_bytes is 0xff becomes
// 0; any other foreground token adds 1, saturating at 254.
__device__ __forceinline__ uint32_t stale_step(uint32_t s, uint32_t fresh_bytes) {
  const uint32_t fgm = (bytes_nonzero(~s) >> 7) * 0xffu;          // 0xff per foreground byte
  const uint32_t inc = bytes_nonzero(~(s | 0x01010101u)) >> 7;     // s < 254
  return (s + inc) & ~(fresh_bytes & fgm);
}

// The pass over the tokens (lane group of 4 per pair word, 8 tokens per
// lane; each wave takes 16 consecutive words per round, blocks stride over
// the words of every (asset, view) row), then in the last block: SCORE ==
// false, forced views first and a - n_forced greedy rounds, the set to out;
// SCORE == true, score[m] for the M sets.  UPDATE: the pass first applies
// one step of the staleness rule with the anchor set anchor_mask to the
// lane's tokens (stored back) and adds their statistics to stats (cleared
// by k_hist_clear) -- the per-row sums of one wave with one atomic each --
// so the histogram, and the selection or scores, are those of the updated
// staleness.
template <bool VEC, bool SCORE, bool UPDATE>
__global__ __launch_bounds__(kHistThreads) void k_cov_hist(const uint32_t* __restrict__ bits,
                                                           uint8_t* __restrict__ stale, int B, int N, int HW,
                                                           int wpr, int64_t n_words, HistState* __restrict__ hs, int a,
                                                           unsigned long long forced, int32_t* __restrict__ out,
                                                           SetMasks sets, int M, unsigned long long* __restrict__ score,
                                                           unsigned long long anchor_mask, int R,
                                                           uint32_t* __restrict__ stats) {
  __shared__ unsigned long long y[kHistBins];     // the last block's subset sums
  __shared__ uint32_t h[kHistBins];               // this block's histogram
  __shared__ int last;
  const int nb = 1 << N;
  for (int i = (int)threadIdx.x; i < nb; i += kHistThreads) h[i] = 0u;
  __syncthreads();
  const int lane = __lane_id();
  const int sub = lane & 3;                       // which 8 tokens of the word
  // the whole wave runs every round (a lane past the end only contributes
  // nothing), so the statistics' wave reductions see every lane
  for (int64_t base = ((int64_t)blockIdx.x * kHistThreads + (threadIdx.x & ~63)) >> 2; base < n_words;
       base += (int64_t)gridDim.x * (kHistThreads / 4)) {
    const int64_t wg = base + (lane >> 2);
    const bool active = wg < n_words;
    const int bv = active ? (int)(wg / wpr) : 0;
    const int wi = active ? (int)(wg - (int64_t)bv * wpr) : 0;
    const int b = bv / N, v = bv - b * N;
    uint32_t d[2] = {~0u, ~0u};   // staleness bytes of the lane's 8 tokens (background past the row)
    if (active) load_8_bytes<VEC>(stale + (int64_t)bv * HW, HW, wi * 32 + 8 * sub, d);
    uint32_t pb[kHistViews];      // the other views' pair bits of these 8 tokens
#pragma unroll
    for (int u = 0; u < kHistViews; ++u)
      pb[u] = (active && u < N && u != v) ? (pair_word(bits, B, N, wpr, u, b, v, wi) >> (8 * sub)) & 0xffu : 0u;
    if constexpr (UPDATE) {
      uint32_t fresh = (anchor_mask >> v) & 1ull ? 0xffu : 0u;
#pragma unroll
      for (int u = 0; u < kHistViews; ++u) fresh |= (anchor_mask >> u) & 1ull ? pb[u] : 0u;
      fresh &= (valid_bits(HW, wi) >> (8 * sub)) & 0xffu;
      uint32_t c_fg = 0u, c_ge = 0u, c_sum = 0u, c_max = 0u;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const uint32_t s0 = d[k];
        const uint32_t n = stale_step(s0, nibble_bytes(fresh, k) * 0xffu);
        d[k] = n;
        const uint32_t fgm = (bytes_nonzero(~s0) >> 7) * 0xffu;
        const uint32_t nf = n & fgm;                               // background reads 0
        c_fg += (uint32_t)__popc(bytes_nonzero(~s0));
        c_sum = __builtin_amdgcn_udot4(nf, 0x01010101u, c_sum, false);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t x = (nf >> (8 * j)) & 0xffu;
          c_ge += x >= (uint32_t)R ? 1u : 0u;
          c_max = max(c_max, x);
        }
      }
      if (active) store_8_bytes<VEC>(stale + (int64_t)bv * HW, HW, wi * 32 + 8 * sub, d);
      // per-row statistics: one atomic per counter for a wave within one row
      const int bv0 = __builtin_amdgcn_readfirstlane(bv);   // lane 0 is always active
      if (__ballot(active && bv != bv0) == 0ull) {
        c_fg = wave_add(c_fg);
        c_ge = wave_add(c_ge);
        c_sum = wave_add(c_sum);
        c_max = wave_max(c_max);
        if (lane == 0) {
          uint32_t* st = stats + (int64_t)bv0 * 4;
          if (c_fg) atomicAdd(st + 0, c_fg);
          if (c_ge) atomicAdd(st + 1, c_ge);
          if (c_sum) atomicAdd(st + 2, c_sum);
          if (c_max) atomicMax(st + 3, c_max);
        }
      } else if (active) {
        uint32_t* st = stats + (int64_t)bv * 4;
        if (c_fg) atomicAdd(st + 0, c_fg);
        if (c_ge) atomicAdd(st + 1, c_ge);
        if (c_sum) atomicAdd(st + 2, c_sum);
        if (c_max) atomicMax(st + 3, c_max);
      }
    }
    const uint32_t w[2] = {bytes_plus_one(d[0]), bytes_plus_one(d[1])};   // weights 1 + staleness, 0: background
    if (!(w[0] | w[1])) continue;
    // neighbouring tokens mostly share a mask: runs of one mask go to LDS as one add
    uint32_t run_m = 0u, run_w = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t wt = (w[j >> 2] >> (8 * (j & 3))) & 0xffu;
      uint32_t m = 1u << v;
#pragma unroll
      for (int u = 0; u < kHistViews; ++u) m |= ((pb[u] >> j) & 1u) << u;
      if (wt) {
        if (m == run_m) {
          run_w += wt;
        } else {
          if (run_w) atomicAdd(&h[run_m], run_w);
          run_m = m;
          run_w = wt;
        }
      }
    }
    if (run_w) atomicAdd(&h[run_m], run_w);
  }
  __syncthreads();
  for (int i = (int)threadIdx.x; i < nb; i += kHistThreads)
    if (h[i]) atomicAdd(&hs->H[i], (unsigned long long)h[i]);
  // The last block to add its bins computes the result (no block waits).
  // The barrier waits for this block's bin atomics; one acquire-release
  // ticket per block orders them before the last block's reads of H.
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(&hs->ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  subset_sums(hs, N, y);
  const unsigned all = (1u << N) - 1u;
  if constexpr (SCORE) {
    if ((int)threadIdx.x < M) score[threadIdx.x] = y[all] - y[all & ~(unsigned)sets.m[threadIdx.x]];
  } else {
    // one thread runs the rounds; per round the N + 1 lookups are issued
    // together (a view outside [0, N) or already chosen looks up its own
    // mask and is no candidate); the larger gain wins, on equal gains the
    // lower view
    if (threadIdx.x != 0) return;
    unsigned chosen = (unsigned)forced;
    for (int n = __popc(chosen); n < a; ++n) {
      const unsigned free_views = all & ~chosen;
      unsigned long long rest[kHistViews];
#pragma unroll
      for (int u = 0; u < kHistViews; ++u) rest[u] = y[free_views & ~(1u << u)];
      const unsigned long long base = y[free_views];
      unsigned long long best_g = 0ull;
      int best = kHistViews;
#pragma unroll
      for (int u = 0; u < kHistViews; ++u) {
        const bool cand = u < N && !((chosen >> u) & 1u);
        const unsigned long long g = base - rest[u];
        const bool take = cand && (best == kHistViews || g > best_g);
        best_g = take ? g : best_g;
        best = take ? u : best;
      }
      chosen |= 1u << best;
    }
    write_set(chosen, N, out);
  }
}

// Reductions over all tokens (selection gains, set scores) run on at most
// kRedBlocks one-wave blocks that stride over the items; lane u of a block
// keeps candidate u's total, written as one partial row of the workspace at
// the end, and one small block adds the rows up.  No global atomics: the
// per-candidate counters would otherwise take an atomic from every block.
constexpr int kRedBlocks = 2048;

// Workspace layout: per-block partial sums, candidate-major (the reducer's
// loads are coalesced), then the selection state.
struct SelState {
  unsigned long long part[GC_MAX_VIEWS][kRedBlocks];   // part[u][block]: gains or scores
  unsigned long long chosen;                           // bit u: view u chosen
};

int red_blocks(int64_t n_items) { return (int)(n_items < kRedBlocks ? n_items : kRedBlocks); }

// 1024 threads: wave w sums candidate u = w, w + 16, ... over the first nblk
// blocks' partials (coalesced, then a wave sum) into out[u] (LDS).
__device__ __forceinline__ void sum_partials(const SelState* st, int n, int nblk, unsigned long long* out) {
  const int wv = threadIdx.x / 64, lane = __lane_id();
  for (int u = wv; u < n; u += 16) {
    unsigned long long acc = 0ull;
#pragma unroll 4
    for (int i = lane; i < nblk; i += 64) acc += st->part[u][i];
    for (int o = 32; o > 0; o >>= 1) acc += (unsigned long long)__shfl_xor((long long)acc, o);
    if (lane == 0) out[u] = acc;
  }
}

// The views chosen before this round: the forced ones in the first round,
// else the set the previous round's pick left in the workspace.
__device__ __forceinline__ unsigned long long chosen_so_far(const SelState* st, unsigned long long forced, int first) {
  return first ? forced : st->chosen;
}

// Per token: weight 1 + staleness if no chosen view covers it (0 for
// background), added to every unchosen candidate that covers it.  Items
// whose view is chosen are covered throughout and add nothing.
template <bool VEC>
__global__ __launch_bounds__(64) void k_sel_gains(const uint32_t* __restrict__ bits, const uint8_t* __restrict__ stale,
                                                  int B, int N, int HW, int wpr, SelState* st,
                                                  unsigned long long forced, int first) {
  const unsigned long long chosen = chosen_so_far(st, forced, first);
  const int lane = (int)threadIdx.x;
  const int cpr = (wpr + 63) / 64;   // items per (asset, view)
  const int64_t n_items = (int64_t)B * N * cpr;
  unsigned long long mine = 0ull;    // lane u: candidate u's total
  for (int64_t it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int bv = (int)(it / cpr);
    const int b = bv / N, v = bv - b * N;
    if ((chosen >> v) & 1ull) continue;   // uniform
    const int wi = (int)(it - (int64_t)bv * cpr) * 64 + lane;
    uint32_t w[8];
    load_word_bytes<VEC>(stale + (int64_t)bv * HW, HW, wi * 32, w);
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = bytes_plus_one(w[k]);
    const bool in = wi < wpr;
    const uint32_t live = in ? valid_bits(HW, wi) & ~set_covers(bits, B, N, wpr, chosen, b, v, wi) : 0u;
    for (int u0 = 0; u0 < N; u0 += 16) {   // uniform; the group's words are loaded together
      uint32_t wd[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int u = u0 + q;
        wd[q] = (u >= N || ((chosen >> u) & 1ull) || !in) ? 0u : (u == v ? ~0u : pair_word(bits, B, N, wpr, u, b, v, wi));
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int u = u0 + q;
        if (u < N) {   // uniform
          const uint32_t g = wave_add(weighted_count(w, wd[q] & live));
          if (lane == u) mine += g;
        }
      }
    }
  }
  if (lane < N) st->part[lane][blockIdx.x] = mine;
}

// 1024 threads: each view's gain is the sum of the blocks' partials; then
// the unchosen view with the largest gain (ties: lower view) is chosen.  The
// last round writes the set to out.
__global__ __launch_bounds__(1024) void k_sel_pick(SelState* st, int N, int nblk, unsigned long long forced, int first,
                                                   int32_t* out) {
  __shared__ unsigned long long gain[GC_MAX_VIEWS];
  sum_partials(st, N, nblk, gain);
  __syncthreads();
  if (threadIdx.x != 0) return;
  unsigned long long chosen = chosen_so_far(st, forced, first);
  int best = -1;
  for (int c = 0; c < N; ++c) {
    if ((chosen >> c) & 1ull) continue;
    if (best < 0 || gain[c] > gain[best]) best = c;
  }
  if (best >= 0) chosen |= 1ull << best;
  st->chosen = chosen;
  if (out) write_set(chosen, N, out);
}

// the forced views are the whole set: no round runs
__global__ void k_sel_forced(unsigned long long forced, int N, int32_t* out) {
  if (threadIdx.x == 0) write_set(forced, N, out);
}

// score[m] partials: 1 + staleness over the foreground tokens set m covers.
template <bool VEC>
__global__ __launch_bounds__(64) void k_cov_score(const uint32_t* __restrict__ bits, const uint8_t* __restrict__ stale,
                                                  int B, int N, int HW, int wpr, SetMasks sets, int M, SelState* st) {
  const int lane = (int)threadIdx.x;
  const int cpr = (wpr + 63) / 64;
  const int64_t n_items = (int64_t)B * N * cpr;
  unsigned long long mine = 0ull;   // lane m: set m's total
  for (int64_t it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int bv = (int)(it / cpr);
    const int b = bv / N, v = bv - b * N;
    const int wi = (int)(it - (int64_t)bv * cpr) * 64 + lane;
    uint32_t w[8];
    load_word_bytes<VEC>(stale + (int64_t)bv * HW, HW, wi * 32, w);
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = bytes_plus_one(w[k]);
    const bool in = wi < wpr;
    const uint32_t vm = in ? valid_bits(HW, wi) : 0u;
    for (int m = 0; m < M; ++m) {   // uniform
      const uint32_t cov = in ? set_covers(bits, B, N, wpr, sets.m[m], b, v, wi) & vm : 0u;
      const uint32_t g = wave_add(weighted_count(w, cov));
      if (lane == m) mine += g;
    }
  }
  if (lane < M) st->part[lane][blockIdx.x] = mine;
}

__global__ __launch_bounds__(1024) void k_score_final(const SelState* st, int M, int nblk,
                                                      unsigned long long* __restrict__ score) {
  __shared__ unsigned long long sum[kMaxSets];
  sum_partials(st, M, nblk, sum);
  __syncthreads();
  if ((int)threadIdx.x < M) score[threadIdx.x] = sum[threadIdx.x];
}

// The histogram path: clear H and the ticket (and the statistics), then the
// pass over the tokens with the last block's rounds (select) or scores
// (score); UPDATE applies the staleness step first (anchor_mask, R, stats).
template <bool SCORE, bool UPDATE>
void launch_hist(const uint32_t* bits, uint8_t* stale, int B, int N, size_t HW, HistState* hs, bool vec, int a,
                 unsigned long long forced, int32_t* out, const SetMasks& sets, int M, unsigned long long* score,
                 unsigned long long anchor_mask, int R, uint32_t* stats, hipStream_t stream) {
  const int wpr = (int)((HW + 31) / 32);
  const int64_t n_words = (int64_t)B * N * wpr;
  int64_t nblk = (n_words * 4 + kHistThreads - 1) / kHistThreads;
  if (nblk > kHistBlocks) nblk = kHistBlocks;
  const int64_t need = (n_words + kHistMaxWords - 1) / kHistMaxWords;
  if (nblk < need) nblk = need;
  const int n_stats = UPDATE ? B * N * 4 : 0;   // B * N <= 65535 (check_grid)
  const int n_clear = (1 << N) > n_stats ? (1 << N) : n_stats;
  hipLaunchKernelGGL(k_hist_clear, dim3((unsigned)((n_clear + 255) / 256)), dim3(256), 0, stream, hs, 1 << N, stats,
                     n_stats);
  if (vec)
    hipLaunchKernelGGL((k_cov_hist<true, SCORE, UPDATE>), dim3((unsigned)nblk), dim3(kHistThreads), 0, stream, bits,
                       stale, B, N, (int)HW, wpr, n_words, hs, a, forced, out, sets, M, score, anchor_mask, R, stats);
  else
    hipLaunchKernelGGL((k_cov_hist<false, SCORE, UPDATE>), dim3((unsigned)nblk), dim3(kHistThreads), 0, stream, bits,
                       stale, B, N, (int)HW, wpr, n_words, hs, a, forced, out, sets, M, score, anchor_mask, R, stats);
}

// The histogram path serves N <= kHistViews (its grid stays below 2^31 blocks for any legal size).
bool hist_path(int N) { return N <= kHistViews; }

// The staleness rows start 16-byte aligned: the token kernels then move
// each lane's 32 bytes with two 16-byte accesses.
bool rows_aligned(const uint8_t* stale, size_t HW) { return ((uintptr_t)stale & 15u) == 0 && HW % 16 == 0; }

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

namespace gc {
namespace {

// Argument checks of one staleness step; mask: the anchor set's views.
int check_update(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a, int R,
                 const uint8_t* stale, const uint32_t* stats, const char* who, unsigned long long* mask) {
  if (!pair_bits || !anchors || !stale || !stats) return fail(GC_ERR_ARG, "%s: null pointer", who);
  int rc = check_grid(B, N, H, W, who);
  if (rc) return rc;
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "%s: a=%d outside [1, N=%d]", who, a, N);
  if (R < 1) return fail(GC_ERR_ARG, "%s: R=%d must be >= 1", who, R);
  *mask = 0;
  for (int s = 0; s < a; ++s) {
    if (anchors[s] < 0 || anchors[s] >= N) return fail(GC_ERR_ARG, "%s: anchor %d outside [0, %d)", who, anchors[s], N);
    if ((*mask >> anchors[s]) & 1ull) return fail(GC_ERR_ARG, "%s: anchor %d listed twice", who, anchors[s]);
    *mask |= 1ull << anchors[s];
  }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  if (overlaps(stats, (size_t)B * N * 16, stale, n_tok) || overlaps(stats, (size_t)B * N * 16, pair_bits, nb) ||
      overlaps(stale, n_tok, pair_bits, nb))
    return fail(GC_ERR_ALIAS, "%s: stale, stats and pair_bits must not overlap", who);
  if (!aligned16(pair_bits) || !aligned16(stats)) return fail(GC_ERR_ALIGN, "%s: pair_bits and stats must be 16-byte aligned", who);
  return GC_OK;
}

// Argument checks of a selection; mask: the forced views.
int check_select(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, int a,
                 const int32_t* forced, int n_forced, const int32_t* anchors_out, const void* workspace,
                 size_t ws_bytes, const char* who, unsigned long long* mask) {
  if (!pair_bits || !stale || !anchors_out || !workspace) return fail(GC_ERR_ARG, "%s: null pointer", who);
  int rc = check_grid(B, N, H, W, who);
  if (rc) return rc;
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "%s: a=%d outside [1, N=%d]", who, a, N);
  if (a > GC_MAX_ANCHORS) return fail(GC_ERR_CAPACITY, "%s: a=%d exceeds %d", who, a, GC_MAX_ANCHORS);
  if (n_forced < 0 || n_forced > a || (n_forced > 0 && !forced))
    return fail(GC_ERR_ARG, "%s: n_forced=%d outside [0, a=%d]", who, n_forced, a);
  if (ws_bytes < gc_coverage_workspace_bytes())
    return fail(GC_ERR_CAPACITY, "%s: workspace of %zu bytes, %zu needed", who, ws_bytes, gc_coverage_workspace_bytes());
  if (!aligned16(workspace) || !aligned16(pair_bits)) return fail(GC_ERR_ALIGN, "%s: workspace and pair_bits must be 16-byte aligned", who);
  *mask = 0;
  for (int j = 0; j < n_forced; ++j) {
    if (forced[j] < 0 || forced[j] >= N) return fail(GC_ERR_ARG, "%s: forced view %d outside [0, %d)", who, forced[j], N);
    if ((*mask >> forced[j]) & 1ull) return fail(GC_ERR_ARG, "%s: forced view %d listed twice", who, forced[j]);
    *mask |= 1ull << forced[j];
  }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  const size_t ws = gc_coverage_workspace_bytes();
  if (overlaps(workspace, ws, pair_bits, nb) || overlaps(workspace, ws, stale, n_tok) ||
      overlaps(anchors_out, (size_t)a * 4, workspace, ws) || overlaps(anchors_out, (size_t)a * 4, pair_bits, nb) ||
      overlaps(anchors_out, (size_t)a * 4, stale, n_tok))
    return fail(GC_ERR_ALIAS, "%s: workspace / anchors_out overlap an input", who);
  return GC_OK;
}

// Argument checks of a scoring call; masks: the candidate sets as view masks.
int check_score(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, const int32_t* sets,
                int M, int a, const uint64_t* scores, const void* workspace, size_t ws_bytes, const char* who,
                SetMasks* masks) {
  if (!pair_bits || !stale || !sets || !scores || !workspace) return fail(GC_ERR_ARG, "%s: null pointer", who);
  int rc = check_grid(B, N, H, W, who);
  if (rc) return rc;
  if (M < 1 || M > kMaxSets) return fail(GC_ERR_CAPACITY, "%s: M=%d outside [1, %d]", who, M, kMaxSets);
  if (a < 1 || a > N) return fail(GC_ERR_ARG, "%s: a=%d outside [1, N=%d]", who, a, N);
  std::memset(masks, 0, sizeof(*masks));
  for (int m = 0; m < M; ++m)
    for (int j = 0; j < a; ++j) {
      const int u = sets[m * a + j];
      if (u < 0 || u >= N) return fail(GC_ERR_ARG, "%s: view %d of set %d outside [0, %d)", who, u, m, N);
      masks->m[m] |= 1ull << u;
    }
  const size_t HW = (size_t)H * W;
  const size_t n_tok = (size_t)B * N * HW, nb = (size_t)gc_coverage_pair_words(B, N, H, W) * 4;
  if (ws_bytes < gc_coverage_workspace_bytes())
    return fail(GC_ERR_CAPACITY, "%s: workspace of %zu bytes, %zu needed", who, ws_bytes, gc_coverage_workspace_bytes());
  const size_t ws = gc_coverage_workspace_bytes();
  if (overlaps(scores, (size_t)M * 8, pair_bits, nb) || overlaps(scores, (size_t)M * 8, stale, n_tok) ||
      overlaps(workspace, ws, pair_bits, nb) || overlaps(workspace, ws, stale, n_tok) ||
      overlaps(workspace, ws, scores, (size_t)M * 8))
    return fail(GC_ERR_ALIAS, "%s: scores / workspace overlap an input or each other", who);
  if (!aligned16(pair_bits) || !aligned16(workspace) || ((uintptr_t)scores & 7u))
    return fail(GC_ERR_ALIGN, "%s: pair_bits and workspace 16-byte, scores 8-byte aligned", who);
  return GC_OK;
}

// The staleness step alone: one block per (asset, view) row, each writing its
// row's statistics.
void launch_update(const uint32_t* pair_bits, int B, int N, size_t HW, unsigned long long mask, int R, uint8_t* stale,
                   uint32_t* stats, hipStream_t stream) {
  const int wpr = (int)((HW + 31) / 32);
  const dim3 grid((unsigned)(B * N));
  if (rows_aligned(stale, HW))
    hipLaunchKernelGGL(k_cov_update<true>, grid, dim3(kRowBlock), 0, stream, pair_bits, B, N, (int)HW, wpr, mask, R,
                       stale, stats);
  else
    hipLaunchKernelGGL(k_cov_update<false>, grid, dim3(kRowBlock), 0, stream, pair_bits, B, N, (int)HW, wpr, mask, R,
                       stale, stats);
}

// The selection on the current staleness (after the optional step of
// mask_upd, R, stats, which the histogram pass applies itself).
void launch_select(const uint32_t* pair_bits, uint8_t* stale, int B, int N, size_t HW, int a, unsigned long long forced,
                   int n_forced, int32_t* anchors_out, void* workspace, bool upd, unsigned long long mask_upd, int R,
                   uint32_t* stats, hipStream_t stream) {
  const bool vec = rows_aligned(stale, HW);
  if (hist_path(N) && n_forced < a) {
    SetMasks none;
    std::memset(&none, 0, sizeof(none));
    HistState* hs = static_cast<HistState*>(workspace);
    if (upd)
      launch_hist<false, true>(pair_bits, stale, B, N, HW, hs, vec, a, forced, anchors_out, none, 0, nullptr, mask_upd,
                               R, stats, stream);
    else
      launch_hist<false, false>(pair_bits, stale, B, N, HW, hs, vec, a, forced, anchors_out, none, 0, nullptr, 0ull, 1,
                                nullptr, stream);
    return;
  }
  if (upd) launch_update(pair_bits, B, N, HW, mask_upd, R, stale, stats, stream);
  if (n_forced == a) {
    hipLaunchKernelGGL(k_sel_forced, dim3(1), dim3(64), 0, stream, forced, N, anchors_out);
    return;
  }
  SelState* st = static_cast<SelState*>(workspace);
  const int wpr = (int)((HW + 31) / 32);
  const int nblk = red_blocks((int64_t)B * N * ((wpr + 63) / 64));
  for (int r = n_forced; r < a; ++r) {   // more views: one pass over the tokens per round
    const int first = r == n_forced;
    int32_t* out = r == a - 1 ? anchors_out : nullptr;
    if (vec)
      hipLaunchKernelGGL(k_sel_gains<true>, dim3(nblk), dim3(64), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, st,
                         forced, first);
    else
      hipLaunchKernelGGL(k_sel_gains<false>, dim3(nblk), dim3(64), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, st,
                         forced, first);
    hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(1024), 0, stream, st, N, nblk, forced, first, out);
  }
}

// The set scores on the current staleness (after the optional step, as above).
void launch_score(const uint32_t* pair_bits, uint8_t* stale, int B, int N, size_t HW, const SetMasks& masks, int M,
                  int a, uint64_t* scores, void* workspace, bool upd, unsigned long long mask_upd, int R,
                  uint32_t* stats, hipStream_t stream) {
  unsigned long long* out = reinterpret_cast<unsigned long long*>(scores);
  if (hist_path(N)) {
    HistState* hs = static_cast<HistState*>(workspace);
    if (upd)
      launch_hist<true, true>(pair_bits, stale, B, N, HW, hs, rows_aligned(stale, HW), a, 0ull, nullptr, masks, M, out,
                              mask_upd, R, stats, stream);
    else
      launch_hist<true, false>(pair_bits, stale, B, N, HW, hs, rows_aligned(stale, HW), a, 0ull, nullptr, masks, M,
                               out, 0ull, 1, nullptr, stream);
    return;
  }
  if (upd) launch_update(pair_bits, B, N, HW, mask_upd, R, stale, stats, stream);
  SelState* st = static_cast<SelState*>(workspace);
  const int wpr = (int)((HW + 31) / 32);
  const int nblk = red_blocks((int64_t)B * N * ((wpr + 63) / 64));
  if (rows_aligned(stale, HW))
    hipLaunchKernelGGL(k_cov_score<true>, dim3(nblk), dim3(64), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, masks,
                       M, st);
  else
    hipLaunchKernelGGL(k_cov_score<false>, dim3(nblk), dim3(64), 0, stream, pair_bits, stale, B, N, (int)HW, wpr, masks,
                       M, st);
  hipLaunchKernelGGL(k_score_final, dim3(1), dim3(1024), 0, stream, st, M, nblk, out);
}

}  // namespace
}  // namespace gc

extern "C" int gc_coverage_update(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a,
                                  int R, uint8_t* stale, uint32_t* stats, hipStream_t stream) {
  clear_error();
  unsigned long long mask = 0;
  const int rc = check_update(pair_bits, B, N, H, W, anchors, a, R, stale, stats, "gc_coverage_update", &mask);
  if (rc) return rc;
  launch_update(pair_bits, B, N, (size_t)H * W, mask, R, stale, stats, stream);
  return after_launch(stream, "gc_coverage_update");
}

extern "C" size_t gc_coverage_workspace_bytes(void) {
  const size_t n = sizeof(SelState) > sizeof(HistState) ? sizeof(SelState) : sizeof(HistState);
  return (n + 255) / 256 * 256;
}

extern "C" int gc_coverage_select(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, int a,
                                  const int32_t* forced, int n_forced, int32_t* anchors_out, void* workspace,
                                  size_t ws_bytes, hipStream_t stream) {
  clear_error();
  unsigned long long mask = 0;
  const int rc = check_select(pair_bits, stale, B, N, H, W, a, forced, n_forced, anchors_out, workspace, ws_bytes,
                              "gc_coverage_select", &mask);
  if (rc) return rc;
  // the pass reads the staleness only (no update): the cast is for the shared kernel
  launch_select(pair_bits, const_cast<uint8_t*>(stale), B, N, (size_t)H * W, a, mask, n_forced, anchors_out, workspace,
                false, 0ull, 1, nullptr, stream);
  return after_launch(stream, "gc_coverage_select");
}

extern "C" int gc_coverage_score(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W,
                                 const int32_t* sets, int M, int a, uint64_t* scores, void* workspace, size_t ws_bytes,
                                 hipStream_t stream) {
  clear_error();
  SetMasks masks;
  const int rc = check_score(pair_bits, stale, B, N, H, W, sets, M, a, scores, workspace, ws_bytes,
                             "gc_coverage_score", &masks);
  if (rc) return rc;
  launch_score(pair_bits, const_cast<uint8_t*>(stale), B, N, (size_t)H * W, masks, M, a, scores, workspace, false, 0ull,
               1, nullptr, stream);
  return after_launch(stream, "gc_coverage_score");
}

extern "C" int gc_coverage_update_select(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors,
                                         int a, int R, uint8_t* stale, uint32_t* stats, int a_next,
                                         const int32_t* forced, int n_forced, int32_t* anchors_out, void* workspace,
                                         size_t ws_bytes, hipStream_t stream) {
  clear_error();
  const char* who = "gc_coverage_update_select";
  unsigned long long mask_upd = 0, mask_forced = 0;
  int rc = check_update(pair_bits, B, N, H, W, anchors, a, R, stale, stats, who, &mask_upd);
  if (rc) return rc;
  rc = check_select(pair_bits, stale, B, N, H, W, a_next, forced, n_forced, anchors_out, workspace, ws_bytes, who,
                    &mask_forced);
  if (rc) return rc;
  const size_t ws = gc_coverage_workspace_bytes();
  if (overlaps(stats, (size_t)B * N * 16, workspace, ws) || overlaps(stats, (size_t)B * N * 16, anchors_out, (size_t)a_next * 4))
    return fail(GC_ERR_ALIAS, "%s: stats overlaps the workspace or anchors_out", who);
  launch_select(pair_bits, stale, B, N, (size_t)H * W, a_next, mask_forced, n_forced, anchors_out, workspace, true,
                mask_upd, R, stats, stream);
  return after_launch(stream, who);
}

extern "C" int gc_coverage_update_score(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors,
                                        int a, int R, uint8_t* stale, uint32_t* stats, const int32_t* sets, int M,
                                        int a_set, uint64_t* scores, void* workspace, size_t ws_bytes,
                                        hipStream_t stream) {
  clear_error();
  const char* who = "gc_coverage_update_score";
  unsigned long long mask_upd = 0;
  int rc = check_update(pair_bits, B, N, H, W, anchors, a, R, stale, stats, who, &mask_upd);
  if (rc) return rc;
  SetMasks masks;
  rc = check_score(pair_bits, stale, B, N, H, W, sets, M, a_set, scores, workspace, ws_bytes, who, &masks);
  if (rc) return rc;
  const size_t ws = gc_coverage_workspace_bytes();
  if (overlaps(stats, (size_t)B * N * 16, workspace, ws) || overlaps(stats, (size_t)B * N * 16, scores, (size_t)M * 8))
    return fail(GC_ERR_ALIAS, "%s: stats overlaps the workspace or scores", who);
  launch_score(pair_bits, stale, B, N, (size_t)H * W, masks, M, a_set, scores, workspace, true, mask_upd, R, stats,
               stream);
  return after_launch(stream, who);
}
