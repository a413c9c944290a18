// Token indexes that let the per-step kernels split their work into
// gathering blocks over a compact list and streaming blocks over everything
// else, which recognise the listed tokens by one bit each.
//
// Visible-token index of a correspondence operator (once per asset and
// anchor set).  G_{A->v} has a non-zero row only for tokens some anchor sees
// (Sec. 3.2: a token with no tap inside the tolerance has an all-zero row);
// the list holds those tokens.
//
// Foreground index of the position maps (once per asset batch).  Only a
// token with a finite position can be seen by an anchor (the operator's
// tolerance test needs its 3D point), so the on-the-fly step evaluates the
// operator for foreground tokens only; the list holds each one's token index
// and position, so that one 16-byte load gives a lane both.
//
// The lists are in tile order: view after view, and inside a view 16 x 16
// tiles of the token grid (bands of 16 rows from the top, tiles from the
// left, narrower or shorter at the grid's right and bottom edges), row-major
// inside a tile.  A block of the per-step kernels takes consecutive list
// entries, so its tokens form a compact patch of the view, whose footprints
// in each anchor view lie close together: their tap reads share cache lines.
//
// Three passes, deterministic:
//   count    per 1024-entry chunk of the list order, listed tokens (ballot +
//            popcount); also writes the bitmask in token order (one 64-bit
//            ballot per wave over consecutive tokens)
//   scan     exclusive prefix over the chunk counts, total -> list length
//   scatter  each chunk writes its tokens at its offset, ranked inside the
//            chunk by (round, wave, mbcnt of the ballot)
#include <mutex>

#include "gc_common.h"

// Scratch of gc_index_correspondence_noalloc (per-chunk counts and offsets),
// one copy per GPU for the life of the process.  Host code never uses this
// name as an address: it takes the device address from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[GC_NOALLOC_SCRATCH_BYTES];

namespace gc {
namespace {

constexpr int kBlock = 256;
constexpr int kRounds = 4;                 // tokens per block = kRounds * kBlock
constexpr int kChunk = kRounds * kBlock;
constexpr int kWaves = kBlock / 64;
constexpr int kTile = 16;                  // tiles of the list order: kTile x kTile tokens

// Position i of the list order -> token index; a bijection of
// [0, n_views * H * W) (no padding: edge tiles are narrower or shorter).
struct TileOrder {
  int H, W;
  int64_t HW;
  __device__ __forceinline__ int64_t token(int64_t i) const {
    const int64_t view = i / HW;
    const int r = (int)(i - view * HW);           // position inside the view
    const int band = r / (kTile * W);             // band of kTile rows (the last may be shorter)
    const int rb = r - band * kTile * W;
    const int bh = min(kTile, H - band * kTile);  // rows of this band
    const int tx = rb / (bh * kTile);             // tile inside the band (the last may be narrower)
    const int q = rb - tx * bh * kTile;
    const int tw = min(kTile, W - tx * kTile);    // columns of this tile
    const int yy = q / tw;
    return view * HW + (int64_t)(band * kTile + yy) * W + tx * kTile + (q - yy * tw);
  }
};

// Listed tokens of the visible-token index: a non-zero correspondence row.
struct VisiblePred {
  const int32_t* corr;
  int a;
  __device__ __forceinline__ bool operator()(int64_t tok) const {
    const int32_t* w = corr + tok * a;
    if (a == 4) {
      const int4 q = *reinterpret_cast<const int4*>(w);
      return (q.x | q.y | q.z | q.w) != 0;
    }
    int32_t any = 0;
    for (int s = 0; s < a; ++s) any |= w[s];
    return any != 0;
  }
  // list entry: the token index
  __device__ __forceinline__ void write(int32_t* list, int32_t at, int64_t tok) const { list[at] = (int32_t)tok; }
};

// Listed tokens of the foreground index: all three position components finite.
struct ForegroundPred {
  const float* pos;
  __device__ __forceinline__ bool operator()(int64_t tok) const {
    const float* q = pos + tok * 3;
    return finite_f(q[0]) && finite_f(q[1]) && finite_f(q[2]);
  }
  // list entry: {token, x, y, z} (positions as float bit patterns), 16 bytes
  __device__ __forceinline__ void write(int32_t* list, int32_t at, int64_t tok) const {
    const float* q = pos + tok * 3;
    *reinterpret_cast<int4*>(list + (int64_t)at * 4) =
        make_int4((int32_t)tok, __float_as_int(q[0]), __float_as_int(q[1]), __float_as_int(q[2]));
  }
};

template <class Pred>
__global__ __launch_bounds__(kBlock) void k_index_count(Pred pred, TileOrder order, int64_t n_tokens,
                                                        uint32_t* __restrict__ bits, int64_t n_words,
                                                        int32_t* __restrict__ counts) {
  __shared__ int32_t wave_cnt[kWaves];
  const int wv = threadIdx.x / 64;
  int32_t total = 0;
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = (int64_t)blockIdx.x * kChunk + r * kBlock + threadIdx.x;
    // the bitmask over consecutive tokens
    const unsigned long long m = __ballot(i < n_tokens && pred(i));
    if (__lane_id() == 0) {
      const int64_t w0 = ((int64_t)blockIdx.x * kChunk + r * kBlock + wv * 64) >> 5;
      if (w0 < n_words) bits[w0] = (uint32_t)m;
      if (w0 + 1 < n_words) bits[w0 + 1] = (uint32_t)(m >> 32);
    }
    // the count over this chunk of the list order
    const unsigned long long c = __ballot(i < n_tokens && pred(order.token(i)));
    if (__lane_id() == 0) wave_cnt[wv] = __popcll(c);
    __syncthreads();
    if (threadIdx.x == 0)
      for (int w = 0; w < kWaves; ++w) total += wave_cnt[w];
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[blockIdx.x] = total;
}

// one block: exclusive scan of counts[n] into offsets[n], total into n_vis
__global__ __launch_bounds__(kBlock) void k_index_scan(const int32_t* __restrict__ counts, int64_t n,
                                                       int32_t* __restrict__ offsets, int32_t* __restrict__ n_vis) {
  __shared__ int32_t buf[kBlock];
  int32_t carry = 0;
  for (int64_t base = 0; base < n; base += kBlock) {
    const int64_t i = base + threadIdx.x;
    const int32_t c = i < n ? counts[i] : 0;
    buf[threadIdx.x] = c;
    __syncthreads();
    // inclusive Hillis-Steele scan over the block
    for (int o = 1; o < kBlock; o <<= 1) {
      const int32_t add = threadIdx.x >= o ? buf[threadIdx.x - o] : 0;
      __syncthreads();
      buf[threadIdx.x] += add;
      __syncthreads();
    }
    if (i < n) offsets[i] = carry + buf[threadIdx.x] - c;
    const int32_t block_total = buf[kBlock - 1];
    __syncthreads();
    carry += block_total;
  }
  if (threadIdx.x == 0) *n_vis = carry;
}

template <class Pred>
__global__ __launch_bounds__(kBlock) void k_index_scatter(Pred pred, TileOrder order, int64_t n_tokens,
                                                          const int32_t* __restrict__ offsets,
                                                          int32_t* __restrict__ list) {
  __shared__ int32_t wave_cnt[kWaves];
  const int wv = threadIdx.x / 64;
  int32_t pos = offsets[blockIdx.x];
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = (int64_t)blockIdx.x * kChunk + r * kBlock + threadIdx.x;
    const int64_t tok = i < n_tokens ? order.token(i) : 0;
    const bool vis = i < n_tokens && pred(tok);
    const unsigned long long m = __ballot(vis);
    if (__lane_id() == 0) wave_cnt[wv] = __popcll(m);
    __syncthreads();
    int32_t before = 0;
    for (int w = 0; w < wv; ++w) before += wave_cnt[w];
    const int32_t rank = (int32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (vis) pred.write(list, pos + before + rank, tok);
    int32_t round_total = 0;
    for (int w = 0; w < kWaves; ++w) round_total += wave_cnt[w];
    __syncthreads();
    pos += round_total;
  }
}

}  // namespace
}  // namespace gc

using namespace gc;

extern "C" size_t gc_index_workspace_bytes(int64_t n_tokens) {
  if (n_tokens <= 0) return 256;
  const int64_t nb = (n_tokens + kChunk - 1) / kChunk;
  return (size_t)(((2 * nb * 4) + 255) / 256 * 256);
}

namespace gc {
namespace {

// Views of H x W tokens: the token count (at most 2^31 - 1) and the list order.
int check_views(int64_t n_views, int H, int W, const char* who, int64_t* n_tokens, TileOrder* order) {
  if (n_views < 0 || H < 1 || W < 1)
    return fail(GC_ERR_SHAPE, "%s: bad shape n_views=%lld H=%d W=%d", who, (long long)n_views, H, W);
  if (H > GC_MAX_GRID || W > GC_MAX_GRID) return fail(GC_ERR_CAPACITY, "%s: grid %dx%d exceeds %d", who, H, W, GC_MAX_GRID);
  if (n_views > 0x7fffffffLL / ((int64_t)H * W))
    return fail(GC_ERR_CAPACITY, "%s: n_views * H * W exceeds 2^31-1", who);
  *n_tokens = n_views * H * W;
  order->H = H;
  order->W = W;
  order->HW = (int64_t)H * W;
  return GC_OK;
}

// Validation of the visible-token index's own arguments (everything but
// the scratch memory).
int check_visible_index(const int32_t* corr, int64_t n_tokens, int a, const uint32_t* vis_bits,
                        const int32_t* vis_list, const int32_t* n_vis, const char* who) {
  if (!n_vis) return fail(GC_ERR_ARG, "%s: null n_vis", who);
  if (a < 1 || a > GC_MAX_ANCHORS) return fail(GC_ERR_ARG, "%s: a=%d outside [1, %d]", who, a, GC_MAX_ANCHORS);
  if (n_tokens > 0 && (!corr || !vis_bits || !vis_list)) return fail(GC_ERR_ARG, "%s: null pointer", who);
  if ((corr && !aligned16(corr)) || (vis_bits && !aligned16(vis_bits)) || (vis_list && !aligned16(vis_list)))
    return fail(GC_ERR_ALIGN, "%s: pointers must be 16-byte aligned", who);
  const int64_t n_words = (n_tokens + 31) / 32;
  const size_t nc = (size_t)n_tokens * a * 4, nl = (size_t)n_tokens * 4, nbits = (size_t)n_words * 4;
  if (overlaps(vis_bits, nbits, corr, nc) || overlaps(vis_list, nl, corr, nc) || overlaps(vis_list, nl, vis_bits, nbits) ||
      overlaps(n_vis, 4, vis_list, nl) || overlaps(n_vis, 4, vis_bits, nbits))
    return fail(GC_ERR_ALIAS, "%s: buffers overlap", who);
  return GC_OK;
}

// The three passes; counts_offsets: 2 * ceil(n_tokens / kChunk) int32 of
// device scratch, fully written before it is read.
void launch_visible_index(const int32_t* corr, int64_t n_tokens, const TileOrder& order, int a, uint32_t* vis_bits,
                          int32_t* vis_list, int32_t* n_vis, int32_t* counts_offsets, hipStream_t stream) {
  const int64_t n_words = (n_tokens + 31) / 32;
  const int64_t nb = n_tokens > 0 ? (n_tokens + kChunk - 1) / kChunk : 0;
  int32_t* counts = counts_offsets;
  int32_t* offsets = counts + nb;
  if (nb > 0)
    hipLaunchKernelGGL(k_index_count<VisiblePred>, dim3((unsigned)nb), dim3(kBlock), 0, stream,
                       VisiblePred{corr, a}, order, n_tokens, vis_bits, n_words, counts);
  hipLaunchKernelGGL(k_index_scan, dim3(1), dim3(kBlock), 0, stream, counts, nb, offsets, n_vis);
  if (nb > 0)
    hipLaunchKernelGGL(k_index_scatter<VisiblePred>, dim3((unsigned)nb), dim3(kBlock), 0, stream,
                       VisiblePred{corr, a}, order, n_tokens, offsets, vis_list);
}

// Device address of this library's scratch array on the current device,
// looked up once per device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(void** out, const char* who) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(GC_ERR_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(GC_ERR_CAPACITY, "%s: device %d beyond %d", who, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(GC_ERR_HIP, "%s: hipGetSymbolAddress of the scratch array: %s", who, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GC_OK;
}

}  // namespace
}  // namespace gc

extern "C" int gc_index_correspondence(const int32_t* corr, int64_t n_views, int H, int W, int a, uint32_t* vis_bits,
                                       int32_t* vis_list, int32_t* n_vis, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream) {
  clear_error();
  const char* who = "gc_index_correspondence";
  if (!workspace) return fail(GC_ERR_ARG, "%s: null workspace", who);
  int64_t n_tokens = 0;
  TileOrder order;
  int rc = check_views(n_views, H, W, who, &n_tokens, &order);
  if (rc) return rc;
  rc = check_visible_index(corr, n_tokens, a, vis_bits, vis_list, n_vis, who);
  if (rc) return rc;
  if (!aligned16(workspace)) return fail(GC_ERR_ALIGN, "%s: pointers must be 16-byte aligned", who);
  if (workspace_bytes < gc_index_workspace_bytes(n_tokens))
    return fail(GC_ERR_CAPACITY, "%s: workspace of %zu bytes is below the %zu required", who, workspace_bytes,
                gc_index_workspace_bytes(n_tokens));
  const size_t nc = (size_t)n_tokens * a * 4, nl = (size_t)n_tokens * 4, nbits = (size_t)(n_tokens + 31) / 32 * 4;
  if (overlaps(workspace, workspace_bytes, corr, nc) || overlaps(workspace, workspace_bytes, vis_list, nl) ||
      overlaps(workspace, workspace_bytes, vis_bits, nbits) || overlaps(workspace, workspace_bytes, n_vis, 4))
    return fail(GC_ERR_ALIAS, "%s: buffers overlap", who);
  launch_visible_index(corr, n_tokens, order, a, vis_bits, vis_list, n_vis, static_cast<int32_t*>(workspace), stream);
  return after_launch(stream, who);
}

extern "C" int gc_index_correspondence_noalloc(const int32_t* corr, int64_t n_views, int H, int W, int a,
                                               uint32_t* vis_bits, int32_t* vis_list, int32_t* n_vis,
                                               hipStream_t stream) {
  clear_error();
  const char* who = "gc_index_correspondence_noalloc";
  int64_t n_tokens = 0;
  TileOrder order;
  int rc = check_views(n_views, H, W, who, &n_tokens, &order);
  if (rc) return rc;
  rc = check_visible_index(corr, n_tokens, a, vis_bits, vis_list, n_vis, who);
  if (rc) return rc;
  if (gc_index_workspace_bytes(n_tokens) > GC_NOALLOC_SCRATCH_BYTES)
    return fail(GC_ERR_CAPACITY, "%s: n_tokens=%lld needs %zu bytes of scratch, above the library's %d", who,
                (long long)n_tokens, gc_index_workspace_bytes(n_tokens), GC_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  rc = scratch_on_current_device(&ws, who);
  if (rc) return rc;
  launch_visible_index(corr, n_tokens, order, a, vis_bits, vis_list, n_vis, static_cast<int32_t*>(ws), stream);
  return after_launch(stream, who);
}

extern "C" int gc_index_foreground(const float* pos, int64_t n_views, int H, int W, uint32_t* fg_bits,
                                   int32_t* fg_recs, int32_t* n_fg, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  clear_error();
  if (!n_fg || !workspace) return fail(GC_ERR_ARG, "foreground index: null n_fg or workspace");
  int64_t n_tokens = 0;
  TileOrder order;
  const int rc = check_views(n_views, H, W, "foreground index", &n_tokens, &order);
  if (rc) return rc;
  if (n_tokens > 0 && (!pos || !fg_bits || !fg_recs)) return fail(GC_ERR_ARG, "foreground index: null pointer");
  if ((pos && !aligned16(pos)) || (fg_bits && !aligned16(fg_bits)) || (fg_recs && !aligned16(fg_recs)) ||
      !aligned16(workspace))
    return fail(GC_ERR_ALIGN, "foreground index: pointers must be 16-byte aligned");
  if (workspace_bytes < gc_index_workspace_bytes(n_tokens))
    return fail(GC_ERR_CAPACITY, "foreground index: workspace of %zu bytes is below the %zu required", workspace_bytes,
                gc_index_workspace_bytes(n_tokens));
  const int64_t n_words = (n_tokens + 31) / 32;
  const size_t np = (size_t)n_tokens * 12, nr = (size_t)n_tokens * 16, nbits = (size_t)n_words * 4;
  if (overlaps(fg_bits, nbits, pos, np) || overlaps(fg_recs, nr, pos, np) || overlaps(fg_recs, nr, fg_bits, nbits) ||
      overlaps(n_fg, 4, fg_recs, nr) || overlaps(n_fg, 4, fg_bits, nbits) || overlaps(n_fg, 4, pos, np) ||
      overlaps(workspace, workspace_bytes, pos, np) || overlaps(workspace, workspace_bytes, fg_recs, nr) ||
      overlaps(workspace, workspace_bytes, fg_bits, nbits) || overlaps(workspace, workspace_bytes, n_fg, 4))
    return fail(GC_ERR_ALIAS, "foreground index: buffers overlap");
  const int64_t nb = n_tokens > 0 ? (n_tokens + kChunk - 1) / kChunk : 0;
  int32_t* counts = static_cast<int32_t*>(workspace);
  int32_t* offsets = counts + nb;
  if (nb > 0)
    hipLaunchKernelGGL(k_index_count<ForegroundPred>, dim3((unsigned)nb), dim3(kBlock), 0, stream,
                       ForegroundPred{pos}, order, n_tokens, fg_bits, n_words, counts);
  hipLaunchKernelGGL(k_index_scan, dim3(1), dim3(kBlock), 0, stream, counts, nb, offsets, n_fg);
  if (nb > 0)
    hipLaunchKernelGGL(k_index_scatter<ForegroundPred>, dim3((unsigned)nb), dim3(kBlock), 0, stream,
                       ForegroundPred{pos}, order, n_tokens, offsets, fg_recs);
  return after_launch(stream, "gc_index_foreground");
}
