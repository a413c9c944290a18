/*
 * geocache.h -- C ABI of the MI355X (gfx950) cross-view delta-transport library.
 *
 * GeoCache ("Training-Free Acceleration of Multi-View Texture Diffusion via
 * Geometric Delta Transport") runs the denoiser on a rotating subset of anchor
 * views at a cached step and carries the anchors' per-step change in the
 * predicted clean signal x0 to every other view through a geometric
 * correspondence built from the views' position maps (Sec. 3.2).  This
 * library implements that per-step path on the GPU:
 *
 *   once per asset       gc_posmap_downsample   render-res position maps -> latent grid
 *                        gc_posmap_bbox         per-asset bbox and squared tolerance
 *                        gc_build_correspondence   G_{A->v} for one anchor set
 *                        gc_index_correspondence   visible-token index of G_{A->v}
 *                        gc_index_correspondence_noalloc   the same without a workspace argument
 *                        gc_index_foreground       foreground-token index of the position maps
 *   every cached step    gc_transport_step      Eq. 1: x0(v) = x0_prev(v) + G[dx0(A)]
 *                        gc_sampler_reconstruct sampler-consistent eps / v / velocity + x_t update
 *                        gc_transport_reconstruct  the two above fused in one pass
 *                        gc_unipc_update, gc_transport_unipc  multistep (UniPC) variant
 *                        gc_transport_step_geom, gc_transport_reconstruct_geom, gc_transport_unipc_geom
 *                                               the same with G_{A->v} computed on the fly
 *   coverage schedule    gc_coverage_pairs, gc_coverage_init, gc_coverage_update, gc_coverage_select,
 *                        gc_coverage_score, gc_schedule_refresh_due
 *                                               token staleness, adaptive anchors and refresh
 *   host schedule        gc_schedule_anchors, gc_schedule_full_steps, gc_sampler_step_times,
 *                        gc_schedule_forced_views, gc_schedule_advance_gaps
 *
 * Conventions shared by every call
 *   - Every call returns GC_OK (0) or a negative GC_ERR_* code and never
 *     throws.  gc_last_error() returns a thread-local description of the last
 *     failure on the calling thread.
 *   - All arguments are validated on the host before anything is launched, so
 *     a call that fails has no side effects on device memory.
 *   - The library never allocates, frees or copies device memory on its own:
 *     every device buffer is owned by the caller, contiguous, and passed as a
 *     plain device pointer.  Host arrays (anchor lists, sampler parameters) are
 *     read during the call only.
 *   - Device work is enqueued on the given HIP stream (0 = the null stream)
 *     and is asynchronous: nothing synchronises.  A launch failure maps to
 *     GC_ERR_HIP; faults during execution surface at the caller's next
 *     synchronisation.  With the environment variable GC_SYNC_CHECK=1 every
 *     call synchronises its stream and checks for errors before returning.
 *   - Calls keep no state between invocations and are safe to issue
 *     concurrently on different streams with disjoint outputs.
 *   - Latent tensors are NHWC per view: [B][views][H][W][C], B assets, C a
 *     multiple of 4 (at most GC_MAX_CHANNELS), stored as float32 (GC_F32) or
 *     bfloat16 (GC_BF16, round-to-nearest-even on output); arithmetic is
 *     float32.  NaN/Inf in latents is data and propagates.
 *   - Position maps are float32 [..][H][W][3] world coordinates of the surface
 *     point seen through each pixel; a pixel with any non-finite component is
 *     background.
 *   - Pointer alignment: latents, position maps, correspondence words and
 *     weights must be 16-byte aligned (GC_ERR_ALIGN otherwise).
 */
#ifndef GEOCACHE_H
#define GEOCACHE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GC_ABI_VERSION 4

/* limits */
#define GC_MAX_VIEWS 64     /* views per asset */
#define GC_MAX_ANCHORS 8    /* anchors per cached step */
#define GC_MAX_GRID 4094    /* latent H and W (12-bit packed tap coordinates) */
#define GC_MAX_CHANNELS 256 /* latent channels */
#define GC_NOALLOC_SCRATCH_BYTES (1 << 20) /* library-held scratch of gc_index_correspondence_noalloc, per GPU */

/* status codes */
#define GC_OK 0
#define GC_ERR_ARG (-1)      /* null pointer, out-of-range scalar, bad anchor list */
#define GC_ERR_SHAPE (-2)    /* inconsistent or unsupported sizes */
#define GC_ERR_DTYPE (-3)    /* unknown latent dtype */
#define GC_ERR_ALIGN (-4)    /* a device pointer is not 16-byte aligned */
#define GC_ERR_ALIAS (-5)    /* an output overlaps an input it must not overlap */
#define GC_ERR_CAPACITY (-6) /* a size exceeds a library limit */
#define GC_ERR_HIP (-7)      /* the HIP runtime reported an error */

/* latent storage types */
#define GC_F32 0
#define GC_BF16 1

/* sampler kinds and optional model-parameterisation outputs */
#define GC_DDIM 0         /* DDIM, eta = 0, linear beta schedule over T steps */
#define GC_FLOW_EULER 1   /* flow matching x = (1 - sigma) x0 + sigma eps, Euler */
#define GC_PRED_NONE 0
#define GC_PRED_EPS 1     /* DDIM: eps */
#define GC_PRED_V 2       /* DDIM: v = sqrt(abar) eps - sqrt(1 - abar) x0 */
#define GC_PRED_VEL 3     /* flow: velocity (x_t - x0) / sigma */

/* full-step rules for gc_schedule_full_steps */
#define GC_FULL_PERIODIC 0      /* steps 0, E, 2E, ... */
#define GC_FULL_HEAD_MID_TAIL 1 /* steps 0, 1, floor(S/2), S-1 */
#define GC_FULL_HEAD_TAIL_E 2   /* steps 0, 1 and the last E steps */

/*
 * A pinhole or orthographic camera (68 bytes, 4-byte aligned): the view
 * camera into which the correspondence operator projects a target token's 3D
 * point to find the anchor pixels that may see it (Sec. 3.2, correspondence
 * operator).  The paper states no camera model; these two cover its
 * renderers' perspective views and the orthographic rigs of the tests.
 * World -> camera: x_c = R * X + t, R row-major; camera axes x right, y down,
 * z forward.  Intrinsics are in latent-pixel units; pixel i spans [i, i+1).
 *   model 0 (pinhole):      u = fx * (x_c / z_c) + cx,  v = fy * (y_c / z_c) + cy,
 *                           a point with z_c <= 0 is not seen
 *   model 1 (orthographic): u = fx * x_c + cx,          v = fy * y_c + cy
 * Any other model value makes the camera see nothing.
 */
typedef struct gc_camera {
  int32_t model;
  float R[9];
  float t[3];
  float fx, fy, cx, cy;
} gc_camera;

/*
 * Sampler description (32 bytes).  kind = GC_DDIM uses T, beta_start and
 * beta_end (beta_i linear in i over 0..T-1, abar_t = prod_{i<=t}(1 - beta_i),
 * abar_{-1} = 1); kind = GC_FLOW_EULER ignores them.  pred_out selects the
 * optional model_out tensor of the reconstruction (GC_PRED_*).
 */
typedef struct gc_sampler {
  int32_t kind;
  int32_t pred_out;
  int32_t T;
  int32_t reserved;
  double beta_start;
  double beta_end;
} gc_sampler;

/* GC_ABI_VERSION of the loaded library. */
int gc_abi_version(void);

/* Description of the last error on this thread ("" if none).  The pointer is
 * valid until the next gc_* call on the same thread. */
const char* gc_last_error(void);

/*
 * Area-downsample render-resolution position maps to the latent grid.
 * Position maps supply each latent token's 3D point (Sec. 3.1, motivating
 * study; Sec. 3.2, correspondence operator); a render at f times the latent
 * resolution is reduced by averaging each f x f block over its foreground
 * samples.  A block with fewer than half foreground samples is background
 * (NaN).  The block mean is accumulated in double and rounded once to float.
 *   pos_hi   device float [n_maps][Hr][Wr][3]
 *   pos_lat  device float [n_maps][Hr/f][Wr/f][3] (output; must not overlap pos_hi)
 *   f        1..64, dividing Hr and Wr; Hr/f and Wr/f at most GC_MAX_GRID.
 */
int gc_posmap_downsample(const float* pos_hi, int64_t n_maps, int Hr, int Wr, int f, float* pos_lat,
                         hipStream_t stream);

/*
 * Per-asset bounding box and squared match tolerance.  The tolerance is
 * tol_frac (the paper uses 1%) of the bounding-box diagonal of the asset
 * (Sec. 3.2, correspondence operator); it is kept squared in float:
 *   e = max - min per axis, d2 = (ex*ex + ey*ey) + ez*ez,
 *   tol2 = (tol_frac*tol_frac) * d2.
 *   pos   device float [B][N][H][W][3] latent-grid position maps
 *   bbox  device float [B][8] output = {min x,y,z, max x,y,z, tol2, 0};
 *         an asset without a foreground sample gets all zeros.
 * 0 < tol_frac <= 1.
 */
int gc_posmap_bbox(const float* pos, int B, int N, int H, int W, float tol_frac, float* bbox,
                   hipStream_t stream);

/*
 * Build the correspondence operator G_{A->v} for every non-anchor view v of
 * every asset, for one anchor set A (Sec. 3.2: correspondence operator,
 * multi-anchor aggregation, invalid matches).  For target token p with 3D
 * point P and anchor slot s (view u = anchors[s]):
 *   - project P into camera u; the 2x2 source pixels whose centres surround
 *     the projection are the candidate taps (g = proj - 0.5, (x0, y0) =
 *     floor(g), taps k = 0..3 at (x0 + (k&1), y0 + (k>>1)));
 *   - a tap is valid if on the grid, foreground and |Q - P|^2 <= tol2
 *     (the per-tap visibility/occlusion test);
 *   - keep the K valid taps nearest in 3D (ties: lower k);
 *   - weights are the taps' overlap areas with a unit pixel centred on the
 *     projection (bilinear weights), renormalised over the kept taps; if all
 *     kept areas are zero the nearest kept tap gets 1; zero-weight taps are
 *     dropped; finally every anchor that sees p is divided by n_vis, the
 *     number of such anchors, so each visible row sums to 1 and rows no
 *     anchor sees are zero.
 * All projection and distance arithmetic is IEEE float in a fixed order.
 *   pos      device float [B][N][H][W][3]
 *   cams     device gc_camera [B][N]
 *   anchors  host int32 [a]: distinct views in [0, N); slot s = position in the list
 *   a        1..min(N, GC_MAX_ANCHORS); a == N is legal and produces empty outputs
 *   K        taps kept per anchor, 1..4
 *   bbox     device float [B][8] from gc_posmap_bbox (only tol2 is read)
 *   corr     device int32 [B][N-a][H][W][a] output, target views in ascending
 *            view order: word = (x0+1) | (y0+1) << 12 | mask << 24, mask bit k
 *            set for each kept tap; 0 iff anchor s contributes nothing
 *   weights  device float [B][N-a][H][W][a][K] output, written for the pairs
 *            whose word is non-zero: final weight of the j-th tap set in the
 *            word (ascending k), 0 beyond.  The weights of a pair whose word is
 *            0 are not written (no transport call reads them), so the buffer
 *            keeps whatever it held there.
 *   stats    nullable device uint32 [B][4] output (zeroed by the call):
 *            {visible (pixel, anchor) pairs, target pixels seen by >= 1 anchor,
 *             foreground target pixels, kept taps}
 * H, W at most GC_MAX_GRID; N at most GC_MAX_VIEWS.
 */
int gc_build_correspondence(const float* pos, const gc_camera* cams, int B, int N, int H, int W,
                            const int32_t* anchors, int a, int K, const float* bbox, int32_t* corr,
                            float* weights, uint32_t* stats, hipStream_t stream);

/*
 * Visible-token index of a correspondence operator (once per asset and
 * anchor set).  A token's row of G_{A->v} is non-zero iff at least one anchor
 * sees it (Sec. 3.2: a token with no tap inside the tolerance has an all-zero
 * row).  The index lets the per-step calls split their work: the visible
 * tokens, listed compactly, get the gathering; every other token is streamed
 * and recognised by one bit instead of its a correspondence words.
 *   corr       device int32 [n_views][H][W][a] words from gc_build_correspondence,
 *              n_views = B * (N - a); n_tokens = n_views * H * W is at most
 *              2^31 - 1, and token i is (view i / (H W), row, column)
 *   vis_bits   device uint32 [ceil(n_tokens / 32)] output: bit (i & 31) of word
 *              i >> 5 is set iff token i has a non-zero word
 *   vis_list   device int32 [n_tokens] output (capacity): the first *n_vis
 *              entries are the visible token indices in tile order: view by
 *              view, and inside a view by 16 x 16 tiles of the grid (bands of
 *              16 rows from the top, tiles from the left, the last band and
 *              column of tiles shorter or narrower when H or W is not a
 *              multiple of 16), row-major inside a tile.  A block of the
 *              step's gather part then holds a compact patch of a view, whose
 *              anchor taps share cache lines.
 *   n_vis      device int32 [1] output
 *   workspace  device scratch of at least gc_index_workspace_bytes(n_tokens)
 *              bytes, owned by the caller; its contents are not meaningful
 *              after the call and calls sharing one workspace must not overlap
 * The result is deterministic.  n_views = 0 is legal (n_vis = 0); H, W >= 1.
 */
size_t gc_index_workspace_bytes(int64_t n_tokens);
int gc_index_correspondence(const int32_t* corr, int64_t n_views, int H, int W, int a, uint32_t* vis_bits,
                            int32_t* vis_list, int32_t* n_vis, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/*
 * gc_index_correspondence without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  The per-chunk counts and offsets
 * go to a scratch array of GC_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends (its address is looked up once
 * per device, on the first call with that device current); the call itself
 * allocates nothing.  Arguments, outputs and result are those of
 * gc_index_correspondence; the current device must be the one that owns the
 * buffers and the stream.  n_tokens is at most 134217728 (the scratch holds
 * 2 * ceil(n_tokens / 1024) int32); larger counts fail with GC_ERR_CAPACITY
 * before anything is launched.  Every call on one GPU shares that GPU's
 * scratch: calls that overlap in time on one GPU (concurrent streams or host
 * threads) race and must be serialised by the caller.  The scratch keeps the
 * last call's contents; every call writes all of the part it reads, so
 * nothing has to be cleared between calls.
 */
int gc_index_correspondence_noalloc(const int32_t* corr, int64_t n_views, int H, int W, int a, uint32_t* vis_bits,
                                    int32_t* vis_list, int32_t* n_vis, hipStream_t stream);

/*
 * Foreground index of latent-grid position maps (once per asset batch; it
 * does not depend on the anchor set).  Only a token with a finite position
 * can pass the operator's tolerance test (Sec. 3.2: the test compares 3D
 * points), so the on-the-fly step (gc_transport_*_geom) can evaluate the
 * operator for the listed tokens only and stream every other one.
 *   pos        device float32 [n_views][H][W][3], n_views = B * N; n_tokens =
 *              n_views * H * W is at most 2^31 - 1; a token is foreground iff
 *              its three components are finite
 *   fg_bits    device uint32 [ceil(n_tokens / 32)] output: bit (i & 31) of
 *              word i >> 5 is set iff token i is foreground
 *   fg_recs    device int32 [n_tokens][4] output (capacity): the first *n_fg
 *              records are {i, x, y, z} for the foreground tokens i in the
 *              tile order of gc_index_correspondence, x, y, z being the
 *              position's float bit patterns
 *   n_fg       device int32 [1] output
 *   workspace  device scratch of at least gc_index_workspace_bytes(n_tokens)
 *              bytes, as for gc_index_correspondence
 * All pointers 16-byte aligned; outputs must not overlap pos or each other.
 * The result is deterministic.  n_views = 0 is legal (n_fg = 0); H, W >= 1.
 */
int gc_index_foreground(const float* pos, int64_t n_views, int H, int W, uint32_t* fg_bits, int32_t* fg_recs,
                        int32_t* n_fg, void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Delta transport, Eq. 1 (Sec. 3.2, delta transport and loop order), for one
 * cached step:
 *   anchor view u = anchors[s]:  x0_out(u) = x0_anchor_new(s)          (copy)
 *   other view v:  x0_out(v) = x0_prev(v) + sum_s sum_k w * (x0_anchor_new(s)[q] - x0_prev(u)[q])
 * accumulated in float (anchors in slot order, taps in ascending k), added to
 * x0_prev(v) and rounded to the storage dtype.  Tokens no anchor sees are a
 * bit copy of x0_prev(v).
 *   x0_prev        device [B][N][H][W][C]  stored x0 of the previous step, all views
 *   x0_anchor_new  device [B][a][H][W][C]  this step's anchor predictions, slot order
 *   corr, weights  as written by gc_build_correspondence for the same anchor list, B, N, H, W, K
 *   vis_bits, vis_list, n_vis
 *                  optional index of corr from gc_index_correspondence (n_vis
 *                  read back to the host); both null for the plain launch.
 *                  With the index the visible tokens are processed by their own
 *                  blocks; the result is bit-identical either way.  The index
 *                  needs n_vis * CV <= 2^31 - 2048, CV being the channel
 *                  vectors per token (C/4 for float32; C/8 for bfloat16 when 8
 *                  divides C, else C/4); larger counts fail with GC_ERR_CAPACITY.
 *                  A step with fewer than 2^18 work items (B*(N-a)*H*W
 *                  target tokens times CV) validates the index and then takes the plain
 *                  launch, which is faster at that size; the environment
 *                  variable GC_SPLIT_MIN_ITEMS, read once per process, moves
 *                  that bound (0: every indexed step takes the split launch).
 *   x0_out         device [B][N][H][W][C]  output; must not overlap x0_prev or x0_anchor_new
 */
int gc_transport_step(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr,
                      const float* weights, const uint32_t* vis_bits, const int32_t* vis_list, int64_t n_vis,
                      int B, int N, int H, int W, int C, const int32_t* anchors, int a, int K, int dtype,
                      void* x0_out, hipStream_t stream);

/*
 * Sampler-consistent reconstruction (Sec. 3.2, after Eq. 1): from x0 and the
 * current state x_t at the step's noise level, recover the sampler's own
 * quantities by the closed forms and take the sampler step.  Elementwise over
 * n_elems values, float32 arithmetic with coefficients computed on the host in
 * double and rounded once to float.
 *   GC_DDIM (eta = 0; t, t_next integer timesteps, t_next = -1 for the end):
 *     eps = (x_t - sqrt(abar_t) x0) / sqrt(1 - abar_t)
 *     x_next = sqrt(abar_n) x0 + sqrt(1 - abar_n) eps
 *     model_out = eps (GC_PRED_EPS) or sqrt(abar_t) eps - sqrt(1 - abar_t) x0 (GC_PRED_V)
 *   GC_FLOW_EULER (t = sigma_t in (0, 1], t_next = sigma_n in [0, t]):
 *     vel = (x_t - x0) / sigma_t,  x_next = x_t + (sigma_n - sigma_t) vel
 *     model_out = vel (GC_PRED_VEL)
 *   x_t, x0    device [n_elems]
 *   x_next     device [n_elems] output; may be x_t itself (in place), must not
 *              otherwise overlap x_t or x0
 *   model_out  nullable device [n_elems] output (required iff pred_out != GC_PRED_NONE)
 *   n_elems    a multiple of 4
 */
int gc_sampler_reconstruct(const void* x_t, const void* x0, void* x_next, void* model_out,
                           int64_t n_elems, int dtype, const gc_sampler* smp, double t, double t_next,
                           hipStream_t stream);

/*
 * gc_transport_step followed by gc_sampler_reconstruct over all B*N views, in
 * one pass (one read of every input, one write of every output): the cached
 * step of the loop order (Sec. 3.2: transport the anchors' increment, then
 * reconstruct every view for the sampler) as one multi-view, multi-asset
 * kernel, the remedy the paper names for a loop that has become launch-bound
 * (Sec. 5, limitations).  The
 * optional index (vis_bits, vis_list, n_vis) is as for gc_transport_step.  The
 * reconstruction consumes x0_out as stored (rounded to the dtype), so the
 * result is bit-identical to the two separate calls.
 *   x_t        device [B][N][H][W][C]
 *   x0_out     device [B][N][H][W][C] output (the next step's x0_prev)
 *   x_next     device [B][N][H][W][C] output; may be x_t itself
 *   model_out  nullable device [B][N][H][W][C] output
 * x0_out, x_next and model_out must not overlap x0_prev, x0_anchor_new or each
 * other (x_next == x_t excepted).
 */
int gc_transport_reconstruct(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr,
                             const float* weights, const uint32_t* vis_bits, const int32_t* vis_list,
                             int64_t n_vis, const void* x_t, int B, int N, int H, int W, int C,
                             const int32_t* anchors, int a, int K, int dtype, const gc_sampler* smp,
                             double t, double t_next, void* x0_out, void* x_next, void* model_out,
                             hipStream_t stream);

/*
 * Multistep (UniPC) sampler-consistent update.
 * The reconstruction keeps the solver's history in the parameterisation it
 * expects (Sec. 3.2, after Eq. 1).  For a multistep solver in data
 * prediction -- UniPC with B(h) = expm1(h) (Zhao et al. 2023), the solver of
 * the paper's headline operating point -- that history is the x0 of earlier
 * steps, i.e. the x0 store: at a cached step the transported x0 of every
 * view enters it directly.  One step k of an S-step trajectory on the DDIM
 * noise schedule (alpha = sqrt(abar), sigma = sqrt(1 - abar), trailing
 * timesteps, sigma = 0 after the last step) is linear in its inputs:
 *   corrector (use_corrector):  x_c = c_xprev x_prev + c_mk2 m_{k-2} + c_mk1 m_{k-1} + c_mk m_k
 *   otherwise:                  x_c = x_cur
 *   predictor:                  x_next = p_xc x_c + p_mk1 m_{k-1} + p_mk m_k
 * with m_j the x0 of step j, x_prev the corrected sample of step k-1 and
 * x_cur the sample step k starts from.  Orders: first order at step 0 and on
 * the last step, otherwise min(order, 2); the corrector uses the previous
 * step's predictor order.  gc_unipc_coeffs computes the coefficients on the
 * host in double; the kernels round them once to float.
 */
typedef struct gc_unipc_step {
  int32_t use_corrector;
  int32_t corrector_order;
  int32_t predictor_order;
  int32_t reserved;
  double c_xprev, c_mk2, c_mk1, c_mk;
  double p_xc, p_mk1, p_mk;
} gc_unipc_step;

/* smp: a GC_DDIM sampler (its T and betas define the schedule); order 1 or 2;
 * corrector 0/1. */
int gc_unipc_coeffs(const gc_sampler* smp, int S, int k, int order, int corrector, gc_unipc_step* out);

/*
 * The update over n_elems values (a full step: x0 of every view given).
 *   x_cur   device [n] (required iff !use_corrector)
 *   x_prev  device [n] (required iff use_corrector)
 *   m_km2, m_km1  device [n], required iff a coefficient of theirs is non-zero
 *   m_k     device [n]
 *   x_c     device [n] output (the next step's x_prev); may be x_prev itself
 *   x_next  device [n] output; may be x_cur itself
 * n_elems a multiple of 4; other outputs must not overlap any input.
 */
int gc_unipc_update(const void* x_cur, const void* x_prev, const void* m_km2, const void* m_km1, const void* m_k,
                    int64_t n_elems, int dtype, const gc_unipc_step* st, void* x_c, void* x_next,
                    hipStream_t stream);

/*
 * A cached step with the UniPC update, fused: gc_transport_step (m_k =
 * x0_out, m_{k-1} = x0_prev) followed by gc_unipc_update over all B*N views
 * in one pass.  Arguments as for gc_transport_step and gc_unipc_update; all
 * latents [B][N][H][W][C].  x_c may be x_prev, x_next may be x_cur.
 */
int gc_transport_unipc(const void* x0_prev, const void* x0_anchor_new, const int32_t* corr, const float* weights,
                       const uint32_t* vis_bits, const int32_t* vis_list, int64_t n_vis, const void* x_cur,
                       const void* x_prev, const void* m_km2, int B, int N, int H, int W, int C,
                       const int32_t* anchors, int a, int K, int dtype, const gc_unipc_step* st, void* x0_out,
                       void* x_c, void* x_next, hipStream_t stream);

/*
 * Cached step with the correspondence computed on the fly (Sec. 3.2: the
 * operator is a function of the position maps and cameras only).  Instead of
 * a stored G_{A->v}, the kernel projects every target token into the anchor
 * cameras and runs the
 * same tap test, selection and weighting as gc_build_correspondence, then
 * applies Eq. 1 (and, for the _reconstruct variant, the sampler step).  The
 * outputs equal gc_build_correspondence + gc_transport_step (+ the sampler
 * step of gc_transport_reconstruct) bit for bit.  Nothing is built or stored
 * per anchor set, which suits anchor sets that do not repeat; the stored
 * operator with its index is cheaper per step when they do.
 *   pos    device float32 [B][N][H][W][3] latent-grid position maps (NaN = background)
 *   cams   device gc_camera [B][N]
 *   bbox   device float32 [B][8] from gc_posmap_bbox (element 6 = squared tolerance)
 *   fg_bits, fg_recs, n_fg
 *          optional foreground index of pos from gc_index_foreground (n_fg
 *          read back to the host); fg_bits and fg_recs null and n_fg 0 for the
 *          blocked launch.  With the index, only the listed tokens of the
 *          target views run the operator and every other token is streamed;
 *          the result is bit-identical either way.  The index must be the one
 *          built from these position maps: a target token whose bit is set is
 *          written only through its record.  A record whose token lies
 *          outside [0, B*N*H*W) is ignored.  The index is used when B * a <= 64
 *          (the launch stages every (asset, anchor) camera); otherwise the
 *          blocked launch runs.  It needs n_fg <= 2^31 - 2048 / G, G being
 *          the channel vectors per token (as for gc_transport_step) rounded
 *          up to a power of two, at most 8; larger counts fail with
 *          GC_ERR_CAPACITY.
 * Other arguments as for gc_transport_step / gc_transport_reconstruct.
 * x0_out, x_next and model_out must not overlap any input (x_next may be
 * x_t); latents, pos, fg_bits and fg_recs 16-byte aligned.
 */
int gc_transport_step_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos, const gc_camera* cams,
                           const float* bbox, const uint32_t* fg_bits, const int32_t* fg_recs, int64_t n_fg, int B,
                           int N, int H, int W, int C, const int32_t* anchors, int a, int K, int dtype, void* x0_out,
                           hipStream_t stream);
int gc_transport_reconstruct_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos,
                                  const gc_camera* cams, const float* bbox, const uint32_t* fg_bits,
                                  const int32_t* fg_recs, int64_t n_fg, const void* x_t, int B, int N, int H, int W,
                                  int C, const int32_t* anchors, int a, int K, int dtype, const gc_sampler* smp,
                                  double t, double t_next, void* x0_out, void* x_next, void* model_out,
                                  hipStream_t stream);

/*
 * The multistep variant of the on-the-fly step: Eq. 1 with G_{A->v} computed
 * on the fly, then the UniPC corrector + predictor on the x0 history
 * (gc_transport_unipc's update), in one pass.  Equals gc_build_correspondence
 * + gc_transport_unipc bit for bit.  Arguments as for gc_transport_unipc and
 * gc_transport_reconstruct_geom: m_{k-1} is x0_prev; x_c may be x_prev and
 * x_next may be x_cur, no other output may overlap an input or another
 * output.
 */
int gc_transport_unipc_geom(const void* x0_prev, const void* x0_anchor_new, const float* pos, const gc_camera* cams,
                            const float* bbox, const uint32_t* fg_bits, const int32_t* fg_recs, int64_t n_fg,
                            const void* x_cur, const void* x_prev, const void* m_km2, int B, int N, int H, int W,
                            int C, const int32_t* anchors, int a, int K, int dtype, const gc_unipc_step* st,
                            void* x0_out, void* x_c, void* x_next, hipStream_t stream);

/*
 * Token staleness and the coverage-driven schedule.
 * A token no anchor sees keeps its state and misses that step's denoising
 * until the next full step (Sec. 3.2, invalid matches); the paper's
 * limitations section names adaptive anchor selection and visibility-aware
 * refresh as the remedy for regions few anchors observe but defines neither.
 * This library's reading:
 *   staleness  uint8 per token [B][N][H][W]: consecutive steps without a fresh
 *              prediction (its view an anchor, or a full step) or a
 *              transported increment (some anchor of the step sees it),
 *              saturating at 254; 255 marks background (non-finite position)
 *              and is never counted;
 *   selection  greedy weighted maximum coverage: view u covers token (b, v, p)
 *              when v = u or anchor u sees it; an uncovered foreground token
 *              weighs 1 + its staleness.  Forced views are taken first, then
 *              the view with the largest gain (ties: the lower view) until a
 *              views are chosen; the set is written in ascending order;
 *   refresh    a full step is due when, over all assets and views, the tokens
 *              with staleness >= R exceed the fraction tau of the foreground.
 * Visibility comes from single-anchor pairs: bit (u, b, v, p) is set when
 * anchor u alone has an in-tolerance tap for token p of view v -- the tap
 * test of gc_build_correspondence, which examines each anchor on its own, so
 * a set sees a token iff one of its anchors does.
 *
 * gc_coverage_pair_words: uint32 words of the pair bits, N * B * N * ceil(H*W/32);
 *   layout [u][b][v][ceil(H*W/32)], token p at bit p % 32 of word p / 32, the
 *   bits of view u in row (u, b, u) zero.  The update, selection and scoring
 *   calls read neither the padding bits past H*W nor the rows (u, b, u) (a
 *   view covers its own tokens), so other producers may leave them unset.
 * gc_coverage_pairs: pos [B][N][H][W][3], cams device gc_camera [B][N], bbox
 *   device [B][8] (gc_posmap_bbox) -> pair_bits (once per asset batch).
 * gc_coverage_init: staleness 0 for foreground tokens, 255 for background.
 * gc_coverage_update: one step with the anchor set anchors (host [a]; all N
 *   views for a full step) -> staleness updated in place and stats
 *   (device uint32 [B][N][4]: foreground tokens, tokens with staleness >= R,
 *   sum and maximum of the staleness), recomputed by the call.
 * gc_coverage_select: the anchor set of the next cached step, written to
 *   anchors_out (device int32 [a], ascending); forced: host [n_forced] views
 *   that must be in it.  a <= GC_MAX_ANCHORS.  workspace: caller-owned device
 *   memory of gc_coverage_workspace_bytes(), 16-byte aligned, any contents;
 *   it holds the coverage histogram (or per-block partial gains), so
 *   concurrent calls need separate workspaces.  With N <= 12 it enqueues two
 *   launches whatever a is: one that clears the histogram, then the pass over
 *   the tokens that builds it -- the weights 1 + staleness summed per cover
 *   mask (the token's own view and the views that see it) -- whose last block
 *   takes its subset sums Y and runs every round, the gain of u given the
 *   chosen set S being Y[all \ S] - Y[all \ (S + u)]; with more views,
 *   2 (a - n_forced) launches.  One launch when every view is forced.  Never
 *   synchronises.
 * gc_coverage_score: scores (device uint64 [M], overwritten) = the weighted
 *   coverage, sum of 1 + staleness over the foreground tokens it covers, of
 *   each candidate set sets (host int32 [M][a]); M <= 64.  workspace as for
 *   gc_coverage_select.  Choosing the rotation's set with the largest score
 *   keeps the rotation's evenly spread anchors while following where the
 *   stale tokens are.  With N <= 12 a set's score is Y[all] - Y[all \ S]
 *   from the same histogram (two launches).
 * gc_coverage_update_select: gc_coverage_update with anchors, a, R, stale,
 *   stats, then gc_coverage_select of a_next views (forced, n_forced,
 *   anchors_out, workspace) on the updated staleness -- the end of one step
 *   and the choice for the next in one pass over the tokens when N <= 12
 *   (two launches; the statistics are summed with integer atomics, so the
 *   result is the same as the two calls').  With more views, the two calls'
 *   launches.  stats must not overlap the workspace or anchors_out.
 * gc_coverage_update_score: gc_coverage_update, then gc_coverage_score of
 *   the M sets of a_set views on the updated staleness, fused as above.
 * gc_schedule_refresh_due: host; stats as written by gc_coverage_update and
 *   copied to the host; *due = 1 when a full step is due.
 */
int64_t gc_coverage_pair_words(int B, int N, int H, int W);
int gc_coverage_pairs(const float* pos, const gc_camera* cams, const float* bbox, int B, int N, int H, int W,
                      uint32_t* pair_bits, hipStream_t stream);
int gc_coverage_init(const float* pos, int B, int N, int H, int W, uint8_t* stale, hipStream_t stream);
int gc_coverage_update(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a, int R,
                       uint8_t* stale, uint32_t* stats, hipStream_t stream);
size_t gc_coverage_workspace_bytes(void);
int gc_coverage_select(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, int a,
                       const int32_t* forced, int n_forced, int32_t* anchors_out, void* workspace, size_t ws_bytes,
                       hipStream_t stream);
int gc_coverage_score(const uint32_t* pair_bits, const uint8_t* stale, int B, int N, int H, int W, const int32_t* sets,
                      int M, int a, uint64_t* scores, void* workspace, size_t ws_bytes, hipStream_t stream);
int gc_coverage_update_select(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a,
                              int R, uint8_t* stale, uint32_t* stats, int a_next, const int32_t* forced, int n_forced,
                              int32_t* anchors_out, void* workspace, size_t ws_bytes, hipStream_t stream);
int gc_coverage_update_score(const uint32_t* pair_bits, int B, int N, int H, int W, const int32_t* anchors, int a,
                             int R, uint8_t* stale, uint32_t* stats, const int32_t* sets, int M, int a_set,
                             uint64_t* scores, void* workspace, size_t ws_bytes, hipStream_t stream);
int gc_schedule_refresh_due(const uint32_t* stats, int B, int N, double tau, int* due);

/*
 * Anchor gaps of the coverage-driven schedule (host; no device work).  The
 * limitations section (Sec. 5) names adaptive anchor selection as the remedy
 * for regions few anchors observe; a purely greedy choice can starve a view,
 * so a caller may force views whose gap -- cached steps since the view was
 * last an anchor (or predicted by a full step) -- reached max_gap, as
 * gc_coverage_select's forced list.
 * gc_schedule_forced_views: gap host int32 [N] (>= 0); writes to forced_out
 *   (host int32, room for a) the views with gap >= max_gap, the longest gap
 *   first, equal gaps in ascending view order, at most a of them, and their
 *   number to *n_forced.  max_gap = 0 forces nothing.
 * gc_schedule_advance_gaps: gap host int32 [N], updated in place after a step
 *   whose denoiser predicted views[0..n_views): those views (every view when
 *   full != 0) go to 0, the others grow by one (saturating at INT32_MAX).
 */
int gc_schedule_forced_views(const int32_t* gap, int N, int a, int max_gap, int32_t* forced_out, int* n_forced);
int gc_schedule_advance_gaps(int32_t* gap, int N, const int32_t* views, int n_views, int full);

/*
 * Host schedule (no device work).
 *
 * gc_schedule_anchors: anchors of cached step c (Sec. 3.2, batch-sliced anchor
 * forward: anchors rotate every step and each view returns to the anchor set
 * within ceil(N/a) steps): A_c = {(c + floor(j*N/a)) mod N : j < a}, written
 * in ascending view order to anchors_out[a].
 *
 * gc_schedule_full_steps: is_full_out[k] = 1 for the full-view steps of an
 * S-step trajectory (Sec. 3.2, drift-bounding schedule; Sec. 4.1,
 * configurations): GC_FULL_PERIODIC every E-th step, GC_FULL_HEAD_MID_TAIL
 * steps {0, 1, floor(S/2), S-1}, GC_FULL_HEAD_TAIL_E steps {0, 1} and the last
 * E steps (E full-view refresh steps at the end, 0 <= E <= S).  Step 0 is
 * always full.
 *
 * gc_sampler_step_times: (t, t_next) of step k of an S-step trajectory.
 * DDIM: trailing timesteps t_k = round((S-k) T / S) - 1 and t_S = -1.
 * Flow: sigma_k = 1 - k/S.
 *
 * gc_sampler_alpha_bar: abar_t of the DDIM schedule (1 for t = -1).
 */
int gc_schedule_anchors(int N, int a, int64_t c, int32_t* anchors_out);
int gc_schedule_full_steps(int rule, int S, int E, uint8_t* is_full_out);
int gc_sampler_step_times(const gc_sampler* smp, int S, int k, double* t, double* t_next);
int gc_sampler_alpha_bar(const gc_sampler* smp, int t, double* abar);

#ifdef __cplusplus
}
#endif

#endif /* GEOCACHE_H */
