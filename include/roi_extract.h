/*
 * roi_extract.h -- C ABI of the MI355X multi-level RoIAlign library.
 *
 * The operator is the RoIExtractor of MMDetection (arXiv 1906.07155, §3.1, model
 * representation): the features of each RoI are pooled from one level of an FPN
 * feature pyramid (§3.1, Neck), the level matched to the RoI's size, by a RoI
 * pooling operator, here RoIAlign (the Mask R-CNN operator, cited among the
 * supported frameworks in §2).  The paper runs these bbox and mask operations on
 * the GPU (§1) and trains with a forward and a backward every iteration (§3.2).
 *
 * Conventions (the paper leaves them open; these are the library's definitions):
 *   - RoI k is 5 binary32 values (batch_index, x1, y1, x2, y2) in input-image
 *     pixels.  batch_index is truncated toward zero; a RoI whose batch index or
 *     level index is outside the valid range yields zeros and no gradient.
 *   - Level rule (threshold form of the FPN rule floor(log2(sqrt(wh)/s0))):
 *     level = #{ j in 1..L-1 : (x2-x1)*(y2-y1) >= (s0*2^j)^2 }, every product and
 *     difference rounded to binary32, s0 = finest_scale (56 for P2..P5); the _ex
 *     entry points can measure boxes in whole pixels instead (RE_BOX_PIXELS).
 *   - On level l with scale s, H x W map, output PH x PW, sampling ratio S:
 *       off = aligned ? 0.5 : 0
 *       x0 = x1*s - off,  xe = x2*s - off,  rw = xe - x0 (>= 1 if !aligned)
 *       bw = rw / PW;     gw = S > 0 ? S : min(ceil(bw), 64)   (same for y)
 *       sample (pw, ix):  x = (x0 + pw*bw) + ((ix + 0.5)*bw) / gw
 *     each operation rounded to binary32 in that order (no fused multiply-add).
 *     A sample with y < -1, y > H, x < -1 or x > W contributes zero; otherwise
 *     y = max(y, 0), yl = (int)y, yh = yl + 1, and if yl >= H-1 then
 *     yl = yh = H-1 and y = yl; ly = y - yl, hy = 1 - ly (same for x).
 *       out[k,c,ph,pw] = (1/count) * sum over samples of
 *           hy*hx*F[yl,xl] + hy*lx*F[yl,xh] + ly*hx*F[yh,xl] + ly*lx*F[yh,xh],
 *       count = max(gh*gw, 1)   (invalid samples are counted).
 *   - Backward is the exact transpose: grad_F[b,c,y*,x*] += g[k,c,ph,pw]*w/count
 *     for every valid sample and corner, summed in fp32 either by atomics (scatter)
 *     or per output tile (gather); the summation order, hence the last bits, may
 *     vary between runs and algorithms.
 *
 * Ownership and execution: the caller owns every buffer; all data pointers are
 * device pointers except the re_level_t arrays, which are read on the host during
 * the call.  Calls enqueue work on `stream` (a hipStream_t; NULL = the null
 * stream) and return without synchronizing.  The library never allocates device
 * memory and keeps no state between calls (one exception: roi_align_fwd_noalloc keeps
 * its plan in a fixed array of the library's device code, see there).  Argument
 * errors are detected on the
 * host before anything is enqueued; a launch failure is reported as
 * RE_ERR_DEVICE.  Device-side content (RoI coordinates, level indices, plan
 * contents) is never reported as an error: out-of-range values are clamped or
 * skipped so every memory access stays inside the buffers described here.
 */
#ifndef ROI_EXTRACT_H
#define ROI_EXTRACT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RE_OK = 0,
    RE_ERR_INVALID_ARG = 1,   /* null pointer, bad shape/stride/dtype/size/scale */
    RE_ERR_UNSUPPORTED = 2,   /* valid request this build does not implement */
    RE_ERR_WORKSPACE = 3,     /* workspace missing or too small */
    RE_ERR_DEVICE = 4         /* a HIP call or kernel launch failed */
} re_status_t;

typedef enum {
    RE_DTYPE_F32 = 0,         /* IEEE binary32 */
    RE_DTYPE_BF16 = 1         /* bfloat16; results are rounded to nearest-even */
} re_dtype_t;

#define RE_MAX_LEVELS 8
#define RE_MAX_OUT 256        /* largest out_h / out_w */
#define RE_MAX_SAMPLING 64    /* largest sampling_ratio; also the adaptive-grid cap */

/* One pyramid level: a logically NCHW tensor [n, c, h, w] with element strides.
 * stride_c == 1 (channels-last, e.g. a PyTorch channels_last tensor) selects the
 * fast path with channel-contiguous loads; any other non-negative strides are
 * accepted and served by a general kernel.  Every level of a pyramid has the same
 * n, c and dtype.  `data` must be aligned to its element size. */
typedef struct {
    void *data;
    int32_t dtype;            /* re_dtype_t */
    int32_t reserved;         /* must be 0 */
    int64_t n, c, h, w;
    int64_t stride_n, stride_c, stride_h, stride_w;
    float spatial_scale;      /* feature pixels per input pixel, e.g. 1/4 for P2 */
    float reserved2;          /* must be 0 */
} re_level_t;

/* a1 -- FPN level of every RoI (§3.1: each RoI is pooled from the pyramid level
 * that matches its size).  rois: device float[num_rois][5]; levels_out: device
 * int32[num_rois], written with values in [0, num_levels).  num_levels in
 * [1, RE_MAX_LEVELS]; finest_scale finite and > 0.  num_rois == 0 is a no-op. */
re_status_t fpn_level_map(const float *rois, int64_t num_rois, int32_t num_levels,
                          float finest_scale, int32_t *levels_out, void *stream);

/* Box conventions of the level rule (the paper does not fix one; the legacy
 * detectors of its era, e.g. Fast R-CNN and the first MMDetection releases, §2,
 * measured boxes in whole pixels):
 *   RE_BOX_CONTINUOUS  sides x2 - x1, y2 - y1 (the default above);
 *   RE_BOX_PIXELS      boxes are inclusive pixel ranges: sides (x2 - x1) + 1 and
 *                      (y2 - y1) + 1, the difference rounded to binary32 first.
 * Only the level rule changes; the sampling geometry is chosen by `aligned`. */
#define RE_BOX_CONTINUOUS 0
#define RE_BOX_PIXELS 1

/* a1 with a box convention: as fpn_level_map, the sides measured by box_convention
 * (RE_BOX_CONTINUOUS or RE_BOX_PIXELS; anything else is RE_ERR_INVALID_ARG, nothing
 * enqueued). */
re_status_t fpn_level_map_ex(const float *rois, int64_t num_rois, int32_t num_levels,
                             float finest_scale, int32_t box_convention, int32_t *levels_out,
                             void *stream);

/* Workspace of the launch plan (a1 + a2, §3.1: the per-level extraction).
 * Bytes of device workspace a plan for num_rois RoIs over the pyramid `levels` needs
 * (host array; only n, h and w are read).  It holds the launch permutation and the
 * tile->RoI lists of the gather backward (8 bytes per RoI, 12 per bin-tile, and 4 per
 * RoI times the largest number of bin-tiles of one image-level) and the plan's own
 * counters (60 KiB).  Where that product exceeds 2^28 the plan keeps no tile lists
 * (the gather backward is then not eligible).  Host-only; writes *bytes.  (A plan needs the level shapes, not
 * only the RoI and level counts, to size its tile lists, hence the level array.) */
re_status_t roi_extract_workspace_size(const re_level_t *levels, int32_t num_levels,
                                       int64_t num_rois, size_t *bytes);

/* a1 + a2 -- the level of every RoI (written to levels_out, as by fpn_level_map)
 * and the launch plan: a permutation of the RoIs ordered by (level, image, coarse
 * spatial cell of the box centre) plus per-level offsets, stored in `workspace`; the
 * plan also lists, for every bin-tile (16 pixels or more a side) of every
 * (level, image), the RoIs whose footprint can reach it, and orders the tiles by
 * decreasing list length (used by the gather backward).  Up to 8192 RoIs (and bucket
 * and tile tables that fit one workgroup's LDS) this is one kernel launch, otherwise
 * five (all on `stream`, nothing allocated).  The forward and backward walk the RoIs in plan order,
 * so neighbouring work shares cache; any valid permutation gives the same
 * results, and RoIs with equal keys may come in any order.  The plan stays valid
 * for as long as rois, levels_out and the level shapes are unchanged, so one plan
 * serves a forward and its backward.
 *   levels: host array of num_levels descriptors (only n, h, w and spatial_scale
 *           are read);  rois: device float[num_rois][5];
 *   levels_out: device int32[num_rois];  workspace: device, at least
 *           roi_extract_workspace_size() bytes. */
re_status_t roi_extract_plan(const re_level_t *levels, int32_t num_levels,
                             const float *rois, int64_t num_rois, float finest_scale,
                             int32_t *levels_out, void *workspace, size_t workspace_bytes,
                             void *stream);

/* a1 + a2 with a box convention for the level rule (see fpn_level_map_ex); otherwise
 * as roi_extract_plan. */
re_status_t roi_extract_plan_ex(const re_level_t *levels, int32_t num_levels,
                                const float *rois, int64_t num_rois, float finest_scale,
                                int32_t box_convention, int32_t *levels_out, void *workspace,
                                size_t workspace_bytes, void *stream);

/* Copy of the plan's per-level offsets: a device int32[num_levels + 1] array
 * (offsets[l] = first position of level l in plan order; offsets[num_levels] =
 * num_rois) is written to `offsets_out` (device).  For inspection and tests. */
re_status_t roi_extract_plan_offsets(const void *workspace, size_t workspace_bytes,
                                     int64_t num_rois, int32_t num_levels,
                                     int32_t *offsets_out, void *stream);

/* Device pointer to the plan's permutation (int32[num_rois]) inside `workspace`,
 * for inspection and tests.  Host-only pointer arithmetic. */
re_status_t roi_extract_plan_perm(const void *workspace, size_t workspace_bytes,
                                  int64_t num_rois, const int32_t **perm_out);

/* a3-a5 -- RoIAlign forward: the RoIExtractor's pooling of every RoI from its level
 * (§3.1, RoIExtractor; RoIAlign is the Mask R-CNN operator of §2), computed as
 * defined under Conventions above.
 *   levels/num_levels: host array of feature levels (same n, c, dtype);
 *   rois: device float[num_rois][5];
 *   roi_levels: device int32[num_rois] (e.g. from roi_extract_plan); may be NULL
 *           only when num_levels == 1;
 *   out_h, out_w in [1, RE_MAX_OUT]; sampling_ratio in [0, RE_MAX_SAMPLING]
 *           (0 = adaptive ceil(bin size), capped at RE_MAX_SAMPLING);
 *   aligned: 0 or 1;
 *   out: device [num_rois][c][out_h][out_w], dense, of out_dtype;
 *   plan: a workspace filled by roi_extract_plan for these RoIs (RoIs are then
 *           visited in plan order), or NULL (visited in index order).
 * Writes every element of out exactly once; results do not depend on the plan. */
re_status_t roi_align_fwd(const re_level_t *levels, int32_t num_levels,
                          const float *rois, int64_t num_rois, const int32_t *roi_levels,
                          int32_t out_h, int32_t out_w, int32_t sampling_ratio,
                          int32_t aligned, void *out, int32_t out_dtype,
                          const void *plan, size_t plan_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): roi_extract_plan's level map and
 * launch order without the tile lists, then roi_align_fwd in that order, with the plan
 * kept in a fixed array of RE_NOALLOC_SCRATCH_BYTES inside the library's device code
 * instead of a caller workspace.  Nothing is allocated (no hipMalloc or hipFree, no
 * allocating library routine); each GPU the library runs on holds its own copy of the
 * array until the process ends.  The copy of the current device is used (`stream` must
 * belong to it); its address is looked up on the first call on each device.
 *   num_rois <= RE_NOALLOC_MAX_ROIS (RE_ERR_UNSUPPORTED above, nothing enqueued);
 *   levels_out: device int32[num_rois], written as by roi_extract_plan (RE_BOX_CONTINUOUS);
 *   the other arguments as roi_extract_plan and roi_align_fwd.
 * Results equal roi_align_fwd's.  Every call on one GPU shares that GPU's array (each
 * call rebuilds the plan in it), so calls that overlap on one GPU -- on two streams or
 * from two host threads -- race and must be serialised by the caller. */
#define RE_NOALLOC_MAX_ROIS 65536
#define RE_NOALLOC_SCRATCH_BYTES 589824   /* 576 KiB per GPU */
re_status_t roi_align_fwd_noalloc(const re_level_t *levels, int32_t num_levels,
                                  const float *rois, int64_t num_rois, float finest_scale,
                                  int32_t *levels_out, int32_t out_h, int32_t out_w,
                                  int32_t sampling_ratio, int32_t aligned, void *out,
                                  int32_t out_dtype, void *stream);

/* a6 -- clear the gradient pyramid (every element of every level set to +0.0), the
 * start of the scatter backward (§3.2).
 * grad_levels: host array; every level RE_DTYPE_F32. */
re_status_t roi_extract_zero_grad(const re_level_t *grad_levels, int32_t num_levels,
                                  void *stream);

/* Backward algorithms. */
#define RE_BWD_AUTO 0       /* gather when eligible, else scatter */
#define RE_BWD_SCATTER 1    /* per-RoI scatter, fp32 atomics (a7) */
#define RE_BWD_GATHER 2     /* per-tile gather, plain stores (needs a plan, gradient
                               levels whose images span less than 2^30 bytes -- channels-
                               last or contiguous NCHW alike -- out 7x7 or 14x14 with
                               sampling_ratio 2, and a plan with tile lists) */

/* a6 + a7 -- RoIAlign backward (§3.2: every training iteration runs the forward and
 * the backward of the RoIExtractor): adds the transpose of the forward applied to
 * grad_out into the gradient pyramid (clears it first when zero_init != 0).
 *   grad_out: device [num_rois][c][out_h][out_w], dense, of grad_out_dtype;
 *   grad_levels: host array of num_levels descriptors, RE_DTYPE_F32, same n, c,
 *           h, w and spatial_scale as the forward's levels;
 *   algorithm: RE_BWD_SCATTER adds every RoI's contributions with fp32 atomics, one
 *           per distinct (pixel, channel) of the RoI, after an optional clearing
 *           pass; RE_BWD_GATHER has each (8x8-pixel quadrant, 64 channels) of the
 *           pyramid sum the RoIs the plan binned to it and write every element once
 *           (no atomics; clearing is part of the same pass), which requires `plan`
 *           built by roi_extract_plan for these RoIs with levels_out == roi_levels;
 *           RE_BWD_AUTO picks gather when eligible.  RE_ERR_UNSUPPORTED if gather is
 *           requested but not eligible.  With a NaN or infinity in grad_out the
 *           scatter follows the definition exactly, while the gather may also put it
 *           on untapped pixels of the rows the RoI's bin row touches in a quadrant;
 *   other arguments as roi_align_fwd. */
re_status_t roi_align_bwd(const void *grad_out, int32_t grad_out_dtype,
                          const float *rois, int64_t num_rois, const int32_t *roi_levels,
                          int32_t out_h, int32_t out_w, int32_t sampling_ratio,
                          int32_t aligned, const re_level_t *grad_levels, int32_t num_levels,
                          int32_t zero_init, int32_t algorithm, const void *plan,
                          size_t plan_bytes, void *stream);

/* f2 -- several heads on one pyramid.  A two-stage detector extracts RoI features
 * from the same FPN levels for more than one RoIHead (§3.1: BBoxHead and MaskHead;
 * the cascaded heads of Cascade R-CNN and HTC, §2), and every head's backward adds
 * into the same gradient pyramid.  One head is one upstream gradient and the RoIs
 * it was extracted for: */
#define RE_MAX_HEADS 8
typedef struct {
    const void *grad_out;     /* device [num_rois][c][out_h][out_w] of grad_out_dtype */
    int32_t grad_out_dtype;   /* re_dtype_t */
    int32_t out_h, out_w;
    int32_t sampling_ratio;
    int32_t aligned;
    int32_t reserved;         /* must be 0 */
    const float *rois;        /* device float[num_rois][5] */
    int64_t num_rois;
    const int32_t *roi_levels;/* device int32[num_rois]; NULL only with one level */
    const void *plan;         /* roi_extract_plan workspace for these RoIs, or NULL */
    size_t plan_bytes;
} re_head_t;

/* Backward of num_heads heads (1..RE_MAX_HEADS) into one gradient pyramid:
 * grad_F += sum over heads of (head's transpose applied to its grad_out), after
 * clearing when zero_init != 0; each head is defined as for roi_align_bwd.  Heads
 * are taken in pairs: when both heads of a pair take the gather (plan, levels the
 * gather can address, 7x7 or 14x14 grid, sampling_ratio 2, one gradient dtype and one tile
 * layout), the pair is a single pass in which every gradient element is written once;
 * otherwise the heads run one after the other (gather or scatter, as roi_align_bwd
 * with RE_BWD_AUTO).  Results equal the sum of the single-head calls up to the fp32
 * summation order. */
re_status_t roi_align_bwd_multi(const re_head_t *heads, int32_t num_heads,
                                const re_level_t *grad_levels, int32_t num_levels,
                                int32_t zero_init, void *stream);

/* f2 -- the forward of several heads in one launch.  The RoIHeads of a two-stage
 * detector extract features from the same pyramid (§3.1: BBoxHead and MaskHead; the
 * cascaded stages of Cascade R-CNN and HTC, §2, extract again from refined boxes): each
 * head has its own RoIs, grid and output, and the forward of all of them is one kernel
 * launch whose workgroups are the heads' (RoI, channel slice) pairs, every head's in its
 * own plan order.  Heads on the channels-last fast path (7x7 or 14x14 grid, sampling
 * ratio 2, every level with stride_c == 1) share the launch, 14x14 heads first; with
 * fp32 features (or an odd channel count) the 7x7 and the 14x14 heads take one launch
 * each, since the 14x14 kernel's register count would lower the 7x7 heads' occupancy.
 * Other heads run one after the other as roi_align_fwd.  Results equal roi_align_fwd's
 * for every head, bit for bit. */
typedef struct {
    const float *rois;        /* device float[num_rois][5] */
    int64_t num_rois;
    const int32_t *roi_levels;/* device int32[num_rois]; NULL only with one level */
    int32_t out_h, out_w;
    int32_t sampling_ratio;
    int32_t aligned;
    void *out;                /* device [num_rois][c][out_h][out_w] of the call's out_dtype */
    const void *plan;         /* roi_extract_plan workspace for these RoIs, or NULL */
    size_t plan_bytes;
} re_fwd_head_t;

/* num_heads in [1, RE_MAX_HEADS]; levels and out_dtype as roi_align_fwd, each head's
 * fields as the arguments of roi_align_fwd. */
re_status_t roi_align_fwd_multi(const re_level_t *levels, int32_t num_levels,
                                const re_fwd_head_t *heads, int32_t num_heads, int32_t out_dtype,
                                void *stream);

/* f3 -- deformable RoI pooling (DCN) and its modulated form (DCNv2), general modules
 * of §2.  Every bin of the RoIAlign grid above is moved by a learned offset given
 * normalized to the box size, and the bin average is scaled by a learned modulation:
 *   dx = (gamma * offset[k,0,ph,pw]) * rw,  dy = (gamma * offset[k,1,ph,pw]) * rh
 *   (rw, rh: the box length on the level, as in the RoIAlign definition)
 *   sample (pw, ix):  x = ((x0 + pw*bw) + dx) + ((ix + 0.5)*bw) / gw   (y likewise)
 * each operation rounded to binary32 in that order; a sample with x or y outside
 * [-1, size] (or not a number) contributes zero but counts; cut, clamp, bilinear
 * weights and count are RoIAlign's, and
 *   out[k,c,ph,pw] = m * (sum of weighted taps) / count,  m = mask[k,ph,pw] (1 if NULL).
 * With every offset 0 and no mask this is roi_align_fwd.
 *   offset: device float[num_rois][2][out_h][out_w] (x then y);
 *   mask: device float[num_rois][out_h][out_w] or NULL;  gamma: finite;
 *   other arguments as roi_align_fwd (out of out_dtype, [num_rois][c][out_h][out_w]). */
re_status_t deform_roi_pool_fwd(const re_level_t *levels, int32_t num_levels, const float *rois,
                                int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                                int32_t out_w, int32_t sampling_ratio, int32_t aligned,
                                const float *offset, const float *mask, float gamma, void *out,
                                int32_t out_dtype, const void *plan, size_t plan_bytes,
                                void *stream);

/* f3 -- gradients of deform_roi_pool_fwd for upstream gradient g:
 *   features (added into grad_levels, cleared first when zero_init != 0):
 *     g * m / count * corner weight, for every valid sample and corner;
 *   grad_offset[k,0,ph,pw] (written) = sum over channels and valid samples of
 *     g * m / count * dV/dx * gamma * rw, where dV/dx = hy*(F[yl,xh] - F[yl,xl]) +
 *     ly*(F[yh,xh] - F[yh,xl]) for a sample not clamped along x (0 <= x and
 *     xl < W-1) and 0 for a clamped one; grad_offset[k,1] likewise along y;
 *   grad_mask[k,ph,pw] (written; NULL allowed, and required when mask is NULL) =
 *     sum over channels of g * (sum of weighted taps) / count.
 * Sums use fp32 atomics, so the last bits may vary between runs.  With a plan that
 * holds tile lists, a 7 x 7 grid, 1 or 2 samples per axis and channels-last levels,
 * the feature gradient is gathered per tile (every gradient element written once,
 * zero_init != 0 needing no separate clearing) and only the taps outside their RoI's
 * tile range are added with atomics; the plan's levels must then be roi_levels (RoIs
 * of another level are not found in the tile lists).
 *   levels: the forward's features (read);  grad_levels: binary32 levels with the
 *   features' n, c, h, w and spatial_scale;  grad_out: [num_rois][c][out_h][out_w]. */
re_status_t deform_roi_pool_bwd(const void *grad_out, int32_t grad_out_dtype,
                                const re_level_t *levels, const re_level_t *grad_levels,
                                int32_t num_levels, const float *rois, int64_t num_rois,
                                const int32_t *roi_levels, int32_t out_h, int32_t out_w,
                                int32_t sampling_ratio, int32_t aligned, const float *offset,
                                const float *mask, float gamma, int32_t zero_init,
                                float *grad_offset, float *grad_mask, const void *plan,
                                size_t plan_bytes, void *stream);

/* f1 -- RoI max pooling, the RoIPool of Fast R-CNN (a two-stage method of §2),
 * the other RoI pooling operator a RoIExtractor uses (§3.1).  On level l (scale
 * s, H x W map), every operation rounded to binary32 in this order:
 *   xs = roundf(x1*s), xe = roundf(x2*s)   (halves away from zero)
 *   len = max(xe - xs + 1, 1)              (both end pixels belong to the box)
 *   bin = len / out_w;  bin pw covers columns [floor(pw*bin) + xs, ceil((pw+1)*bin) + xs)
 *   clipped to [0, W]; rows likewise with y1, y2, out_h, H.
 * out[k,c,ph,pw] is the largest value of the bin: the pixels are scanned row by row,
 * each row left to right, and a value replaces the running maximum only if it is
 * strictly larger (so the first maximum wins and a NaN is never chosen; the running
 * maximum starts at -FLT_MAX).  argmax[k,c,ph,pw] = y*W + x of the chosen pixel.
 * An empty bin gives 0 and argmax -1; a non-empty bin without a value larger than
 * -FLT_MAX (all NaN or -inf) gives -FLT_MAX (bf16 output: the most negative finite
 * bf16) and argmax -1.  A RoI whose batch or level index is invalid gives 0 / -1.
 *   levels, rois, roi_levels, plan: as roi_align_fwd (every H*W below 2^31);
 *   out: device [num_rois][c][out_h][out_w] of out_dtype (bf16: features rounded to
 *        nearest even, so bf16 features are stored exactly);
 *   argmax: device int32 [num_rois][c][out_h][out_w].
 * Writes every element of out and argmax once; results do not depend on the plan. */
re_status_t roi_pool_fwd(const re_level_t *levels, int32_t num_levels, const float *rois,
                         int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                         int32_t out_w, void *out, int32_t out_dtype, int32_t *argmax,
                         const void *plan, size_t plan_bytes, void *stream);

/* f1 -- RoI max pooling backward: grad_F_l[b, c, argmax / W, argmax % W] +=
 * grad_out[k, c, ph, pw] for every element whose argmax is in [0, H*W) (no gradient
 * for -1).  The summation order, hence the last bits, may vary between runs.  Two
 * forms:
 *   - with a plan that holds tile lists (see roi_extract_workspace_size), a 7 x 7 grid
 *     and gradient levels whose images span less than 2^30 bytes: per tile and 64
 *     channels, the RoIs binned to the tile are added in LDS and every gradient element
 *     is written once (zero_init != 0: no separate clearing).  The plan's levels must
 *     be roi_levels (RoIs of another level are not found in the tile lists), and only
 *     an argmax inside the RoI's bins, as roi_pool_fwd writes it, is certain to be
 *     added;
 *   - otherwise the gradient pyramid is cleared first when zero_init != 0 and every
 *     element is added with an fp32 atomic.
 *   grad_out: device [num_rois][c][out_h][out_w] of grad_out_dtype;
 *   argmax: device int32, as written by roi_pool_fwd for the same RoIs and levels;
 *   grad_levels: binary32 levels with the forward's n, c, h, w;
 *   other arguments as roi_pool_fwd. */
re_status_t roi_pool_bwd(const void *grad_out, int32_t grad_out_dtype, const int32_t *argmax,
                         const float *rois, int64_t num_rois, const int32_t *roi_levels,
                         int32_t out_h, int32_t out_w, const re_level_t *grad_levels,
                         int32_t num_levels, int32_t zero_init, const void *plan,
                         size_t plan_bytes, void *stream);

/* f4 -- greedy non-maximum suppression, the step that turns a dense head's scored
 * boxes into the proposals whose RoI features the functions above extract (the paper
 * runs its bbox operations on the GPU, §1).  Boxes are ranked by score, highest first:
 * scores compare by the IEEE total order of their bits (-0 below +0), NaN ranks after
 * every number, equal scores rank by index.  In rank order a box is kept unless a kept
 * box of the same category overlaps it with IoU > iou_threshold, IoU decided in binary32
 * with one rounding per operation in this order:
 *   iw = max(min(x2a, x2b) - max(x1a, x1b), 0), ih likewise, inter = iw * ih,
 *   area = (x2 - x1) * (y2 - y1), union = (area_a + area_b) - inter, iou = inter / union
 * (a NaN IoU, e.g. of two zero-area boxes, removes nothing).  Boxes of different
 * categories never interact, so several images or classes go in one call by giving
 * each its own category.
 *   boxes: device float[num_boxes][4] (x1, y1, x2, y2);  scores: device float[num_boxes];
 *   categories: device int32[num_boxes] or NULL (one category);
 *   num_boxes in [0, RE_MAX_NMS_BOXES] (RE_ERR_UNSUPPORTED above);
 *   keep_out: device int32[min(num_boxes, max_keep)]: the kept box indices in rank
 *     order, then -1;  num_keep_out: device int32[1], the number kept (at most
 *     max_keep >= 0);  iou_threshold: not NaN;
 *   workspace: device, 256-byte aligned, box_nms_workspace_size() bytes. */
#define RE_MAX_NMS_BOXES 8192
re_status_t box_nms_workspace_size(int64_t num_boxes, size_t *bytes);
re_status_t box_nms(const float *boxes, const float *scores, const int32_t *categories,
                    int64_t num_boxes, float iou_threshold, int64_t max_keep, int32_t *keep_out,
                    int32_t *num_keep_out, void *workspace, size_t workspace_bytes,
                    void *stream);

/* f4 -- per-category proposal selection: greedy NMS or Soft-NMS over a batch in one
 * call.  A two-stage detector selects proposals per image (and detections per class)
 * with NMS before extracting their RoI features; the paper runs these bbox operations
 * on the GPU (§1) and lists Soft-NMS among its general modules (§2).  Each box belongs
 * to one category (an image, or an image and class), and categories never interact.
 * For every category c in [0, num_categories):
 *   candidates: the boxes of category c whose score is >= score_threshold (a NaN score,
 *     or a category outside the range, never is), ranked by score as in box_nms (IEEE
 *     total order of the bits, highest first; equal scores by index);
 *   RE_NMS_HARD: greedy NMS over the candidates in rank order -- a box is kept unless
 *     a kept box overlaps it with IoU > iou_threshold (IoU as in box_nms);
 *   RE_NMS_LINEAR / RE_NMS_GAUSSIAN (Soft-NMS): while candidates remain and fewer than
 *     max_keep are kept, the candidate with the largest current score (same order;
 *     equal current scores by rank) is output with that score and removed, and every
 *     remaining candidate is decayed, s = s * w rounded to binary32, with
 *       linear:   w = 1 - iou when iou > iou_threshold (else s is unchanged),
 *       gaussian: w = exp(-iou^2 / sigma) evaluated in double by scaling and squaring
 *                 (halve the argument into [-1/2, 0], degree-16 Taylor polynomial in
 *                 Horner form, square back; 0 below -128), rounded to binary32;
 *     a NaN IoU leaves s unchanged; a candidate whose score falls below
 *     score_threshold is dropped.
 * Outputs (dense, [num_categories][max_keep]): keep_out = the kept box indices of each
 * category in selection order (RE_NMS_HARD: rank order), then -1; scores_out = the
 * score of each at its selection (RE_NMS_HARD: its input score), then 0; num_keep_out
 * [num_categories] = the number kept (<= max_keep).
 *   boxes: device float[num_boxes][4] (x1, y1, x2, y2); scores: device float[num_boxes];
 *   categories: device int32[num_boxes], or NULL with num_categories == 1;
 *   num_boxes in [0, RE_MAX_NMS_BATCH_BOXES]; num_categories in [1, RE_MAX_NMS_CATEGORIES];
 *   iou_threshold, score_threshold not NaN; sigma finite > 0 (RE_NMS_GAUSSIAN);
 *   max_keep >= 0 with max_keep * num_categories < 2^31;
 *   workspace: device, 256-byte aligned, box_nms_batched_workspace_size() bytes (about
 *   48 bytes per box).
 * A category is handled by one workgroup: its candidates are sorted in LDS up to 8192
 * (above that in the workspace, slower); greedy selection tests blocks of 64 candidates
 * against the growing kept list, Soft-NMS runs one workgroup-wide iteration per
 * selection. */
#define RE_NMS_HARD 0
#define RE_NMS_LINEAR 1
#define RE_NMS_GAUSSIAN 2
#define RE_MAX_NMS_BATCH_BOXES (1 << 24)
#define RE_MAX_NMS_CATEGORIES 8192
re_status_t box_nms_batched_workspace_size(int64_t num_boxes, int32_t num_categories,
                                           size_t *bytes);
re_status_t box_nms_batched(const float *boxes, const float *scores, const int32_t *categories,
                            int64_t num_boxes, int32_t num_categories, int32_t method,
                            float iou_threshold, float sigma, float score_threshold,
                            int32_t max_keep, int32_t *keep_out, float *scores_out,
                            int32_t *num_keep_out, void *workspace, size_t workspace_bytes,
                            void *stream);

/* Static description of a status code. */
const char *roi_extract_status_str(re_status_t status);

/* Library version string. */
const char *roi_extract_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ROI_EXTRACT_H */
