// internal.hpp -- argument blocks and launchers shared by the host API and the
// kernel translation units.  Not part of the public ABI.
#pragma once

#include "common.hpp"

namespace rex {

constexpr int kPlanThreads = 1024;
// The one-launch plan's bands of tile rows (see plan.hip): at most kBandTiles tiles
// (LDS cursors), about kBandTarget aimed at; kBandCand RoIs of a band kept in LDS.
constexpr int kBandTiles = 2048;   // LDS cursors of one band
#ifndef REX_BAND_CAND
#define REX_BAND_CAND 2048
#endif
constexpr int kBandCand = REX_BAND_CAND;   // RoIs of one band kept in LDS (beyond: a second scan)
#ifndef REX_BAND_TARGET
#define REX_BAND_TARGET 64
#endif
constexpr int kBandTarget = REX_BAND_TARGET;   // tiles per band aimed at
constexpr int kPlanMaxBins = 15360;   // LDS histogram + scan scratch of the plan kernel = 64 KiB

struct PlanArgs {
    const float *rois;
    int32_t *levels_out;
    int32_t *keys;
    int32_t *perm;
    int32_t *offsets;      // [L + 1]
    int32_t K;
    int32_t L;
    float finest_scale;
    int32_t N;
    int32_t nbins;
    int32_t cell_shift;    // spatial cell = 2^cell_shift feature pixels
    int32_t batch_in_key;
    int32_t box_plus1;     // level rule on inclusive pixel boxes
    int32_t H[kMaxLevels], W[kMaxLevels];
    int32_t ncx[kMaxLevels], ncy[kMaxLevels], base[kMaxLevels];
    float scale[kMaxLevels];
    // Tile binning for the gather backward: bin-tiles of 2^tile_shift pixels per
    // (level, image); tile_rois[tile_start[t], tile_end[t]) lists the RoIs whose
    // (conservative) footprint box meets tile t.
    int32_t *tile_start;   // [ntiles]
    int32_t *tile_end;     // [ntiles] (the fill's cursors until the lists are done)
    int32_t *tile_rois;    // [capacity]
    int32_t *tile_order;   // [ntiles]: tiles by decreasing list length
    int32_t *key_count;    // [nbins] scratch: bucket counts, then cursors
    int32_t ntiles;
    int32_t capacity;
    int32_t tile_shift;
    int32_t pad2;
    int32_t ntx[kMaxLevels], nty[kMaxLevels], tbase[kMaxLevels + 1];
    // One-launch plan: bands of band_rows[l] tile rows of one (level, image), band ids
    // [band_base[l], band_base[l + 1]) on level l; the list-length difference grids,
    // (nty + 1) x (ntx + 1) per (level, image), level l's from dbase[l], ndiff in all.
    int32_t nbands;
    int32_t ndiff;
    int32_t band_base[kMaxLevels + 1];
    int32_t band_rows[kMaxLevels];
    int32_t dbase[kMaxLevels];
};

// Tile layout shared by the plan and the gather backward (a function of the level
// shapes and the batch size only).
struct TileLayout {
    int32_t shift;
    int32_t ntiles;
    int64_t capacity;
    int32_t ntx[kMaxLevels], nty[kMaxLevels], tbase[kMaxLevels + 1];
};

// One head's RoIs for the gather backward (its upstream gradient and its plan).
struct GatherHead {
    const void *gout;            // [K][C][PH][PW]
    const int32_t *argmax;       // RoI max pooling: [K][C][PH][PW] pixel indices
    const float *rois;
    const int32_t *roi_levels;
    const int32_t *tile_start;   // the head's plan: tile -> RoI lists
    const int32_t *tile_end;
    const int32_t *tile_rois;
    int32_t K;
    int32_t aligned;
    int32_t capacity;
    int32_t PH, PW;
    int32_t pad;
};

// Division by a divisor fixed at launch, for the block-id decoding of the gather
// kernels: n / d = (t + ((n - t) >> s1)) >> s2 with t = umulhi(n, m), exact for every
// 32-bit n (Granlund and Montgomery, division by invariant integers, 1994).  The
// scalar unit has no divide instruction; this takes five scalar operations.
// The two shifts are packed as s1 | s2 << 8.  Per-level divisors are kept as plain
// integer arrays (a switch over a struct array in the kernel arguments can make the
// compiler copy the arguments to scratch memory to index them).
struct FastDiv {
    uint32_t m;
    int32_t sh;
};

inline FastDiv make_fastdiv(uint32_t d) {   // d >= 1
    int l = 0;
    while ((uint64_t(1) << l) < d) ++l;   // ceil(log2 d)
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{static_cast<uint32_t>(m), (l < 1 ? l : 1) | (l > 1 ? l - 1 : 0) << 8};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, uint32_t m, int32_t sh) {
    const uint32_t t = __umulhi(n, m);
    return (t + ((n - t) >> (sh & 0xff))) >> (sh >> 8);
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) { return fdiv(n, f.m, f.sh); }

struct GatherArgs {
    LevelTable lv;               // gradient levels (binary32, channels-last)
    GatherHead head[2];          // head 1 is used by the two-head kernel only
    const int32_t *tile_order;   // head 0's plan: tiles by decreasing list length
    int32_t nheads;
    int32_t PH, PW, S;           // head 0's grid (both heads sample with S)
    int32_t zero_init;
    int32_t ntiles;
    int32_t tile_shift;
    int32_t qside;               // 8x8 quadrants per bin-tile side
    int32_t ncg;                 // 64-channel groups
    int32_t wg_per_tile;
    int32_t gout_dtype1;         // head 1's upstream-gradient dtype
    int32_t ntx[kMaxLevels], nty[kMaxLevels], tbase[kMaxLevels + 1];
    // set at launch: block-id decoding without integer division
    int32_t qs_shift;            // log2 qside
    int32_t wgpt_shift;          // log2 wg_per_tile
    FastDiv div_tile;            // by ncg * wg_per_tile
    uint32_t img_m[kMaxLevels];  // by the tiles of one image of a level
    int32_t img_sh[kMaxLevels];
    uint32_t row_m[kMaxLevels];  // by the tiles of one row of a level
    int32_t row_sh[kMaxLevels];
    uint32_t wid_m[kMaxLevels];  // by the width of a level (pixel index -> row)
    int32_t wid_sh[kMaxLevels];
};

struct FwdArgs {
    LevelTable lv;
    const float *rois;
    const int32_t *roi_levels;   // may be null when lv.num == 1
    const int32_t *perm;         // plan order or null
    void *out;
    int32_t K;
    int32_t PH, PW, S;
    int32_t aligned;
    int32_t nslices;             // channel slices per RoI (fast kernels)
    int32_t wg_per_roi;          // workgroups per RoI (fast kernels)
    int32_t spw;                 // slices per workgroup (channels-last forward)
};

// One head of a multi-head forward (the pyramid is shared): its RoIs, output and the
// slicing of its channels, and the first logical block id of its workgroups.
constexpr int kMaxFwdHeads = 8;
struct FwdHeadArgs {
    const float *rois;
    const int32_t *roi_levels;
    const int32_t *perm;         // plan order or null
    void *out;
    int32_t K;
    int32_t PH, PW, S;
    int32_t aligned;
    int32_t nslices;
    int32_t wg_per_roi;
    int32_t spw;
    int32_t first;               // first logical block of the head
    int32_t pad;
};

struct FwdMultiArgs {
    LevelTable lv;
    FwdHeadArgs head[kMaxFwdHeads];
    int32_t nheads;
    int32_t pad;
};

// Heads on the channels-last fast path (fwd_fast_available grids) in one launch; the
// heads' K, PH, PW, S, aligned, rois, roi_levels, perm and out must be set.
hipError_t launch_fwd_multi(FwdMultiArgs m, int feat_dtype, int out_dtype, hipStream_t stream);

struct BwdArgs {
    LevelTable lv;               // gradient levels (binary32, written with atomics)
    const void *gout;
    const float *rois;
    const int32_t *roi_levels;
    const int32_t *perm;
    int32_t K;
    int32_t PH, PW, S;
    int32_t aligned;
    int32_t nslices;
    int32_t wg_per_roi;
    int32_t pad;
};

// RoI max pooling (forward and backward share the block).
constexpr int kPoolFastBins = 96;   // largest out_h * out_w of the channels-last kernels

struct PoolArgs {
    LevelTable lv;               // features (forward) or binary32 gradients (backward)
    const float *rois;
    const int32_t *roi_levels;
    const int32_t *perm;         // plan order or null
    void *out;                   // forward: [K][C][PH][PW]
    int32_t *argmax;             // [K][C][PH][PW]; read-only in the backward
    const void *gout;            // backward: [K][C][PH][PW]
    int32_t K;
    int32_t PH, PW;
    int32_t nslices;
};

bool pool_fwd_fast_available(int PH, int PW);
hipError_t launch_pool_fwd(PoolArgs a, int feat_dtype, int out_dtype, bool fast,
                           hipStream_t stream);
hipError_t launch_pool_bwd(PoolArgs a, int gout_dtype, bool fast, hipStream_t stream);
// The tile-gather backward of RoI max pooling (head 0 of `a`, with its argmax).
bool pool_gather_available(int PH, int PW);
hipError_t launch_pool_gather(GatherArgs a, int gout_dtype, hipStream_t stream);

// Deformable (modulated) RoI pooling, forward and backward.
struct DeformArgs {
    LevelTable lv;               // features
    LevelTable glv;              // backward: binary32 gradient levels
    const float *rois;
    const int32_t *roi_levels;
    const int32_t *perm;         // plan order or null
    const float *offset;         // [K][2][PH][PW]
    const float *mask;           // [K][PH][PW] or null
    void *out;                   // forward output [K][C][PH][PW]
    const void *gout;            // backward upstream gradient [K][C][PH][PW]
    float *grad_offset;          // backward, [K][2][PH][PW] (cleared first, then summed)
    float *grad_mask;            // backward, [K][PH][PW] or null
    float gamma;
    int32_t K;
    int32_t PH, PW, S;
    int32_t aligned;
    int32_t nslices;
    // backward after the tile gather: the feature gradient of every tap whose tile is in
    // its RoI's tile range (roi_tile_range) is already written; add only the others
    int32_t gathered;
    int32_t tile_shift;
    int32_t ntx[kMaxLevels], nty[kMaxLevels];
};

hipError_t launch_deform_fwd(DeformArgs a, int feat_dtype, int out_dtype, bool fast,
                             hipStream_t stream);
// The feature gradient of deformable pooling as a tile gather (7x7 bins, 1 or 2 samples
// per axis): every tap whose tile is in its RoI's tile range, written once per element.
bool deform_gather_available(int PH, int PW, int S);
hipError_t launch_deform_gather(GatherArgs g, const DeformArgs &d, int gout_dtype,
                                hipStream_t stream);
// Clears grad_offset / grad_mask, then adds the gradients (features with atomics).
hipError_t launch_deform_bwd(DeformArgs a, int feat_dtype, int gout_dtype, bool fast,
                             hipStream_t stream);

// Greedy non-maximum suppression.
constexpr int kNmsMaxBoxes = 8192;   // boxes per call: the sort's 64-bit items fill 64 KiB of LDS

struct NmsArgs {
    const float *boxes;          // [N][4]
    const float *scores;         // [N]
    const int32_t *categories;   // [N] or null
    int32_t *order;              // workspace: box index of every rank
    float4 *sboxes;              // workspace: boxes in rank order
    int32_t *scats;              // workspace: categories in rank order
    uint64_t *mask;              // workspace: [N][nw] overlap bits of the upper triangle
    int32_t *keep;               // [min(N, max_keep)]
    int32_t *num_keep;           // [1]
    int64_t max_keep;
    float threshold;
    int32_t N;
    int32_t nw;                  // 64-box blocks
};

hipError_t launch_nms(NmsArgs a, hipStream_t stream);

// Rank key of a score: IEEE total order of the bits, largest first; NaN after every
// number.
__device__ __forceinline__ uint32_t nms_key(float s) {
    const uint32_t u = __float_as_uint(s);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0xffffffffu;
    const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ~asc;
}

// Binary32 IoU, one rounding per operation in the order of the definition.
__device__ __forceinline__ float nms_iou(float4 a, float4 b) {
    const float ix1 = fmaxf(a.x, b.x);
    const float iy1 = fmaxf(a.y, b.y);
    const float ix2 = fminf(a.z, b.z);
    const float iy2 = fminf(a.w, b.w);
    float iw = ix2 - ix1;
    float ih = iy2 - iy1;
    iw = fmaxf(iw, 0.0f);
    ih = fmaxf(ih, 0.0f);
    const float inter = iw * ih;
    const float wa = a.z - a.x;
    const float ha = a.w - a.y;
    const float wb = b.z - b.x;
    const float hb = b.w - b.y;
    const float area_a = wa * ha;
    const float area_b = wb * hb;
    const float sum = area_a + area_b;
    const float uni = sum - inter;
    return inter / uni;
}

// Per-category proposal selection (greedy NMS or Soft-NMS), many categories per call.
constexpr int kNmsHard = 0, kNmsLinear = 1, kNmsGaussian = 2;

struct NmsBatchArgs {
    const float *boxes;          // [N][4]
    const float *scores;         // [N]
    const int32_t *categories;   // [N] or null (one category)
    int32_t *keep;               // [C][max_keep]
    float *kept_scores;          // [C][max_keep]
    int32_t *num_keep;           // [C]
    // workspace
    int32_t *count;              // [C] candidates per category, then the placement cursor
    int32_t *start;              // [C + 1] first sorted position of each category
    int32_t *sidx;               // [N] box index of every sorted position
    uint64_t *skey;              // [N] sort keys (categories too long for LDS)
    float4 *sbox;                // [N] boxes in sorted order
    float *sscore;               // [N] scores in sorted order (Soft-NMS: current scores)
    float4 *kbox;                // [N] kept boxes of each category (greedy)
    int32_t N, C;
    int32_t method;
    int32_t max_keep;
    float iou_threshold, sigma, score_threshold;
    int32_t pad;
};

hipError_t launch_nms_batched(const NmsBatchArgs &a, hipStream_t stream);

// Inclusive prefix sum across the 64 lanes of a wavefront, in DPP moves: shifts by
// 1, 2, 4 and 8 lanes inside each row of 16 (lanes shifted in from outside the row
// add the old value, 0), then the last lane of row 0 (and of row 2) broadcast into
// row 1 (and row 3), then the last lane of row 1 into rows 2 and 3.
__device__ __forceinline__ int wave_inclusive_scan(int v, int /*lane*/) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

// Exclusive scan of hist[0, n) in place by the whole workgroup: per-thread chunk
// sums, a wavefront scan of the sums, a scan of the wavefront totals by wave 0,
// then the chunk prefixes.  part[] holds the wavefront totals.  Returns the total.
__device__ __forceinline__ int block_exclusive_scan(int32_t *hist, int n, int32_t *part) {
    constexpr int kWaves = kPlanThreads / 64;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int per = (n + kPlanThreads - 1) / kPlanThreads;
    const int lo = min(tid * per, n);
    const int hi = min(lo + per, n);
    int s = 0;
    for (int i = lo; i < hi; ++i) s += hist[i];
    const int incl = wave_inclusive_scan(s, lane);
    if (lane == 63) part[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const int w = lane < kWaves ? part[lane] : 0;
        const int wi = wave_inclusive_scan(w, lane);
        if (lane < kWaves) part[kWaves + lane] = wi - w;   // exclusive wave prefix
        if (lane == kWaves - 1) part[2 * kWaves] = wi;     // total
    }
    __syncthreads();
    int run = part[kWaves + wave] + incl - s;
    for (int i = lo; i < hi; ++i) {
        const int c = hist[i];
        hist[i] = run;
        run += c;
    }
    const int total = part[2 * kWaves];
    __syncthreads();
    return total;
}

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t box_plus1, int32_t *out, hipStream_t stream);
hipError_t launch_plan(const PlanArgs &a, hipStream_t stream);
void plan_bands(PlanArgs &a);   // fills nbands, ndiff, band_base, band_rows, dbase

// Forward: `fast` selects the channels-last kernels (every level stride_c == 1 and
// (PH, PW, S) in the specialised set); otherwise the general strided kernel.
bool fwd_fast_available(int PH, int PW, int S);
hipError_t launch_fwd(FwdArgs a, int feat_dtype, int out_dtype, bool fast, hipStream_t stream);

bool bwd_fast_available(int PH, int PW, int S);
hipError_t launch_bwd(BwdArgs a, int gout_dtype, bool fast, hipStream_t stream);

// Tile-gather backward (channels-last levels, specialised grids, a plan with tiles).
bool gather_available(int PH, int PW, int S);
hipError_t launch_gather(GatherArgs a, int gout_dtype, hipStream_t stream);

// Zero every element of the (binary32) levels in `lv`; `numel[l]` and `dense[l]`
// describe each level (dense levels are cleared as flat arrays).
hipError_t launch_zero(const LevelTable &lv, const int64_t *numel, const int *dense,
                       hipStream_t stream);

}  // namespace rex
