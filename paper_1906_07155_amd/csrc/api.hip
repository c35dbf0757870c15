// api.hip -- the C ABI declared in include/roi_extract.h.
//
// Every argument is validated on the host before anything is enqueued, and no
// HIP runtime call is made on an error path, so argument errors are reported the
// same way with or without a GPU.  The library allocates nothing and keeps no
// state: all scratch lives in the caller's workspace.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "internal.hpp"
#include "roi_extract.h"

namespace rex {

// Bands and difference grids of the one-launch plan (nbands = 0 when a level is wider
// than one band's cursors).
void plan_bands(PlanArgs &a) {
    a.nbands = 0;
    a.ndiff = 0;
    int nb = 0, nd = 0;
    for (int l = 0; l < kMaxLevels; ++l) {
        a.band_base[l] = nb;
        a.dbase[l] = nd;
        a.band_rows[l] = 1;
        if (l >= a.L || a.ntiles <= 0) continue;
        if (a.ntx[l] > kBandTiles) return;
        const int rows = std::min(a.nty[l], std::max(1, kBandTarget / a.ntx[l]));
        a.band_rows[l] = rows;
        nb += a.N * ((a.nty[l] + rows - 1) / rows);
        nd += a.N * (a.nty[l] + 1) * (a.ntx[l] + 1);
    }
    a.band_base[kMaxLevels] = nb;
    a.nbands = nb;
    a.ndiff = nd;
}

}  // namespace rex

using namespace rex;

namespace {

// Workspace layout: [0, 256) per-level offsets, then perm[K], keys[K],
// tile_start[ntiles], tile_end[ntiles], tile_order[ntiles], tile_rois[capacity], and
// the plan's scratch: bucket counters[kPlanMaxBins], each region aligned to 256 bytes.
constexpr size_t kHeader = 256;
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
size_t perm_offset() { return kHeader; }
size_t keys_offset(int64_t K) { return kHeader + align256(static_cast<size_t>(K) * 4); }
size_t tiles_offset(int64_t K) { return kHeader + 2 * align256(static_cast<size_t>(K) * 4); }
size_t tile_end_offset(int64_t K, const TileLayout &t) {
    return tiles_offset(K) + align256(static_cast<size_t>(t.ntiles) * 4);
}
size_t tile_order_offset(int64_t K, const TileLayout &t) {
    return tile_end_offset(K, t) + align256(static_cast<size_t>(t.ntiles) * 4);
}
size_t tile_rois_offset(int64_t K, const TileLayout &t) {
    return tile_order_offset(K, t) + align256(static_cast<size_t>(t.ntiles) * 4);
}
size_t key_count_offset(int64_t K, const TileLayout &t) {
    return tile_rois_offset(K, t) + align256(static_cast<size_t>(t.capacity) * 4);
}
size_t workspace_bytes_for(int64_t K, const TileLayout &t) {
    return key_count_offset(K, t) + align256(static_cast<size_t>(kPlanMaxBins) * 4);
}

// Bin-tiles of 2^shift pixels per (level, image): the smallest shift >= 4 whose tile
// count fits the plan kernel's LDS histogram.  capacity bounds the slots of the tile
// lists: the lists of the RoIs of one (level, image) take that bucket's RoI count
// times its tiles, at most K times the most tiles of one image-level.  Binning is
// switched off (ntiles = 0) when that bound would exceed 2^28 pairs.
constexpr int64_t kMaxPairs = int64_t(1) << 28;

// No bin-tiles: the plan is the forward's launch order only.
TileLayout no_tiles() {
    TileLayout off{};
    off.shift = 4;
    for (int l = 0; l <= kMaxLevels; ++l) {
        if (l < kMaxLevels) {
            off.ntx[l] = 1;
            off.nty[l] = 1;
        }
        off.tbase[l] = 0;
    }
    return off;
}

TileLayout tile_layout(const LevelTable &t, int64_t K) {
    TileLayout L{};
    for (int shift = 4; shift <= 24; ++shift) {
        int64_t n = 0, most = 1;
        for (int l = 0; l < t.num; ++l) {
            const int64_t nx = (t.l[l].W + (int64_t(1) << shift) - 1) >> shift;
            const int64_t ny = (t.l[l].H + (int64_t(1) << shift) - 1) >> shift;
            n += int64_t(t.N) * nx * ny;
            most = std::max(most, nx * ny);
        }
        if (n > kPlanMaxBins) continue;
        if (K * most > kMaxPairs) break;
        L.shift = shift;
        L.ntiles = static_cast<int32_t>(n);
        L.capacity = std::max<int64_t>(1, K * most);
        int32_t base = 0;
        for (int l = 0; l < kMaxLevels; ++l) {
            if (l < t.num) {
                L.ntx[l] = static_cast<int32_t>((t.l[l].W + (1 << shift) - 1) >> shift);
                L.nty[l] = static_cast<int32_t>((t.l[l].H + (1 << shift) - 1) >> shift);
                L.tbase[l] = base;
                base += t.N * L.ntx[l] * L.nty[l];
            } else {
                L.ntx[l] = 1;
                L.nty[l] = 1;
                L.tbase[l] = base;
            }
        }
        L.tbase[kMaxLevels] = base;
        return L;
    }
    return no_tiles();   // ntiles = 0: no binning
}

constexpr int64_t kMaxRois = int64_t(1) << 22;
constexpr int64_t kMaxExtent = int64_t(1) << 24;   // H, W exactly representable in binary32

bool valid_dtype(int32_t d) { return d == RE_DTYPE_F32 || d == RE_DTYPE_BF16; }
size_t dtype_size(int32_t d) { return d == RE_DTYPE_BF16 ? 2 : 4; }

// Validates a pyramid and fills the kernel table.  `need_data`: data must be non-null.
re_status_t check_levels(const re_level_t *levels, int32_t num_levels, bool need_data,
                         LevelTable *t, bool *all_channels_last, int64_t *numel,
                         int *dense) {
    if (!levels) return RE_ERR_INVALID_ARG;
    if (num_levels < 1 || num_levels > RE_MAX_LEVELS) return RE_ERR_INVALID_ARG;
    std::memset(t, 0, sizeof(*t));
    bool cl = true;
    for (int l = 0; l < num_levels; ++l) {
        const re_level_t &v = levels[l];
        if (v.reserved != 0 || v.reserved2 != 0.0f) return RE_ERR_INVALID_ARG;
        if (!valid_dtype(v.dtype)) return RE_ERR_INVALID_ARG;
        if (v.n < 1 || v.c < 1 || v.h < 1 || v.w < 1) return RE_ERR_INVALID_ARG;
        if (v.n > INT32_MAX || v.c > INT32_MAX || v.h >= kMaxExtent || v.w >= kMaxExtent)
            return RE_ERR_INVALID_ARG;
        if (v.stride_n < 0 || v.stride_c < 0 || v.stride_h < 0 || v.stride_w < 0)
            return RE_ERR_INVALID_ARG;
        if (!std::isfinite(v.spatial_scale) || !(v.spatial_scale > 0.0f)) return RE_ERR_INVALID_ARG;
        if (l > 0 && (v.n != levels[0].n || v.c != levels[0].c || v.dtype != levels[0].dtype))
            return RE_ERR_INVALID_ARG;
        if (need_data && !v.data) return RE_ERR_INVALID_ARG;
        if (v.data && reinterpret_cast<uintptr_t>(v.data) % dtype_size(v.dtype) != 0)
            return RE_ERR_INVALID_ARG;
        // largest element offset must fit int64 comfortably
        const double span = double(v.n - 1) * v.stride_n + double(v.c - 1) * v.stride_c +
                            double(v.h - 1) * v.stride_h + double(v.w - 1) * v.stride_w;
        if (span > 9.0e18) return RE_ERR_INVALID_ARG;
        LevelArg &a = t->l[l];
        a.data = v.data;
        a.sn = v.stride_n;
        a.sc = v.stride_c;
        a.sh = v.stride_h;
        a.sw = v.stride_w;
        a.H = static_cast<int32_t>(v.h);
        a.W = static_cast<int32_t>(v.w);
        a.scale = v.spatial_scale;
        if (v.stride_c != 1 && v.c != 1) cl = false;   // a single channel has no stride
        // the channels-last kernels address one image of a level with 32-bit byte
        // offsets below 2^30
        const double img = (double(v.c - 1) * v.stride_c + double(v.h - 1) * v.stride_h +
                            double(v.w - 1) * v.stride_w + 1.0) * dtype_size(v.dtype);
        if (img < double(kBufMaxBytes)) a.img_bytes = static_cast<uint32_t>(img);
        else cl = false;
        if (numel) numel[l] = v.n * v.c * v.h * v.w;
        if (dense) {
            // dense: the strides are those of a contiguous tensor for some order of dims
            int64_t ext[4] = {v.n, v.c, v.h, v.w};
            int64_t str[4] = {v.stride_n, v.stride_c, v.stride_h, v.stride_w};
            int order[4] = {0, 1, 2, 3};
            for (int i = 0; i < 4; ++i)
                for (int j = i + 1; j < 4; ++j)
                    if (str[order[j]] < str[order[i]] ||
                        (str[order[j]] == str[order[i]] && ext[order[j]] < ext[order[i]])) {
                        const int tmp = order[i];
                        order[i] = order[j];
                        order[j] = tmp;
                    }
            int64_t expect = 1;
            bool ok = true;
            for (int i = 0; i < 4; ++i) {
                const int d = order[i];
                if (ext[d] == 1) continue;
                if (str[d] != expect) ok = false;
                expect *= ext[d];
            }
            dense[l] = ok ? 1 : 0;
        }
    }
    t->num = num_levels;
    t->N = static_cast<int32_t>(levels[0].n);
    t->C = static_cast<int32_t>(levels[0].c);
    if (all_channels_last) *all_channels_last = cl;
    return RE_OK;
}

re_status_t check_common(const float *rois, int64_t K, const int32_t *roi_levels,
                         int32_t num_levels, int32_t out_h, int32_t out_w,
                         int32_t sampling_ratio, int32_t aligned) {
    if (K < 0 || K > kMaxRois) return RE_ERR_INVALID_ARG;
    if (K > 0 && !rois) return RE_ERR_INVALID_ARG;
    if (K > 0 && num_levels > 1 && !roi_levels) return RE_ERR_INVALID_ARG;
    if (out_h < 1 || out_w < 1 || out_h > RE_MAX_OUT || out_w > RE_MAX_OUT)
        return RE_ERR_INVALID_ARG;
    if (sampling_ratio < 0 || sampling_ratio > RE_MAX_SAMPLING) return RE_ERR_INVALID_ARG;
    if (aligned != 0 && aligned != 1) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(rois) % 4 != 0) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(roi_levels) % 4 != 0) return RE_ERR_INVALID_ARG;
    return RE_OK;
}

re_status_t check_plan(const void *plan, size_t plan_bytes, int64_t K, const LevelTable &t) {
    if (!plan) return RE_OK;
    if (reinterpret_cast<uintptr_t>(plan) % 256 != 0) return RE_ERR_WORKSPACE;
    if (plan_bytes < workspace_bytes_for(K, tile_layout(t, K))) return RE_ERR_WORKSPACE;
    return RE_OK;
}

re_status_t from_hip(hipError_t e) { return e == hipSuccess ? RE_OK : RE_ERR_DEVICE; }

// Plan arguments for the RoIs over pyramid t, the plan stored in `ws` with the tile
// layout tl (ntiles = 0: no tile lists, the forward's launch order only).
re_status_t plan_args(const LevelTable &t, const float *rois, int64_t num_rois, float finest_scale,
                      int32_t box_convention, int32_t *levels_out, char *ws, const TileLayout &tl,
                      PlanArgs *out) {
    const int32_t num_levels = t.num;
    PlanArgs a{};
    a.rois = rois;
    a.levels_out = levels_out;
    a.offsets = reinterpret_cast<int32_t *>(ws);
    a.perm = reinterpret_cast<int32_t *>(ws + perm_offset());
    a.keys = reinterpret_cast<int32_t *>(ws + keys_offset(num_rois));
    a.K = static_cast<int32_t>(num_rois);
    a.L = num_levels;
    a.finest_scale = finest_scale;
    a.box_plus1 = box_convention == RE_BOX_PIXELS ? 1 : 0;
    a.N = t.N;
    // Cell size 2^shift feature pixels: the smallest shift >= 4 whose bucket count fits.
    a.batch_in_key = 1;
    int shift = 4;
    int64_t nbins = 0;
    for (;; ++shift) {
        nbins = 0;
        for (int l = 0; l < num_levels; ++l) {
            const int64_t ncx = (t.l[l].W + (int64_t(1) << shift) - 1) >> shift;
            const int64_t ncy = (t.l[l].H + (int64_t(1) << shift) - 1) >> shift;
            nbins += (a.batch_in_key ? t.N : 1) * ncx * ncy;
        }
        if (nbins <= kPlanMaxBins) break;
        if (shift >= 24) {
            if (!a.batch_in_key) return RE_ERR_UNSUPPORTED;
            a.batch_in_key = 0;   // very large batches: bucket by level and cell only
            shift = 3;
        }
    }
    a.cell_shift = shift;
    a.nbins = static_cast<int32_t>(nbins);
    int32_t base = 0;
    for (int l = 0; l < num_levels; ++l) {
        a.H[l] = t.l[l].H;
        a.W[l] = t.l[l].W;
        a.scale[l] = t.l[l].scale;
        a.ncx[l] = static_cast<int32_t>((t.l[l].W + (1 << shift) - 1) >> shift);
        a.ncy[l] = static_cast<int32_t>((t.l[l].H + (1 << shift) - 1) >> shift);
        a.base[l] = base;
        base += (a.batch_in_key ? t.N : 1) * a.ncx[l] * a.ncy[l];
    }
    a.tile_start = reinterpret_cast<int32_t *>(ws + tiles_offset(num_rois));
    a.tile_end = reinterpret_cast<int32_t *>(ws + tile_end_offset(num_rois, tl));
    a.tile_rois = reinterpret_cast<int32_t *>(ws + tile_rois_offset(num_rois, tl));
    a.tile_order = reinterpret_cast<int32_t *>(ws + tile_order_offset(num_rois, tl));
    a.key_count = reinterpret_cast<int32_t *>(ws + key_count_offset(num_rois, tl));
    // the tile lists are bucketed by (level, image): every tile's bucket must be one
    // key range (always so when the tiles fit: cells then fit at a shift no larger)
    if (tl.ntiles > 0 && !a.batch_in_key) return RE_ERR_UNSUPPORTED;
    a.ntiles = tl.ntiles;
    a.capacity = static_cast<int32_t>(tl.capacity);
    a.tile_shift = tl.shift;
    for (int l = 0; l < kMaxLevels; ++l) {
        a.ntx[l] = tl.ntx[l];
        a.nty[l] = tl.nty[l];
        a.tbase[l] = tl.tbase[l];
    }
    a.tbase[kMaxLevels] = tl.tbase[kMaxLevels];
    plan_bands(a);
    *out = a;
    return RE_OK;
}

}  // namespace

extern "C" {

const char *roi_extract_version(void) { return "roi_extract 0.1 (gfx950)"; }

const char *roi_extract_status_str(re_status_t s) {
    switch (s) {
        case RE_OK: return "ok";
        case RE_ERR_INVALID_ARG: return "invalid argument";
        case RE_ERR_UNSUPPORTED: return "unsupported";
        case RE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case RE_ERR_DEVICE: return "HIP runtime or kernel launch error";
    }
    return "unknown status";
}

re_status_t roi_extract_workspace_size(const re_level_t *levels, int32_t num_levels,
                                       int64_t num_rois, size_t *bytes) {
    if (!bytes || num_rois < 0 || num_rois > kMaxRois) return RE_ERR_INVALID_ARG;
    LevelTable t;
    re_status_t st = check_levels(levels, num_levels, false, &t, nullptr, nullptr, nullptr);
    if (st != RE_OK) return st;
    *bytes = workspace_bytes_for(num_rois, tile_layout(t, num_rois));
    return RE_OK;
}

re_status_t fpn_level_map(const float *rois, int64_t num_rois, int32_t num_levels,
                          float finest_scale, int32_t *levels_out, void *stream) {
    return fpn_level_map_ex(rois, num_rois, num_levels, finest_scale, RE_BOX_CONTINUOUS,
                            levels_out, stream);
}

re_status_t fpn_level_map_ex(const float *rois, int64_t num_rois, int32_t num_levels,
                             float finest_scale, int32_t box_convention, int32_t *levels_out,
                             void *stream) {
    if (box_convention != RE_BOX_CONTINUOUS && box_convention != RE_BOX_PIXELS)
        return RE_ERR_INVALID_ARG;
    if (num_rois < 0 || num_rois > kMaxRois) return RE_ERR_INVALID_ARG;
    if (num_levels < 1 || num_levels > RE_MAX_LEVELS) return RE_ERR_INVALID_ARG;
    if (!std::isfinite(finest_scale) || !(finest_scale > 0.0f)) return RE_ERR_INVALID_ARG;
    if (num_rois == 0) return RE_OK;
    if (!rois || !levels_out) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(rois) % 4 || reinterpret_cast<uintptr_t>(levels_out) % 4)
        return RE_ERR_INVALID_ARG;
    return from_hip(launch_level_map(rois, static_cast<int32_t>(num_rois), num_levels,
                                     finest_scale, box_convention == RE_BOX_PIXELS ? 1 : 0,
                                     levels_out, static_cast<hipStream_t>(stream)));
}

re_status_t roi_extract_plan(const re_level_t *levels, int32_t num_levels, const float *rois,
                             int64_t num_rois, float finest_scale, int32_t *levels_out,
                             void *workspace, size_t workspace_bytes, void *stream) {
    return roi_extract_plan_ex(levels, num_levels, rois, num_rois, finest_scale,
                               RE_BOX_CONTINUOUS, levels_out, workspace, workspace_bytes, stream);
}

re_status_t roi_extract_plan_ex(const re_level_t *levels, int32_t num_levels, const float *rois,
                                int64_t num_rois, float finest_scale, int32_t box_convention,
                                int32_t *levels_out, void *workspace, size_t workspace_bytes,
                                void *stream) {
    if (box_convention != RE_BOX_CONTINUOUS && box_convention != RE_BOX_PIXELS)
        return RE_ERR_INVALID_ARG;
    LevelTable t;
    re_status_t st = check_levels(levels, num_levels, false, &t, nullptr, nullptr, nullptr);
    if (st != RE_OK) return st;
    if (num_rois < 0 || num_rois > kMaxRois) return RE_ERR_INVALID_ARG;
    if (!std::isfinite(finest_scale) || !(finest_scale > 0.0f)) return RE_ERR_INVALID_ARG;
    if (!workspace) return RE_ERR_WORKSPACE;
    if ((st = check_plan(workspace, workspace_bytes, num_rois, t)) != RE_OK) return st;
    if (num_rois > 0 && (!rois || !levels_out)) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(rois) % 4 || reinterpret_cast<uintptr_t>(levels_out) % 4)
        return RE_ERR_INVALID_ARG;

    PlanArgs a;
    if ((st = plan_args(t, rois, num_rois, finest_scale, box_convention, levels_out,
                        static_cast<char *>(workspace), tile_layout(t, num_rois), &a)) != RE_OK)
        return st;
    return from_hip(launch_plan(a, static_cast<hipStream_t>(stream)));
}

re_status_t roi_extract_plan_perm(const void *workspace, size_t workspace_bytes,
                                  int64_t num_rois, const int32_t **perm_out) {
    if (!perm_out || !workspace) return RE_ERR_INVALID_ARG;
    if (num_rois < 0 || num_rois > kMaxRois) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return RE_ERR_WORKSPACE;
    if (workspace_bytes < tiles_offset(num_rois)) return RE_ERR_WORKSPACE;
    *perm_out = reinterpret_cast<const int32_t *>(static_cast<const char *>(workspace) +
                                                  perm_offset());
    return RE_OK;
}

re_status_t roi_extract_plan_offsets(const void *workspace, size_t workspace_bytes,
                                     int64_t num_rois, int32_t num_levels,
                                     int32_t *offsets_out, void *stream) {
    if (!workspace || !offsets_out) return RE_ERR_INVALID_ARG;
    if (num_rois < 0 || num_rois > kMaxRois) return RE_ERR_INVALID_ARG;
    if (num_levels < 1 || num_levels > RE_MAX_LEVELS) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return RE_ERR_WORKSPACE;
    if (workspace_bytes < tiles_offset(num_rois)) return RE_ERR_WORKSPACE;
    return from_hip(hipMemcpyAsync(offsets_out, workspace, (num_levels + 1) * sizeof(int32_t),
                                   hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream)));
}

re_status_t roi_align_fwd(const re_level_t *levels, int32_t num_levels, const float *rois,
                          int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                          int32_t out_w, int32_t sampling_ratio, int32_t aligned, void *out,
                          int32_t out_dtype, const void *plan, size_t plan_bytes,
                          void *stream) {
    LevelTable t;
    bool cl = false;
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if ((st = check_common(rois, num_rois, roi_levels, num_levels, out_h, out_w,
                           sampling_ratio, aligned)) != RE_OK)
        return st;
    if (!valid_dtype(out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && !out) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(out) % dtype_size(out_dtype)) return RE_ERR_INVALID_ARG;
    if ((st = check_plan(plan, plan_bytes, num_rois, t)) != RE_OK) return st;
    if (num_rois == 0) return RE_OK;

    FwdArgs a{};
    a.lv = t;
    a.rois = rois;
    a.roi_levels = roi_levels;
    a.perm = plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(plan) +
                                                      perm_offset())
                  : nullptr;
    a.out = out;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    a.S = sampling_ratio;
    a.aligned = aligned;
    const bool fast = cl && fwd_fast_available(out_h, out_w, sampling_ratio);
    return from_hip(launch_fwd(a, levels[0].dtype, out_dtype, fast,
                               static_cast<hipStream_t>(stream)));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free forward
// ---------------------------------------------------------------------------
//
// roi_align_fwd_noalloc keeps its launch plan in `scratch`, a fixed array in the
// library's device code instead of a caller workspace.  In host code the name
// `scratch` only stands in for the symbol: the device address of each GPU's copy is
// looked up once per device (hipGetSymbolAddress with that device current) and only
// that address is passed to kernels.  The plan kernels clear every counter they use
// themselves (no memset), so the array's previous contents do not matter.

static_assert(RE_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[RE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on first use).
re_status_t scratch_address(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RE_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return RE_ERR_DEVICE;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return RE_OK;
}
}  // namespace

extern "C" {

re_status_t roi_align_fwd_noalloc(const re_level_t *levels, int32_t num_levels, const float *rois,
                                  int64_t num_rois, float finest_scale, int32_t *levels_out,
                                  int32_t out_h, int32_t out_w, int32_t sampling_ratio,
                                  int32_t aligned, void *out, int32_t out_dtype, void *stream) {
    LevelTable t;
    bool cl = false;
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if (num_rois > RE_NOALLOC_MAX_ROIS) return RE_ERR_UNSUPPORTED;
    if ((st = check_common(rois, num_rois, levels_out, 2, out_h, out_w, sampling_ratio,
                           aligned)) != RE_OK)
        return st;
    if (!std::isfinite(finest_scale) || !(finest_scale > 0.0f)) return RE_ERR_INVALID_ARG;
    if (!valid_dtype(out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && !out) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(out) % dtype_size(out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois == 0) return RE_OK;
    const TileLayout tl = no_tiles();
    if (workspace_bytes_for(num_rois, tl) > RE_NOALLOC_SCRATCH_BYTES) return RE_ERR_UNSUPPORTED;

    void *ws = nullptr;
    if ((st = scratch_address(&ws)) != RE_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    PlanArgs pa;
    if ((st = plan_args(t, rois, num_rois, finest_scale, RE_BOX_CONTINUOUS, levels_out,
                        static_cast<char *>(ws), tl, &pa)) != RE_OK)
        return st;
    if ((st = from_hip(launch_plan(pa, s))) != RE_OK) return st;

    FwdArgs a{};
    a.lv = t;
    a.rois = rois;
    a.roi_levels = levels_out;
    a.perm = reinterpret_cast<const int32_t *>(static_cast<const char *>(ws) + perm_offset());
    a.out = out;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    a.S = sampling_ratio;
    a.aligned = aligned;
    const bool fast = cl && fwd_fast_available(out_h, out_w, sampling_ratio);
    return from_hip(launch_fwd(a, levels[0].dtype, out_dtype, fast, s));
}

re_status_t roi_align_fwd_multi(const re_level_t *levels, int32_t num_levels,
                                const re_fwd_head_t *heads, int32_t num_heads, int32_t out_dtype,
                                void *stream) {
    LevelTable t;
    bool cl = false;
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if (!heads || num_heads < 1 || num_heads > RE_MAX_HEADS) return RE_ERR_INVALID_ARG;
    if (!valid_dtype(out_dtype)) return RE_ERR_INVALID_ARG;
    for (int i = 0; i < num_heads; ++i) {
        const re_fwd_head_t &h = heads[i];
        if ((st = check_common(h.rois, h.num_rois, h.roi_levels, num_levels, h.out_h, h.out_w,
                               h.sampling_ratio, h.aligned)) != RE_OK)
            return st;
        if (h.num_rois > 0 && !h.out) return RE_ERR_INVALID_ARG;
        if (reinterpret_cast<uintptr_t>(h.out) % dtype_size(out_dtype)) return RE_ERR_INVALID_ARG;
        if ((st = check_plan(h.plan, h.plan_bytes, h.num_rois, t)) != RE_OK) return st;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    FwdMultiArgs m{};
    m.lv = t;
    int64_t fused_wgs = 0;   // upper bound of the shared launch's workgroups
    for (int i = 0; i < num_heads; ++i) {
        const re_fwd_head_t &h = heads[i];
        if (h.num_rois == 0) continue;
        const int32_t *perm = h.plan ? reinterpret_cast<const int32_t *>(
                                           static_cast<const char *>(h.plan) + perm_offset())
                                     : nullptr;
        // fast-path heads share the launch while its grid stays within one dispatch
        const int64_t wgs = h.num_rois * ((t.C + 63) / 64);
        if (cl && fwd_fast_available(h.out_h, h.out_w, h.sampling_ratio) &&
            fused_wgs + wgs < (int64_t(1) << 24)) {
            fused_wgs += wgs;
            FwdHeadArgs &a = m.head[m.nheads++];
            a.rois = h.rois;
            a.roi_levels = h.roi_levels;
            a.perm = perm;
            a.out = h.out;
            a.K = static_cast<int32_t>(h.num_rois);
            a.PH = h.out_h;
            a.PW = h.out_w;
            a.S = h.sampling_ratio;
            a.aligned = h.aligned;
            continue;
        }
        FwdArgs a{};
        a.lv = t;
        a.rois = h.rois;
        a.roi_levels = h.roi_levels;
        a.perm = perm;
        a.out = h.out;
        a.K = static_cast<int32_t>(h.num_rois);
        a.PH = h.out_h;
        a.PW = h.out_w;
        a.S = h.sampling_ratio;
        a.aligned = h.aligned;
        const bool fast = cl && fwd_fast_available(h.out_h, h.out_w, h.sampling_ratio);
        if ((st = from_hip(launch_fwd(a, levels[0].dtype, out_dtype, fast, s))) != RE_OK) return st;
    }
    if (m.nheads == 0) return RE_OK;
    return from_hip(launch_fwd_multi(m, levels[0].dtype, out_dtype, s));
}

re_status_t roi_extract_zero_grad(const re_level_t *grad_levels, int32_t num_levels,
                                  void *stream) {
    LevelTable t;
    int64_t numel[RE_MAX_LEVELS] = {0};
    int dense[RE_MAX_LEVELS] = {0};
    re_status_t st = check_levels(grad_levels, num_levels, true, &t, nullptr, numel, dense);
    if (st != RE_OK) return st;
    for (int l = 0; l < num_levels; ++l)
        if (grad_levels[l].dtype != RE_DTYPE_F32) return RE_ERR_UNSUPPORTED;
    return from_hip(launch_zero(t, numel, dense, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

// One head of a backward, validated.
struct BwdHead {
    const void *gout;
    int32_t gdt;
    const float *rois;
    int64_t K;
    const int32_t *roi_levels;
    int32_t out_h, out_w, S, aligned;
    const void *plan;
    size_t plan_bytes;
};

re_status_t check_head(const BwdHead &h, int32_t num_levels, const LevelTable &t) {
    re_status_t st;
    if ((st = check_common(h.rois, h.K, h.roi_levels, num_levels, h.out_h, h.out_w, h.S,
                           h.aligned)) != RE_OK)
        return st;
    if (!valid_dtype(h.gdt)) return RE_ERR_INVALID_ARG;
    if (h.K > 0 && !h.gout) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(h.gout) % dtype_size(h.gdt)) return RE_ERR_INVALID_ARG;
    return check_plan(h.plan, h.plan_bytes, h.K, t);
}

// The gather stores through a buffer resource over one image of a level, so it takes
// any strides for which an image spans less than 2^30 bytes (img_bytes != 0): the
// channels-last pyramid and contiguous NCHW alike.
bool levels_buffered(const LevelTable &t) {
    for (int l = 0; l < t.num; ++l)
        if (t.l[l].img_bytes == 0) return false;
    return true;
}

bool head_gather_ok(const BwdHead &h, const LevelTable &t, const TileLayout &tl) {
    return h.plan && levels_buffered(t) && tl.ntiles > 0 && h.K > 0 &&
           gather_available(h.out_h, h.out_w, h.S);
}

GatherHead gather_head(const BwdHead &h, const TileLayout &tl) {
    GatherHead g{};
    const char *ws = static_cast<const char *>(h.plan);
    g.gout = h.gout;
    g.rois = h.rois;
    g.roi_levels = h.roi_levels;
    g.tile_start = reinterpret_cast<const int32_t *>(ws + tiles_offset(h.K));
    g.tile_end = reinterpret_cast<const int32_t *>(ws + tile_end_offset(h.K, tl));
    g.tile_rois = reinterpret_cast<const int32_t *>(ws + tile_rois_offset(h.K, tl));
    g.K = static_cast<int32_t>(h.K);
    g.aligned = h.aligned;
    g.capacity = static_cast<int32_t>(tl.capacity);
    g.PH = h.out_h;
    g.PW = h.out_w;
    return g;
}

GatherArgs gather_args(const LevelTable &t, const BwdHead &h0, const TileLayout &tl,
                       int32_t zero_init) {
    GatherArgs g{};
    g.lv = t;
    g.head[0] = gather_head(h0, tl);
    g.tile_order = reinterpret_cast<const int32_t *>(static_cast<const char *>(h0.plan) +
                                                     tile_order_offset(h0.K, tl));
    g.nheads = 1;
    g.PH = h0.out_h;
    g.PW = h0.out_w;
    g.S = h0.S;
    g.zero_init = zero_init;
    g.ntiles = tl.ntiles;
    g.tile_shift = tl.shift;
    g.qside = 1 << (tl.shift - 3);
    for (int l = 0; l < kMaxLevels; ++l) {
        g.ntx[l] = tl.ntx[l];
        g.nty[l] = tl.nty[l];
        g.tbase[l] = tl.tbase[l];
    }
    g.tbase[kMaxLevels] = tl.tbase[kMaxLevels];
    return g;
}

// One validated head: gather when eligible and not refused by `algorithm`, else the
// scatter (after clearing when zero_init).
re_status_t bwd_head(const BwdHead &h, const LevelTable &t, bool cl, const int64_t *numel,
                     const int *dense, int32_t zero_init, int32_t algorithm, hipStream_t s) {
    const TileLayout tl = tile_layout(t, h.K);
    const bool gather_ok = head_gather_ok(h, t, tl);
    if (algorithm == RE_BWD_GATHER && !gather_ok && h.K > 0) return RE_ERR_UNSUPPORTED;
    if (gather_ok && algorithm != RE_BWD_SCATTER)
        return from_hip(launch_gather(gather_args(t, h, tl, zero_init), h.gdt, s));
    re_status_t st;
    if (zero_init) {
        if ((st = from_hip(launch_zero(t, numel, dense, s))) != RE_OK) return st;
    }
    if (h.K == 0) return RE_OK;
    BwdArgs a{};
    a.lv = t;
    a.gout = h.gout;
    a.rois = h.rois;
    a.roi_levels = h.roi_levels;
    a.perm = h.plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(h.plan) +
                                                        perm_offset())
                    : nullptr;
    a.K = static_cast<int32_t>(h.K);
    a.PH = h.out_h;
    a.PW = h.out_w;
    a.S = h.S;
    a.aligned = h.aligned;
    const bool fast = cl && bwd_fast_available(h.out_h, h.out_w, h.S);
    return from_hip(launch_bwd(a, h.gdt, fast, s));
}

re_status_t check_grad_levels(const re_level_t *grad_levels, int32_t num_levels, LevelTable *t,
                              bool *cl, int64_t *numel, int *dense) {
    re_status_t st = check_levels(grad_levels, num_levels, true, t, cl, numel, dense);
    if (st != RE_OK) return st;
    for (int l = 0; l < num_levels; ++l)
        if (grad_levels[l].dtype != RE_DTYPE_F32) return RE_ERR_UNSUPPORTED;
    return RE_OK;
}

}  // namespace

extern "C" {

re_status_t roi_align_bwd(const void *grad_out, int32_t grad_out_dtype, const float *rois,
                          int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                          int32_t out_w, int32_t sampling_ratio, int32_t aligned,
                          const re_level_t *grad_levels, int32_t num_levels, int32_t zero_init,
                          int32_t algorithm, const void *plan, size_t plan_bytes, void *stream) {
    LevelTable t;
    bool cl = false;
    int64_t numel[RE_MAX_LEVELS] = {0};
    int dense[RE_MAX_LEVELS] = {0};
    re_status_t st = check_grad_levels(grad_levels, num_levels, &t, &cl, numel, dense);
    if (st != RE_OK) return st;
    const BwdHead h{grad_out, grad_out_dtype, rois,    num_rois, roi_levels, out_h,
                    out_w,    sampling_ratio, aligned, plan,     plan_bytes};
    if ((st = check_head(h, num_levels, t)) != RE_OK) return st;
    if (zero_init != 0 && zero_init != 1) return RE_ERR_INVALID_ARG;
    if (algorithm != RE_BWD_AUTO && algorithm != RE_BWD_SCATTER && algorithm != RE_BWD_GATHER)
        return RE_ERR_INVALID_ARG;
    return bwd_head(h, t, cl, numel, dense, zero_init, algorithm,
                    static_cast<hipStream_t>(stream));
}

re_status_t roi_align_bwd_multi(const re_head_t *heads, int32_t num_heads,
                                const re_level_t *grad_levels, int32_t num_levels,
                                int32_t zero_init, void *stream) {
    LevelTable t;
    bool cl = false;
    int64_t numel[RE_MAX_LEVELS] = {0};
    int dense[RE_MAX_LEVELS] = {0};
    re_status_t st = check_grad_levels(grad_levels, num_levels, &t, &cl, numel, dense);
    if (st != RE_OK) return st;
    if (!heads || num_heads < 1 || num_heads > RE_MAX_HEADS) return RE_ERR_INVALID_ARG;
    if (zero_init != 0 && zero_init != 1) return RE_ERR_INVALID_ARG;
    BwdHead hs[RE_MAX_HEADS];
    for (int i = 0; i < num_heads; ++i) {
        const re_head_t &u = heads[i];
        if (u.reserved != 0) return RE_ERR_INVALID_ARG;
        hs[i] = BwdHead{u.grad_out, u.grad_out_dtype, u.rois,    u.num_rois, u.roi_levels,
                        u.out_h,    u.out_w,          u.sampling_ratio, u.aligned, u.plan,
                        u.plan_bytes};
        if ((st = check_head(hs[i], num_levels, t)) != RE_OK) return st;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    // Heads in pairs: a pair whose heads both take the gather on the same tile layout
    // (and one gradient dtype) is one pass over the pyramid; anything else runs head
    // by head.  Only the first pass clears.
    int32_t clear = zero_init;
    for (int i = 0; i < num_heads;) {
        if (i + 1 < num_heads) {
            const BwdHead &a = hs[i], &b = hs[i + 1];
            const TileLayout ta = tile_layout(t, a.K), tb = tile_layout(t, b.K);
            if (head_gather_ok(a, t, ta) && head_gather_ok(b, t, tb) &&
                ta.shift == tb.shift && ta.ntiles == tb.ntiles && a.gdt == b.gdt &&
                a.S == b.S) {
                GatherArgs g = gather_args(t, a, ta, clear);
                g.head[1] = gather_head(b, tb);
                g.nheads = 2;
                g.gout_dtype1 = b.gdt;
                if ((st = from_hip(launch_gather(g, a.gdt, s))) != RE_OK) return st;
                clear = 0;
                i += 2;
                continue;
            }
        }
        if ((st = bwd_head(hs[i], t, cl, numel, dense, clear, RE_BWD_AUTO, s)) != RE_OK) return st;
        clear = 0;
        ++i;
    }
    return RE_OK;
}

// ---------------------------------------------------------------------------
// RoI max pooling
// ---------------------------------------------------------------------------

namespace {
// The argmax is a 32-bit index y * W + x into one (level, image, channel) plane.
bool planes_fit_int32(const LevelTable &t) {
    for (int l = 0; l < t.num; ++l)
        if (int64_t(t.l[l].H) * t.l[l].W > INT32_MAX) return false;
    return true;
}
}  // namespace

re_status_t roi_pool_fwd(const re_level_t *levels, int32_t num_levels, const float *rois,
                         int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                         int32_t out_w, void *out, int32_t out_dtype, int32_t *argmax,
                         const void *plan, size_t plan_bytes, void *stream) {
    LevelTable t;
    bool cl = false;
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if ((st = check_common(rois, num_rois, roi_levels, num_levels, out_h, out_w, 0, 0)) != RE_OK)
        return st;
    if (!planes_fit_int32(t)) return RE_ERR_INVALID_ARG;
    if (!valid_dtype(out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && (!out || !argmax)) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(out) % dtype_size(out_dtype)) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(argmax) % 4) return RE_ERR_INVALID_ARG;
    if ((st = check_plan(plan, plan_bytes, num_rois, t)) != RE_OK) return st;
    if (num_rois == 0) return RE_OK;

    PoolArgs a{};
    a.lv = t;
    a.rois = rois;
    a.roi_levels = roi_levels;
    a.perm = plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(plan) +
                                                      perm_offset())
                  : nullptr;
    a.out = out;
    a.argmax = argmax;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    // the channels-last kernel keeps pixel indices in 24 bits
    bool small_maps = true;
    for (int l = 0; l < num_levels; ++l)
        if (int64_t(t.l[l].H) * t.l[l].W >= (int64_t(1) << 24)) small_maps = false;
    const bool fast = cl && small_maps && pool_fwd_fast_available(out_h, out_w);
    return from_hip(launch_pool_fwd(a, levels[0].dtype, out_dtype, fast,
                                    static_cast<hipStream_t>(stream)));
}

re_status_t roi_pool_bwd(const void *grad_out, int32_t grad_out_dtype, const int32_t *argmax,
                         const float *rois, int64_t num_rois, const int32_t *roi_levels,
                         int32_t out_h, int32_t out_w, const re_level_t *grad_levels,
                         int32_t num_levels, int32_t zero_init, const void *plan,
                         size_t plan_bytes, void *stream) {
    LevelTable t;
    bool cl = false;
    int64_t numel[RE_MAX_LEVELS] = {0};
    int dense[RE_MAX_LEVELS] = {0};
    re_status_t st = check_levels(grad_levels, num_levels, true, &t, &cl, numel, dense);
    if (st != RE_OK) return st;
    for (int l = 0; l < num_levels; ++l)
        if (grad_levels[l].dtype != RE_DTYPE_F32) return RE_ERR_UNSUPPORTED;
    if ((st = check_common(rois, num_rois, roi_levels, num_levels, out_h, out_w, 0, 0)) != RE_OK)
        return st;
    if (!planes_fit_int32(t)) return RE_ERR_INVALID_ARG;
    if (!valid_dtype(grad_out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && (!grad_out || !argmax)) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(grad_out) % dtype_size(grad_out_dtype))
        return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(argmax) % 4) return RE_ERR_INVALID_ARG;
    if (zero_init != 0 && zero_init != 1) return RE_ERR_INVALID_ARG;
    if ((st = check_plan(plan, plan_bytes, num_rois, t)) != RE_OK) return st;

    hipStream_t s = static_cast<hipStream_t>(stream);
    // With a plan that holds tile lists: the tile gather, which writes every gradient
    // element once (clearing included)
    const TileLayout tl = tile_layout(t, num_rois);
    if (plan && num_rois > 0 && tl.ntiles > 0 && levels_buffered(t) &&
        pool_gather_available(out_h, out_w)) {
        BwdHead h{};
        h.gout = grad_out;
        h.gdt = grad_out_dtype;
        h.rois = rois;
        h.K = num_rois;
        h.roi_levels = roi_levels;
        h.out_h = out_h;
        h.out_w = out_w;
        h.plan = plan;
        h.plan_bytes = plan_bytes;
        GatherArgs g = gather_args(t, h, tl, zero_init);
        g.head[0].argmax = argmax;
        return from_hip(launch_pool_gather(g, grad_out_dtype, s));
    }
    if (zero_init) {
        if ((st = from_hip(launch_zero(t, numel, dense, s))) != RE_OK) return st;
    }
    if (num_rois == 0) return RE_OK;
    PoolArgs a{};
    a.lv = t;
    a.rois = rois;
    a.roi_levels = roi_levels;
    a.perm = plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(plan) +
                                                      perm_offset())
                  : nullptr;
    a.argmax = const_cast<int32_t *>(argmax);
    a.gout = grad_out;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    const bool fast = cl && pool_fwd_fast_available(out_h, out_w);
    return from_hip(launch_pool_bwd(a, grad_out_dtype, fast, s));
}

// ---------------------------------------------------------------------------
// Deformable (modulated) RoI pooling
// ---------------------------------------------------------------------------

namespace {
constexpr int kDeformFastBins = 196;   // LDS of the channels-last kernels: 64 * bins * 4 bytes

re_status_t check_deform(const float *offset, const float *mask, float gamma, int64_t K) {
    if (K > 0 && !offset) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(offset) % 4 || reinterpret_cast<uintptr_t>(mask) % 4)
        return RE_ERR_INVALID_ARG;
    if (!std::isfinite(gamma)) return RE_ERR_INVALID_ARG;
    return RE_OK;
}
}  // namespace

re_status_t deform_roi_pool_fwd(const re_level_t *levels, int32_t num_levels, const float *rois,
                                int64_t num_rois, const int32_t *roi_levels, int32_t out_h,
                                int32_t out_w, int32_t sampling_ratio, int32_t aligned,
                                const float *offset, const float *mask, float gamma, void *out,
                                int32_t out_dtype, const void *plan, size_t plan_bytes,
                                void *stream) {
    LevelTable t;
    bool cl = false;
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if ((st = check_common(rois, num_rois, roi_levels, num_levels, out_h, out_w,
                           sampling_ratio, aligned)) != RE_OK)
        return st;
    if ((st = check_deform(offset, mask, gamma, num_rois)) != RE_OK) return st;
    if (!valid_dtype(out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && !out) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(out) % dtype_size(out_dtype)) return RE_ERR_INVALID_ARG;
    if ((st = check_plan(plan, plan_bytes, num_rois, t)) != RE_OK) return st;
    if (num_rois == 0) return RE_OK;
    DeformArgs a{};
    a.lv = t;
    a.rois = rois;
    a.roi_levels = roi_levels;
    a.perm = plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(plan) +
                                                      perm_offset())
                  : nullptr;
    a.offset = offset;
    a.mask = mask;
    a.out = out;
    a.gamma = gamma;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    a.S = sampling_ratio;
    a.aligned = aligned;
    const bool fast = cl && out_h * out_w <= kDeformFastBins;
    return from_hip(launch_deform_fwd(a, levels[0].dtype, out_dtype, fast,
                                      static_cast<hipStream_t>(stream)));
}

re_status_t deform_roi_pool_bwd(const void *grad_out, int32_t grad_out_dtype,
                                const re_level_t *levels, const re_level_t *grad_levels,
                                int32_t num_levels, const float *rois, int64_t num_rois,
                                const int32_t *roi_levels, int32_t out_h, int32_t out_w,
                                int32_t sampling_ratio, int32_t aligned, const float *offset,
                                const float *mask, float gamma, int32_t zero_init,
                                float *grad_offset, float *grad_mask, const void *plan,
                                size_t plan_bytes, void *stream) {
    LevelTable t, g;
    bool cl = false, gcl = false;
    int64_t numel[RE_MAX_LEVELS] = {0};
    int dense[RE_MAX_LEVELS] = {0};
    re_status_t st = check_levels(levels, num_levels, true, &t, &cl, nullptr, nullptr);
    if (st != RE_OK) return st;
    if ((st = check_levels(grad_levels, num_levels, true, &g, &gcl, numel, dense)) != RE_OK)
        return st;
    for (int l = 0; l < num_levels; ++l) {
        if (grad_levels[l].dtype != RE_DTYPE_F32) return RE_ERR_UNSUPPORTED;
        if (grad_levels[l].n != levels[l].n || grad_levels[l].c != levels[l].c ||
            grad_levels[l].h != levels[l].h || grad_levels[l].w != levels[l].w ||
            grad_levels[l].spatial_scale != levels[l].spatial_scale)
            return RE_ERR_INVALID_ARG;
    }
    if ((st = check_common(rois, num_rois, roi_levels, num_levels, out_h, out_w,
                           sampling_ratio, aligned)) != RE_OK)
        return st;
    if ((st = check_deform(offset, mask, gamma, num_rois)) != RE_OK) return st;
    if (!valid_dtype(grad_out_dtype)) return RE_ERR_INVALID_ARG;
    if (num_rois > 0 && (!grad_out || !grad_offset)) return RE_ERR_INVALID_ARG;
    if (grad_mask && !mask) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(grad_out) % dtype_size(grad_out_dtype) ||
        reinterpret_cast<uintptr_t>(grad_offset) % 4 || reinterpret_cast<uintptr_t>(grad_mask) % 4)
        return RE_ERR_INVALID_ARG;
    if (zero_init != 0 && zero_init != 1) return RE_ERR_INVALID_ARG;
    if ((st = check_plan(plan, plan_bytes, num_rois, t)) != RE_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool fast = cl && gcl && out_h * out_w <= kDeformFastBins &&
                      num_rois * ((levels[0].c + 63) / 64) < (int64_t(1) << 24);
    // With a plan that holds tile lists: the feature gradient by the tile gather, which
    // writes every gradient element once (clearing included); the per-RoI kernel then
    // adds the taps the lists do not reach
    const TileLayout tl = tile_layout(g, num_rois);
    const bool gather = fast && plan && num_rois > 0 && tl.ntiles > 0 && levels_buffered(g) &&
                        deform_gather_available(out_h, out_w, sampling_ratio);
    if (zero_init && !gather) {
        if ((st = from_hip(launch_zero(g, numel, dense, s))) != RE_OK) return st;
    }
    if (num_rois == 0) return RE_OK;
    DeformArgs a{};
    a.lv = t;
    a.glv = g;
    a.rois = rois;
    a.roi_levels = roi_levels;
    a.perm = plan ? reinterpret_cast<const int32_t *>(static_cast<const char *>(plan) +
                                                      perm_offset())
                  : nullptr;
    a.offset = offset;
    a.mask = mask;
    a.gout = grad_out;
    a.grad_offset = grad_offset;
    a.grad_mask = grad_mask;
    a.gamma = gamma;
    a.K = static_cast<int32_t>(num_rois);
    a.PH = out_h;
    a.PW = out_w;
    a.S = sampling_ratio;
    a.aligned = aligned;
    if (gather) {
        BwdHead h{};
        h.gout = grad_out;
        h.gdt = grad_out_dtype;
        h.rois = rois;
        h.K = num_rois;
        h.roi_levels = roi_levels;
        h.out_h = out_h;
        h.out_w = out_w;
        h.S = sampling_ratio;
        h.aligned = aligned;
        h.plan = plan;
        h.plan_bytes = plan_bytes;
        if ((st = from_hip(launch_deform_gather(gather_args(g, h, tl, zero_init), a,
                                                grad_out_dtype, s))) != RE_OK)
            return st;
        a.gathered = 1;
        a.tile_shift = tl.shift;
        for (int l = 0; l < kMaxLevels; ++l) {
            a.ntx[l] = tl.ntx[l];
            a.nty[l] = tl.nty[l];
        }
    }
    return from_hip(launch_deform_bwd(a, levels[0].dtype, grad_out_dtype, fast, s));
}

// ---------------------------------------------------------------------------
// Non-maximum suppression
// ---------------------------------------------------------------------------

namespace {
struct NmsLayout {
    size_t order, sboxes, scats, mask, total;
};
static NmsLayout nms_layout(int64_t N) {
    NmsLayout L{};
    const int64_t nw = (N + 63) / 64;
    L.order = 0;
    L.sboxes = align256(static_cast<size_t>(N) * 4);
    L.scats = L.sboxes + align256(static_cast<size_t>(N) * 16);
    L.mask = L.scats + align256(static_cast<size_t>(N) * 4);
    L.total = L.mask + align256(static_cast<size_t>(N) * static_cast<size_t>(nw) * 8);
    return L;
}
}  // namespace

re_status_t box_nms_workspace_size(int64_t num_boxes, size_t *bytes) {
    if (!bytes || num_boxes < 0 || num_boxes > kNmsMaxBoxes) return RE_ERR_INVALID_ARG;
    *bytes = std::max<size_t>(nms_layout(num_boxes).total, 256);
    return RE_OK;
}

re_status_t box_nms(const float *boxes, const float *scores, const int32_t *categories,
                    int64_t num_boxes, float iou_threshold, int64_t max_keep, int32_t *keep_out,
                    int32_t *num_keep_out, void *workspace, size_t workspace_bytes,
                    void *stream) {
    if (num_boxes < 0) return RE_ERR_INVALID_ARG;
    if (num_boxes > kNmsMaxBoxes) return RE_ERR_UNSUPPORTED;
    if (max_keep < 0 || !num_keep_out || std::isnan(iou_threshold)) return RE_ERR_INVALID_ARG;
    if (num_boxes > 0 && (!boxes || !scores)) return RE_ERR_INVALID_ARG;
    if (num_boxes > 0 && max_keep > 0 && !keep_out) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(boxes) % 4 || reinterpret_cast<uintptr_t>(scores) % 4 ||
        reinterpret_cast<uintptr_t>(categories) % 4 || reinterpret_cast<uintptr_t>(keep_out) % 4 ||
        reinterpret_cast<uintptr_t>(num_keep_out) % 4)
        return RE_ERR_INVALID_ARG;
    const NmsLayout lay = nms_layout(num_boxes);
    if (num_boxes > 0) {
        if (!workspace || reinterpret_cast<uintptr_t>(workspace) % 256) return RE_ERR_WORKSPACE;
        if (workspace_bytes < lay.total) return RE_ERR_WORKSPACE;
    }
    char *ws = static_cast<char *>(workspace);
    NmsArgs a{};
    a.boxes = boxes;
    a.scores = scores;
    a.categories = categories;
    if (num_boxes > 0) {
        a.order = reinterpret_cast<int32_t *>(ws + lay.order);
        a.sboxes = reinterpret_cast<float4 *>(ws + lay.sboxes);
        a.scats = reinterpret_cast<int32_t *>(ws + lay.scats);
        a.mask = reinterpret_cast<uint64_t *>(ws + lay.mask);
    }
    a.keep = keep_out;
    a.num_keep = num_keep_out;
    a.max_keep = max_keep;
    a.threshold = iou_threshold;
    a.N = static_cast<int32_t>(num_boxes);
    a.nw = static_cast<int32_t>((num_boxes + 63) / 64);
    return from_hip(launch_nms(a, static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------------------
// Per-category proposal selection
// ---------------------------------------------------------------------------

namespace {
struct NmsBatchLayout {
    size_t count, start, sidx, skey, sbox, sscore, kbox, total;
};
static NmsBatchLayout nmsb_layout(int64_t N, int32_t C) {
    NmsBatchLayout L{};
    const size_t n = static_cast<size_t>(std::max<int64_t>(N, 1));
    L.count = 0;
    L.start = align256(static_cast<size_t>(C) * 4);
    L.sidx = L.start + align256(static_cast<size_t>(C + 1) * 4);
    L.skey = L.sidx + align256(n * 4);
    L.sbox = L.skey + align256(n * 8);
    L.sscore = L.sbox + align256(n * 16);
    L.kbox = L.sscore + align256(n * 4);
    L.total = L.kbox + align256(n * 16);
    return L;
}
static bool nmsb_sizes_ok(int64_t N, int32_t C) {
    return N >= 0 && N <= RE_MAX_NMS_BATCH_BOXES && C >= 1 && C <= RE_MAX_NMS_CATEGORIES;
}
}  // namespace

re_status_t box_nms_batched_workspace_size(int64_t num_boxes, int32_t num_categories,
                                           size_t *bytes) {
    if (!bytes || !nmsb_sizes_ok(num_boxes, num_categories)) return RE_ERR_INVALID_ARG;
    *bytes = nmsb_layout(num_boxes, num_categories).total;
    return RE_OK;
}

re_status_t box_nms_batched(const float *boxes, const float *scores, const int32_t *categories,
                            int64_t num_boxes, int32_t num_categories, int32_t method,
                            float iou_threshold, float sigma, float score_threshold,
                            int32_t max_keep, int32_t *keep_out, float *scores_out,
                            int32_t *num_keep_out, void *workspace, size_t workspace_bytes,
                            void *stream) {
    if (!nmsb_sizes_ok(num_boxes, num_categories)) return RE_ERR_INVALID_ARG;
    if (!categories && num_categories != 1) return RE_ERR_INVALID_ARG;
    if (method != RE_NMS_HARD && method != RE_NMS_LINEAR && method != RE_NMS_GAUSSIAN)
        return RE_ERR_INVALID_ARG;
    if (std::isnan(iou_threshold) || std::isnan(score_threshold)) return RE_ERR_INVALID_ARG;
    if (method == RE_NMS_GAUSSIAN && (!std::isfinite(sigma) || !(sigma > 0.0f)))
        return RE_ERR_INVALID_ARG;
    if (max_keep < 0 || int64_t(max_keep) * num_categories > INT32_MAX) return RE_ERR_INVALID_ARG;
    if (!num_keep_out) return RE_ERR_INVALID_ARG;
    if (max_keep > 0 && (!keep_out || !scores_out)) return RE_ERR_INVALID_ARG;
    if (num_boxes > 0 && (!boxes || !scores)) return RE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(boxes) % 4 || reinterpret_cast<uintptr_t>(scores) % 4 ||
        reinterpret_cast<uintptr_t>(categories) % 4 || reinterpret_cast<uintptr_t>(keep_out) % 4 ||
        reinterpret_cast<uintptr_t>(scores_out) % 4 || reinterpret_cast<uintptr_t>(num_keep_out) % 4)
        return RE_ERR_INVALID_ARG;
    const NmsBatchLayout lay = nmsb_layout(num_boxes, num_categories);
    if (!workspace || reinterpret_cast<uintptr_t>(workspace) % 256) return RE_ERR_WORKSPACE;
    if (workspace_bytes < lay.total) return RE_ERR_WORKSPACE;
    char *ws = static_cast<char *>(workspace);
    NmsBatchArgs a{};
    a.boxes = boxes;
    a.scores = scores;
    a.categories = categories;
    a.keep = keep_out;
    a.kept_scores = scores_out;
    a.num_keep = num_keep_out;
    a.count = reinterpret_cast<int32_t *>(ws + lay.count);
    a.start = reinterpret_cast<int32_t *>(ws + lay.start);
    a.sidx = reinterpret_cast<int32_t *>(ws + lay.sidx);
    a.skey = reinterpret_cast<uint64_t *>(ws + lay.skey);
    a.sbox = reinterpret_cast<float4 *>(ws + lay.sbox);
    a.sscore = reinterpret_cast<float *>(ws + lay.sscore);
    a.kbox = reinterpret_cast<float4 *>(ws + lay.kbox);
    a.N = static_cast<int32_t>(num_boxes);
    a.C = num_categories;
    a.method = method;
    a.max_keep = max_keep;
    a.iou_threshold = iou_threshold;
    a.sigma = sigma;
    a.score_threshold = score_threshold;
    return from_hip(launch_nms_batched(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
