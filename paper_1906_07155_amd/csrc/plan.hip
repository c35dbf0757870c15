// plan.hip -- FPN level assignment and the RoI launch plan.
//
// Level assignment: §3.1 of MMDetection (SingleRoIExtractor reads each RoI from
// "the corresponding level" of the FPN pyramid); the rule is the FPN rule in its
// threshold form, see include/roi_extract.h.
//
// The plan is a counting sort of the RoIs by (level, image, spatial cell of the box
// centre): RoIs that read the same feature rows end up next to each other in launch
// order, and the XCD-aware block mapping of the forward/backward then keeps them on
// one XCD's L2.  The order of RoIs with equal keys is whatever the atomics give;
// only the keys' order and the per-level offsets are defined.
//
// The plan also bins the RoIs into square bin-tiles of every (level, image) for
// the gather backward: a CSR list of the RoIs whose footprint can reach each
// tile (a superset: a listed RoI may contribute nothing to the tile).
#include "internal.hpp"

namespace rex {

__global__ __launch_bounds__(256) void level_map_kernel(const float *__restrict__ rois,
                                                        int32_t K, int32_t L, float finest_scale,
                                                        int32_t box_plus1,
                                                        int32_t *__restrict__ out) {
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x) {
        const float *r = rois + 5 * static_cast<int64_t>(k);
        out[k] = fpn_level(r[1], r[2], r[3], r[4], L, finest_scale, box_plus1);
    }
}

// Per-level tables of the plan arguments, staged in LDS at kernel start: indexing the
// argument arrays with a per-lane level would make every lane load from the
// kernel-argument segment after its RoI's level is known; the staging loads are issued
// at once, alongside the first RoI loads.
struct LevelTab {
    float scale[kMaxLevels];
    int32_t W[kMaxLevels], H[kMaxLevels], ncx[kMaxLevels], ncy[kMaxLevels], base[kMaxLevels];
    int32_t tbase[kMaxLevels], ntx[kMaxLevels], nty[kMaxLevels];
};

// Threads 0..kMaxLevels-1 fill the table; a barrier must follow before it is read.
__device__ __forceinline__ void load_tab(const PlanArgs &a, LevelTab &t) {
    const int i = threadIdx.x;
    if (i < kMaxLevels) {
        t.scale[i] = a.scale[i];
        t.W[i] = a.W[i];
        t.H[i] = a.H[i];
        t.ncx[i] = a.ncx[i];
        t.ncy[i] = a.ncy[i];
        t.base[i] = a.base[i];
        t.tbase[i] = a.tbase[i];
        t.ntx[i] = a.ntx[i];
        t.nty[i] = a.nty[i];
    }
}

// Bin-tiles met by a conservative box around the footprint of a RoI on its level.
// Every sample of the RoI lies between the (shifted) box edges for any output size,
// sampling ratio and alignment; taps add one pixel, and a 1.5-pixel margin absorbs
// rounding.  Non-finite boxes cover the whole map.
__device__ void roi_tile_box(const PlanArgs &a, const LevelTab &tb, int lvl, float x1, float y1, float x2, float y2,
                             int &tx0, int &tx1, int &ty0, int &ty1) {
    const float s = tb.scale[lvl];
    const float W = static_cast<float>(tb.W[lvl] - 1);
    const float H = static_cast<float>(tb.H[lvl] - 1);
    float lx = 0.0f, hx = W, ly = 0.0f, hy = H;
    if (isfinite(x1) && isfinite(x2) && isfinite(y1) && isfinite(y2)) {
        lx = fminf(fmaxf(fminf(x1, x2) * s - 1.5f, 0.0f), W);
        hx = fminf(fmaxf(fmaxf(fmaxf(x1, x2) * s, x1 * s + 1.0f) + 2.5f, 0.0f), W);
        ly = fminf(fmaxf(fminf(y1, y2) * s - 1.5f, 0.0f), H);
        hy = fminf(fmaxf(fmaxf(fmaxf(y1, y2) * s, y1 * s + 1.0f) + 2.5f, 0.0f), H);
    }
    tx0 = static_cast<int>(lx) >> a.tile_shift;
    tx1 = max(static_cast<int>(hx) >> a.tile_shift, tx0);
    ty0 = static_cast<int>(ly) >> a.tile_shift;
    ty1 = max(static_cast<int>(hy) >> a.tile_shift, ty0);
    tx1 = min(tx1, tb.ntx[lvl] - 1);
    ty1 = min(ty1, tb.nty[lvl] - 1);
}

// Sort key of a RoI: level bucket + image + spatial cell of the box centre.
__device__ __forceinline__ int plan_key(const PlanArgs &a, const LevelTab &tb, float x1, float y1, float x2, float y2,
                                        int lvl, int bb) {
    const int b = (bb < 0 || !a.batch_in_key) ? 0 : bb;
    float cx = (x1 + x2) * 0.5f * tb.scale[lvl];
    float cy = (y1 + y2) * 0.5f * tb.scale[lvl];
    cx = fminf(fmaxf(cx, 0.0f), static_cast<float>(tb.W[lvl] - 1));   // NaN -> 0
    cy = fminf(fmaxf(cy, 0.0f), static_cast<float>(tb.H[lvl] - 1));
    const int gx = min(static_cast<int>(cx) >> a.cell_shift, tb.ncx[lvl] - 1);
    const int gy = min(static_cast<int>(cy) >> a.cell_shift, tb.ncy[lvl] - 1);
    return tb.base[lvl] + (b * tb.ncy[lvl] + gy) * tb.ncx[lvl] + gx;
}

// The tile phases give each RoI kPlanLanes consecutive lanes, which split its tiles,
// so the atomics of one RoI are in flight together.
constexpr int kPlanLanes = 16;
constexpr int kPlanSmall = kPlanThreads * 2;

// Small plans (K <= kPlanSmall) run in one 1024-thread workgroup with LDS
// histograms, which avoids the launch latency of the four-kernel plan; each thread
// keeps the keys of up to kCached RoIs in registers between the phases.
constexpr int kCached = 2;

__global__ __launch_bounds__(kPlanThreads) void plan_small_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;                           // [max(nbins, ntiles)]
    int32_t *part = hist + max(a.nbins, a.ntiles);  // [kPlanThreads]
    int32_t *box = part + kPlanThreads;             // [3 * kPlanSmall]: tile box per RoI
    __shared__ LevelTab tb;
    const int tid = threadIdx.x;
    int ckey[kCached];

    // the RoIs are loaded before the first barrier, alongside the level tables
    float rv[kCached][5];
#pragma unroll
    for (int i = 0; i < kCached; ++i) {
        const int32_t k = tid + i * kPlanThreads;
        if (k < a.K) {
            const float *r = a.rois + 5 * static_cast<int64_t>(k);
#pragma unroll
            for (int j = 0; j < 5; ++j) rv[i][j] = r[j];
        }
    }
    load_tab(a, tb);
    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = 0;
    __syncthreads();

    // a1: level of every RoI; key = level bucket + image + spatial cell; the tile box
    // of its footprint (first tile, packed x and y ranges; first tile -1: no tiles).
#pragma unroll
    for (int i = 0; i < kCached; ++i) {
        const int32_t k = tid + i * kPlanThreads;
        if (k < a.K) {
            const float b0 = rv[i][0], x1 = rv[i][1], y1 = rv[i][2], x2 = rv[i][3], y2 = rv[i][4];
            const int lvl = fpn_level(x1, y1, x2, y2, a.L, a.finest_scale, a.box_plus1);
            a.levels_out[k] = lvl;
            const int bb = roi_batch(b0, a.N);
            ckey[i] = plan_key(a, tb, x1, y1, x2, y2, lvl, bb);
            atomicAdd(&hist[ckey[i]], 1);
            int first = -1, xr = 0, yr = 0;
            if (a.ntiles > 0 && bb >= 0) {
                int tx0, tx1, ty0, ty1;
                roi_tile_box(a, tb, lvl, x1, y1, x2, y2, tx0, tx1, ty0, ty1);
                first = tb.tbase[lvl] + (bb * tb.nty[lvl] + ty0) * tb.ntx[lvl] + tx0;
                xr = (tx1 - tx0 + 1) | (tb.ntx[lvl] << 16);
                yr = ty1 - ty0 + 1;
            }
            box[3 * k] = first;
            box[3 * k + 1] = xr;
            box[3 * k + 2] = yr;
        }
    }
    __syncthreads();

    block_exclusive_scan(hist, a.nbins, part);

    // Per-level offsets: the first slot of each level's bucket range.
    if (tid < a.L) a.offsets[tid] = hist[tb.base[tid]];
    if (tid == 0) a.offsets[a.L] = a.K;
    __syncthreads();

    // a2: scatter RoI indices to their slots.
#pragma unroll
    for (int i = 0; i < kCached; ++i) {
        const int32_t k = tid + i * kPlanThreads;
        if (k < a.K) a.perm[atomicAdd(&hist[ckey[i]], 1)] = k;
    }
    if (a.ntiles <= 0) return;   // uniform
    __syncthreads();

    // Tile binning: count the (tile, RoI) pairs, scan, then fill the CSR lists.  Each
    // RoI gets kSmallLanes consecutive lanes, which split its tiles.
    constexpr int kSmallLanes = 4;
    constexpr int kPer = kPlanThreads / kSmallLanes;   // RoIs per pass
    const int sub = tid % kSmallLanes;
    auto for_tiles = [&](auto &&fn) {
        for (int32_t k = tid / kSmallLanes; k < a.K; k += kPer) {
            const int first = box[3 * k];
            if (first < 0) continue;
            const int w = box[3 * k + 1] & 0xffff;
            const int ntx = box[3 * k + 1] >> 16;
            const int n = w * box[3 * k + 2];
            for (int i = sub; i < n; i += kSmallLanes) {
                const int dy = i / w;
                fn(first + dy * ntx + (i - dy * w), k);
            }
        }
    };
    for (int i = tid; i < a.ntiles; i += kPlanThreads) hist[i] = 0;
    __syncthreads();
    for_tiles([&](int t, int) { atomicAdd(&hist[t], 1); });
    __syncthreads();
    // Launch order of the tiles: longest lists first (counting sort on the list
    // length, capped at 255), so the longest sequential chains start earliest.
    constexpr int kLenBins = 256;
    int32_t *lenh = part + 2 * (kPlanThreads / 64) + 1;   // [kLenBins], after the scan scratch
    for (int i = tid; i < kLenBins; i += kPlanThreads) lenh[i] = 0;
    __syncthreads();
    for (int i = tid; i < a.ntiles; i += kPlanThreads)
        atomicAdd(&lenh[kLenBins - 1 - min(hist[i], kLenBins - 1)], 1);
    __syncthreads();
    block_exclusive_scan(lenh, kLenBins, part);
    for (int i = tid; i < a.ntiles; i += kPlanThreads) {
        const int pos = atomicAdd(&lenh[kLenBins - 1 - min(hist[i], kLenBins - 1)], 1);
        a.tile_order[pos] = i;
    }
    __syncthreads();
    const int total = block_exclusive_scan(hist, a.ntiles, part);
    for (int i = tid; i < a.ntiles; i += kPlanThreads) a.tile_start[i] = hist[i];
    if (tid == 0) a.tile_start[a.ntiles] = total;
    __syncthreads();
    for_tiles([&](int t, int k) {
        const int pos = atomicAdd(&hist[t], 1);
        if (pos < a.capacity) a.tile_rois[pos] = k;
    });
}

// Larger plans run as four short kernels over the whole GPU: clear the counters;
// per RoI, its level, sort key and the tiles its footprint box meets, counted with
// device-scope integer atomics; one workgroup turns the counts into bucket starts,
// per-level offsets, tile list starts and the longest-first tile order; per RoI,
// its slot in the permutation and in each of its tiles' lists.

__global__ __launch_bounds__(256) void plan_clear_kernel(int32_t *__restrict__ a, int32_t na,
                                                         int32_t *__restrict__ b, int32_t nb) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < na + nb;
         i += gridDim.x * blockDim.x) {
        if (i < na) a[i] = 0;
        else b[i - na] = 0;
    }
}

__global__ __launch_bounds__(256) void plan_count_kernel(PlanArgs a) {
    __shared__ LevelTab tb;
    load_tab(a, tb);
    __syncthreads();
    const int sub = threadIdx.x % kPlanLanes;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (256 / kPlanLanes);
    for (int64_t k = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) / kPlanLanes; k < a.K;
         k += stride) {
        const float *r = a.rois + 5 * k;
        const float b0 = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
        const int lvl = fpn_level(x1, y1, x2, y2, a.L, a.finest_scale, a.box_plus1);
        const int bb = roi_batch(b0, a.N);
        if (sub == 0) {
            a.levels_out[k] = lvl;
            const int key = plan_key(a, tb, x1, y1, x2, y2, lvl, bb);
            a.keys[k] = key;
            atomicAdd(&a.key_count[key], 1);
        }
        if (a.ntiles > 0 && bb >= 0) {
            int tx0, tx1, ty0, ty1;
            roi_tile_box(a, tb, lvl, x1, y1, x2, y2, tx0, tx1, ty0, ty1);
            const int w = tx1 - tx0 + 1;
            const int n = w * (ty1 - ty0 + 1);
            const int base = tb.tbase[lvl] + bb * tb.nty[lvl] * tb.ntx[lvl];
            for (int i = sub; i < n; i += kPlanLanes) {
                const int dy = i / w;
                atomicAdd(&a.tile_start[base + (ty0 + dy) * tb.ntx[lvl] + tx0 + (i - dy * w)], 1);
            }
        }
    }
}

__global__ __launch_bounds__(kPlanThreads) void plan_scan_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;                           // [max(nbins, ntiles)]
    int32_t *part = smem + max(a.nbins, a.ntiles);  // [kPlanThreads]
    const int tid = threadIdx.x;

    // Bucket starts (the fill kernel's cursors) and per-level offsets.
    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = a.key_count[i];
    __syncthreads();
    block_exclusive_scan(hist, a.nbins, part);
    for (int i = tid; i < a.nbins; i += kPlanThreads) a.key_count[i] = hist[i];
    if (tid < a.L) a.offsets[tid] = hist[a.base[tid]];
    if (tid == 0) a.offsets[a.L] = a.K;
    if (a.ntiles <= 0) return;   // uniform
    __syncthreads();

    // Tile list starts and cursors; launch order of the tiles: longest lists first
    // (counting sort on the list length, capped at 255), so the longest sequential
    // chains start earliest.
    constexpr int kLenBins = 256;
    int32_t *lenh = part + 2 * (kPlanThreads / 64) + 1;   // [kLenBins], after the scan scratch
    for (int i = tid; i < kLenBins; i += kPlanThreads) lenh[i] = 0;
    for (int i = tid; i < a.ntiles; i += kPlanThreads) hist[i] = a.tile_start[i];
    __syncthreads();
    for (int i = tid; i < a.ntiles; i += kPlanThreads)
        atomicAdd(&lenh[kLenBins - 1 - min(hist[i], kLenBins - 1)], 1);
    __syncthreads();
    block_exclusive_scan(lenh, kLenBins, part);
    for (int i = tid; i < a.ntiles; i += kPlanThreads) {
        const int pos = atomicAdd(&lenh[kLenBins - 1 - min(hist[i], kLenBins - 1)], 1);
        a.tile_order[pos] = i;
    }
    __syncthreads();
    const int total = block_exclusive_scan(hist, a.ntiles, part);
    for (int i = tid; i < a.ntiles; i += kPlanThreads) {
        a.tile_start[i] = hist[i];
        a.tile_cursor[i] = hist[i];
    }
    if (tid == 0) a.tile_start[a.ntiles] = total;
}

__global__ __launch_bounds__(256) void plan_fill_kernel(PlanArgs a) {
    __shared__ LevelTab tb;
    load_tab(a, tb);
    __syncthreads();
    const int sub = threadIdx.x % kPlanLanes;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (256 / kPlanLanes);
    for (int64_t k = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) / kPlanLanes; k < a.K;
         k += stride) {
        if (sub == 0) {
            const int pos = atomicAdd(&a.key_count[a.keys[k]], 1);
            a.perm[pos] = static_cast<int32_t>(k);
        }
        if (a.ntiles > 0) {
            const float *r = a.rois + 5 * k;
            const int bb = roi_batch(r[0], a.N);
            if (bb < 0) continue;
            const int lvl = a.levels_out[k];
            int tx0, tx1, ty0, ty1;
            roi_tile_box(a, tb, lvl, r[1], r[2], r[3], r[4], tx0, tx1, ty0, ty1);
            const int w = tx1 - tx0 + 1;
            const int n = w * (ty1 - ty0 + 1);
            const int base = tb.tbase[lvl] + bb * tb.nty[lvl] * tb.ntx[lvl];
            for (int i = sub; i < n; i += kPlanLanes) {
                const int dy = i / w;
                const int t = base + (ty0 + dy) * tb.ntx[lvl] + tx0 + (i - dy * w);
                const int p = atomicAdd(&a.tile_cursor[t], 1);
                if (p < a.capacity) a.tile_rois[p] = static_cast<int32_t>(k);
            }
        }
    }
}

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t box_plus1, int32_t *out, hipStream_t stream) {
    const int blocks = min((K + 255) / 256, 4096);
    level_map_kernel<<<blocks, 256, 0, stream>>>(rois, K, L, finest_scale, box_plus1, out);
    return hipGetLastError();
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
    if (a.K <= kPlanSmall) {
        const size_t shmem =
            static_cast<size_t>(max(a.nbins, a.ntiles) + kPlanThreads + 3 * kPlanSmall) *
            sizeof(int32_t);
        plan_small_kernel<<<1, kPlanThreads, shmem, stream>>>(a);
        return hipGetLastError();
    }
    // key counts, and the tile counts that become tile_start
    const int ntc = a.ntiles > 0 ? a.ntiles + 1 : 0;
    const int nclear = a.nbins + ntc;
    plan_clear_kernel<<<max(1, min((nclear + 255) / 256, 1024)), 256, 0, stream>>>(
        a.key_count, a.nbins, a.tile_start, ntc);
    const int blocks = max(1, min((a.K + 256 / kPlanLanes - 1) / (256 / kPlanLanes), 4096));
    plan_count_kernel<<<blocks, 256, 0, stream>>>(a);
    const size_t shmem =
        static_cast<size_t>(max(a.nbins, a.ntiles) + kPlanThreads) * sizeof(int32_t);
    plan_scan_kernel<<<1, kPlanThreads, shmem, stream>>>(a);
    plan_fill_kernel<<<blocks, 256, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
