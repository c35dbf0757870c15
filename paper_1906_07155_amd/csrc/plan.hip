// plan.hip -- FPN level assignment and the RoI launch plan.
//
// Level assignment: §3.1 of MMDetection (SingleRoIExtractor reads each RoI from
// "the corresponding level" of the FPN pyramid); the rule is the FPN rule in its
// threshold form, see include/roi_extract.h.
//
// The plan is a counting sort of the RoIs by (level, image, spatial cell of the box
// centre), done by one 1024-thread workgroup with an LDS histogram: RoIs that read
// the same feature rows end up next to each other in launch order, and the
// XCD-aware block mapping of the forward/backward then keeps them on one XCD's L2.
// The order of RoIs with equal keys is whatever the LDS atomics give; only the
// keys' order and the per-level offsets are defined.
//
// The same kernel also bins the RoIs into square bin-tiles of every (level, image)
// for the gather backward: a CSR list of the RoIs whose footprint can reach each
// tile (a superset: a listed RoI may contribute nothing to the tile).
#include "internal.hpp"

namespace rex {

__global__ __launch_bounds__(256) void level_map_kernel(const float *__restrict__ rois,
                                                        int32_t K, int32_t L, float finest_scale,
                                                        int32_t *__restrict__ out) {
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x) {
        const float *r = rois + 5 * static_cast<int64_t>(k);
        out[k] = fpn_level(r[1], r[2], r[3], r[4], L, finest_scale);
    }
}

// Exclusive scan of hist[0, n) in place by the whole workgroup (per-thread chunk
// sums, a block scan of the sums, then the chunk prefixes).  Returns the total.
__device__ int block_exclusive_scan(int32_t *hist, int n, int32_t *part) {
    const int tid = threadIdx.x;
    const int per = (n + kPlanThreads - 1) / kPlanThreads;
    const int lo = min(tid * per, n);
    const int hi = min(lo + per, n);
    int s = 0;
    for (int i = lo; i < hi; ++i) s += hist[i];
    part[tid] = s;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        const int v = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    int run = tid == 0 ? 0 : part[tid - 1];
    for (int i = lo; i < hi; ++i) {
        const int c = hist[i];
        hist[i] = run;
        run += c;
    }
    const int total = part[kPlanThreads - 1];
    __syncthreads();
    return total;
}

// Bin-tiles met by a conservative box around the footprint of a RoI on its level.
// Every sample of the RoI lies between the (shifted) box edges for any output size,
// sampling ratio and alignment; taps add one pixel, and a 1.5-pixel margin absorbs
// rounding.  Non-finite boxes cover the whole map.
__device__ void roi_tile_box(const PlanArgs &a, int lvl, float x1, float y1, float x2, float y2,
                             int &tx0, int &tx1, int &ty0, int &ty1) {
    const float s = a.scale[lvl];
    const float W = static_cast<float>(a.W[lvl] - 1);
    const float H = static_cast<float>(a.H[lvl] - 1);
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
    tx1 = min(tx1, a.ntx[lvl] - 1);
    ty1 = min(ty1, a.nty[lvl] - 1);
}

// RoIs per thread kept in registers between the phases (K <= kPlanThreads * kCached);
// larger K re-reads them from memory.
constexpr int kCached = 8;

template <bool CACHED>
__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;                           // [max(nbins, ntiles)]
    int32_t *part = smem + max(a.nbins, a.ntiles);  // [kPlanThreads]
    const int tid = threadIdx.x;
    constexpr int R = CACHED ? kCached : 1;
    float cx1[R], cy1[R], cx2[R], cy2[R];
    int cb[R], clv[R], ckey[R];

    // Loads RoI k: from the cache when CACHED (slot i), else from memory.
    auto roi = [&](int i, int k, float &x1, float &y1, float &x2, float &y2, int &b, int &lvl) {
        if constexpr (CACHED) {
            x1 = cx1[i];
            y1 = cy1[i];
            x2 = cx2[i];
            y2 = cy2[i];
            b = cb[i];
            lvl = clv[i];
        } else {
            const float *r = a.rois + 5 * static_cast<int64_t>(k);
            x1 = r[1];
            y1 = r[2];
            x2 = r[3];
            y2 = r[4];
            b = roi_batch(r[0], a.N);
            lvl = a.levels_out[k];
        }
    };

    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = 0;
    __syncthreads();

    // a1: level of every RoI; key = level bucket + image + spatial cell.
#pragma unroll
    for (int i = 0; i < R; ++i) {
        for (int32_t k = tid + i * kPlanThreads; k < a.K; k += R * kPlanThreads) {
            const float *r = a.rois + 5 * static_cast<int64_t>(k);
            const float b0 = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
            const int lvl = fpn_level(x1, y1, x2, y2, a.L, a.finest_scale);
            a.levels_out[k] = lvl;
            const int bb = roi_batch(b0, a.N);
            const int b = (bb < 0 || !a.batch_in_key) ? 0 : bb;
            float cx = (x1 + x2) * 0.5f * a.scale[lvl];
            float cy = (y1 + y2) * 0.5f * a.scale[lvl];
            cx = fminf(fmaxf(cx, 0.0f), static_cast<float>(a.W[lvl] - 1));   // NaN -> 0
            cy = fminf(fmaxf(cy, 0.0f), static_cast<float>(a.H[lvl] - 1));
            const int gx = min(static_cast<int>(cx) >> a.cell_shift, a.ncx[lvl] - 1);
            const int gy = min(static_cast<int>(cy) >> a.cell_shift, a.ncy[lvl] - 1);
            const int key = a.base[lvl] + (b * a.ncy[lvl] + gy) * a.ncx[lvl] + gx;
            if constexpr (CACHED) {
                cx1[i] = x1;
                cy1[i] = y1;
                cx2[i] = x2;
                cy2[i] = y2;
                cb[i] = bb;
                clv[i] = lvl;
                ckey[i] = key;
            } else {
                a.keys[k] = key;
            }
            atomicAdd(&hist[key], 1);
        }
    }
    __syncthreads();

    block_exclusive_scan(hist, a.nbins, part);

    // Per-level offsets: the first slot of each level's bucket range.
    if (tid < a.L) a.offsets[tid] = hist[a.base[tid]];
    if (tid == 0) a.offsets[a.L] = a.K;
    __syncthreads();

    // a2: scatter RoI indices to their slots.
#pragma unroll
    for (int i = 0; i < R; ++i) {
        for (int32_t k = tid + i * kPlanThreads; k < a.K; k += R * kPlanThreads) {
            int key;
            if constexpr (CACHED)
                key = ckey[i];
            else
                key = a.keys[k];
            const int pos = atomicAdd(&hist[key], 1);
            a.perm[pos] = k;
        }
    }
    if (a.ntiles <= 0) return;   // uniform
    __syncthreads();

    // Tile binning: count the (tile, RoI) pairs, scan, then fill the CSR lists.
    for (int i = tid; i < a.ntiles; i += kPlanThreads) hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < R; ++i) {
        for (int32_t k = tid + i * kPlanThreads; k < a.K; k += R * kPlanThreads) {
            float x1, y1, x2, y2;
            int b, lvl;
            roi(i, k, x1, y1, x2, y2, b, lvl);
            if (b < 0) continue;
            int tx0, tx1, ty0, ty1;
            roi_tile_box(a, lvl, x1, y1, x2, y2, tx0, tx1, ty0, ty1);
            const int base = a.tbase[lvl] + b * a.nty[lvl] * a.ntx[lvl];
            for (int ty = ty0; ty <= ty1; ++ty)
                for (int tx = tx0; tx <= tx1; ++tx) atomicAdd(&hist[base + ty * a.ntx[lvl] + tx], 1);
        }
    }
    __syncthreads();
    const int total = block_exclusive_scan(hist, a.ntiles, part);
    for (int i = tid; i < a.ntiles; i += kPlanThreads) a.tile_start[i] = hist[i];
    if (tid == 0) a.tile_start[a.ntiles] = total;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < R; ++i) {
        for (int32_t k = tid + i * kPlanThreads; k < a.K; k += R * kPlanThreads) {
            float x1, y1, x2, y2;
            int b, lvl;
            roi(i, k, x1, y1, x2, y2, b, lvl);
            if (b < 0) continue;
            int tx0, tx1, ty0, ty1;
            roi_tile_box(a, lvl, x1, y1, x2, y2, tx0, tx1, ty0, ty1);
            const int base = a.tbase[lvl] + b * a.nty[lvl] * a.ntx[lvl];
            for (int ty = ty0; ty <= ty1; ++ty)
                for (int tx = tx0; tx <= tx1; ++tx) {
                    const int pos = atomicAdd(&hist[base + ty * a.ntx[lvl] + tx], 1);
                    if (pos < a.capacity) a.tile_rois[pos] = k;
                }
        }
    }
    __syncthreads();

    // Launch order of the tiles: longest lists first (counting sort on the list
    // length, capped at 255), so the longest sequential chains start earliest.  After
    // the fill, hist[i] is the end of tile i's list and hist[i - 1] its start.
    constexpr int kLenBins = 256;
    for (int i = tid; i < kLenBins; i += kPlanThreads) part[i] = 0;
    __syncthreads();
    for (int i = tid; i < a.ntiles; i += kPlanThreads) {
        const int len = min(hist[i] - (i > 0 ? hist[i - 1] : 0), kLenBins - 1);
        atomicAdd(&part[kLenBins - 1 - len], 1);
    }
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int i = 0; i < kLenBins; ++i) {
            const int c = part[i];
            part[i] = run;
            run += c;
        }
    }
    __syncthreads();
    for (int i = tid; i < a.ntiles; i += kPlanThreads) {
        const int len = min(hist[i] - (i > 0 ? hist[i - 1] : 0), kLenBins - 1);
        const int pos = atomicAdd(&part[kLenBins - 1 - len], 1);
        a.tile_order[pos] = i;
    }
}

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t *out, hipStream_t stream) {
    const int blocks = min((K + 255) / 256, 4096);
    level_map_kernel<<<blocks, 256, 0, stream>>>(rois, K, L, finest_scale, out);
    return hipGetLastError();
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
    const size_t shmem =
        static_cast<size_t>(max(a.nbins, a.ntiles) + kPlanThreads) * sizeof(int32_t);
    if (a.K <= kPlanThreads * kCached)
        plan_kernel<true><<<1, kPlanThreads, shmem, stream>>>(a);
    else
        plan_kernel<false><<<1, kPlanThreads, shmem, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
