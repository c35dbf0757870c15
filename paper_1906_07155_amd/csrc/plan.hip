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

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;              // [nbins]
    int32_t *part = smem + a.nbins;    // [kPlanThreads]
    const int tid = threadIdx.x;

    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = 0;
    __syncthreads();

    // a1: level of every RoI; key = level bucket + image + spatial cell.
    for (int32_t k = tid; k < a.K; k += kPlanThreads) {
        const float *r = a.rois + 5 * static_cast<int64_t>(k);
        const float b0 = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
        const int lvl = fpn_level(x1, y1, x2, y2, a.L, a.finest_scale);
        a.levels_out[k] = lvl;
        int b = roi_batch(b0, a.N);
        if (b < 0 || !a.batch_in_key) b = 0;
        float cx = (x1 + x2) * 0.5f * a.scale[lvl];
        float cy = (y1 + y2) * 0.5f * a.scale[lvl];
        cx = fminf(fmaxf(cx, 0.0f), static_cast<float>(a.W[lvl] - 1));   // NaN -> 0
        cy = fminf(fmaxf(cy, 0.0f), static_cast<float>(a.H[lvl] - 1));
        const int gx = min(static_cast<int>(cx) >> a.cell_shift, a.ncx[lvl] - 1);
        const int gy = min(static_cast<int>(cy) >> a.cell_shift, a.ncy[lvl] - 1);
        const int key = a.base[lvl] + (b * a.ncy[lvl] + gy) * a.ncx[lvl] + gx;
        a.keys[k] = key;
        atomicAdd(&hist[key], 1);
    }
    __syncthreads();

    // Exclusive scan of the histogram: per-thread chunk sums, a block scan of the
    // sums, then the chunk prefixes.
    const int per = (a.nbins + kPlanThreads - 1) / kPlanThreads;
    const int lo = min(tid * per, a.nbins);
    const int hi = min(lo + per, a.nbins);
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
    __syncthreads();

    // Per-level offsets: the first slot of each level's bucket range.
    if (tid < a.L) a.offsets[tid] = hist[a.base[tid]];
    if (tid == 0) a.offsets[a.L] = a.K;
    __syncthreads();

    // a2: scatter RoI indices to their slots.
    for (int32_t k = tid; k < a.K; k += kPlanThreads) {
        const int pos = atomicAdd(&hist[a.keys[k]], 1);
        a.perm[pos] = k;
    }
}

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t *out, hipStream_t stream) {
    const int blocks = min((K + 255) / 256, 4096);
    level_map_kernel<<<blocks, 256, 0, stream>>>(rois, K, L, finest_scale, out);
    return hipGetLastError();
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
    const size_t shmem = static_cast<size_t>(a.nbins + kPlanThreads) * sizeof(int32_t);
    plan_kernel<<<1, kPlanThreads, shmem, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
