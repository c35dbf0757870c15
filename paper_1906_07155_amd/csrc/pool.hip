// pool.hip -- RoI max pooling forward and backward.
//
// RoIPool is the other RoI pooling operator of the RoIExtractor (MMDetection
// §3.1): Fast R-CNN (listed among the two-stage methods in §2) quantizes the box to
// whole feature pixels, cuts it into out_h x out_w bins and keeps each bin's maximum.
// Definition, tie rule and sentinels are stated in include/roi_extract.h.
//
// Kernels:
//   pool_fwd_cl_kernel     channels-last levels, out_h * out_w <= kPoolFastBins.  One
//                          workgroup = one RoI x one slice of 64 channels; lanes run
//                          over channels, so every pixel read is one coalesced load,
//                          and each wave scans the pixels of its bins in row-major order
//                          with sixteen loads in flight.  Values and argmax leave through
//                          an LDS transpose so the [C][PH][PW] blocks are stored
//                          contiguously at the RoI's original index.
//   pool_fwd_generic_kernel any strides and grid sizes: one thread per output element.
//   pool_bwd_cl_kernel     channels-last gradient levels: the RoI's gradient and argmax
//                          blocks are read coalesced through LDS, then every lane adds
//                          its channel's gradients to the argmax pixels with no-return
//                          fp32 atomics (each channel has its own argmax, so the targets
//                          of one instruction are scattered).
//   pool_bwd_generic_kernel any strides: one thread per upstream-gradient element.
#include <float.h>

#include "internal.hpp"

namespace rex {

constexpr int kPoolBatch = 16;   // pixel loads of one bin in flight at a time

// Pixel range [lo, hi) of bin p along one axis, binary32, one rounding per operation:
// the box end points are rounded to whole pixels (halves away from zero), the box
// spans both of them, and the bin edges are floor / ceil of p * len / P, shifted by
// the box start and clipped to [0, size].
struct PoolRange {
    int lo, hi;
};

__device__ __forceinline__ PoolRange pool_bin(float c1, float c2, float scale, int P, int p,
                                              int size) {
    const float s = roundf(c1 * scale);
    const float e = roundf(c2 * scale);
    float len = e - s;
    len = len + 1.0f;
    len = fmaxf(len, 1.0f);
    const float bin = len / static_cast<float>(P);
    const float a = static_cast<float>(p) * bin;
    const float b = static_cast<float>(p + 1) * bin;
    const int si = static_cast<int>(s);
    const int lo = static_cast<int>(floorf(a)) + si;
    const int hi = static_cast<int>(ceilf(b)) + si;
    PoolRange r;
    r.lo = min(max(lo, 0), size);
    r.hi = min(max(hi, 0), size);
    return r;
}

// Bit pattern stored for the "no comparable value" sentinel -FLT_MAX: binary32 as is;
// bfloat16 takes the most negative finite bf16 (-FLT_MAX rounded toward zero), since
// rounding to nearest would give -inf.
template <typename TO> __device__ __forceinline__ void store_pool(gptr<TO> p, float v);
template <> __device__ __forceinline__ void store_pool<float>(gptr<float> p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_pool<uint16_t>(gptr<uint16_t> p, float v) {
    *p = (v == -FLT_MAX) ? static_cast<uint16_t>(0xFF7Fu) : f32_to_bf16(v);
}

// ---------------------------------------------------------------------------
// General strided forward
// ---------------------------------------------------------------------------

template <typename T, typename TO>
__global__ __launch_bounds__(256) void pool_fwd_generic_kernel(PoolArgs a) {
    const int PH = a.PH, PW = a.PW;
    const int64_t NB = static_cast<int64_t>(PH) * PW;
    const int64_t CNB = static_cast<int64_t>(a.lv.C) * NB;
    const int64_t total = static_cast<int64_t>(a.K) * CNB;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t k = e / CNB;
        const int64_t rem = e - k * CNB;
        const int64_t c = rem / NB;
        const int j = static_cast<int>(rem - c * NB);
        const int ph = j / PW, pw = j - (j / PW) * PW;
        float best = 0.0f;
        int arg = -1;
        const float *r = a.rois + 5 * k;
        const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
        if (lvl >= 0 && lvl < a.lv.num) {
            const LevelArg L = level_at(a.lv, lvl);
            const int b = roi_batch(r[0], a.lv.N);
            if (b >= 0) {
                const PoolRange ry = pool_bin(r[2], r[4], L.scale, PH, ph, L.H);
                const PoolRange rx = pool_bin(r[1], r[3], L.scale, PW, pw, L.W);
                if (ry.hi > ry.lo && rx.hi > rx.lo) {
                    best = -FLT_MAX;
                    const gcptr<T> base = as_global<T>(L.data) + b * L.sn + c * L.sc;
                    for (int y = ry.lo; y < ry.hi; ++y)
                        for (int x = rx.lo; x < rx.hi; ++x) {
                            const float v = load_f32(base + y * L.sh + x * L.sw);
                            if (v > best) {
                                best = v;
                                arg = y * L.W + x;
                            }
                        }
                }
            }
        }
        store_pool<TO>(as_global_mut<TO>(a.out) + e, best);
        a.argmax[e] = arg;
    }
}

// ---------------------------------------------------------------------------
// Channels-last forward
// ---------------------------------------------------------------------------

template <typename T, typename TO>
__global__ __launch_bounds__(256) void pool_fwd_cl_kernel(PoolArgs a) {
    // [64][NB] values then [64][NB] argmax; sized at launch (64 * NB * 8 bytes)
    extern __shared__ __align__(16) float s_pool[];
    const int PH = a.PH, PW = a.PW;
    const int NB = PH * PW;
    float *const s_val = s_pool;
    int *const s_arg = reinterpret_cast<int *>(s_pool + 64 * NB);
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int slot = static_cast<int>(lid / static_cast<uint32_t>(a.nslices));
    const int slice = static_cast<int>(lid) - slot * a.nslices;
    int k = a.perm ? a.perm[slot] : slot;
    const bool kvalid = k >= 0 && k < a.K;
    if (!kvalid) k = 0;
    const float *r = a.rois + 5 * static_cast<int64_t>(k);
    const float rb = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
    const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
    const bool lvalid = lvl >= 0 && lvl < a.lv.num;
    const LevelArg L = level_at(a.lv, lvalid ? lvl : 0);
    const int b = roi_batch(rb, a.lv.N);
    const bool active = kvalid && lvalid && b >= 0;

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int c = slice * 64 + lane;
    const int nch = min(64, a.lv.C - slice * 64);
    // one image of the level through a buffer resource; lanes past the last channel
    // read out of range (zero) and their results are never stored
    const char *img = static_cast<const char *>(L.data) +
                      static_cast<int64_t>(active ? b : 0) * L.sn * static_cast<int64_t>(sizeof(T));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(img, L.img_bytes);
    const uint32_t vo = lane < nch ? static_cast<uint32_t>(c) * uint32_t(sizeof(T)) : kBufOOB;
    const uint32_t sh = static_cast<uint32_t>(L.sh) * uint32_t(sizeof(T));
    const uint32_t sw = static_cast<uint32_t>(L.sw) * uint32_t(sizeof(T));

    // bins dealt round-robin to the four waves
    for (int jb = wave; jb < NB; jb += 4) {
        const int ph = jb / PW, pw = jb - (jb / PW) * PW;
        {
            const PoolRange ry = pool_bin(y1, y2, L.scale, PH, ph, L.H);
            const PoolRange rx = pool_bin(x1, x2, L.scale, PW, pw, L.W);
            float best = 0.0f;
            int arg = -1;
            if (active && ry.hi > ry.lo && rx.hi > rx.lo) {
                best = -FLT_MAX;
                // The bin's pixels in row-major order, kPoolBatch loads in flight at a
                // time, then compared in order so the first maximum wins.  A position
                // past the bin takes the out-of-range lane offset and reads zero without
                // a memory access (the hardware range check covers the lane offset only,
                // never the scalar one, so the scalar offset is always an in-map pixel);
                // its value is skipped.
                const int nx = rx.hi - rx.lo;
                const int n = (ry.hi - ry.lo) * nx;
                int y = ry.lo, x = rx.lo;
                for (int i0 = 0; i0 < n; i0 += kPoolBatch) {
                    float v[kPoolBatch];
                    int yy = y, xx = x;
#pragma unroll
                    for (int j = 0; j < kPoolBatch; ++j) {
                        const bool in_bin = i0 + j < n;
                        const uint32_t off = in_bin ? static_cast<uint32_t>(yy) * sh +
                                                          static_cast<uint32_t>(xx) * sw
                                                    : 0u;
                        v[j] = raw_to_f32<T>(buf_load_raw_s<T>(rs, in_bin ? vo : kBufOOB, off));
                        if (++xx == rx.hi) {
                            xx = rx.lo;
                            ++yy;
                        }
                    }
#pragma unroll
                    for (int j = 0; j < kPoolBatch; ++j) {
                        if (i0 + j < n && v[j] > best) {
                            best = v[j];
                            arg = y * L.W + x;
                        }
                        if (++x == rx.hi) {
                            x = rx.lo;
                            ++y;
                        }
                    }
                }
            }
            s_val[lane * NB + ph * PW + pw] = best;
            s_arg[lane * NB + ph * PW + pw] = arg;
        }
    }
    __syncthreads();
    if (!kvalid) return;   // uniform over the workgroup, after the last barrier
    // [nch][NB] block of RoI k, contiguous in out and argmax
    const int64_t o0 = (static_cast<int64_t>(k) * a.lv.C + static_cast<int64_t>(slice) * 64) * NB;
    const gptr<TO> out = as_global_mut<TO>(a.out) + o0;
    gptr<int32_t> am = as_global_mut<int32_t>(a.argmax) + o0;
    for (int e = threadIdx.x; e < nch * NB; e += 256) {
        store_pool<TO>(out + e, s_val[e]);
        am[e] = s_arg[e];
    }
}

bool pool_fwd_fast_available(int PH, int PW) { return PH * PW <= kPoolFastBins; }

hipError_t launch_pool_fwd(PoolArgs a, int feat_dtype, int out_dtype, bool fast,
                           hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    if (fast) {
        a.nslices = (a.lv.C + 63) / 64;
        const int64_t grid = static_cast<int64_t>(a.K) * a.nslices;
        if (grid < (int64_t(1) << 24)) {
            const uint32_t g = static_cast<uint32_t>(grid);
            const size_t lds = static_cast<size_t>(64) * a.PH * a.PW * 8;
            if (feat_dtype == kF32 && out_dtype == kF32)
                pool_fwd_cl_kernel<float, float><<<g, 256, lds, stream>>>(a);
            else if (feat_dtype == kF32)
                pool_fwd_cl_kernel<float, uint16_t><<<g, 256, lds, stream>>>(a);
            else if (out_dtype == kF32)
                pool_fwd_cl_kernel<uint16_t, float><<<g, 256, lds, stream>>>(a);
            else
                pool_fwd_cl_kernel<uint16_t, uint16_t><<<g, 256, lds, stream>>>(a);
            return hipGetLastError();
        }
    }
    const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * a.PH * a.PW;
    const uint32_t blocks = static_cast<uint32_t>(std::min<int64_t>((total + 255) / 256, 16384));
    if (feat_dtype == kF32 && out_dtype == kF32)
        pool_fwd_generic_kernel<float, float><<<blocks, 256, 0, stream>>>(a);
    else if (feat_dtype == kF32)
        pool_fwd_generic_kernel<float, uint16_t><<<blocks, 256, 0, stream>>>(a);
    else if (out_dtype == kF32)
        pool_fwd_generic_kernel<uint16_t, float><<<blocks, 256, 0, stream>>>(a);
    else
        pool_fwd_generic_kernel<uint16_t, uint16_t><<<blocks, 256, 0, stream>>>(a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backward: gradient to the argmax pixels
// ---------------------------------------------------------------------------

template <typename TG>
__global__ __launch_bounds__(256) void pool_bwd_generic_kernel(PoolArgs a) {
    const int64_t NB = static_cast<int64_t>(a.PH) * a.PW;
    const int64_t CNB = static_cast<int64_t>(a.lv.C) * NB;
    const int64_t total = static_cast<int64_t>(a.K) * CNB;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t k = e / CNB;
        const int64_t c = (e - k * CNB) / NB;
        const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
        if (lvl < 0 || lvl >= a.lv.num) continue;
        const LevelArg L = level_at(a.lv, lvl);
        const int b = roi_batch(a.rois[5 * k], a.lv.N);
        if (b < 0) continue;
        const int am = a.argmax[e];
        if (am < 0 || am >= L.H * L.W) continue;
        const int y = am / L.W, x = am - (am / L.W) * L.W;
        const float g = load_f32(as_global<TG>(a.gout) + e);
        unsafeAtomicAdd(static_cast<float *>(const_cast<void *>(L.data)) + b * L.sn + c * L.sc +
                            y * L.sh + x * L.sw,
                        g);
    }
}

template <typename TG>
__global__ __launch_bounds__(256) void pool_bwd_cl_kernel(PoolArgs a) {
    extern __shared__ __align__(16) float s_pool[];   // 64 * NB * 8 bytes, as the forward
    const int NB = a.PH * a.PW;
    float *const s_g = s_pool;
    int *const s_am = reinterpret_cast<int *>(s_pool + 64 * NB);
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int slot = static_cast<int>(lid / static_cast<uint32_t>(a.nslices));
    const int slice = static_cast<int>(lid) - slot * a.nslices;
    const int k = a.perm ? a.perm[slot] : slot;
    if (k < 0 || k >= a.K) return;   // uniform over the workgroup, before any barrier
    const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
    if (lvl < 0 || lvl >= a.lv.num) return;
    const LevelArg L = level_at(a.lv, lvl);
    const int b = roi_batch(a.rois[5 * static_cast<int64_t>(k)], a.lv.N);
    if (b < 0) return;

    const int nch = min(64, a.lv.C - slice * 64);
    const int64_t o0 = (static_cast<int64_t>(k) * a.lv.C + static_cast<int64_t>(slice) * 64) * NB;
    const gcptr<TG> gsrc = as_global<TG>(a.gout) + o0;
    const gcptr<int32_t> asrc = as_global<int32_t>(a.argmax) + o0;
    for (int e = threadIdx.x; e < nch * NB; e += 256) {
        s_g[e] = load_f32(gsrc + e);
        s_am[e] = asrc[e];
    }
    __syncthreads();

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    if (lane >= nch) return;
    const int c = slice * 64 + lane;
    const int HW = L.H * L.W;
    float *const base = static_cast<float *>(const_cast<void *>(L.data)) + b * L.sn + c;
    for (int j = wave; j < NB; j += 4) {
        const int am = s_am[lane * NB + j];
        if (am < 0 || am >= HW) continue;
        const int y = am / L.W, x = am - (am / L.W) * L.W;
        unsafeAtomicAdd(base + y * L.sh + x * L.sw, s_g[lane * NB + j]);
    }
}

hipError_t launch_pool_bwd(PoolArgs a, int gout_dtype, bool fast, hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    if (fast) {
        a.nslices = (a.lv.C + 63) / 64;
        const int64_t grid = static_cast<int64_t>(a.K) * a.nslices;
        if (grid < (int64_t(1) << 24)) {
            const uint32_t g = static_cast<uint32_t>(grid);
            const size_t lds = static_cast<size_t>(64) * a.PH * a.PW * 8;
            if (gout_dtype == kF32)
                pool_bwd_cl_kernel<float><<<g, 256, lds, stream>>>(a);
            else
                pool_bwd_cl_kernel<uint16_t><<<g, 256, lds, stream>>>(a);
            return hipGetLastError();
        }
    }
    const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * a.PH * a.PW;
    const uint32_t blocks = static_cast<uint32_t>(std::min<int64_t>((total + 255) / 256, 16384));
    if (gout_dtype == kF32)
        pool_bwd_generic_kernel<float><<<blocks, 256, 0, stream>>>(a);
    else
        pool_bwd_generic_kernel<uint16_t><<<blocks, 256, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
