// pool.hip -- RoI max pooling forward and backward.
//
// RoIPool is the other RoI pooling operator of the RoIExtractor (MMDetection
// §3.1): Fast R-CNN (listed among the two-stage methods in §2) quantizes the box to
// whole feature pixels, cuts it into out_h x out_w bins and keeps each bin's maximum.
// Definition, tie rule and sentinels are stated in include/roi_extract.h.
//
// Kernels:
//   pool_fwd_cl_kernel     channels-last levels, out_h * out_w <= kPoolFastBins, maps
//                          of fewer than 2^24 pixels.  One workgroup = one RoI x one
//                          slice of 64 channels; lanes run over channels, so every
//                          pixel read is one coalesced load, and each wave walks the
//                          pixels of its bins as one sequence with two batches of loads
//                          in flight.  Values and argmax leave through an LDS transpose
//                          so the [C][PH][PW] blocks are stored contiguously at the
//                          RoI's original index.
//   pool_fwd_generic_kernel any strides and grid sizes: one thread per output element.
//   pool_bwd_cl_kernel     channels-last gradient levels: the RoI's gradient and argmax
//                          blocks are read coalesced through LDS, then every lane adds
//                          its channel's gradients to the argmax pixels with no-return
//                          fp32 atomics (each channel has its own argmax, so the targets
//                          of one instruction are scattered).
//   pool_gather_kernel     the backward with a plan that holds tile lists (7x7 bins):
//                          per (tile region, 64 channels), the RoIs binned to the tile
//                          are added into LDS accumulators and every gradient element
//                          is stored once (no device atomics, no separate clearing);
//                          see the comment above the kernel.
//   pool_bwd_generic_kernel any strides: one thread per upstream-gradient element.
#include <float.h>

#include "gather.hpp"

namespace rex {

constexpr int kPoolBatch = 16;   // pixel loads per batch (two batches in flight)
constexpr int kPoolWaveBins = (kPoolFastBins + 3) / 4;   // bins of one wave of the forward

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
__device__ __forceinline__ uint16_t pool_bf16(float v) {
    return (v == -FLT_MAX) ? static_cast<uint16_t>(0xFF7Fu) : f32_to_bf16(v);
}
template <typename TO> __device__ __forceinline__ void store_pool(gptr<TO> p, float v);
template <> __device__ __forceinline__ void store_pool<float>(gptr<float> p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_pool<uint16_t>(gptr<uint16_t> p, float v) {
    *p = pool_bf16(v);
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
    __shared__ int s_rng[4][kPoolFastBins];   // per bin row: first, end row; per column: first, end
    __shared__ int s_wbin[4][kPoolWaveBins * 5 + 1];   // per wave: its bins' layout, its element count
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

    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
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

    // The bins' pixel ranges, once per workgroup (bin (ph, pw) covers rows
    // [s_rng[0][ph], s_rng[1][ph]) and columns [s_rng[2][pw], s_rng[3][pw])), and the
    // results of an empty bin (0, -1) in every slot this wave owns.
    if (tid < PH) {
        const PoolRange rr = pool_bin(y1, y2, L.scale, PH, tid, L.H);
        s_rng[0][tid] = rr.lo;
        s_rng[1][tid] = rr.hi;
    } else if (tid < PH + PW) {
        const PoolRange rr = pool_bin(x1, x2, L.scale, PW, tid - PH, L.W);
        s_rng[2][tid - PH] = rr.lo;
        s_rng[3][tid - PH] = rr.hi;
    }
    for (int jb = wave; jb < NB; jb += 4) {
        s_val[lane * NB + jb] = 0.0f;
        s_arg[lane * NB + jb] = -1;
    }
    __syncthreads();

    // Wave w takes bins w, w + 4, ... and streams their pixels as one sequence, each bin
    // row by row, each row left to right: two batches of kPoolBatch loads are in
    // flight, across bin boundaries, while the oldest batch is compared in order (so
    // the first maximum of a bin still wins).  Where each element of the sequence lies
    // is worked out 64 elements at a time, one element per lane (its bin by a search
    // of the bins' starts, then row and column), and read back one element at a time
    // with a lane read, so the walk costs no scalar bookkeeping per pixel.
    //   per wave and bin i: start of the bin in the sequence, first row, first column,
    //   width, pixel count
    int *const wb = s_wbin[wave];
    const int nbw = active && wave < NB ? (NB - wave + 3) >> 2 : 0;   // this wave's bins
    {
        int area = 0, ylo = 0, xlo = 0, w = 1;
        if (lane < nbw) {
            const int jb = wave + 4 * lane;
            const int ph = jb / PW, pw = jb - ph * PW;
            ylo = s_rng[0][ph];
            xlo = s_rng[2][pw];
            const int h = s_rng[1][ph] - ylo;
            w = s_rng[3][pw] - xlo;
            area = h > 0 && w > 0 ? h * w : 0;
            if (w <= 0) w = 1;
        }
        const int incl = wave_inclusive_scan(area, lane);
        if (lane < nbw) {
            wb[lane * 5 + 0] = incl - area;
            wb[lane * 5 + 1] = ylo;
            wb[lane * 5 + 2] = xlo;
            wb[lane * 5 + 3] = w;
            wb[lane * 5 + 4] = area;
        }
        wb[kPoolWaveBins * 5] = __shfl(incl, 63);   // elements of this wave
    }
    wave_sync();
    const int n_w = uniform_i(wb[kPoolWaveBins * 5]);
    const uint32_t Wu = static_cast<uint32_t>(L.W);
    // Element e0 + lane of the sequence: its byte offset in the image, and its argmax
    // index with, in the top 8 bits, 1 + the bin's number when it is the bin's last
    // pixel (0 otherwise).  Elements past the end load pixel 0 and end no bin.
    auto locate = [&](int e0, uint32_t &off, uint32_t &pixf) {
        const int e = e0 + lane;
        int bi = 0;
        for (int q = 1; q < nbw; ++q) bi = e >= uniform_i(wb[q * 5]) ? q : bi;
        off = 0;
        pixf = 0;
        if (e < n_w) {
            const int local = e - wb[bi * 5];
            const int w = wb[bi * 5 + 3];
            // row = local / w: the binary32 estimate (local < 2^24, exact as a float; the
            // reciprocal and the product add under two units of the last place of a
            // quotient below 2^23 when w >= 2, none when w = 1) is within two of it
            int row = static_cast<int>(static_cast<float>(local) * __builtin_amdgcn_rcpf(static_cast<float>(w)));
            if (row * w > local) --row;
            if (row * w > local) --row;
            if ((row + 1) * w <= local) ++row;
            if ((row + 1) * w <= local) ++row;
            const uint32_t y = static_cast<uint32_t>(wb[bi * 5 + 1] + row);
            const uint32_t x = static_cast<uint32_t>(wb[bi * 5 + 2] + (local - row * w));
            off = y * sh + x * sw;
            const bool last = local == wb[bi * 5 + 4] - 1;
            pixf = (y * Wu + x) | (last ? static_cast<uint32_t>(bi + 1) << 24 : 0u);
        }
    };
    float best = -FLT_MAX;
    int arg = -1;
    auto issue = [&](uint32_t (&v)[kPoolBatch], uint32_t off, int base) {
#pragma unroll
        for (int j = 0; j < kPoolBatch; ++j)
            v[j] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(off, base + j));
    };
    auto consume = [&](const uint32_t (&v)[kPoolBatch], uint32_t pixf, int base) {
#pragma unroll
        for (int j = 0; j < kPoolBatch; ++j) {
            const uint32_t pf = __builtin_amdgcn_readlane(pixf, base + j);
            const float f = raw_to_f32<T>(v[j]);
            if (f > best) {
                best = f;
                arg = static_cast<int>(pf & 0xFFFFFFu);
            }
            if (pf >> 24) {   // the bin's last pixel: its results, then the next bin
                const int jb = wave + 4 * static_cast<int>((pf >> 24) - 1);
                s_val[lane * NB + jb] = best;
                s_arg[lane * NB + jb] = arg;
                best = -FLT_MAX;
                arg = -1;
            }
        }
    };
    static_assert(4 * kPoolBatch == 64, "a located chunk is four batches");
    if (n_w > 0) {
        uint32_t off, pixf, off_n, pixf_n;
        uint32_t va[kPoolBatch], vb[kPoolBatch];
        locate(0, off, pixf);
        issue(va, off, 0);
        issue(vb, off, kPoolBatch);
        for (int e0 = 0; e0 < n_w; e0 += 64) {
            // batches 0-1 of this chunk are in flight; 2-3 follow, then the next chunk's 0-1
            consume(va, pixf, 0);
            if (e0 + 2 * kPoolBatch < n_w) issue(va, off, 2 * kPoolBatch);
            consume(vb, pixf, kPoolBatch);
            if (e0 + 3 * kPoolBatch < n_w) issue(vb, off, 3 * kPoolBatch);
            const bool more = e0 + 64 < n_w;
            if (more) locate(e0 + 64, off_n, pixf_n);
            if (e0 + 2 * kPoolBatch >= n_w) break;
            consume(va, pixf, 2 * kPoolBatch);
            if (more) issue(va, off_n, 0);
            if (e0 + 3 * kPoolBatch >= n_w) break;
            consume(vb, pixf, 3 * kPoolBatch);
            if (more) issue(vb, off_n, kPoolBatch);
            off = off_n;
            pixf = pixf_n;
        }
    }
    __syncthreads();
    if (!kvalid) return;   // uniform over the workgroup, after the last barrier
    // [nch][NB] block of RoI k, contiguous in out and argmax
    const int64_t o0 = (static_cast<int64_t>(k) * a.lv.C + static_cast<int64_t>(slice) * 64) * NB;
    const gptr<TO> out = as_global_mut<TO>(a.out) + o0;
    gptr<int32_t> am = as_global_mut<int32_t>(a.argmax) + o0;
    const int n = nch * NB;
    int done = 0;
    // Four elements per store where both blocks are aligned to 4 elements (always for a
    // multiple of 4 channels): 16-byte argmax stores, 16- or 8-byte value stores.  The
    // values are never read back by this operator, so they stream past the caches; the
    // argmax is read by the backward and is stored as usual.
    if ((reinterpret_cast<uintptr_t>(out) & (4 * sizeof(TO) - 1)) == 0 &&
        (reinterpret_cast<uintptr_t>(am) & 15u) == 0) {
        const int nv = n >> 2;
        for (int v = threadIdx.x; v < nv; v += 256) {
            const float4 f = *reinterpret_cast<const float4 *>(s_val + 4 * v);
            const u32x4 g = *reinterpret_cast<const u32x4 *>(s_arg + 4 * v);
            *reinterpret_cast<REX_GLOBAL u32x4 *>(am + 4 * v) = g;
            if constexpr (sizeof(TO) == 4) {
                const u32x4 w = {__float_as_uint(f.x), __float_as_uint(f.y), __float_as_uint(f.z),
                                 __float_as_uint(f.w)};
                __builtin_nontemporal_store(w, reinterpret_cast<REX_GLOBAL u32x4 *>(out + 4 * v));
            } else {
                const u32x2 w = {static_cast<uint32_t>(pool_bf16(f.x)) | (static_cast<uint32_t>(pool_bf16(f.y)) << 16),
                                 static_cast<uint32_t>(pool_bf16(f.z)) | (static_cast<uint32_t>(pool_bf16(f.w)) << 16)};
                __builtin_nontemporal_store(w, reinterpret_cast<REX_GLOBAL u32x2 *>(out + 4 * v));
            }
        }
        done = nv << 2;
    }
    for (int e = done + static_cast<int>(threadIdx.x); e < n; e += 256) {
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

// ---------------------------------------------------------------------------
// Backward, tile-gather form
// ---------------------------------------------------------------------------
// The gradient of a pixel is the sum of the upstream gradients of every (RoI, bin)
// whose argmax it is, for its channel.  With the plan's tile lists a workgroup owns the
// 256 pixels of a tile region and 64 channels, accumulated in LDS, and walks the RoIs
// binned to the tile: each RoI's gradient and argmax blocks ([64 channels][bins],
// contiguous in memory) are read coalesced into registers, those of the next two RoIs
// while the current one is added, and every element whose argmax lies in the region is
// added to its (channel, pixel) accumulator with an LDS atomic.  No bin geometry is needed: the tile lists
// hold every RoI whose bins can reach the tile.  The accumulators then leave through
// the quadrant store of the align gather, so every gradient element is written once,
// which replaces both the clearing and the device-scope atomics of the per-RoI form
// (many bins of overlapping RoIs share their maximum pixel, and device-scope atomics
// on one address are serialised).

constexpr int kPoolGatherBins = 49;      // 7 x 7 grids
constexpr int kPoolAccPitch = 260;       // LDS words per channel: 256 pixels + 4, 16-byte
                                         // rows whose channels start in different banks
constexpr int kPoolBlock = 64 * kPoolGatherBins;                  // elements of one block
constexpr int kPoolThreads = 512;                                // 8 waves
constexpr int kPoolPerThread = (kPoolBlock + kPoolThreads - 1) / kPoolThreads;   // 7

bool pool_gather_available(int PH, int PW) { return PH * PW == kPoolGatherBins && PH == 7; }

template <typename TG>
__global__ __launch_bounds__(kPoolThreads) void pool_gather_kernel(GatherArgs a) {
    constexpr int NB = kPoolGatherBins;
    constexpr int P = kPoolAccPitch;
    constexpr int E = kPoolPerThread;
    __shared__ __align__(16) float s_acc[64 * P];   // [channel][pixel of the region]
    __shared__ int s_k[64];
    __shared__ int s_n;
    static_assert(64 * P >= 4 * 512, "store scratch in the accumulators");
    GatherTile x;
    const int t = gather_tile(a, a.tile_order, x);
    const GatherHead &h = a.head[0];
    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
    // waves 0-3 own the region's quadrants; waves 4-7 only read and add
    if (wave >= 4) x.wave_on = false;
    const LevelArg &L = x.L;
    static_assert(P % 4 == 0, "16-byte accumulator rows");
    for (int e = tid; e < 64 * P / 4; e += kPoolThreads)
        reinterpret_cast<float4 *>(s_acc)[e] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);

    int s0 = h.tile_start[t];
    int s1 = h.tile_end[t];
    s0 = max(0, min(s0, h.capacity));
    s1 = max(s0, min(s1, h.capacity));
    const int64_t kstride = static_cast<int64_t>(a.lv.C) * NB;
    const uint32_t nvalid = static_cast<uint32_t>(x.nch * NB);
    // The region's origin as an argmax index, its size, and the level width divisor.
    const int RW = x.WC1 - x.WC0, RH = x.WR1 - x.WR0;   // RW * RH = 256
    const uint32_t W = static_cast<uint32_t>(L.W);
    const uint32_t wm = pick(a.wid_m, x.l);
    const int32_t wsh = pick(a.wid_sh, x.l);
    // Per element of this thread: its channel row of the accumulators (or -1 past the
    // block), fixed for the whole walk.
    int crow[E];
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const int e = tid + kPoolThreads * i;
        crow[i] = e < kPoolBlock ? (e / NB) * P : -1;
    }
    uint32_t gv[3][E], av[3][E];
    auto fetch = [&](int j, uint32_t (&g)[E], uint32_t (&am)[E]) {
        const int k = uniform_i(s_k[j]);
        const int64_t e0 = static_cast<int64_t>(x.cg) * 64 * NB + static_cast<int64_t>(k) * kstride;
        const __amdgpu_buffer_rsrc_t rg = make_rsrc(
            static_cast<const char *>(h.gout) + e0 * int64_t(sizeof(TG)), nvalid * uint32_t(sizeof(TG)));
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(
            reinterpret_cast<const char *>(h.argmax) + e0 * 4, nvalid * 4u);
#pragma unroll
        for (int i = 0; i < E; ++i) {
            const uint32_t e = static_cast<uint32_t>(tid + kPoolThreads * i);
            g[i] = buf_load_raw<TG>(rg, e * uint32_t(sizeof(TG)));
            am[i] = __builtin_amdgcn_raw_buffer_load_b32(ra, e * 4u, 0, 0);
        }
    };
    // Adds one staged RoI: an element whose argmax (y W + x) lies in the region goes to
    // its accumulator.  -1 (an empty bin) and indices off the level give rows past it.
    auto add = [&](const uint32_t (&g)[E], const uint32_t (&am)[E]) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
            const uint32_t u = am[i];
            const uint32_t y = fdiv(u, wm, wsh);
            const uint32_t xx = u - y * W;
            const uint32_t ly = y - static_cast<uint32_t>(x.WR0);
            const uint32_t lx = xx - static_cast<uint32_t>(x.WC0);
            if (crow[i] >= 0 && ly < static_cast<uint32_t>(RH) && lx < static_cast<uint32_t>(RW))
                atomicAdd(&s_acc[crow[i] + static_cast<int>(ly) * RW + static_cast<int>(lx)],
                          raw_to_f32<TG>(g[i]));
        }
    };

    for (int base = s0; base < s1; base += 64) {
        const int n = min(64, s1 - base);
        __syncthreads();   // the previous batch's records are no longer read
        // Records of this batch (wave 0): RoIs of this tile's level and image, compacted.
        if (wave == 0) {
            bool keep = false;
            int k = 0;
            if (lane < n) {
                k = h.tile_rois[base + lane];
                if (k >= 0 && k < h.K) {
                    const int lvl = h.roi_levels ? h.roi_levels[k] : 0;
                    keep = lvl == x.l && roi_batch(h.rois[5 * static_cast<int64_t>(k)], a.lv.N) == x.b;
                }
            }
            const uint64_t km = __ballot(keep);
            if (keep) {
                const int pos = static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                    static_cast<uint32_t>(km >> 32),
                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(km), 0u)));
                s_k[pos] = k;
            }
            if (lane == 0) s_n = __builtin_popcountll(km);
        }
        __syncthreads();
        const int nk = s_n;
        if (nk == 0) continue;
        // Unrolled by three so that each register set is named statically: the loads
        // of RoIs j + 1 and j + 2 are in flight while RoI j is added.
        fetch(0, gv[0], av[0]);
        if (nk > 1) fetch(1, gv[1], av[1]);
        for (int j = 0; j < nk; j += 3) {
            if (j + 2 < nk) fetch(j + 2, gv[2], av[2]);
            add(gv[0], av[0]);
            if (j + 1 >= nk) break;
            if (j + 3 < nk) fetch(j + 3, gv[0], av[0]);
            add(gv[1], av[1]);
            if (j + 2 >= nk) break;
            if (j + 4 < nk) fetch(j + 4, gv[1], av[1]);
            add(gv[2], av[2]);
        }
    }
    __syncthreads();   // every addition is done
    float acc[8][8] = {};
    if (x.wave_on) {
        // a quadrant row is 8 words at a multiple of 8 (RW and the quadrant's origin are
        // multiples of 8): two 16-byte reads
        const int p0 = (x.R0 - x.WR0) * RW + (x.Q0 - x.WC0);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const float4 lo = *reinterpret_cast<const float4 *>(s_acc + lane * P + p0 + r * RW);
            const float4 hi = *reinterpret_cast<const float4 *>(s_acc + lane * P + p0 + r * RW + 4);
            acc[r][0] = lo.x;
            acc[r][1] = lo.y;
            acc[r][2] = lo.z;
            acc[r][3] = lo.w;
            acc[r][4] = hi.x;
            acc[r][5] = hi.y;
            acc[r][6] = hi.z;
            acc[r][7] = hi.w;
        }
    }
    __syncthreads();   // the accumulators are read: the store may reuse them as scratch
    if (wave < 4) gather_store(x, a.zero_init, acc, s_acc + wave * 512);
}

hipError_t launch_pool_gather(GatherArgs a, int gout_dtype, hipStream_t stream) {
    if (!gather_prepare(a)) return hipErrorInvalidConfiguration;
    const int64_t grid = static_cast<int64_t>(a.ntiles) * a.wg_per_tile * a.ncg;
    if (grid <= 0) return hipSuccess;
    if (grid >= (int64_t(1) << 24) || !pool_gather_available(a.PH, a.PW))
        return hipErrorInvalidConfiguration;
    const uint32_t g = static_cast<uint32_t>(grid);
    if (gout_dtype == kF32)
        pool_gather_kernel<float><<<g, kPoolThreads, 0, stream>>>(a);
    else
        pool_gather_kernel<uint16_t><<<g, kPoolThreads, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
