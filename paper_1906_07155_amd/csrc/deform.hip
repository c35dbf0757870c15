// deform.hip -- deformable RoI pooling and its modulated form.
//
// DCN's deformable RoI pooling and DCNv2's modulated variant (general modules of
// MMDetection, §2) move every bin of the RoIAlign grid by a learned offset,
// normalized to the box size, and scale the bin average by a learned modulation.
// Definition and gradients are stated in include/roi_extract.h.
//
// Kernels:
//   deform_fwd_stream_kernel channels-last features, a fixed grid of up to 4 x 4 samples:
//                            as deform_fwd_cl_kernel, but each wave walks the samples of
//                            its bins as one sequence with two batches of corner loads
//                            in flight (see the comment above the kernel).
//   deform_fwd_cl_kernel     channels-last features.  One workgroup = one RoI x one
//                            slice of 64 channels; lanes run over channels, so every tap
//                            is one coalesced load; the bins are dealt round-robin to
//                            the four waves; results leave through an LDS transpose so
//                            the [C][PH][PW] block is stored contiguously.
//   deform_bwd_cl_kernel     channels-last features and gradients.  Same decomposition;
//                            the slice's upstream gradient block is read through LDS,
//                            feature gradients go out as no-return fp32 atomics (64
//                            consecutive channels of one pixel per instruction), and the
//                            offset and modulation gradients of a bin are summed over
//                            the wave's channels with lane shuffles and added once per
//                            wave.
//   deform_gather_kernel     the feature gradient with a plan that holds tile lists (7x7,
//                            1-2 samples per axis): per (tile region, 64 channels) the
//                            RoIs of the tile's list are added into register
//                            accumulators and every element is stored once.
//   deform_bwd_stream_kernel after the gather: offset and modulation gradients, and the
//                            taps outside their RoI's tile range, walking the samples as
//                            deform_fwd_stream_kernel does.
//   deform_*_generic_kernel  any strides: one thread per output element.
#include "gather.hpp"

namespace rex {

// One sample of a shifted bin along one axis.  Binary32, one rounding per operation:
//   x = ((start + p*bin) + shift) + ((i + 1/2)*bin) / grid.
// A sample outside [-1, size] (or not a number) is invalid; otherwise it is clamped
// like RoIAlign's, and `slope` says whether the value is bilinear in the coordinate
// (not clamped), which is where the offset gradient is nonzero.
struct DTap {
    int lo, hi;
    float wlo, whi;
    bool valid;
    bool slope;
};

__device__ __forceinline__ DTap deform_tap(const Axis &a, float shift, int p, int i, int size) {
    const float pos = static_cast<float>(p) * a.bin;
    const float b = a.start + pos;
    const float b2 = b + shift;
    const float half = static_cast<float>(i) + 0.5f;
    const float e0 = half * a.bin;
    const float e = e0 / static_cast<float>(a.grid);
    float v = b2 + e;
    DTap t;
    t.lo = t.hi = 0;
    t.wlo = t.whi = 0.0f;
    t.valid = false;
    t.slope = false;
    if (!(v >= -1.0f) || v > static_cast<float>(size)) return t;
    t.valid = true;
    t.slope = v >= 0.0f;
    v = fmaxf(v, 0.0f);
    int lo = static_cast<int>(v);
    int hi;
    if (lo >= size - 1) {
        lo = size - 1;
        hi = size - 1;
        v = static_cast<float>(lo);
        t.slope = false;
    } else {
        hi = lo + 1;
    }
    const float frac = v - static_cast<float>(lo);
    t.lo = lo;
    t.hi = hi;
    t.wlo = 1.0f - frac;
    t.whi = frac;
    return t;
}

// Shift of a bin along one axis: (gamma * offset) * box length.
__device__ __forceinline__ float deform_shift(float gamma, float off, float len) {
    const float t = gamma * off;
    return t * len;
}

// Sum over the 64 lanes by DPP moves (VALU only, no LDS round trips): an inclusive scan
// within rows of 16 lanes, then across rows, and the total read from lane 63.  Every
// lane of the wave must be active.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK,
                                                          0xf, false));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
    v = dpp_add<0x111, 0xf>(v);   // row_shr:1
    v = dpp_add<0x112, 0xf>(v);   // row_shr:2
    v = dpp_add<0x114, 0xf>(v);   // row_shr:4
    v = dpp_add<0x118, 0xf>(v);   // row_shr:8
    v = dpp_add<0x142, 0xa>(v);   // row_bcast:15
    v = dpp_add<0x143, 0xc>(v);   // row_bcast:31
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Gradient level `l` of the table, by constant indices only (as level_at).
__device__ __forceinline__ void grad_level(const DeformArgs &a, int l, float *&data, int64_t &sn,
                                           int64_t &sc, int64_t &sh, int64_t &sw) {
#define REX_GRAD_LEVEL(i)                                              \
    case i:                                                             \
        data = static_cast<float *>(const_cast<void *>(a.glv.l[i].data)); \
        sn = a.glv.l[i].sn;                                             \
        sc = a.glv.l[i].sc;                                             \
        sh = a.glv.l[i].sh;                                             \
        sw = a.glv.l[i].sw;                                             \
        break;
    switch (l) {
        REX_GRAD_LEVEL(1)
        REX_GRAD_LEVEL(2)
        REX_GRAD_LEVEL(3)
        REX_GRAD_LEVEL(4)
        REX_GRAD_LEVEL(5)
        REX_GRAD_LEVEL(6)
        REX_GRAD_LEVEL(7)
        default:
            data = static_cast<float *>(const_cast<void *>(a.glv.l[0].data));
            sn = a.glv.l[0].sn;
            sc = a.glv.l[0].sc;
            sh = a.glv.l[0].sh;
            sw = a.glv.l[0].sw;
    }
#undef REX_GRAD_LEVEL
}

// ---------------------------------------------------------------------------
// General strided kernels
// ---------------------------------------------------------------------------

template <typename T, typename TO>
__global__ __launch_bounds__(256) void deform_fwd_generic_kernel(DeformArgs a) {
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
        float val = 0.0f;
        const float *r = a.rois + 5 * k;
        const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
        if (lvl >= 0 && lvl < a.lv.num) {
            const LevelArg L = level_at(a.lv, lvl);
            const int b = roi_batch(r[0], a.lv.N);
            if (b >= 0) {
                const Axis ax = axis_setup(r[1], r[3], L.scale, a.aligned, PW, a.S);
                const Axis ay = axis_setup(r[2], r[4], L.scale, a.aligned, PH, a.S);
                const float sx = deform_shift(a.gamma, a.offset[(k * 2 + 0) * NB + j], ax.len);
                const float sy = deform_shift(a.gamma, a.offset[(k * 2 + 1) * NB + j], ay.len);
                const gcptr<T> base = as_global<T>(L.data) + b * L.sn + c * L.sc;
                float sum = 0.0f;
                for (int iy = 0; iy < ay.grid; ++iy) {
                    const DTap ty = deform_tap(ay, sy, ph, iy, L.H);
                    if (!ty.valid) continue;
                    for (int ix = 0; ix < ax.grid; ++ix) {
                        const DTap tx = deform_tap(ax, sx, pw, ix, L.W);
                        if (!tx.valid) continue;
                        sum = fmaf(ty.wlo * tx.wlo, load_f32(base + ty.lo * L.sh + tx.lo * L.sw), sum);
                        sum = fmaf(ty.wlo * tx.whi, load_f32(base + ty.lo * L.sh + tx.hi * L.sw), sum);
                        sum = fmaf(ty.whi * tx.wlo, load_f32(base + ty.hi * L.sh + tx.lo * L.sw), sum);
                        sum = fmaf(ty.whi * tx.whi, load_f32(base + ty.hi * L.sh + tx.hi * L.sw), sum);
                    }
                }
                const int count = max(ay.grid * ax.grid, 1);
                const float m = a.mask ? a.mask[k * NB + j] : 1.0f;
                val = m * (sum / static_cast<float>(count));
            }
        }
        store_f32<TO>(as_global_mut<TO>(a.out) + e, val);
    }
}

template <typename T, typename TG>
__global__ __launch_bounds__(256) void deform_bwd_generic_kernel(DeformArgs a) {
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
        const float *r = a.rois + 5 * k;
        const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
        if (lvl < 0 || lvl >= a.lv.num) continue;
        const LevelArg L = level_at(a.lv, lvl);
        float *gdata;
        int64_t gsn, gsc, gsh, gsw;
        grad_level(a, lvl, gdata, gsn, gsc, gsh, gsw);
        const int b = roi_batch(r[0], a.lv.N);
        if (b < 0) continue;
        const Axis ax = axis_setup(r[1], r[3], L.scale, a.aligned, PW, a.S);
        const Axis ay = axis_setup(r[2], r[4], L.scale, a.aligned, PH, a.S);
        const float sx = deform_shift(a.gamma, a.offset[(k * 2 + 0) * NB + j], ax.len);
        const float sy = deform_shift(a.gamma, a.offset[(k * 2 + 1) * NB + j], ay.len);
        const int count = max(ay.grid * ax.grid, 1);
        const float m = a.mask ? a.mask[k * NB + j] : 1.0f;
        const float gv = load_f32(as_global<TG>(a.gout) + e);
        const float gq = (gv * m) / static_cast<float>(count);
        const gcptr<T> base = as_global<T>(L.data) + b * L.sn + c * L.sc;
        float *const gbase = gdata + b * gsn + c * gsc;
        float px = 0.0f, py = 0.0f, pm = 0.0f;
        for (int iy = 0; iy < ay.grid; ++iy) {
            const DTap ty = deform_tap(ay, sy, ph, iy, L.H);
            if (!ty.valid) continue;
            for (int ix = 0; ix < ax.grid; ++ix) {
                const DTap tx = deform_tap(ax, sx, pw, ix, L.W);
                if (!tx.valid) continue;
                const float v11 = load_f32(base + ty.lo * L.sh + tx.lo * L.sw);
                const float v12 = load_f32(base + ty.lo * L.sh + tx.hi * L.sw);
                const float v21 = load_f32(base + ty.hi * L.sh + tx.lo * L.sw);
                const float v22 = load_f32(base + ty.hi * L.sh + tx.hi * L.sw);
                unsafeAtomicAdd(gbase + ty.lo * gsh + tx.lo * gsw, gq * (ty.wlo * tx.wlo));
                unsafeAtomicAdd(gbase + ty.lo * gsh + tx.hi * gsw, gq * (ty.wlo * tx.whi));
                unsafeAtomicAdd(gbase + ty.hi * gsh + tx.lo * gsw, gq * (ty.whi * tx.wlo));
                unsafeAtomicAdd(gbase + ty.hi * gsh + tx.hi * gsw, gq * (ty.whi * tx.whi));
                if (tx.slope) px += ty.wlo * (v12 - v11) + ty.whi * (v22 - v21);
                if (ty.slope) py += tx.wlo * (v21 - v11) + tx.whi * (v22 - v12);
                pm += ty.wlo * tx.wlo * v11 + ty.wlo * tx.whi * v12 + ty.whi * tx.wlo * v21 +
                      ty.whi * tx.whi * v22;
            }
        }
        unsafeAtomicAdd(a.grad_offset + (k * 2 + 0) * NB + j, gq * px * (a.gamma * ax.len));
        unsafeAtomicAdd(a.grad_offset + (k * 2 + 1) * NB + j, gq * py * (a.gamma * ay.len));
        if (a.grad_mask) unsafeAtomicAdd(a.grad_mask + k * NB + j, gv * pm / static_cast<float>(count));
    }
}

// ---------------------------------------------------------------------------
// Channels-last kernels
// ---------------------------------------------------------------------------

struct DeformRoi {
    int k, slice, nch;
    bool kvalid, active;
    LevelArg L;
    int b;
    Axis ax, ay;
};

__device__ __forceinline__ DeformRoi deform_roi(const DeformArgs &a) {
    DeformRoi d;
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int slot = static_cast<int>(lid / static_cast<uint32_t>(a.nslices));
    d.slice = static_cast<int>(lid) - slot * a.nslices;
    int k = a.perm ? a.perm[slot] : slot;
    d.kvalid = k >= 0 && k < a.K;
    if (!d.kvalid) k = 0;
    d.k = k;
    const float *r = a.rois + 5 * static_cast<int64_t>(k);
    const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
    const bool lvalid = lvl >= 0 && lvl < a.lv.num;
    d.L = level_at(a.lv, lvalid ? lvl : 0);
    d.b = roi_batch(r[0], a.lv.N);
    d.active = d.kvalid && lvalid && d.b >= 0;
    d.ax = axis_setup(r[1], r[3], d.L.scale, a.aligned, a.PW, a.S);
    d.ay = axis_setup(r[2], r[4], d.L.scale, a.aligned, a.PH, a.S);
    d.nch = min(64, a.lv.C - d.slice * 64);
    return d;
}

template <typename T, typename TO>
__global__ __launch_bounds__(256) void deform_fwd_cl_kernel(DeformArgs a) {
    extern __shared__ __align__(16) float s_out[];   // [64][NB]
    const int NB = a.PH * a.PW;
    const DeformRoi d = deform_roi(a);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const LevelArg &L = d.L;
    const char *img = static_cast<const char *>(L.data) +
                      static_cast<int64_t>(d.active ? d.b : 0) * L.sn * static_cast<int64_t>(sizeof(T));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(img, L.img_bytes);
    const uint32_t vo =
        lane < d.nch ? static_cast<uint32_t>(d.slice * 64 + lane) * uint32_t(sizeof(T)) : kBufOOB;
    const uint32_t sh = static_cast<uint32_t>(L.sh) * uint32_t(sizeof(T));
    const uint32_t sw = static_cast<uint32_t>(L.sw) * uint32_t(sizeof(T));
    const int count = max(d.ay.grid * d.ax.grid, 1);
    for (int jb = wave; jb < NB; jb += 4) {
        float val = 0.0f;
        if (d.active) {
            const int ph = jb / a.PW, pw = jb - (jb / a.PW) * a.PW;
            const int64_t kb = static_cast<int64_t>(d.k) * NB + jb;
            const float sx = deform_shift(a.gamma, a.offset[2 * static_cast<int64_t>(d.k) * NB + jb],
                                          d.ax.len);
            const float sy = deform_shift(
                a.gamma, a.offset[(2 * static_cast<int64_t>(d.k) + 1) * NB + jb], d.ay.len);
            float sum = 0.0f;
            for (int iy = 0; iy < d.ay.grid; ++iy) {
                const DTap ty = deform_tap(d.ay, sy, ph, iy, L.H);
                if (!ty.valid) continue;
                const uint32_t r0 = static_cast<uint32_t>(ty.lo) * sh;
                const uint32_t r1 = static_cast<uint32_t>(ty.hi) * sh;
                for (int ix = 0; ix < d.ax.grid; ++ix) {
                    const DTap tx = deform_tap(d.ax, sx, pw, ix, L.W);
                    if (!tx.valid) continue;
                    const uint32_t c0 = static_cast<uint32_t>(tx.lo) * sw;
                    const uint32_t c1 = static_cast<uint32_t>(tx.hi) * sw;
                    const float v11 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r0 + c0));
                    const float v12 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r0 + c1));
                    const float v21 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r1 + c0));
                    const float v22 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r1 + c1));
                    sum = fmaf(ty.wlo * tx.wlo, v11, sum);
                    sum = fmaf(ty.wlo * tx.whi, v12, sum);
                    sum = fmaf(ty.whi * tx.wlo, v21, sum);
                    sum = fmaf(ty.whi * tx.whi, v22, sum);
                }
            }
            const float m = a.mask ? a.mask[kb] : 1.0f;
            val = m * (sum / static_cast<float>(count));
        }
        s_out[lane * NB + jb] = val;
    }
    __syncthreads();
    if (!d.kvalid) return;   // uniform over the workgroup, after the last barrier
    const int64_t o0 =
        (static_cast<int64_t>(d.k) * a.lv.C + static_cast<int64_t>(d.slice) * 64) * NB;
    const gptr<TO> out = as_global_mut<TO>(a.out) + o0;
    for (int e = threadIdx.x; e < d.nch * NB; e += 256) store_f32<TO>(out + e, s_out[e]);
}

// The forward for a fixed grid of S x S samples per bin (S <= 4), pipelined: wave w
// takes bins w, w + 4, ... and walks their samples as one sequence (each bin's samples
// row by row), the four corner loads of two batches of kDeformBatch samples in flight
// across bin boundaries while the oldest batch is summed in the order of the
// definition.  Where each sample lies (its four byte offsets, its four weights, whether
// it is valid and whether it ends its bin) is worked out 64 samples at a time, one per
// lane, and read back per sample with lane reads.  Taps, weights and the bin sum are
// those of deform_fwd_cl_kernel, operation for operation.
constexpr int kDeformBatch = 4;              // samples per batch: 16 loads
constexpr int kDeformStreamBins = 196;       // bins of the channels-last kernels

struct DeformMeta {
    uint32_t o11, o12, o21, o22;             // byte offsets of the corners in the image
    uint32_t w11, w12, w21, w22;             // their weights (binary32 bits)
    uint32_t flags;                          // 1: valid, 2: last sample of its bin, bin << 2
};

template <typename T, typename TO>
__global__ __launch_bounds__(256) void deform_fwd_stream_kernel(DeformArgs a) {
    extern __shared__ __align__(16) float s_out[];   // [64][NB]
    __shared__ float s_sx[kDeformStreamBins], s_sy[kDeformStreamBins], s_m[kDeformStreamBins];
    const int PW = a.PW;
    const int NB = a.PH * PW;
    const DeformRoi d = deform_roi(a);
    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
    const LevelArg &L = d.L;
    const char *img = static_cast<const char *>(L.data) +
                      static_cast<int64_t>(d.active ? d.b : 0) * L.sn * static_cast<int64_t>(sizeof(T));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(img, L.img_bytes);
    const uint32_t vo =
        lane < d.nch ? static_cast<uint32_t>(d.slice * 64 + lane) * uint32_t(sizeof(T)) : kBufOOB;
    const uint32_t sh = static_cast<uint32_t>(L.sh) * uint32_t(sizeof(T));
    const uint32_t sw = static_cast<uint32_t>(L.sw) * uint32_t(sizeof(T));
    // the bins' shifts and modulation, once per workgroup; an inactive RoI stores zeros
    if (d.active && tid < NB) {
        const int64_t k = d.k;
        s_sx[tid] = deform_shift(a.gamma, a.offset[2 * k * NB + tid], d.ax.len);
        s_sy[tid] = deform_shift(a.gamma, a.offset[(2 * k + 1) * NB + tid], d.ay.len);
        s_m[tid] = a.mask ? a.mask[k * NB + tid] : 1.0f;
    }
    for (int jb = wave; jb < NB; jb += 4) s_out[lane * NB + jb] = 0.0f;
    __syncthreads();

    const int S = a.S, G = S * S;
    const int nbw = d.active && wave < NB ? (NB - wave + 3) >> 2 : 0;   // this wave's bins
    const int n_w = nbw * G;                                            // and their samples
    const float fcount = static_cast<float>(max(d.ay.grid * d.ax.grid, 1));
    // floor(n / D) = (n * ceil(2^16 / D)) >> 16 exactly for the small n and D used here
    // (n < 2^10, D <= 196: the rounding up adds less than 1/D to the quotient)
    const uint32_t mG = (65536u + G - 1) / G, mS = (65536u + S - 1) / S;
    const uint32_t mPW = (65536u + PW - 1) / PW;
    auto locate = [&](int e0, DeformMeta &m) {
        const int e = e0 + lane;
        m.o11 = m.o12 = m.o21 = m.o22 = 0;
        m.w11 = m.w12 = m.w21 = m.w22 = 0;
        m.flags = 0;
        if (e < n_w) {
            const int i = static_cast<int>((static_cast<uint32_t>(e) * mG) >> 16);
            const int sm = e - i * G;
            const int iy = static_cast<int>((static_cast<uint32_t>(sm) * mS) >> 16);
            const int ix = sm - iy * S;
            const int jb = wave + 4 * i;
            const int ph = static_cast<int>((static_cast<uint32_t>(jb) * mPW) >> 16);
            const int pw = jb - ph * PW;
            const DTap ty = deform_tap(d.ay, s_sy[jb], ph, iy, L.H);
            const DTap tx = deform_tap(d.ax, s_sx[jb], pw, ix, L.W);
            const bool valid = ty.valid && tx.valid;
            if (valid) {
                const uint32_t r0 = static_cast<uint32_t>(ty.lo) * sh, r1 = static_cast<uint32_t>(ty.hi) * sh;
                const uint32_t c0 = static_cast<uint32_t>(tx.lo) * sw, c1 = static_cast<uint32_t>(tx.hi) * sw;
                m.o11 = r0 + c0;
                m.o12 = r0 + c1;
                m.o21 = r1 + c0;
                m.o22 = r1 + c1;
                m.w11 = __float_as_uint(ty.wlo * tx.wlo);
                m.w12 = __float_as_uint(ty.wlo * tx.whi);
                m.w21 = __float_as_uint(ty.whi * tx.wlo);
                m.w22 = __float_as_uint(ty.whi * tx.whi);
            }
            m.flags = (valid ? 1u : 0u) | (sm == G - 1 ? 2u : 0u) | (static_cast<uint32_t>(i) << 2);
        }
    };
    auto issue = [&](uint32_t (&v)[4 * kDeformBatch], const DeformMeta &m, int base) {
#pragma unroll
        for (int j = 0; j < kDeformBatch; ++j) {
            v[4 * j + 0] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o11, base + j));
            v[4 * j + 1] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o12, base + j));
            v[4 * j + 2] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o21, base + j));
            v[4 * j + 3] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o22, base + j));
        }
    };
    float sum = 0.0f;
    auto consume = [&](const uint32_t (&v)[4 * kDeformBatch], const DeformMeta &m, int base) {
#pragma unroll
        for (int j = 0; j < kDeformBatch; ++j) {
            const uint32_t f = __builtin_amdgcn_readlane(m.flags, base + j);
            if (f & 1u) {
                sum = fmaf(__uint_as_float(__builtin_amdgcn_readlane(m.w11, base + j)),
                           raw_to_f32<T>(v[4 * j + 0]), sum);
                sum = fmaf(__uint_as_float(__builtin_amdgcn_readlane(m.w12, base + j)),
                           raw_to_f32<T>(v[4 * j + 1]), sum);
                sum = fmaf(__uint_as_float(__builtin_amdgcn_readlane(m.w21, base + j)),
                           raw_to_f32<T>(v[4 * j + 2]), sum);
                sum = fmaf(__uint_as_float(__builtin_amdgcn_readlane(m.w22, base + j)),
                           raw_to_f32<T>(v[4 * j + 3]), sum);
            }
            if (f & 2u) {   // the bin's last sample
                const int jb = wave + 4 * static_cast<int>(f >> 2);
                s_out[lane * NB + jb] = s_m[jb] * (sum / fcount);
                sum = 0.0f;
            }
        }
    };
    if (n_w > 0) {
        constexpr int kPerChunk = 64 / kDeformBatch;   // batches per located chunk
        DeformMeta cur, nxt;
        locate(0, cur);
        if (n_w > 64) locate(64, nxt);
        const int nbatch = (n_w + kDeformBatch - 1) / kDeformBatch;
        uint32_t va[4 * kDeformBatch], vb[4 * kDeformBatch];
        issue(va, cur, 0);
        if (nbatch > 1) issue(vb, cur, kDeformBatch);
        int c0 = 0;   // first batch of the current chunk
        for (int q = 0; q < nbatch; q += 2) {
            const int qs = q - c0;
            consume(va, cur, qs * kDeformBatch);
            if (q + 2 < nbatch) {
                if (qs + 2 < kPerChunk) issue(va, cur, (qs + 2) * kDeformBatch);
                else issue(va, nxt, (qs + 2 - kPerChunk) * kDeformBatch);
            }
            if (q + 1 >= nbatch) break;
            consume(vb, cur, (qs + 1) * kDeformBatch);
            if (q + 3 < nbatch) {
                if (qs + 3 < kPerChunk) issue(vb, cur, (qs + 3) * kDeformBatch);
                else issue(vb, nxt, (qs + 3 - kPerChunk) * kDeformBatch);
            }
            if (qs + 2 == kPerChunk) {   // the next chunk becomes the current one
                cur = nxt;
                c0 += kPerChunk;
                if ((c0 + kPerChunk) * kDeformBatch < n_w) locate((c0 + kPerChunk) * kDeformBatch, nxt);
            }
        }
    }
    __syncthreads();
    if (!d.kvalid) return;   // uniform over the workgroup, after the last barrier
    const int64_t o0 =
        (static_cast<int64_t>(d.k) * a.lv.C + static_cast<int64_t>(d.slice) * 64) * NB;
    const gptr<TO> out = as_global_mut<TO>(a.out) + o0;
    for (int e = threadIdx.x; e < d.nch * NB; e += 256) store_f32<TO>(out + e, s_out[e]);
}

template <typename T, typename TG>
__global__ __launch_bounds__(256) void deform_bwd_cl_kernel(DeformArgs a) {
    extern __shared__ __align__(16) float s_g[];   // [64][NB] upstream gradient of the slice
    const int NB = a.PH * a.PW;
    const DeformRoi d = deform_roi(a);
    if (!d.active) return;   // uniform over the workgroup, before any barrier
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int64_t o0 =
        (static_cast<int64_t>(d.k) * a.lv.C + static_cast<int64_t>(d.slice) * 64) * NB;
    const gcptr<TG> gsrc = as_global<TG>(a.gout) + o0;
    for (int e = threadIdx.x; e < d.nch * NB; e += 256) s_g[e] = load_f32(gsrc + e);
    __syncthreads();

    const bool lane_on = lane < d.nch;
    const LevelArg &L = d.L;
    float *gdata;
    int64_t gsn, gsc, gsh, gsw;
    grad_level(a, a.roi_levels ? a.roi_levels[d.k] : 0, gdata, gsn, gsc, gsh, gsw);
    const char *img = static_cast<const char *>(L.data) +
                      static_cast<int64_t>(d.b) * L.sn * static_cast<int64_t>(sizeof(T));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(img, L.img_bytes);
    const uint32_t vo =
        lane_on ? static_cast<uint32_t>(d.slice * 64 + lane) * uint32_t(sizeof(T)) : kBufOOB;
    const uint32_t sh = static_cast<uint32_t>(L.sh) * uint32_t(sizeof(T));
    const uint32_t sw = static_cast<uint32_t>(L.sw) * uint32_t(sizeof(T));
    float *const gbase = gdata + static_cast<int64_t>(d.b) * gsn + (d.slice * 64 + (lane_on ? lane : 0));
    const int count = max(d.ay.grid * d.ax.grid, 1);
    // After the tile gather, a tap whose tile lies in the RoI's tile range is written
    // already: only the others are added here.
    int tx0 = 0, tx1 = -1, ty0 = 0, ty1 = -1;
    if (a.gathered) {
        const int lvl = a.roi_levels ? a.roi_levels[d.k] : 0;
        const float *r = a.rois + 5 * static_cast<int64_t>(d.k);
        roi_tile_range(r[1], r[2], r[3], r[4], L.scale, L.W, L.H, a.tile_shift, pick(a.ntx, lvl),
                       pick(a.nty, lvl), tx0, tx1, ty0, ty1);
    }
    auto gathered_px = [&](int y, int x) {
        const int ty = y >> a.tile_shift, tx = x >> a.tile_shift;
        return ty >= ty0 && ty <= ty1 && tx >= tx0 && tx <= tx1;
    };
    const float jx = a.gamma * d.ax.len, jy = a.gamma * d.ay.len;
    for (int jb = wave; jb < NB; jb += 4) {
        const int ph = jb / a.PW, pw = jb - (jb / a.PW) * a.PW;
        const int64_t kb = static_cast<int64_t>(d.k) * NB + jb;
        const float sx = deform_shift(a.gamma, a.offset[2 * static_cast<int64_t>(d.k) * NB + jb],
                                      d.ax.len);
        const float sy = deform_shift(
            a.gamma, a.offset[(2 * static_cast<int64_t>(d.k) + 1) * NB + jb], d.ay.len);
        const float m = a.mask ? a.mask[kb] : 1.0f;
        const float gv = lane_on ? s_g[lane * NB + jb] : 0.0f;
        const float gq = (gv * m) / static_cast<float>(count);
        float px = 0.0f, py = 0.0f, pm = 0.0f;
        // One sample: its four taps feed the offset and modulation gradients, and, when
        // `scatter`, its four feature-gradient atomics.
        auto sample = [&](const DTap &ty, const DTap &tx, bool scatter) {
            const uint32_t r0 = static_cast<uint32_t>(ty.lo) * sh;
            const uint32_t r1 = static_cast<uint32_t>(ty.hi) * sh;
            const uint32_t c0 = static_cast<uint32_t>(tx.lo) * sw;
            const uint32_t c1 = static_cast<uint32_t>(tx.hi) * sw;
            const float v11 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r0 + c0));
            const float v12 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r0 + c1));
            const float v21 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r1 + c0));
            const float v22 = raw_to_f32<T>(buf_load_raw_s<T>(rs, vo, r1 + c1));
            if (scatter && lane_on) {
                if (!gathered_px(ty.lo, tx.lo))
                    unsafeAtomicAdd(gbase + ty.lo * gsh + tx.lo * gsw, gq * (ty.wlo * tx.wlo));
                if (!gathered_px(ty.lo, tx.hi))
                    unsafeAtomicAdd(gbase + ty.lo * gsh + tx.hi * gsw, gq * (ty.wlo * tx.whi));
                if (!gathered_px(ty.hi, tx.lo))
                    unsafeAtomicAdd(gbase + ty.hi * gsh + tx.lo * gsw, gq * (ty.whi * tx.wlo));
                if (!gathered_px(ty.hi, tx.hi))
                    unsafeAtomicAdd(gbase + ty.hi * gsh + tx.hi * gsw, gq * (ty.whi * tx.whi));
            }
            if (tx.slope) px += ty.wlo * (v12 - v11) + ty.whi * (v22 - v21);
            if (ty.slope) py += tx.wlo * (v21 - v11) + tx.whi * (v22 - v12);
            pm += ty.wlo * tx.wlo * v11 + ty.wlo * tx.whi * v12 + ty.whi * tx.wlo * v21 +
                  ty.whi * tx.whi * v22;
        };
        if (d.ay.grid <= 2 && d.ax.grid <= 2) {
            // At most two samples per axis.  Validity and weights are separable, so the
            // bin's feature gradient is gq * Wy[y] * Wx[x], Wy / Wx summing the tap weights
            // of the valid samples per pixel row / column.  Sample taps are monotone, so
            // they fit a window of 4 pixels from the first valid sample's low tap unless
            // the samples are more than 2 pixels apart (then per-sample atomics).  A window
            // slot any valid sample taps is `present` even with weight zero, so a
            // non-finite gradient reaches exactly the pixels of the definition.
            DTap ty[2], tx[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                ty[i] = deform_tap(d.ay, sy, ph, i, L.H);
                tx[i] = deform_tap(d.ax, sx, pw, i, L.W);
                if (i >= d.ay.grid) ty[i].valid = false;
                if (i >= d.ax.grid) tx[i].valid = false;
            }
            float wy[4] = {0.0f, 0.0f, 0.0f, 0.0f}, wx[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            bool hy[4] = {false, false, false, false}, hx[4] = {false, false, false, false};
            const int by = ty[0].valid ? ty[0].lo : ty[1].lo;
            const int bx = tx[0].valid ? tx[0].lo : tx[1].lo;
            bool fits = true;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int ylo = ty[i].lo - by, yhi = ty[i].hi - by;
                const int xlo = tx[i].lo - bx, xhi = tx[i].hi - bx;
                if (ty[i].valid) fits = fits && ylo >= 0 && yhi <= 3;
                if (tx[i].valid) fits = fits && xlo >= 0 && xhi <= 3;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (ty[i].valid) {
                        wy[e] += (ylo == e ? ty[i].wlo : 0.0f) + (yhi == e ? ty[i].whi : 0.0f);
                        hy[e] = hy[e] || ylo == e || yhi == e;
                    }
                    if (tx[i].valid) {
                        wx[e] += (xlo == e ? tx[i].wlo : 0.0f) + (xhi == e ? tx[i].whi : 0.0f);
                        hx[e] = hx[e] || xlo == e || xhi == e;
                    }
                }
            }
#pragma unroll
            for (int iy = 0; iy < 2; ++iy)
#pragma unroll
                for (int ix = 0; ix < 2; ++ix)
                    if (ty[iy].valid && tx[ix].valid) sample(ty[iy], tx[ix], !fits);
            if (fits && lane_on) {
#pragma unroll
                for (int ey = 0; ey < 4; ++ey)
#pragma unroll
                    for (int ex = 0; ex < 4; ++ex)
                        if (hy[ey] && hx[ex] && !gathered_px(by + ey, bx + ex))
                            unsafeAtomicAdd(gbase + (by + ey) * gsh + (bx + ex) * gsw,
                                            gq * (wy[ey] * wx[ex]));
            }
        } else {
            for (int iy = 0; iy < d.ay.grid; ++iy) {
                const DTap ty = deform_tap(d.ay, sy, ph, iy, L.H);
                if (!ty.valid) continue;
                for (int ix = 0; ix < d.ax.grid; ++ix) {
                    const DTap tx = deform_tap(d.ax, sx, pw, ix, L.W);
                    if (!tx.valid) continue;
                    sample(ty, tx, true);
                }
            }
        }
        // lanes past the last channel have gv = 0 and read zeros, so they add nothing
        const float sx_sum = wave_sum_dpp(gq * px);
        const float sy_sum = wave_sum_dpp(gq * py);
        const float sm_sum = wave_sum_dpp(gv * pm);
        if (lane == 0) {
            unsafeAtomicAdd(a.grad_offset + 2 * static_cast<int64_t>(d.k) * NB + jb, sx_sum * jx);
            unsafeAtomicAdd(a.grad_offset + (2 * static_cast<int64_t>(d.k) + 1) * NB + jb,
                            sy_sum * jy);
            if (a.grad_mask) unsafeAtomicAdd(a.grad_mask + kb, sm_sum / static_cast<float>(count));
        }
    }
}

// After the tile gather (DeformArgs::gathered), the rest of the backward for a fixed
// grid of S x S samples per bin (S <= 2, the grids the gather takes): the offset and
// modulation gradients, and the feature gradient of the taps outside the RoI's tile
// range.  Samples are walked as in deform_fwd_stream_kernel (the four corner loads of
// two batches in flight across bin boundaries, each sample located by a lane and read
// back with lane reads); per bin the sums over the wave's channels and their atomics
// are those of deform_bwd_cl_kernel, operation for operation.
struct DeformBwdMeta {
    uint32_t o11, o12, o21, o22;   // byte offsets of the corners in the image
    uint32_t wyl, wyh, wxl, wxh;   // tap weights (binary32 bits): rows lo / hi, columns lo / hi
    uint32_t ylo, yhi, xlo, xhi;   // tap pixels
    uint32_t flags;                // 1 valid, 2 last of its bin, 4 x slope, 8 y slope,
                                   // 16 a corner outside the tile range, bin << 5
};

template <typename T, typename TG>
__global__ __launch_bounds__(256) void deform_bwd_stream_kernel(DeformArgs a) {
    extern __shared__ __align__(16) float s_g[];   // [64][NB] upstream gradient of the slice
    __shared__ float s_sx[kDeformStreamBins], s_sy[kDeformStreamBins], s_m[kDeformStreamBins];
    const int PW = a.PW;
    const int NB = a.PH * PW;
    const DeformRoi d = deform_roi(a);
    if (!d.active) return;   // uniform over the workgroup, before any barrier
    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
    const int64_t o0 =
        (static_cast<int64_t>(d.k) * a.lv.C + static_cast<int64_t>(d.slice) * 64) * NB;
    const gcptr<TG> gsrc = as_global<TG>(a.gout) + o0;
    for (int e = tid; e < d.nch * NB; e += 256) s_g[e] = load_f32(gsrc + e);
    for (int jb = tid; jb < NB; jb += 256) {
        const int64_t k = d.k;
        s_sx[jb] = deform_shift(a.gamma, a.offset[2 * k * NB + jb], d.ax.len);
        s_sy[jb] = deform_shift(a.gamma, a.offset[(2 * k + 1) * NB + jb], d.ay.len);
        s_m[jb] = a.mask ? a.mask[k * NB + jb] : 1.0f;
    }
    __syncthreads();

    const bool lane_on = lane < d.nch;
    const LevelArg &L = d.L;
    const int lvl = a.roi_levels ? a.roi_levels[d.k] : 0;
    float *gdata;
    int64_t gsn, gsc, gsh, gsw;
    grad_level(a, lvl, gdata, gsn, gsc, gsh, gsw);
    const char *img = static_cast<const char *>(L.data) +
                      static_cast<int64_t>(d.b) * L.sn * static_cast<int64_t>(sizeof(T));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(img, L.img_bytes);
    const uint32_t vo =
        lane_on ? static_cast<uint32_t>(d.slice * 64 + lane) * uint32_t(sizeof(T)) : kBufOOB;
    const uint32_t sh = static_cast<uint32_t>(L.sh) * uint32_t(sizeof(T));
    const uint32_t sw = static_cast<uint32_t>(L.sw) * uint32_t(sizeof(T));
    float *const gbase = gdata + static_cast<int64_t>(d.b) * gsn + (d.slice * 64 + (lane_on ? lane : 0));
    const int count = max(d.ay.grid * d.ax.grid, 1);
    const float jx = a.gamma * d.ax.len, jy = a.gamma * d.ay.len;
    int tx0, tx1, ty0, ty1;
    {
        const float *r = a.rois + 5 * static_cast<int64_t>(d.k);
        roi_tile_range(r[1], r[2], r[3], r[4], L.scale, L.W, L.H, a.tile_shift, pick(a.ntx, lvl),
                       pick(a.nty, lvl), tx0, tx1, ty0, ty1);
    }
    auto in_range = [&](int y, int x) {
        const int ty = y >> a.tile_shift, tx = x >> a.tile_shift;
        return ty >= ty0 && ty <= ty1 && tx >= tx0 && tx <= tx1;
    };

    const int S = a.S, G = S * S;
    const int nbw = wave < NB ? (NB - wave + 3) >> 2 : 0;
    const int n_w = nbw * G;
    const uint32_t mG = (65536u + G - 1) / G, mS = (65536u + S - 1) / S;
    const uint32_t mPW = (65536u + PW - 1) / PW;
    auto locate = [&](int e0, DeformBwdMeta &m) {
        const int e = e0 + lane;
        m.o11 = m.o12 = m.o21 = m.o22 = 0;
        m.wyl = m.wyh = m.wxl = m.wxh = 0;
        m.ylo = m.yhi = m.xlo = m.xhi = 0;
        m.flags = 0;
        if (e < n_w) {
            const int i = static_cast<int>((static_cast<uint32_t>(e) * mG) >> 16);
            const int sm = e - i * G;
            const int iy = static_cast<int>((static_cast<uint32_t>(sm) * mS) >> 16);
            const int ix = sm - iy * S;
            const int jb = wave + 4 * i;
            const int ph = static_cast<int>((static_cast<uint32_t>(jb) * mPW) >> 16);
            const int pw = jb - ph * PW;
            const DTap ty = deform_tap(d.ay, s_sy[jb], ph, iy, L.H);
            const DTap tx = deform_tap(d.ax, s_sx[jb], pw, ix, L.W);
            const bool valid = ty.valid && tx.valid;
            uint32_t f = (sm == G - 1 ? 2u : 0u) | (static_cast<uint32_t>(i) << 5);
            if (valid) {
                const uint32_t r0 = static_cast<uint32_t>(ty.lo) * sh, r1 = static_cast<uint32_t>(ty.hi) * sh;
                const uint32_t c0 = static_cast<uint32_t>(tx.lo) * sw, c1 = static_cast<uint32_t>(tx.hi) * sw;
                m.o11 = r0 + c0;
                m.o12 = r0 + c1;
                m.o21 = r1 + c0;
                m.o22 = r1 + c1;
                m.wyl = __float_as_uint(ty.wlo);
                m.wyh = __float_as_uint(ty.whi);
                m.wxl = __float_as_uint(tx.wlo);
                m.wxh = __float_as_uint(tx.whi);
                m.ylo = ty.lo;
                m.yhi = ty.hi;
                m.xlo = tx.lo;
                m.xhi = tx.hi;
                const bool out = !in_range(ty.lo, tx.lo) || !in_range(ty.lo, tx.hi) ||
                                 !in_range(ty.hi, tx.lo) || !in_range(ty.hi, tx.hi);
                f |= 1u | (tx.slope ? 4u : 0u) | (ty.slope ? 8u : 0u) | (out ? 16u : 0u);
            }
            m.flags = f;
        }
    };
    auto issue = [&](uint32_t (&v)[4 * kDeformBatch], const DeformBwdMeta &m, int base) {
#pragma unroll
        for (int j = 0; j < kDeformBatch; ++j) {
            v[4 * j + 0] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o11, base + j));
            v[4 * j + 1] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o12, base + j));
            v[4 * j + 2] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o21, base + j));
            v[4 * j + 3] = buf_load_raw_s<T>(rs, vo, __builtin_amdgcn_readlane(m.o22, base + j));
        }
    };
    float px = 0.0f, py = 0.0f, pm = 0.0f;
    auto rdf = [&](uint32_t v, int l) { return __uint_as_float(__builtin_amdgcn_readlane(v, l)); };
    auto consume = [&](const uint32_t (&v)[4 * kDeformBatch], const DeformBwdMeta &m, int base) {
#pragma unroll
        for (int j = 0; j < kDeformBatch; ++j) {
            const int l = base + j;
            const uint32_t f = __builtin_amdgcn_readlane(m.flags, l);
            const int jb = wave + 4 * static_cast<int>(f >> 5);
            if (f & 1u) {
                const float v11 = raw_to_f32<T>(v[4 * j + 0]), v12 = raw_to_f32<T>(v[4 * j + 1]);
                const float v21 = raw_to_f32<T>(v[4 * j + 2]), v22 = raw_to_f32<T>(v[4 * j + 3]);
                const float wyl = rdf(m.wyl, l), wyh = rdf(m.wyh, l);
                const float wxl = rdf(m.wxl, l), wxh = rdf(m.wxh, l);
                if (f & 16u) {   // corners the gather does not reach
                    const int ylo = static_cast<int>(__builtin_amdgcn_readlane(m.ylo, l));
                    const int yhi = static_cast<int>(__builtin_amdgcn_readlane(m.yhi, l));
                    const int xlo = static_cast<int>(__builtin_amdgcn_readlane(m.xlo, l));
                    const int xhi = static_cast<int>(__builtin_amdgcn_readlane(m.xhi, l));
                    const float gv = lane_on ? s_g[lane * NB + jb] : 0.0f;
                    const float gq = (gv * s_m[jb]) / static_cast<float>(count);
                    if (lane_on) {
                        if (!in_range(ylo, xlo))
                            unsafeAtomicAdd(gbase + ylo * gsh + xlo * gsw, gq * (wyl * wxl));
                        if (!in_range(ylo, xhi))
                            unsafeAtomicAdd(gbase + ylo * gsh + xhi * gsw, gq * (wyl * wxh));
                        if (!in_range(yhi, xlo))
                            unsafeAtomicAdd(gbase + yhi * gsh + xlo * gsw, gq * (wyh * wxl));
                        if (!in_range(yhi, xhi))
                            unsafeAtomicAdd(gbase + yhi * gsh + xhi * gsw, gq * (wyh * wxh));
                    }
                }
                if (f & 4u) px += wyl * (v12 - v11) + wyh * (v22 - v21);
                if (f & 8u) py += wxl * (v21 - v11) + wxh * (v22 - v12);
                pm += wyl * wxl * v11 + wyl * wxh * v12 + wyh * wxl * v21 + wyh * wxh * v22;
            }
            if (f & 2u) {   // the bin's last sample: its sums over the wave's channels
                const float gv = lane_on ? s_g[lane * NB + jb] : 0.0f;
                const float gq = (gv * s_m[jb]) / static_cast<float>(count);
                const float sx_sum = wave_sum_dpp(gq * px);
                const float sy_sum = wave_sum_dpp(gq * py);
                const float sm_sum = wave_sum_dpp(gv * pm);
                if (lane == 0) {
                    const int64_t kb = static_cast<int64_t>(d.k) * NB + jb;
                    unsafeAtomicAdd(a.grad_offset + 2 * static_cast<int64_t>(d.k) * NB + jb, sx_sum * jx);
                    unsafeAtomicAdd(a.grad_offset + (2 * static_cast<int64_t>(d.k) + 1) * NB + jb,
                                    sy_sum * jy);
                    if (a.grad_mask) unsafeAtomicAdd(a.grad_mask + kb, sm_sum / static_cast<float>(count));
                }
                px = py = pm = 0.0f;
            }
        }
    };
    if (n_w > 0) {
        constexpr int kPerChunk = 64 / kDeformBatch;
        DeformBwdMeta cur, nxt;
        locate(0, cur);
        if (n_w > 64) locate(64, nxt);
        const int nbatch = (n_w + kDeformBatch - 1) / kDeformBatch;
        uint32_t va[4 * kDeformBatch], vb[4 * kDeformBatch];
        issue(va, cur, 0);
        if (nbatch > 1) issue(vb, cur, kDeformBatch);
        int c0 = 0;
        for (int q = 0; q < nbatch; q += 2) {
            const int qs = q - c0;
            consume(va, cur, qs * kDeformBatch);
            if (q + 2 < nbatch) {
                if (qs + 2 < kPerChunk) issue(va, cur, (qs + 2) * kDeformBatch);
                else issue(va, nxt, (qs + 2 - kPerChunk) * kDeformBatch);
            }
            if (q + 1 >= nbatch) break;
            consume(vb, cur, (qs + 1) * kDeformBatch);
            if (q + 3 < nbatch) {
                if (qs + 3 < kPerChunk) issue(vb, cur, (qs + 3) * kDeformBatch);
                else issue(vb, nxt, (qs + 3 - kPerChunk) * kDeformBatch);
            }
            if (qs + 2 == kPerChunk) {
                cur = nxt;
                c0 += kPerChunk;
                if ((c0 + kPerChunk) * kDeformBatch < n_w) locate((c0 + kPerChunk) * kDeformBatch, nxt);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Feature gradient, tile-gather form
// ---------------------------------------------------------------------------
// With the plan's tile lists, a workgroup owns one tile region and 64 channels (each
// wave an 8x8 quadrant, accumulators in registers) and walks the RoIs binned to the
// tile.  Within a bin, validity and tap weights are separable (RoIAlign's sampling,
// shifted), so the bin adds to the quadrant the outer product
//   acc[r][q] += Wy[r] * (gq * Wx[q]),   gq = g[c][bin] * m / count,
// with Wy[r] (Wx[q]) the summed tap weights of the bin's valid y (x) samples on row
// R0 + r (column Q0 + q), over the rows and columns some valid sample taps (so a
// non-finite gradient reaches the tapped pixels only).  Every element of the region
// is then written once.  A tap whose tile is not in its RoI's tile range (a shift
// larger than the range's margins) is never listed here; the per-RoI kernel adds those
// with atomics afterwards (DeformArgs::gathered).

constexpr int kDeformGatherBins = 49;   // 7 x 7 grids
constexpr int kDeformGatherS = 2;       // at most 2 samples per axis

bool deform_gather_available(int PH, int PW, int S) {
    return PH == 7 && PW == 7 && S >= 1 && S <= kDeformGatherS;
}

struct DeformGatherArgs {
    GatherArgs g;
    const float *offset;
    const float *mask;
    float gamma;
    int32_t S;
    int32_t aligned;
};

struct DeformGatherTaps {
    Tap ty[kDeformGatherBins][kDeformGatherS];   // invalid taps: lo = hi = -1
    Tap tx[kDeformGatherBins][kDeformGatherS];
    float m[kDeformGatherBins];
};

struct DeformGatherSmem {
    int k[64];
    int n;
};

template <typename TG>
__global__ __launch_bounds__(256) void deform_gather_kernel(DeformGatherArgs dg) {
    constexpr int PH = 7, PW = 7, NB = kDeformGatherBins;
    const GatherArgs &a = dg.g;
    __shared__ DeformGatherSmem sm;
    // two staging slots (gradient block and taps of one RoI each), separate variables so
    // the compiler can tell that reading one does not wait for the copy into the other
    __shared__ __align__(16) uint32_t blk0[64 * NB];
    __shared__ __align__(16) uint32_t blk1[64 * NB];
    __shared__ DeformGatherTaps tp0, tp1;
    GatherTile x;
    const int t = gather_tile(a, a.tile_order, x);
    const GatherHead &h = a.head[0];
    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
    const LevelArg &L = x.L;
    const int R0 = x.R0, Q0 = x.Q0;
    const int S = dg.S;
    const float fcount = static_cast<float>(S * S);
    float acc[8][8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[r][q] = 0.0f;

    int s0 = h.tile_start[t];
    int s1 = h.tile_end[t];
    s0 = max(0, min(s0, h.capacity));
    s1 = max(s0, min(s1, h.capacity));
    const int64_t kstride = static_cast<int64_t>(a.lv.C) * NB;
    const uint32_t nvalid = static_cast<uint32_t>(x.nch * NB);
    const bool wide = sizeof(TG) == 4 && (a.lv.C & 3) == 0 &&
                      (reinterpret_cast<uintptr_t>(h.gout) & 15u) == 0;

    // the gradient block of RoI k (channel group cg) into LDS, one 32-bit word per
    // element: runs of 256 words as 16-byte copies when `wide`, else runs of 64
    auto fetch = [&](int k, uint32_t *blk) {
        const char *src = static_cast<const char *>(h.gout) +
                          (static_cast<int64_t>(x.cg) * 64 * NB + static_cast<int64_t>(k) * kstride) *
                              int64_t(sizeof(TG));
        const __amdgpu_buffer_rsrc_t rs = make_rsrc(src, nvalid * uint32_t(sizeof(TG)));
        int w0 = 0;
        if (wide) {
            constexpr int NR = 64 * NB / 256;
#pragma unroll
            for (int m = 0; m < (NR + 3) / 4; ++m) {
                const int run = wave + 4 * m;
                if (m < NR / 4 || run < NR) {
                    auto *d = (__attribute__((address_space(3))) void *)(blk + 256 * run);
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        rs, d, 16, static_cast<uint32_t>(256 * run + lane * 4) * 4u, 0, 0, 0);
                }
            }
            w0 = NR * 256;
        }
        const int nr = (64 * NB - w0) / 64;
        for (int run = wave; run < nr; run += 4) {
            auto *d = (__attribute__((address_space(3))) void *)(blk + w0 + 64 * run);
            const uint32_t off = static_cast<uint32_t>(w0 + 64 * run + lane) * uint32_t(sizeof(TG));
            if constexpr (sizeof(TG) == 4)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 4, off, 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, d, 2, off, 0, 0, 0);
        }
    };

    for (int base = s0; base < s1; base += 64) {
        const int n = min(64, s1 - base);
        __syncthreads();   // the previous batch is fully consumed
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
                sm.k[pos] = k;
            }
            if (lane == 0) sm.n = __builtin_popcountll(km);
        }
        __syncthreads();
        const int nk = sm.n;
        if (nk == 0) continue;
        // Per RoI: its block copied by the buffer unit, its RoI record and shifts loaded
        // into registers (threads of a bin x axis x sample), then, after the previous RoI
        // is consumed, the taps worked out into the slot's tap table.
        struct TapIn {
            float c1, c2, off, m;
            int k;
        };
        auto load_taps = [&](int k, TapIn &in) {
            in.k = k;
            if (tid < NB * 2 * kDeformGatherS) {
                const int b = tid % NB, ax = (tid / NB) & 1;
                const float *r = h.rois + 5 * static_cast<int64_t>(k);
                in.c1 = ax ? r[2] : r[1];
                in.c2 = ax ? r[4] : r[3];
                in.off = dg.offset[(2 * static_cast<int64_t>(k) + ax) * NB + b];
                in.m = dg.mask ? dg.mask[static_cast<int64_t>(k) * NB + b] : 1.0f;
            }
        };
        auto store_taps = [&](const TapIn &in, DeformGatherTaps &tb) {
            if (tid < NB * 2 * kDeformGatherS) {
                const int b = tid % NB, ax = (tid / NB) & 1, i = tid / (2 * NB);
                const int ph = b / PW, pw = b - (b / PW) * PW;
                Tap tp;
                tp.lo = tp.hi = -1;
                tp.wlo = tp.whi = 0.0f;
                if (i < S) {
                    const Axis axis = axis_setup(in.c1, in.c2, L.scale, dg.aligned, ax ? PH : PW, S);
                    const DTap d = deform_tap(axis, deform_shift(dg.gamma, in.off, axis.len),
                                              ax ? ph : pw, i, ax ? L.H : L.W);
                    if (d.valid) {
                        tp.lo = d.lo;
                        tp.hi = d.hi;
                        tp.wlo = d.wlo;
                        tp.whi = d.whi;
                    }
                }
                if (ax) tb.ty[b][i] = tp;
                else tb.tx[b][i] = tp;
                if (ax == 0 && i == 0) tb.m[b] = in.m;
            }
        };
        auto consume = [&](const uint32_t *blk, const DeformGatherTaps &tb) {
            if (!x.wave_on) return;
            // bins with a valid tap on a row and on a column of the quadrant
            bool reach = false;
            if (lane < NB) {
                bool ry = false, rx = false;
#pragma unroll
                for (int i = 0; i < kDeformGatherS; ++i) {
                    const Tap a_ = tb.ty[lane][i], b_ = tb.tx[lane][i];
                    ry = ry || (a_.lo >= 0 && a_.hi >= R0 && a_.lo < R0 + 8);
                    rx = rx || (b_.lo >= 0 && b_.hi >= Q0 && b_.lo < Q0 + 8);
                }
                reach = ry && rx;
            }
            uint64_t bins = __ballot(reach);
            while (bins) {
                // up to four bins per pass: lane group g (16 lanes) builds bin bs[g]'s
                // weights, lanes 0-7 of the group Wy and whether a valid sample taps row
                // R0 + lane, lanes 8-15 the same for the columns
                int bs[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    bs[g] = bins ? __builtin_ctzll(bins) : -1;
                    bins &= bins - 1;   // no-op once empty
                }
                const int g_l = lane >> 4, sub = lane & 15;
                const int b_l = g_l == 0 ? bs[0] : g_l == 1 ? bs[1] : g_l == 2 ? bs[2] : bs[3];
                float w = 0.0f;
                bool hit = false;
                if (b_l >= 0) {
                    const int pos = sub < 8 ? R0 + sub : Q0 + sub - 8;
#pragma unroll
                    for (int i = 0; i < kDeformGatherS; ++i) {
                        const Tap tp = sub < 8 ? tb.ty[b_l][i] : tb.tx[b_l][i];
                        const bool a_ = tp.lo == pos, c_ = tp.hi == pos;   // invalid: -1
                        w += a_ ? tp.wlo : 0.0f;
                        w += c_ ? tp.whi : 0.0f;
                        hit = hit || a_ || c_;
                    }
                }
                const uint64_t hits = __ballot(hit);
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int b = bs[g];
                    if (b < 0) break;
                    const uint32_t rows = static_cast<uint32_t>(hits >> (16 * g)) & 0xffu;
                    const uint32_t cols = static_cast<uint32_t>(hits >> (16 * g + 8)) & 0xffu;
                    if (rows == 0 || cols == 0) continue;
                    const float gq = (raw_to_f32<TG>(blk[lane * NB + b]) * tb.m[b]) / fcount;
                    // a column no valid sample taps has Wx = 0, so gq * Wx is a zero that
                    // leaves the sums as they are unless gq is not finite
                    const bool finite = __ballot(!isfinite(gq)) == 0;
                    float X[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const float wx = __uint_as_float(
                            __builtin_amdgcn_readlane(__float_as_uint(w), 16 * g + 8 + q));
                        X[q] = gq * wx;
                    }
                    if (!finite) {
#pragma unroll
                        for (int q = 0; q < 8; ++q) X[q] = (cols >> q & 1u) ? X[q] : 0.0f;
                    }
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        if (!(rows >> r & 1u)) continue;
                        const float wy = __uint_as_float(
                            __builtin_amdgcn_readlane(__float_as_uint(w), 16 * g + r));
#pragma unroll
                        for (int q = 0; q < 8; ++q) acc[r][q] = fmaf(wy, X[q], acc[r][q]);
                    }
                }
            }
        };
        auto fetch_wait = [&]() { __builtin_amdgcn_s_waitcnt(0x0F70); };
        TapIn in;
        // Unrolled by two so that each slot is named statically: RoI j + 1 is staged
        // into one slot while RoI j is read from the other.
        fetch(uniform_i(sm.k[0]), blk0);
        load_taps(uniform_i(sm.k[0]), in);
        store_taps(in, tp0);
        fetch_wait();
        __syncthreads();
        for (int j = 0; j < nk; j += 2) {
            if (j + 1 < nk) {
                fetch(uniform_i(sm.k[j + 1]), blk1);
                load_taps(uniform_i(sm.k[j + 1]), in);
            }
            consume(blk0, tp0);
            if (j + 1 < nk) store_taps(in, tp1);
            fetch_wait();
            __syncthreads();   // slot 0 consumed, slot 1 staged
            if (j + 1 >= nk) break;
            if (j + 2 < nk) {
                fetch(uniform_i(sm.k[j + 2]), blk0);
                load_taps(uniform_i(sm.k[j + 2]), in);
            }
            consume(blk1, tp1);
            if (j + 2 < nk) store_taps(in, tp0);
            fetch_wait();
            __syncthreads();
        }
    }
    __syncthreads();   // the slots are free: the store uses one as scratch
    static_assert(64 * NB >= 4 * 512, "store scratch in a slot");
    gather_store(x, a.zero_init, acc, reinterpret_cast<float *>(blk0) + wave * 512);
}

hipError_t launch_deform_gather(GatherArgs g, const DeformArgs &d, int gout_dtype,
                                hipStream_t stream) {
    if (!gather_prepare(g)) return hipErrorInvalidConfiguration;
    const int64_t grid = static_cast<int64_t>(g.ntiles) * g.wg_per_tile * g.ncg;
    if (grid <= 0) return hipSuccess;
    if (grid >= (int64_t(1) << 24) || !deform_gather_available(d.PH, d.PW, d.S))
        return hipErrorInvalidConfiguration;
    DeformGatherArgs dg;
    dg.g = g;
    dg.offset = d.offset;
    dg.mask = d.mask;
    dg.gamma = d.gamma;
    dg.S = d.S;
    dg.aligned = d.aligned;
    const uint32_t n = static_cast<uint32_t>(grid);
    if (gout_dtype == kF32)
        deform_gather_kernel<float><<<n, 256, 0, stream>>>(dg);
    else
        deform_gather_kernel<uint16_t><<<n, 256, 0, stream>>>(dg);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void deform_clear_kernel(float *p, int64_t n, float *q,
                                                          int64_t m) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n + m;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (i < n)
            p[i] = 0.0f;
        else
            q[i - n] = 0.0f;
    }
}

template <typename T, typename TO>
static void fwd_typed(const DeformArgs &a, bool fast, hipStream_t stream) {
    const int NB = a.PH * a.PW;
    if (fast) {
        const uint32_t g = static_cast<uint32_t>(static_cast<int64_t>(a.K) * a.nslices);
        if (a.S >= 1 && a.S <= 4 && NB <= kDeformStreamBins)
            deform_fwd_stream_kernel<T, TO><<<g, 256, static_cast<size_t>(64) * NB * 4, stream>>>(a);
        else
            deform_fwd_cl_kernel<T, TO><<<g, 256, static_cast<size_t>(64) * NB * 4, stream>>>(a);
    } else {
        const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * NB;
        const uint32_t blocks = static_cast<uint32_t>(std::min<int64_t>((total + 255) / 256, 16384));
        deform_fwd_generic_kernel<T, TO><<<blocks, 256, 0, stream>>>(a);
    }
}

hipError_t launch_deform_fwd(DeformArgs a, int feat_dtype, int out_dtype, bool fast,
                             hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    a.nslices = (a.lv.C + 63) / 64;
    if (static_cast<int64_t>(a.K) * a.nslices >= (int64_t(1) << 24)) fast = false;
    if (feat_dtype == kF32 && out_dtype == kF32)
        fwd_typed<float, float>(a, fast, stream);
    else if (feat_dtype == kF32)
        fwd_typed<float, uint16_t>(a, fast, stream);
    else if (out_dtype == kF32)
        fwd_typed<uint16_t, float>(a, fast, stream);
    else
        fwd_typed<uint16_t, uint16_t>(a, fast, stream);
    return hipGetLastError();
}

template <typename T, typename TG>
static void bwd_typed(const DeformArgs &a, bool fast, hipStream_t stream) {
    const int NB = a.PH * a.PW;
    if (fast) {
        const uint32_t g = static_cast<uint32_t>(static_cast<int64_t>(a.K) * a.nslices);
        if (a.gathered && a.S >= 1 && a.S <= 4 && NB <= kDeformStreamBins)
            deform_bwd_stream_kernel<T, TG><<<g, 256, static_cast<size_t>(64) * NB * 4, stream>>>(a);
        else
            deform_bwd_cl_kernel<T, TG><<<g, 256, static_cast<size_t>(64) * NB * 4, stream>>>(a);
    } else {
        const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * NB;
        const uint32_t blocks = static_cast<uint32_t>(std::min<int64_t>((total + 255) / 256, 16384));
        deform_bwd_generic_kernel<T, TG><<<blocks, 256, 0, stream>>>(a);
    }
}

hipError_t launch_deform_bwd(DeformArgs a, int feat_dtype, int gout_dtype, bool fast,
                             hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    const int64_t NB = static_cast<int64_t>(a.PH) * a.PW;
    const int64_t n_off = static_cast<int64_t>(a.K) * 2 * NB;
    const int64_t n_mask = a.grad_mask ? static_cast<int64_t>(a.K) * NB : 0;
    const uint32_t cb =
        static_cast<uint32_t>(std::min<int64_t>((n_off + n_mask + 255) / 256, 4096));
    deform_clear_kernel<<<cb, 256, 0, stream>>>(a.grad_offset, n_off, a.grad_mask, n_mask);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    a.nslices = (a.lv.C + 63) / 64;
    if (static_cast<int64_t>(a.K) * a.nslices >= (int64_t(1) << 24)) fast = false;
    // only the channels-last kernel knows which taps the gather has written
    if (a.gathered && !fast) return hipErrorInvalidConfiguration;
    if (feat_dtype == kF32 && gout_dtype == kF32)
        bwd_typed<float, float>(a, fast, stream);
    else if (feat_dtype == kF32)
        bwd_typed<float, uint16_t>(a, fast, stream);
    else if (gout_dtype == kF32)
        bwd_typed<uint16_t, float>(a, fast, stream);
    else
        bwd_typed<uint16_t, uint16_t>(a, fast, stream);
    return hipGetLastError();
}

}  // namespace rex
