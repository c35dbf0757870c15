// fwd.hip -- RoIAlign forward (rows a3-a5 of the hot path).
//
// Operator: the RoIExtractor of MMDetection §3.1 in its RoIAlign form; definition
// and conventions in include/roi_extract.h.
//
// Two kernels:
//   fwd_cl_kernel       channels-last levels (stride_c == 1), specialised output
//                       grids.  One workgroup = one RoI x up to 4 channel slices
//                       (one wavefront each).  The RoI's sample geometry (bilinear
//                       indices and weights of every sample row and column) is
//                       computed once into LDS and shared by every channel; lanes
//                       run over channels, so each corner tap is one coalesced,
//                       channel-contiguous load.  Results are transposed through a
//                       small per-wave LDS tile so the [C][PH][PW] block of the RoI is
//                       stored contiguously at its original RoI index.
//   fwd_generic_kernel  any strides, output size and sampling ratio: one thread per
//                       output element.
#include "internal.hpp"

namespace rex {

// ---------------------------------------------------------------------------
// General strided kernel
// ---------------------------------------------------------------------------

template <typename T, typename TO>
__global__ __launch_bounds__(256) void fwd_generic_kernel(FwdArgs a) {
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
        float sum = 0.0f;
        const float *r = a.rois + 5 * k;
        const int lvl = a.roi_levels ? a.roi_levels[k] : 0;
        if (lvl >= 0 && lvl < a.lv.num) {
            const LevelArg L = level_at(a.lv, lvl);
            const int b = roi_batch(r[0], a.lv.N);
            if (b >= 0) {
                const Axis ax = axis_setup(r[1], r[3], L.scale, a.aligned, PW, a.S);
                const Axis ay = axis_setup(r[2], r[4], L.scale, a.aligned, PH, a.S);
                const gcptr<T> base = as_global<T>(L.data) + b * L.sn + c * L.sc;
                for (int iy = 0; iy < ay.grid; ++iy) {
                    const Tap ty = axis_tap(ay, ph, iy, L.H);
                    if (ty.lo < 0) continue;
                    const gcptr<T> r0 = base + ty.lo * L.sh;
                    const gcptr<T> r1 = base + ty.hi * L.sh;
                    for (int ix = 0; ix < ax.grid; ++ix) {
                        const Tap tx = axis_tap(ax, pw, ix, L.W);
                        if (tx.lo < 0) continue;
                        sum = fmaf(ty.wlo * tx.wlo, load_f32(r0 + tx.lo * L.sw), sum);
                        sum = fmaf(ty.wlo * tx.whi, load_f32(r0 + tx.hi * L.sw), sum);
                        sum = fmaf(ty.whi * tx.wlo, load_f32(r1 + tx.lo * L.sw), sum);
                        sum = fmaf(ty.whi * tx.whi, load_f32(r1 + tx.hi * L.sw), sum);
                    }
                }
                const int count = max(ay.grid * ax.grid, 1);
                sum = sum / static_cast<float>(count);
            }
        }
        store_f32(as_global_mut<TO>(a.out) + e, sum);
    }
}

// ---------------------------------------------------------------------------
// Channels-last kernel
// ---------------------------------------------------------------------------

// Channels per LDS transpose chunk: the largest divisor of CL whose chunk holds at
// most 800 floats.
__host__ __device__ constexpr int chunk_channels(int CL, int NB) {
    int c = CL;
    while (c > 1 && c * NB > 800) c /= 2;
    return c;
}

template <typename T, typename TO, int PH, int PW, int S, int CL>
__global__ __launch_bounds__(256) void fwd_cl_kernel(FwdArgs a) {
    constexpr int NG = 64 / CL;                 // bin groups per wavefront
    constexpr int NB = PH * PW;
    constexpr int BPL = (NB + NG - 1) / NG;     // bins per lane
    constexpr int NR = PH * S;
    constexpr int NCOL = PW * S;
    constexpr int CHK = chunk_channels(CL, NB);
    static_assert(NR + NCOL <= 256, "geometry must fit one pass of the workgroup");

    __shared__ Tap srow[NR];
    __shared__ Tap scol[NCOL];
    __shared__ float stile[4][CHK * NB];

    // Which RoI: XCD-aware block order, then the plan's permutation.
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int slot = static_cast<int>(lid / static_cast<uint32_t>(a.wg_per_roi));
    const int sub = static_cast<int>(lid) - slot * a.wg_per_roi;
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

    // a3: sample geometry of the RoI, once, shared by every channel.
    {
        const Axis ax = axis_setup(x1, x2, L.scale, a.aligned, PW, S);
        const Axis ay = axis_setup(y1, y2, L.scale, a.aligned, PH, S);
        const int t = threadIdx.x;
        if (t < NR) {
            srow[t] = axis_tap(ay, t / S, t % S, L.H);
        } else if (t < NR + NCOL) {
            const int u = t - NR;
            scol[u] = axis_tap(ax, u / S, u % S, L.W);
        }
    }
    __syncthreads();

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int slice = sub * 4 + wave;
    const bool wave_on = slice < a.nslices;
    const int cc = lane % CL;
    const int bg = lane / CL;
    const int c = slice * CL + cc;
    const bool lane_on = active && wave_on && c < a.lv.C;
    const gcptr<T> base = as_global<T>(L.data) + (lane_on ? (b * L.sn + c) : 0);
    const int64_t sh = L.sh, sw = L.sw;

    // a4: gather and average.  Every load is issued unconditionally (an invalid
    // sample reads pixel 0 and its contribution is discarded by a select), which
    // keeps the body straight-line so many loads are in flight at once.
    float acc[BPL];
#pragma clang loop unroll(full)
    for (int i = 0; i < BPL; ++i) {
        const int j = bg + NG * i;
        float s = 0.0f;
        if (lane_on && j < NB) {
            const int ph = j / PW;
            const int pw = j - ph * PW;
#pragma unroll
            for (int iy = 0; iy < S; ++iy) {
                const Tap ty = srow[ph * S + iy];
                const bool vy = ty.lo >= 0;
                const gcptr<T> p0 = base + (vy ? ty.lo : 0) * sh;
                const gcptr<T> p1 = base + (vy ? ty.hi : 0) * sh;
#pragma unroll
                for (int ix = 0; ix < S; ++ix) {
                    const Tap tx = scol[pw * S + ix];
                    const bool v = vy && tx.lo >= 0;
                    const int64_t xl = (tx.lo >= 0 ? tx.lo : 0) * sw;
                    const int64_t xh = (tx.lo >= 0 ? tx.hi : 0) * sw;
                    const float v00 = load_f32(p0 + xl);
                    const float v01 = load_f32(p0 + xh);
                    const float v10 = load_f32(p1 + xl);
                    const float v11 = load_f32(p1 + xh);
                    float q = (ty.wlo * tx.wlo) * v00;
                    q = fmaf(ty.wlo * tx.whi, v01, q);
                    q = fmaf(ty.whi * tx.wlo, v10, q);
                    q = fmaf(ty.whi * tx.whi, v11, q);
                    s += v ? q : 0.0f;
                }
            }
            s = s / static_cast<float>(S * S);
        }
        acc[i] = s;
    }

    // a5: transpose through LDS and store [CL][PH][PW] contiguously at RoI k.
    const gptr<TO> out_blk = as_global_mut<TO>(a.out) +
                        (static_cast<int64_t>(k) * a.lv.C + static_cast<int64_t>(slice) * CL) * NB;
    const int nch = min(CL, a.lv.C - slice * CL);
    float *tile = stile[wave];
#pragma unroll
    for (int c0 = 0; c0 < CL; c0 += CHK) {
        if (cc >= c0 && cc < c0 + CHK) {
#pragma unroll
            for (int i = 0; i < BPL; ++i) {
                const int j = bg + NG * i;
                if (j < NB) tile[(cc - c0) * NB + j] = acc[i];
            }
        }
        wave_sync();
        const int ne = max(0, min(CHK, nch - c0)) * NB;
        if (kvalid && wave_on) {
            for (int e = lane; e < ne; e += 64) store_f32(out_blk + c0 * NB + e, tile[e]);
        }
        wave_sync();
    }
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------

bool fwd_fast_available(int PH, int PW, int S) {
    return S == 2 && ((PH == 7 && PW == 7) || (PH == 14 && PW == 14));
}

template <typename T, typename TO>
static hipError_t launch_fwd_typed(FwdArgs a, bool fast, hipStream_t stream) {
    if (fast) {
        const int CL = (a.PH == 7) ? 64 : 16;
        a.nslices = (a.lv.C + CL - 1) / CL;
        a.wg_per_roi = (a.nslices + 3) / 4;
        const int64_t grid = static_cast<int64_t>(a.K) * a.wg_per_roi;
        // a dispatch holds fewer than 2^32 work-items; beyond that, the strided kernel
        if (grid >= (int64_t(1) << 24)) return launch_fwd_typed<T, TO>(a, false, stream);
        if (a.PH == 7)
            fwd_cl_kernel<T, TO, 7, 7, 2, 64><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
        else
            fwd_cl_kernel<T, TO, 14, 14, 2, 16><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
    } else {
        const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * a.PH * a.PW;
        const int64_t blocks = std::min<int64_t>((total + 255) / 256, 16384);
        fwd_generic_kernel<T, TO><<<static_cast<uint32_t>(blocks), 256, 0, stream>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_fwd(FwdArgs a, int feat_dtype, int out_dtype, bool fast, hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    if (feat_dtype == kF32 && out_dtype == kF32) return launch_fwd_typed<float, float>(a, fast, stream);
    if (feat_dtype == kF32 && out_dtype == kBF16)
        return launch_fwd_typed<float, uint16_t>(a, fast, stream);
    if (feat_dtype == kBF16 && out_dtype == kF32)
        return launch_fwd_typed<uint16_t, float>(a, fast, stream);
    return launch_fwd_typed<uint16_t, uint16_t>(a, fast, stream);
}

}  // namespace rex
