// bwd.hip -- RoIAlign backward (rows a6-a7 of the hot path).
//
// The backward of the RoIExtractor (MMDetection §3.2 runs forward and backward
// every iteration) is the transpose of the forward: every valid sample adds
// g[k,c,ph,pw] * w / count into the four pixels the forward read.
//
// Kernels:
//   bwd_cl_kernel       channels-last gradient levels, specialised grids.  Lanes run
//                       over channels, so the 64 lanes of one atomic instruction hit
//                       64 consecutive floats of one pixel.  Contributions of one RoI
//                       to the same (pixel, channel) are merged before any atomic: the
//                       sample geometry is separable (weight = wy * wx), so the kernel
//                       first folds the RoI's gradient rows into per-tap-row profiles
//                       (y direction), then folds each profile into per-tap-column
//                       sums (x direction), and issues exactly one fp32 atomic per
//                       distinct tap pixel and channel.  Both folds are small state
//                       machines over the monotone sequence of tap rows/columns; their
//                       branches depend only on the RoI, so they are wave-uniform.
//   bwd_generic_kernel  any strides / sizes: one thread per gradient element, four
//                       atomics per valid sample.
//   zero kernels        clear the gradient pyramid.
#include "internal.hpp"

namespace rex {

__device__ __forceinline__ void atomic_add_f32(gptr<float> p, float v) {
    unsafeAtomicAdd((float *)p, v);
}

// ---------------------------------------------------------------------------
// General strided kernel
// ---------------------------------------------------------------------------

template <typename TG>
__global__ __launch_bounds__(256) void bwd_generic_kernel(BwdArgs a) {
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
        const int b = roi_batch(r[0], a.lv.N);
        if (b < 0) continue;
        const Axis ax = axis_setup(r[1], r[3], L.scale, a.aligned, PW, a.S);
        const Axis ay = axis_setup(r[2], r[4], L.scale, a.aligned, PH, a.S);
        const int count = max(ay.grid * ax.grid, 1);
        const float g = load_f32(as_global<TG>(a.gout) + e) / static_cast<float>(count);
        const gptr<float> base = as_global_mut<float>(const_cast<void *>(L.data)) + b * L.sn + c * L.sc;
        for (int iy = 0; iy < ay.grid; ++iy) {
            const Tap ty = axis_tap(ay, ph, iy, L.H);
            if (ty.lo < 0) continue;
            const gptr<float> r0 = base + ty.lo * L.sh;
            const gptr<float> r1 = base + ty.hi * L.sh;
            for (int ix = 0; ix < ax.grid; ++ix) {
                const Tap tx = axis_tap(ax, pw, ix, L.W);
                if (tx.lo < 0) continue;
                atomic_add_f32(r0 + tx.lo * L.sw, g * (ty.wlo * tx.wlo));
                atomic_add_f32(r0 + tx.hi * L.sw, g * (ty.wlo * tx.whi));
                atomic_add_f32(r1 + tx.lo * L.sw, g * (ty.whi * tx.wlo));
                atomic_add_f32(r1 + tx.hi * L.sw, g * (ty.whi * tx.whi));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Channels-last kernel with merged contributions
// ---------------------------------------------------------------------------

// Fold one finished tap row (profile P over the PW bins) into per-column sums and
// add each distinct column once.  `grow` points at (row, channel) of the lane.
template <int PW, int S>
__device__ __forceinline__ void emit_row(gptr<float> grow, int64_t sw, const Tap *scol,
                                         const float (&P)[PW], bool lane_on) {
    int q0 = -4;
    bool h0 = false, h1 = false;
    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
    for (int pw = 0; pw < PW; ++pw) {
#pragma unroll
        for (int ix = 0; ix < S; ++ix) {
            const Tap tx = scol[pw * S + ix];
            const int lo = uniform_i(tx.lo);
            if (lo < 0) continue;
            const int hi = uniform_i(tx.hi);
            const float wlo = uniform_f(tx.wlo), whi = uniform_f(tx.whi);
            const float v = P[pw];
            if (lo != q0) {
                if (lo == q0 + 1) {
                    if (h0 && lane_on) atomic_add_f32(grow + q0 * sw, a0);
                    a0 = a1;
                    h0 = h1;
                } else {
                    if (h0 && lane_on) atomic_add_f32(grow + q0 * sw, a0);
                    if (h1 && lane_on) atomic_add_f32(grow + (q0 + 1) * sw, a1);
                    a0 = 0.0f;
                    h0 = false;
                }
                a1 = 0.0f;
                h1 = false;
                q0 = lo;
            }
            a0 = fmaf(wlo, v, a0);
            h0 = true;
            if (hi != lo) {
                a1 = fmaf(whi, v, a1);
                h1 = true;
            } else {
                a0 = fmaf(whi, v, a0);
            }
        }
    }
    if (h0 && lane_on) atomic_add_f32(grow + q0 * sw, a0);
    if (h1 && lane_on) atomic_add_f32(grow + (q0 + 1) * sw, a1);
}

template <typename TG, int PH, int PW, int S>
__global__ __launch_bounds__(256) void bwd_cl_kernel(BwdArgs a) {
    constexpr int NB = PH * PW;
    constexpr int NR = PH * S;
    constexpr int NCOL = PW * S;
    constexpr int GS = PW | 1;   // odd LDS row stride: conflict-free per-lane reads
    static_assert(NR + NCOL <= 256, "geometry must fit one pass of the workgroup");

    __shared__ Tap srow[NR];
    __shared__ Tap scol[NCOL];
    __shared__ float sg[4][64 * GS];

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
    if (!active) return;   // uniform over the workgroup; no barrier follows

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int slice = sub * 4 + wave;
    if (slice >= a.nslices) return;   // uniform over the wavefront
    const int c = slice * 64 + lane;
    const bool lane_on = c < a.lv.C;
    const int nch = min(64, a.lv.C - slice * 64);
    const gptr<float> gbase =
        as_global_mut<float>(const_cast<void *>(L.data)) + b * L.sn + (lane_on ? c : 0);
    const int64_t sh = L.sh, sw = L.sw;
    const gcptr<TG> gsrc = as_global<TG>(a.gout) +
                           (static_cast<int64_t>(k) * a.lv.C + static_cast<int64_t>(slice) * 64) * NB;
    constexpr float inv_count = 1.0f / static_cast<float>(S * S);
    float *const stage = sg[wave];

    // Upstream gradient of one bin row for the wave's 64 channels: element
    // e = lane + 64*i of the [64][PW] row block.
    float nxt[PW];
    auto fetch_row = [&](int ph) {
#pragma unroll
        for (int i = 0; i < PW; ++i) {
            const int e = lane + 64 * i;
            const int ch = e / PW;
            const int pw = e - ch * PW;
            nxt[i] = ch < nch ? load_f32(gsrc + ch * NB + ph * PW + pw) : 0.0f;
        }
    };
    fetch_row(0);

    float P0[PW], P1[PW];
#pragma unroll
    for (int i = 0; i < PW; ++i) {
        P0[i] = 0.0f;
        P1[i] = 0.0f;
    }
    int r0 = -4;
    bool h0 = false, h1 = false;

    for (int ph = 0; ph < PH; ++ph) {
#pragma unroll
        for (int i = 0; i < PW; ++i) {
            const int e = lane + 64 * i;
            const int ch = e / PW;
            stage[ch * GS + (e - ch * PW)] = nxt[i];
        }
        wave_sync();
        float gr[PW];
#pragma unroll
        for (int i = 0; i < PW; ++i) gr[i] = stage[lane * GS + i] * inv_count;
        wave_sync();
        if (ph + 1 < PH) fetch_row(ph + 1);

#pragma unroll
        for (int iy = 0; iy < S; ++iy) {
            const Tap ty = srow[ph * S + iy];
            const int lo = uniform_i(ty.lo);
            if (lo < 0) continue;
            const int hi = uniform_i(ty.hi);
            const float wlo = uniform_f(ty.wlo), whi = uniform_f(ty.whi);
            if (lo != r0) {
                if (lo == r0 + 1) {
                    if (h0) emit_row<PW, S>(gbase + r0 * sh, sw, scol, P0, lane_on);
#pragma unroll
                    for (int i = 0; i < PW; ++i) P0[i] = P1[i];
                    h0 = h1;
                } else {
                    if (h0) emit_row<PW, S>(gbase + r0 * sh, sw, scol, P0, lane_on);
                    if (h1) emit_row<PW, S>(gbase + (r0 + 1) * sh, sw, scol, P1, lane_on);
#pragma unroll
                    for (int i = 0; i < PW; ++i) P0[i] = 0.0f;
                    h0 = false;
                }
#pragma unroll
                for (int i = 0; i < PW; ++i) P1[i] = 0.0f;
                h1 = false;
                r0 = lo;
            }
#pragma unroll
            for (int i = 0; i < PW; ++i) P0[i] = fmaf(wlo, gr[i], P0[i]);
            h0 = true;
            if (hi != lo) {
#pragma unroll
                for (int i = 0; i < PW; ++i) P1[i] = fmaf(whi, gr[i], P1[i]);
                h1 = true;
            } else {
#pragma unroll
                for (int i = 0; i < PW; ++i) P0[i] = fmaf(whi, gr[i], P0[i]);
            }
        }
    }
    if (h0) emit_row<PW, S>(gbase + r0 * sh, sw, scol, P0, lane_on);
    if (h1) emit_row<PW, S>(gbase + (r0 + 1) * sh, sw, scol, P1, lane_on);
}

// ---------------------------------------------------------------------------
// Zero fill
// ---------------------------------------------------------------------------

struct ZeroDense {
    float *ptr[kMaxLevels];
    int64_t start4[kMaxLevels + 1];   // prefix of float4 counts
    int64_t n[kMaxLevels];
    int32_t num;
};

__global__ __launch_bounds__(256) void zero_dense_kernel(ZeroDense z) {
    const int64_t total4 = z.start4[z.num];
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total4;
         i += stride) {
        int l = 0;
#pragma unroll
        for (int t = 1; t < kMaxLevels; ++t)
            if (t < z.num && i >= z.start4[t]) l = t;
        float *p = z.ptr[0];
        int64_t s = z.start4[0];
#pragma unroll
        for (int t = 1; t < kMaxLevels; ++t)
            if (t == l) {
                p = z.ptr[t];
                s = z.start4[t];
            }
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        as_global_mut<f32x4>(p)[i - s] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    // tails (numel % 4)
    if (blockIdx.x == 0) {
        for (int l = 0; l < z.num; ++l) {
            const int64_t n4 = (z.start4[l + 1] - z.start4[l]) * 4;
            if (threadIdx.x < z.n[l] - n4) as_global_mut<float>(z.ptr[l])[n4 + threadIdx.x] = 0.0f;
        }
    }
}

__global__ __launch_bounds__(256) void zero_strided_kernel(LevelArg L, int64_t n, int64_t c) {
    const int64_t total = n * c * L.H * L.W;
    const gptr<float> base = as_global_mut<float>(const_cast<void *>(L.data));
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        int64_t t = e;
        const int64_t x = t % L.W;
        t /= L.W;
        const int64_t y = t % L.H;
        t /= L.H;
        const int64_t ch = t % c;
        const int64_t b = t / c;
        base[b * L.sn + ch * L.sc + y * L.sh + x * L.sw] = 0.0f;
    }
}

hipError_t launch_zero(const LevelTable &lv, const int64_t *numel, const int *dense,
                       hipStream_t stream) {
    ZeroDense z{};
    int nd = 0;
    int64_t acc = 0;
    for (int l = 0; l < lv.num; ++l) {
        float *p = static_cast<float *>(const_cast<void *>(lv.l[l].data));
        if (dense[l] && (reinterpret_cast<uintptr_t>(p) % 16) == 0) {
            z.ptr[nd] = p;
            z.start4[nd] = acc;
            z.n[nd] = numel[l];
            acc += numel[l] / 4;
            ++nd;
        } else {
            const int64_t blocks = std::min<int64_t>((numel[l] + 255) / 256, 16384);
            zero_strided_kernel<<<static_cast<uint32_t>(blocks), 256, 0, stream>>>(
                lv.l[l], lv.N, lv.C);
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    if (nd == 0) return hipSuccess;
    z.num = nd;
    z.start4[nd] = acc;
    const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((acc + 255) / 256, 8192));
    zero_dense_kernel<<<static_cast<uint32_t>(blocks), 256, 0, stream>>>(z);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------

bool bwd_fast_available(int PH, int PW, int S) {
    return S == 2 && ((PH == 7 && PW == 7) || (PH == 14 && PW == 14));
}

template <typename TG>
static hipError_t launch_bwd_typed(BwdArgs a, bool fast, hipStream_t stream) {
    if (fast) {
        a.nslices = (a.lv.C + 63) / 64;
        a.wg_per_roi = (a.nslices + 3) / 4;
        const int64_t grid = static_cast<int64_t>(a.K) * a.wg_per_roi;
        // a dispatch holds fewer than 2^32 work-items; beyond that, the strided kernel
        if (grid >= (int64_t(1) << 24)) return launch_bwd_typed<TG>(a, false, stream);
        if (a.PH == 7)
            bwd_cl_kernel<TG, 7, 7, 2><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
        else
            bwd_cl_kernel<TG, 14, 14, 2><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
    } else {
        const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * a.PH * a.PW;
        const int64_t blocks = std::min<int64_t>((total + 255) / 256, 16384);
        bwd_generic_kernel<TG><<<static_cast<uint32_t>(blocks), 256, 0, stream>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_bwd(BwdArgs a, int gout_dtype, bool fast, hipStream_t stream) {
    if (a.K == 0) return hipSuccess;
    if (gout_dtype == kF32) return launch_bwd_typed<float>(a, fast, stream);
    return launch_bwd_typed<uint16_t>(a, fast, stream);
}

}  // namespace rex
