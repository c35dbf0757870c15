// bwd.hip -- RoIAlign backward (rows a6-a7 of the hot path).
//
// The backward of the RoIExtractor (MMDetection §3.2 runs forward and backward
// every iteration) is the transpose of the forward: every valid sample adds
// g[k,c,ph,pw] * w / count into the four pixels the forward read.
//
// Kernels:
//   bwd_gather_kernel   the default: per (bin-tile, 64 channels), the RoIs binned to the
//                       tile are gathered into register accumulators and every gradient
//                       element is stored once (no atomics, clearing included); see
//                       "Tile-gather backward" below.
//   bwd_gather2_kernel  the same for two heads on one pyramid in one pass.
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
#include <algorithm>

#include "gather.hpp"

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
// Tile-gather backward
// ---------------------------------------------------------------------------
//
// Device-scope fp32 atomics are executed beyond the per-XCD L2 on this part and
// saturate at about 1.2 TB/s of payload, so the scatter form of the backward is
// bound by atomic transactions.  This kernel inverts the loop: a wavefront owns an
// 8x8-pixel quadrant of one (level, image) for 64 channels, keeps its 64 sums in
// registers, walks the RoIs the plan binned to the enclosing bin-tile, and stores
// every pixel once with plain coalesced stores (which also replaces the zero fill).
// For each RoI the quadrant's separable weights are built in LDS:
//   Wy[ph][r] = sum over the samples of bin row ph of the bilinear weight they put on
//               row R0 + r (divided by the sample count), likewise Wx[pw][q],
// and the contribution is  acc[r][q] += sum_ph Wy[ph][r] * sum_pw Wx[pw][q] * g[ph][pw].

// First / last set bit of a multi-word ballot, -1 if none (uniform scalar values).
template <int P>
__device__ __forceinline__ int first_set(const uint64_t (&b)[P]) {
#pragma unroll
    for (int p = 0; p < P; ++p)
        if (b[p]) return p * 64 + __builtin_ctzll(b[p]);
    return -1;
}
template <int P>
__device__ __forceinline__ int last_set(const uint64_t (&b)[P]) {
#pragma unroll
    for (int p = P - 1; p >= 0; --p)
        if (b[p]) return p * 64 + 63 - __builtin_clzll(b[p]);
    return -1;
}

// acc[r][q] += yrow[r] * X[q] for the rows r0 .. r0 + NR - 1 of the quadrant.
template <int R0, int NR>
__device__ __forceinline__ void outer_rows(float (&acc)[8][8], const float *yrow,
                                           const float (&X)[8]) {
    static_assert(R0 % 4 == 0 && NR % 4 == 0, "rows in aligned groups of 4");
    float yr[8];
#pragma unroll
    for (int h = R0 / 4; h < (R0 + NR) / 4; ++h) {
        const float4 y = *reinterpret_cast<const float4 *>(yrow + 4 * h);
        yr[4 * h] = y.x;
        yr[4 * h + 1] = y.y;
        yr[4 * h + 2] = y.z;
        yr[4 * h + 3] = y.w;
    }
#pragma unroll
    for (int rr = R0; rr < R0 + NR; ++rr)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[rr][q] = fmaf(yr[rr], X[q], acc[rr][q]);
}

// One RoI's contribution to a wave's 8x8 quadrant, for the bin rows pha..phb that
// reach the quadrant's rows and the npw bin columns pwa.. that reach its columns:
//   X[q] = sum over pw of Wx[pw][q] * g[ph][pw]
//   acc[r][q] += Wy[ph][r] * X[q]
// gl points at g[0][pwa] of this lane's channel, wxa at Wx[pwa][0], wy at Wy[0][0];
// yb holds the nonzero pattern of Wy (bit ph * 8 + r), which decides the half
// quadrants (rows 0-3, 4-7) a bin row updates.
template <typename TG, int PW, int YP>
__device__ __forceinline__ void gather_rows(float (&acc)[8][8], const uint32_t *gl,
                                            const float *wxa, const float *wy,
                                            const uint64_t (&yb)[YP], int pha, int phb, int npw) {
    for (int ph = pha; ph <= phb; ++ph) {
        const uint32_t rb = static_cast<uint32_t>(yb[YP == 1 ? 0 : ph >> 3] >> ((ph & 7) * 8)) & 0xffu;
        if (rb == 0) continue;
        const uint32_t *gr = gl + ph * PW;
        // The run of bins is unrolled up to its longest possible length, so every
        // LDS address is a fixed offset from gr / wxa (no loop-carried pointers, which
        // would hide from the compiler that these reads do not touch the slot being
        // filled by the copy in flight).
        float X[8];
#pragma unroll
        for (int i = 0; i < PW; ++i) {
            if (i >= npw) break;
            const float gv = raw_to_f32<TG>(gr[i]);
            const float4 w0 = *reinterpret_cast<const float4 *>(wxa + i * 8);
            const float4 w1 = *reinterpret_cast<const float4 *>(wxa + i * 8 + 4);
            const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
            for (int q = 0; q < 8; ++q) X[q] = i == 0 ? w[q] * gv : fmaf(w[q], gv, X[q]);
        }
        // rows 0-3 and 4-7 of the quadrant are updated only if the bin row reaches them
        if (rb & 0x0fu) outer_rows<0, 4>(acc, wy + ph * 8, X);
        if (rb & 0xf0u) outer_rows<4, 4>(acc, wy + ph * 8, X);
    }
}

// LDS of one head's pass over a tile (see gather_phase).
template <typename TG, int PH, int PW, int S>
struct GatherSmem {
    static constexpr int NR = PH * S;
    static constexpr int NCOL = PW * S;
    static constexpr int T = 8;
    static constexpr int NB = PH * PW;
    static constexpr int GB = 64 * NB;   // 32-bit words of one RoI's gradient block
    // The block is copied in runs of RUN elements, one copy instruction per run:
    // 16 bytes per lane for binary32, one element per lane for bf16.  A slot holds
    // whole runs (GBP words); the words past the block are never read.
    static constexpr int RUN = sizeof(TG) == 4 ? 256 : 64;
    static constexpr int NRUN = (GB + RUN - 1) / RUN;
    static constexpr int GBP = NRUN * RUN;
    // The staged gradient blocks form a ring of NBUF: the next RoI's block is copied
    // into the other slot by the buffer unit while the current one is consumed, when
    // two blocks fit in 52 KiB.  The copy gives every lane a 32-bit LDS slot whatever
    // the element size, so a block holds one 32-bit word per element (a bf16 value in
    // its low half).
    static constexpr int NBUF = 2 * GBP * 4 <= 53248 ? 2 : 1;
    Tap tap[2][NR + NCOL];
    __align__(16) float wy[4][PH * T];
    __align__(16) float wx[4][PW * T];
    int k[64];
    float ax[64][4];
    int rng[64][4];   // per kept RoI: tap extent ymin, ymax, xmin, xmax
    int n;
};

// One staged gradient block.  The ring's slots are separate LDS variables, so the
// compiler can tell that reading one slot does not depend on the copy into the other.
template <typename TG, int PH, int PW, int S>
struct GatherBlock {
    __align__(16) uint32_t g[GatherSmem<TG, PH, PW, S>::GBP];
};

// One head's RoIs binned to tile t, added into this wave's quadrant accumulators:
//   acc[r][q] += sum over RoIs, bins: Wy[ph][r] * sum_pw Wx[pw][q] * g[ph][pw].
// Every wave of the workgroup calls it (it holds workgroup barriers).
template <typename TG, int PH, int PW, int S>
__device__ __forceinline__ void gather_phase(const GatherHead &h, const LevelTable &lv, int t,
                                             const GatherTile &x, float (&acc)[8][8],
                                             GatherSmem<TG, PH, PW, S> &sm, uint32_t *slot0,
                                             uint32_t *slot1) {
    using SM = GatherSmem<TG, PH, PW, S>;
    constexpr int NR = SM::NR, NCOL = SM::NCOL, T = SM::T, NB = SM::NB, GB = SM::GB;
    constexpr int NBUF = SM::NBUF;
    constexpr int YP = (PH * T + 63) / 64;   // ballot passes for the row weights
    constexpr int XP = (PW * T + 63) / 64;
    static_assert(NR + NCOL <= 64, "taps are computed by one wavefront");
    static_assert(PH <= 32 && PW <= 32, "bin masks are 32-bit");

    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const int lane = tid & 63;
    const LevelArg &L = x.L;
    const int l = x.l, b = x.b, R0 = x.R0, Q0 = x.Q0;
    int s0 = h.tile_start[t];
    int s1 = h.tile_end[t];
    s0 = max(0, min(s0, h.capacity));
    s1 = max(s0, min(s1, h.capacity));
    constexpr float inv_count = 1.0f / static_cast<float>(S * S);
    float *wy = sm.wy[wave];
    float *wx = sm.wx[wave];
    const int64_t kstride = static_cast<int64_t>(lv.C) * NB;

    // Coalesced copy of kept RoI j's gradient block (nch x NB values) into LDS
    // through a buffer resource over exactly that block: run r = wave + 4 m goes to
    // words [RUN r, RUN r + RUN), lane i writing the RUN / 64 elements from RUN r +
    // i RUN / 64 on (the LDS address is the uniform run base plus the lane's bytes, in
    // lane order; the global offset is the lane's own); the range check, which works
    // per dword, supplies the zeros past the valid channels.
    const int nvalid = x.nch * NB;
    // 16-byte copies need every block 16-byte aligned: a multiple of 4 channels and an
    // aligned gradient (binary32 only)
    const bool wide = sizeof(TG) == 4 && (lv.C & 3) == 0 &&
                      (reinterpret_cast<uintptr_t>(h.gout) & 15u) == 0;
    auto fetch = [&](int j, uint32_t *gdst) {
        const int k = uniform_i(sm.k[j]);   // one resource for the wave, no waterfall
        const char *src = static_cast<const char *>(h.gout) +
                          (static_cast<int64_t>(x.cg) * 64 * NB + static_cast<int64_t>(k) * kstride) *
                              int64_t(sizeof(TG));
        const __amdgpu_buffer_rsrc_t rs = make_rsrc(src, static_cast<uint32_t>(nvalid) * uint32_t(sizeof(TG)));
        constexpr int RUN = SM::RUN, NRUN = SM::NRUN;
        if (RUN == 256 && wide) {
#pragma unroll
            for (int m = 0; m < (NRUN + 3) / 4; ++m) {
                const int run = wave + 4 * m;
                if (m < NRUN / 4 || run < NRUN) {
                    auto *dst = (__attribute__((address_space(3))) void *)(gdst + RUN * run);
                    const uint32_t off = static_cast<uint32_t>(RUN * run + lane * 4) * 4u;
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 16, off, 0, 0, 0);
                }
            }
        } else {
            // one element per lane and instruction (bf16, or blocks not 16-byte aligned)
            constexpr int NR64 = GB / 64;
#pragma unroll
            for (int m = 0; m < (NR64 + 3) / 4; ++m) {
                const int run = wave + 4 * m;
                if (m < NR64 / 4 || run < NR64) {
                    auto *dst = (__attribute__((address_space(3))) void *)(gdst + 64 * run);
                    const uint32_t off = static_cast<uint32_t>(64 * run + lane) * uint32_t(sizeof(TG));
                    if constexpr (sizeof(TG) == 4)
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 4, off, 0, 0, 0);
                    else
                        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst, 2, off, 0, 0, 0);
                }
            }
        }
    };
    // The copies of this wave are complete (vmcnt 0); a barrier then publishes them.
    auto fetch_wait = [&]() { __builtin_amdgcn_s_waitcnt(0x0F70); };
    // Sample taps of kept RoI j into tap buffer tb (lanes of wave 0).
    auto taps = [&](int j, int tb) {
        if (tid < NR + NCOL) {
            Axis ax;
            ax.grid = S;
            if (tid < NR) {
                ax.start = sm.ax[j][2];
                ax.bin = sm.ax[j][3];
                sm.tap[tb][tid] = axis_tap(ax, tid / S, tid % S, L.H);
            } else {
                ax.start = sm.ax[j][0];
                ax.bin = sm.ax[j][1];
                sm.tap[tb][tid] = axis_tap(ax, (tid - NR) / S, (tid - NR) % S, L.W);
            }
        }
    };
    // Contribution of kept RoI j to this wave's quadrant.
    auto consume = [&](int j, const uint32_t *gsrc, int tb) {
        const int ymin = sm.rng[j][0], ymax = sm.rng[j][1];
        const int xmin = sm.rng[j][2], xmax = sm.rng[j][3];
        if (!x.wave_on || ymax < R0 || ymin >= R0 + T || xmax < Q0 || xmin >= Q0 + T) return;
        // This quadrant's separable weights and which bin rows / columns reach it.
        // Ballot bit p * 64 + i marks a nonzero weight of lane u = p * 64 + i
        // (u = bin * 8 + row or column of the quadrant).
        uint64_t yb[YP], xb[XP];
#pragma unroll
        for (int p = 0; p < YP; ++p) {
            const int u = p * 64 + lane;
            bool hit = false;
            if (u < PH * T) {
                const int ph = u / T;
                const int R = R0 + (u % T);
                float w = 0.0f;
#pragma unroll
                for (int iy = 0; iy < S; ++iy) {
                    // branch-free: an invalid tap has lo = hi = -1 and matches no row
                    const Tap tp = sm.tap[tb][ph * S + iy];
                    const bool a = tp.lo == R, c = tp.hi == R;
                    w += a ? tp.wlo : 0.0f;
                    w += c ? tp.whi : 0.0f;
                    hit = hit || a || c;
                }
                wy[u] = w * inv_count;
            }
            yb[p] = __ballot(hit);
        }
#pragma unroll
        for (int p = 0; p < XP; ++p) {
            const int u = p * 64 + lane;
            bool hit = false;
            if (u < PW * T) {
                const int pw = u / T;
                const int Q = Q0 + (u % T);
                float w = 0.0f;
#pragma unroll
                for (int ix = 0; ix < S; ++ix) {
                    const Tap tp = sm.tap[tb][NR + pw * S + ix];
                    const bool a = tp.lo == Q, c = tp.hi == Q;
                    w += a ? tp.wlo : 0.0f;
                    w += c ? tp.whi : 0.0f;
                    hit = hit || a || c;
                }
                wx[u] = w;
            }
            xb[p] = __ballot(hit);
        }
        // Sample positions grow with the bin index, so the bins reaching the quadrant's
        // rows (columns) form one run [pha, phb] ([pwa, pwb]).
        const int pha = first_set(yb) / T, phb = last_set(yb) / T;
        const int pwa = first_set(xb) / T, pwb = last_set(xb) / T;
        if (pha < 0 || pwa < 0) return;
        wave_sync();

        const uint32_t *gl = gsrc + lane * NB + pwa;   // this lane's channel, stride NB (odd)
        const float *wxa = wx + pwa * T;
        gather_rows<TG, PW>(acc, gl, wxa, wy, yb, pha, phb, pwb - pwa + 1);
        // the weights are rewritten for the next RoI only after the next barrier
    };

    for (int base = s0; base < s1; base += 64) {
        const int n = min(64, s1 - base);
        __syncthreads();   // previous batch fully consumed
        // RoI records of this batch (wave 0): validity, axis parameters and tap extent.
        // RoIs whose tap extent misses the workgroup's region reach none of its pixels
        // and are dropped; the rest are compacted.
        if (wave == 0) {
            bool keep = false;
            int k = 0, ymin = INT32_MAX, ymax = -1, xmin = INT32_MAX, xmax = -1;
            float ax_s = 0.0f, ax_b = 0.0f, ay_s = 0.0f, ay_b = 0.0f;
            if (lane < n) {
                k = h.tile_rois[base + lane];
                if (k >= 0 && k < h.K) {
                    const float *r = h.rois + 5 * static_cast<int64_t>(k);
                    const float r0 = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
                    const int lvl = h.roi_levels ? h.roi_levels[k] : 0;
                    if (lvl == l && roi_batch(r0, lv.N) == b) {
                        const Axis ax = axis_setup(x1, x2, L.scale, h.aligned, PW, S);
                        const Axis ay = axis_setup(y1, y2, L.scale, h.aligned, PH, S);
                        ax_s = ax.start;
                        ax_b = ax.bin;
                        ay_s = ay.start;
                        ay_b = ay.bin;
                        // Tap extent from the first and last sample of each axis (taps
                        // are monotone in the sample index); an end sample outside the
                        // map widens the extent to the map edge, so it is a superset.
                        const Tap fy = axis_tap(ay, 0, 0, L.H);
                        const Tap ly = axis_tap(ay, PH - 1, S - 1, L.H);
                        const Tap fx = axis_tap(ax, 0, 0, L.W);
                        const Tap lx = axis_tap(ax, PW - 1, S - 1, L.W);
                        ymin = fy.lo >= 0 ? fy.lo : 0;
                        ymax = ly.lo >= 0 ? ly.hi : L.H - 1;
                        xmin = fx.lo >= 0 ? fx.lo : 0;
                        xmax = lx.lo >= 0 ? lx.hi : L.W - 1;
                        const bool yhit = ymax >= x.WR0 && ymin < x.WR1;
                        const bool xhit = xmax >= x.WC0 && xmin < x.WC1;
                        keep = yhit && xhit;
                    }
                }
            }
            const uint64_t km = __ballot(keep);
            if (keep) {
                const int pos = static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                    static_cast<uint32_t>(km >> 32),
                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(km), 0u)));
                sm.k[pos] = k;
                sm.ax[pos][0] = ax_s;
                sm.ax[pos][1] = ax_b;
                sm.ax[pos][2] = ay_s;
                sm.ax[pos][3] = ay_b;
                sm.rng[pos][0] = ymin;
                sm.rng[pos][1] = ymax;
                sm.rng[pos][2] = xmin;
                sm.rng[pos][3] = xmax;
            }
            if (lane == 0) sm.n = __builtin_popcountll(km);
        }
        __syncthreads();
        const int nk = sm.n;
        if (nk == 0) continue;
        if constexpr (NBUF == 2) {
            // Unrolled by two so that each slot is named statically: the copy of RoI
            // j + 1 into one slot lands while RoI j is read from the other.
            fetch(0, slot0);
            taps(0, 0);
            fetch_wait();
            __syncthreads();
            for (int j = 0; j < nk; j += 2) {
                if (j + 1 < nk) {
                    fetch(j + 1, slot1);
                    taps(j + 1, 1);   // the other tap buffer is idle
                }
                consume(j, slot0, 0);
                fetch_wait();
                __syncthreads();   // staged block, taps and weights are reused next
                if (j + 1 >= nk) break;
                if (j + 2 < nk) {
                    fetch(j + 2, slot0);
                    taps(j + 2, 0);
                }
                consume(j + 1, slot1, 1);
                fetch_wait();
                __syncthreads();
            }
        } else {
            for (int j = 0; j < nk; ++j) {
                if (j > 0) __syncthreads();   // the previous block is fully consumed
                fetch(j, slot0);
                taps(j, j & 1);
                fetch_wait();
                __syncthreads();
                consume(j, slot0, j & 1);
            }
        }
    }
}


template <typename TG, int PH, int PW, int S>
__global__ __launch_bounds__(256) void bwd_gather_kernel(GatherArgs a) {
    __shared__ GatherSmem<TG, PH, PW, S> sm;
    __shared__ GatherBlock<TG, PH, PW, S> blk0;
    constexpr bool two = GatherSmem<TG, PH, PW, S>::NBUF == 2;
    __shared__ GatherBlock<TG, two ? PH : 1, two ? PW : 1, S> blk1;
    GatherTile x;
    const int t = gather_tile(a, a.tile_order, x);
    float acc[8][8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[r][q] = 0.0f;
    gather_phase<TG, PH, PW, S>(a.head[0], a.lv, t, x, acc, sm, blk0.g,
                                two ? blk1.g : nullptr);
    static_assert(GatherSmem<TG, PH, PW, S>::GBP >= 4 * 512, "store scratch in the first slot");
    __syncthreads();   // the staging slots are free: every wave has consumed its last RoI
    gather_store(x, a.zero_init, acc,
                 reinterpret_cast<float *>(blk0.g) + (threadIdx.x >> 6) * 512);
}

// Two heads on one pyramid (e.g. the 7x7 box head and the 14x14 mask head of a Mask
// R-CNN step): the workgroup walks head 0's RoIs of its tile, then head 1's, into the
// same accumulators, and writes every gradient element once.  Tiles follow head 0's
// order.
template <typename TG, int PH0, int PW0, int PH1, int PW1>
__global__ __launch_bounds__(256) void bwd_gather2_kernel(GatherArgs a) {
    using SM0 = GatherSmem<TG, PH0, PW0, 2>;
    using SM1 = GatherSmem<TG, PH1, PW1, 2>;
    union Smem {
        SM0 h0;
        SM1 h1;
    };
    __shared__ Smem sm;
    // the staging ring of whichever head is being walked
    constexpr int kStage0 = SM0::NBUF * SM0::GBP, kStage1 = SM1::NBUF * SM1::GBP;
    __shared__ __align__(16) uint32_t stage[kStage0 > kStage1 ? kStage0 : kStage1];
    GatherTile x;
    const int t = gather_tile(a, a.tile_order, x);
    float acc[8][8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[r][q] = 0.0f;
    gather_phase<TG, PH0, PW0, 2>(a.head[0], a.lv, t, x, acc, sm.h0, stage,
                                  SM0::NBUF == 2 ? stage + SM0::GBP : nullptr);
    __syncthreads();   // head 0's LDS is no longer read
    gather_phase<TG, PH1, PW1, 2>(a.head[1], a.lv, t, x, acc, sm.h1, stage,
                                  SM1::NBUF == 2 ? stage + SM1::GBP : nullptr);
    static_assert(kStage0 >= 4 * 512 && kStage1 >= 4 * 512, "store scratch in the ring");
    __syncthreads();   // the staging ring is free
    gather_store(x, a.zero_init, acc,
                 reinterpret_cast<float *>(stage) + (threadIdx.x >> 6) * 512);
}

bool gather_available(int PH, int PW, int S) {
    return S == 2 && ((PH == 7 && PW == 7) || (PH == 14 && PW == 14));
}

template <typename TG>
static void launch_gather2_typed(const GatherArgs &a, uint32_t g, hipStream_t stream) {
    const bool b0 = a.PH == 7, b1 = a.head[1].PH == 7;
    if (b0 && b1)
        bwd_gather2_kernel<TG, 7, 7, 7, 7><<<g, 256, 0, stream>>>(a);
    else if (b0)
        bwd_gather2_kernel<TG, 7, 7, 14, 14><<<g, 256, 0, stream>>>(a);
    else if (b1)
        bwd_gather2_kernel<TG, 14, 14, 7, 7><<<g, 256, 0, stream>>>(a);
    else
        bwd_gather2_kernel<TG, 14, 14, 14, 14><<<g, 256, 0, stream>>>(a);
}

hipError_t launch_gather(GatherArgs a, int gout_dtype, hipStream_t stream) {
    if (!gather_prepare(a)) return hipErrorInvalidConfiguration;
    const int64_t grid = static_cast<int64_t>(a.ntiles) * a.wg_per_tile * a.ncg;
    if (grid <= 0) return hipSuccess;
    if (grid >= (int64_t(1) << 24)) return hipErrorInvalidConfiguration;
    const uint32_t g = static_cast<uint32_t>(grid);
    if (a.nheads == 2) {
        // both heads' gradients have one dtype here (the host checks it)
        if (gout_dtype == kF32)
            launch_gather2_typed<float>(a, g, stream);
        else
            launch_gather2_typed<uint16_t>(a, g, stream);
        return hipGetLastError();
    }
    if (gout_dtype == kF32) {
        if (a.PH == 7)
            bwd_gather_kernel<float, 7, 7, 2><<<g, 256, 0, stream>>>(a);
        else
            bwd_gather_kernel<float, 14, 14, 2><<<g, 256, 0, stream>>>(a);
    } else {
        if (a.PH == 7)
            bwd_gather_kernel<uint16_t, 7, 7, 2><<<g, 256, 0, stream>>>(a);
        else
            bwd_gather_kernel<uint16_t, 14, 14, 2><<<g, 256, 0, stream>>>(a);
    }
    return hipGetLastError();
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
