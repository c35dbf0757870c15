// fwd.hip -- RoIAlign forward (rows a3-a5 of the hot path).
//
// Operator: the RoIExtractor of MMDetection §3.1 in its RoIAlign form; definition
// and conventions in include/roi_extract.h.
//
// Two kernels:
//   fwd_cl_kernel       channels-last levels (stride_c == 1), specialised output
//                       grids.  One workgroup = one RoI x 1-4 slices of 64 channels
//                       (128 for bf16 on the 7x7 grid, two channels per lane); lanes
//                       run over channels, so every pixel read is one coalesced,
//                       channel-contiguous load.  The RoI's sample
//                       geometry is reduced once into LDS to its distinct tap rows
//                       and columns with summed weights (the footprint), every
//                       footprint pixel is loaded once, and the bins are formed as
//                       two small separable products.  Results are transposed
//                       through LDS so the [C][PH][PW] block of the RoI is stored
//                       contiguously at its original RoI index.
//   fwd_nchw_kernel     other strides (channels in separate planes), 7x7 / 14x14 with
//                       sampling ratio 2: a RoI's distinct tap rows x columns staged in
//                       LDS per channel, lanes along x.
//   fwd_generic_kernel  any strides, output size and sampling ratio: one thread per
//                       output element.
#include "internal.hpp"

namespace rex {

// Units of footprint loads a forward wave keeps in flight ahead of the one it
// reduces, and distinct columns per unit.
#ifndef REX_FWD_DEPTH
#define REX_FWD_DEPTH 2
#endif
#ifndef REX_FWD_CX
#define REX_FWD_CX 8
#endif
// channels per workgroup of the NCHW kernel (7x7, 14x14 grids): the kernel waits on
// dependent loads, so more resident workgroups (less LDS each) beat fewer, fuller ones
// (batch-2 box head: 2 channels 244 us, 4: 164, 8: 183, 16: 260; mask head 1 or 2: 138,
// 146)
#ifndef REX_NCHW_CC7
#define REX_NCHW_CC7 4
#endif
#ifndef REX_NCHW_CC14
#define REX_NCHW_CC14 1
#endif
// columns per load unit and units in flight with two bf16 channels per lane (7x7 grid)
#ifndef REX_FWD_CX2_BF16
#define REX_FWD_CX2_BF16 4
#endif
#ifndef REX_FWD_DEPTH2_BF16
#define REX_FWD_DEPTH2_BF16 4
#endif

constexpr int kFwdDepth = REX_FWD_DEPTH;
constexpr int kFwdCX = REX_FWD_CX;


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
// Channels-last kernel: footprint-exact separable gather
// ---------------------------------------------------------------------------
//
// With the sample geometry separable, the average over one bin is
//     out[ph][pw] = sum_y sum_x Wy[ph][y] * Wx[pw][x] * F[y][x]
// where y runs over the distinct tap rows and x over the distinct tap columns of
// the RoI, and Wy[ph][y] (Wx[pw][x]) is the summed bilinear weight, divided by S,
// that the samples of bin row ph (bin column pw) give to row y (column x).  Each
// pixel of the footprint is therefore loaded exactly once per channel, however
// many samples share it, and the weights are applied as two small dense products.

struct SampleTap {               // one sample row / column: taps and weights
    int32_t lo;                  // -1: sample outside the map
    int32_t hi;
    float w_lo;
    float w_hi;
};

// Distinct tap positions of `ns` consecutive samples (lane s < ns holds sample s;
// S samples per bin), computed by one wavefront.  Sample coordinates are
// non-decreasing, so the taps are too: a position is new exactly when it exceeds
// the previous sample's upper tap, and its rank among the distinct positions
// follows from two ballots.  If the taps are not monotone (a degenerate RoI whose
// rounded coordinates step backwards), every tap simply gets a slot of its own.
// Writes the byte offset of each distinct position to off[] and, for each bin b,
// the summed weight (times wscale) of each position to w[rank * RS + b * BS]; both
// arrays must be pre-set to the out-of-range offset and to zero.  With `touch`, also
// sets bit b of touch[rank] for every bin b one of whose samples has the position as
// a tap, whatever its weight (touch pre-set to zero).  Returns the count.
template <int S, int RS, int BS>
__device__ __forceinline__ int distinct_taps(const SampleTap *taps, int ns, int lane,
                                             uint32_t stride_b, float wscale, uint32_t *off,
                                             float *w, uint32_t *touch) {
    SampleTap st, pv;
    st.lo = pv.lo = -1;
    st.hi = pv.hi = -1;
    st.w_lo = st.w_hi = pv.w_lo = pv.w_hi = 0.0f;
    if (lane < ns) st = taps[lane];
    if (lane < ns && lane > 0) pv = taps[lane - 1];
    const bool valid = st.lo >= 0;
    const bool pvalid = pv.lo >= 0;
    const uint64_t vm = __builtin_amdgcn_ballot_w64(valid);
    const bool down = valid && pvalid && (st.lo < pv.lo || st.hi < pv.hi);
    const uint64_t run = vm ? (vm >> __builtin_ctzll(vm)) : 0;
    const bool mono = __builtin_amdgcn_ballot_w64(down) == 0 && ((run + 1) & run) == 0;
    int r_lo, r_hi, n;
    if (mono) {
        const bool new_lo = valid && (!pvalid || st.lo > pv.hi);
        const bool new_hi = valid && st.hi > st.lo && (!pvalid || st.hi > pv.hi);
        const uint64_t bl = __builtin_amdgcn_ballot_w64(new_lo);
        const uint64_t bh = __builtin_amdgcn_ballot_w64(new_hi);
        const int below = static_cast<int>(
            __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(bl >> 32),
                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bl), 0u)) +
            __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(bh >> 32),
                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bh), 0u)));
        r_lo = new_lo ? below : below - 1 - (pv.hi - st.lo);
        r_hi = r_lo + (st.hi - st.lo);
        n = __builtin_popcountll(bl) + __builtin_popcountll(bh);
        if (new_lo) off[r_lo] = static_cast<uint32_t>(st.lo) * stride_b;
        if (new_hi) off[r_hi] = static_cast<uint32_t>(st.hi) * stride_b;
    } else {
        r_lo = 2 * lane;
        r_hi = 2 * lane + 1;
        n = 2 * ns;
        if (valid) {
            off[r_lo] = static_cast<uint32_t>(st.lo) * stride_b;
            off[r_hi] = static_cast<uint32_t>(st.hi) * stride_b;
        }
    }
    if (touch && valid) {
        atomicOr(&touch[r_lo], 1u << (lane / S));
        if (r_hi != r_lo) atomicOr(&touch[r_hi], 1u << (lane / S));
    }
    // Per bin, its first lane sums the weights of the bin's samples in sample order
    // (lo before hi), so the result does not depend on scheduling.  The ranks one
    // bin touches span at most 2S consecutive slots.
    const float wl = valid ? st.w_lo * wscale : 0.0f;
    const float wh = valid ? st.w_hi * wscale : 0.0f;
    int rl[S], rh[S];
    float fl[S], fh[S];
    bool ok[S];
#pragma unroll
    for (int t = 0; t < S; ++t) {
        const int src = min(lane + t, 63);
        rl[t] = __shfl(r_lo, src);
        rh[t] = __shfl(r_hi, src);
        fl[t] = __shfl(wl, src);
        fh[t] = __shfl(wh, src);
        ok[t] = __shfl(valid ? 1 : 0, src) != 0 && lane + t < ns;
    }
    if (lane < ns && lane % S == 0) {
        int base = INT32_MAX;
#pragma unroll
        for (int t = 0; t < S; ++t)
            if (ok[t]) base = min(base, rl[t]);
        if (base != INT32_MAX) {
            float win[2 * S];
#pragma unroll
            for (int e = 0; e < 2 * S; ++e) win[e] = 0.0f;
#pragma unroll
            for (int t = 0; t < S; ++t) {
                if (!ok[t]) continue;
#pragma unroll
                for (int e = 0; e < 2 * S; ++e) win[e] += (rl[t] - base == e) ? fl[t] : 0.0f;
#pragma unroll
                for (int e = 0; e < 2 * S; ++e) win[e] += (rh[t] - base == e) ? fh[t] : 0.0f;
            }
            const int bin = lane / S;
#pragma unroll
            for (int e = 0; e < 2 * S; ++e)
                if (base + e < n) w[(base + e) * RS + bin * BS] = win[e];
        }
    }
    return n;
}

// Raw bits of CPL adjacent channels of one pixel: one load per pixel and lane (32 bits
// for one binary32 or one or two bf16 values, 64 bits for two binary32 values), then
// unpacked to binary32 when consumed.
template <typename T, int CPL>
struct RawPix {
    static constexpr int W = (static_cast<int>(sizeof(T)) * CPL + 3) / 4;
    uint32_t w[W];
};

template <typename T, int CPL>
__device__ __forceinline__ void load_pix(__amdgpu_buffer_rsrc_t r, uint32_t off, RawPix<T, CPL> &p) {
    if constexpr (sizeof(T) * CPL == 8) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
        p.w[0] = v[0];
        p.w[1] = v[1];
    } else if constexpr (sizeof(T) * CPL == 4) {
        p.w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    } else {
        p.w[0] = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
    }
}

// Channel j of the pixel (the element at the lower address is channel 0).
template <typename T, int CPL>
__device__ __forceinline__ float unpack_pix(const RawPix<T, CPL> &p, int j) {
    if constexpr (sizeof(T) == 4) {
        return __uint_as_float(p.w[j]);
    } else if constexpr (CPL == 1) {
        return __uint_as_float(p.w[0] << 16);
    } else {
        return __uint_as_float(j == 0 ? (p.w[0] << 16) : (p.w[0] & 0xffff0000u));
    }
}

// One workgroup per (RoI, run of spw slices of 64 * CPL channels); lane i holds channels
// CPL*i .. CPL*i + CPL - 1 of the slice, adjacent in memory, so every pixel read is one
// coalesced load per lane.  Wave w owns bin rows [w*RPW, min(PH, (w+1)*RPW)) and loads
// the distinct tap rows of those bin rows times all distinct tap columns of the RoI, in
// chunks of CX columns, with the next unit's loads issued before the current one is
// reduced.
// LDS of one forward workgroup.
template <int PH, int PW, int S, int CX, int CHK>
struct FwdSmem {
    static constexpr int NB = PH * PW;
    static constexpr int NR = PH * S;
    static constexpr int NCOL = PW * S;
    static constexpr int RPW = (PH + 3) / 4;
    static constexpr int RPWP = (RPW + 3) & ~3;
    static constexpr int MAXY = 2 * RPW * S;
    static constexpr int MAXX = ((2 * NCOL + CX - 1) / CX) * CX;
    static constexpr int PWP = (PW + 3) & ~3;
    SampleTap srow[NR];
    SampleTap scol[NCOL];
    __align__(16) uint32_t s_xoff[MAXX];
    __align__(16) float s_wx[PWP][MAXX];   // [bin column][distinct column]
    uint32_t s_yoff[4][MAXY];
    __align__(16) float s_wy[4][MAXY][RPWP];
    int32_t s_nx;
    int32_t s_ny[4];
    uint32_t s_xbins[MAXX];        // bit q: a sample of bin column q has this tap column
    uint32_t s_cmask[MAXX / CX];   // the same, over each chunk of CX columns
    __align__(16) float stile[CHK * NB];
};

// The forward of workgroup `lid` (in logical order) of a launch over the RoIs of `a`
// (FwdArgs or FwdHeadArgs: RoIs, levels, plan order, output and slicing) on pyramid lv.
template <typename T, typename TO, int PH, int PW, int S, int CX, int CHK, int CPL, typename A,
          int D = kFwdDepth>
__device__ __forceinline__ void fwd_cl_body(const A &a, const LevelTable &lv, uint32_t lid,
                                            FwdSmem<PH, PW, S, CX, CHK> &sm) {
    using SM = FwdSmem<PH, PW, S, CX, CHK>;
    constexpr int NB = SM::NB;
    constexpr int NR = SM::NR;                   // sample rows
    constexpr int NCOL = SM::NCOL;               // sample columns
    constexpr int RPW = SM::RPW;                 // bin rows per wave
    constexpr int RPWP = SM::RPWP;
    constexpr int MAXY = SM::MAXY;               // distinct tap rows per wave
    constexpr int MAXX = SM::MAXX;               // distinct tap columns, padded
    constexpr int PWP = SM::PWP;                 // padded for 16-byte LDS reads
    constexpr int SLICE = 64 * CPL;              // channels of one slice
    static_assert(NR + NCOL <= 256 && NCOL <= 64 && RPW * S <= 64 && MAXX <= 64, "geometry sizes");
    static_assert(SLICE % CHK == 0 && CHK % CPL == 0 && CX % 4 == 0, "tiling");
    SampleTap *const srow = sm.srow;
    SampleTap *const scol = sm.scol;
    uint32_t *const s_xoff = sm.s_xoff;
    float (*const s_wx)[MAXX] = sm.s_wx;
    uint32_t (*const s_yoff)[MAXY] = sm.s_yoff;
    float (*const s_wy)[MAXY][RPWP] = sm.s_wy;
    float *const stile = sm.stile;

    // Which RoI and slice: the logical block id, then the plan's permutation.
    const int slot = static_cast<int>(lid / static_cast<uint32_t>(a.wg_per_roi));
    const int sub = static_cast<int>(lid) - slot * a.wg_per_roi;
    const int slice0 = sub * a.spw;                          // this workgroup's slices
    const int slice1 = min(a.nslices, slice0 + a.spw);
    int k = uniform_i(a.perm ? a.perm[slot] : slot);
    const bool kvalid = k >= 0 && k < a.K;
    if (!kvalid) k = 0;
    const float *r = a.rois + 5 * static_cast<int64_t>(k);
    const float rb = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
    const int lvl = uniform_i(a.roi_levels ? a.roi_levels[k] : 0);
    const bool lvalid = lvl >= 0 && lvl < lv.num;
    const LevelArg L = level_at(lv, lvalid ? lvl : 0);
    const int b = roi_batch(rb, lv.N);
    const bool active = kvalid && lvalid && b >= 0;

    const int t = threadIdx.x;
    const int wave = t >> 6;
    const int lane = t & 63;
    const int p0 = wave * RPW;
    const int p1 = min(PH, p0 + RPW);
    const uint32_t sh_b = static_cast<uint32_t>(L.sh * int64_t(sizeof(T)));
    const uint32_t sw_b = static_cast<uint32_t>(L.sw * int64_t(sizeof(T)));

    // a3: sample geometry, once per workgroup (an inactive RoI gets no valid
    // sample, so its outputs are zero), and cleared footprint tables.
    {
        const Axis ax = axis_setup(x1, x2, L.scale, a.aligned, PW, S);
        const Axis ay = axis_setup(y1, y2, L.scale, a.aligned, PH, S);
        if (t < NR + NCOL) {
            const bool isrow = t < NR;
            const int u = isrow ? t : t - NR;
            const Tap tp = axis_tap(isrow ? ay : ax, u / S, u % S, isrow ? L.H : L.W);
            SampleTap st;
            st.lo = active ? tp.lo : -1;
            st.hi = tp.hi;
            st.w_lo = tp.wlo;
            st.w_hi = tp.whi;
            if (isrow) srow[u] = st;
            else scol[u] = st;
        }
        for (int e = t; e < MAXX * PWP; e += 256) (&s_wx[0][0])[e] = 0.0f;
        for (int e = t; e < MAXX; e += 256) sm.s_xbins[e] = 0u;
        for (int e = t; e < 4 * MAXY * RPWP; e += 256) (&s_wy[0][0][0])[e] = 0.0f;
        for (int e = t; e < MAXX; e += 256) s_xoff[e] = kBufOOB;
        for (int e = t; e < 4 * MAXY; e += 256) (&s_yoff[0][0])[e] = kBufOOB;
    }
    __syncthreads();
    // Footprint: distinct tap rows of each wave's bin rows, distinct tap columns of
    // the RoI (wave 0); weights carry the 1/S of the sample average along their axis.
    constexpr float kInvS = 1.0f / static_cast<float>(S);
    {
        const int ny = distinct_taps<S, RPWP, 1>(srow + p0 * S, (p1 - p0) * S, lane, sh_b, kInvS,
                                                 s_yoff[wave], &s_wy[wave][0][0], nullptr);
        if (lane == 0) sm.s_ny[wave] = ny;
        if (wave == 0) {
            const int nx = distinct_taps<S, 1, MAXX>(scol, NCOL, lane, sw_b, kInvS, s_xoff,
                                                     &s_wx[0][0], sm.s_xbins);
            if (lane == 0) sm.s_nx = nx;
            // Which bin columns each chunk of CX distinct columns reaches (a column is a
            // tap of a run of at most a few adjacent bins): the column reduction skips
            // the others, whose products the definition never takes.
            wave_sync();
            if (lane < MAXX / CX) {
                uint32_t m = 0;
#pragma unroll
                for (int x = 0; x < CX; ++x) m |= sm.s_xbins[lane * CX + x];
                sm.s_cmask[lane] = m;
            }
        }
    }
    __syncthreads();

    // wave-uniform counts in scalar registers: the pipeline below branches on them
    const int ny = uniform_i(sm.s_ny[wave]);
    const int nch = uniform_i((sm.s_nx + CX - 1) / CX);
    // The geometry above serves every slice of the workgroup.
    for (int slice = slice0; slice < slice1; ++slice) {
        if (slice > slice0) __syncthreads();   // the previous slice's output tile is stored
        // the lane's first channel; with CPL > 1 the channel count is a multiple of CPL,
        // so a lane holds either all of its channels or none
        const int c = slice * SLICE + lane * CPL;
        const bool lane_on = active && c < lv.C;
        // One buffer resource per image of the level; a lane with no channel reads out
        // of range (zeros) instead of branching.
        const char *img = static_cast<const char *>(L.data) +
                          (active ? static_cast<int64_t>(b) * L.sn * int64_t(sizeof(T)) : 0);
        const __amdgpu_buffer_rsrc_t res = make_rsrc(img, L.img_bytes);
        const uint32_t vbase = lane_on ? static_cast<uint32_t>(c) * uint32_t(sizeof(T)) : kBufOOB;

        // a4: gather.  Chunk-major over the footprint: for each chunk of CX distinct
        // columns, every distinct row of the wave is loaded (work unit = (chunk, row))
        // and reduced over rows first, H[x][p] = sum_y Wy[p][y] F[y][x]; at the end of
        // the chunk the columns are reduced into the bins, acc[p][q] += Wx[q][x] H[x][p].
        // Columns past the footprint read zeros (out-of-range offsets, zero weights).
        float acc[CPL][RPW][PW];
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int p = 0; p < RPW; ++p)
#pragma unroll
                for (int q = 0; q < PW; ++q) acc[j][p][q] = 0.0f;
        float H[CPL][CX][RPW];
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int x = 0; x < CX; ++x)
#pragma unroll
                for (int p = 0; p < RPW; ++p) H[j][x][p] = 0.0f;

        auto issue = [&](int ch, int yi, RawPix<T, CPL> (&v)[CX]) {
            const uint32_t rowb = vbase + s_yoff[wave][yi];
            const uint32_t *xo = s_xoff + ch * CX;
#pragma unroll
            for (int x = 0; x < CX; ++x) load_pix<T, CPL>(res, rowb + xo[x], v[x]);
        };
        auto consume = [&](int ch, int yi, const RawPix<T, CPL> (&v)[CX]) {
            const float *wy = s_wy[wave][yi];
#pragma unroll
            for (int x = 0; x < CX; ++x) {
#pragma unroll
                for (int j = 0; j < CPL; ++j) {
                    const float f = unpack_pix<T, CPL>(v[x], j);
#pragma unroll
                    for (int p = 0; p < RPW; ++p) H[j][x][p] = fmaf(wy[p], f, H[j][x][p]);
                }
            }
            if (yi == ny - 1) {
                // acc[p][q] += sum over the chunk's columns x of Wx[q][x] H[x][p], for the
                // bin columns q the chunk reaches (uniform mask); the sum over x runs in
                // column order, chunk after chunk, for every bin
                const uint32_t m = static_cast<uint32_t>(uniform_i(static_cast<int>(sm.s_cmask[ch])));
#pragma unroll
                for (int q = 0; q < PW; ++q) {
                    if (!((m >> q) & 1u)) continue;
                    float wq[CX];
#pragma unroll
                    for (int x4 = 0; x4 < CX; x4 += 4) {
                        const float4 w4 = *reinterpret_cast<const float4 *>(&s_wx[q][ch * CX + x4]);
                        wq[x4] = w4.x;
                        wq[x4 + 1] = w4.y;
                        wq[x4 + 2] = w4.z;
                        wq[x4 + 3] = w4.w;
                    }
#pragma unroll
                    for (int x = 0; x < CX; ++x)
#pragma unroll
                        for (int j = 0; j < CPL; ++j)
#pragma unroll
                            for (int p = 0; p < RPW; ++p)
                                acc[j][p][q] = fmaf(wq[x], H[j][x][p], acc[j][p][q]);
                    // one bin column's weights live at a time
                    __builtin_amdgcn_sched_barrier(0);
                }
#pragma unroll
                for (int x = 0; x < CX; ++x)
#pragma unroll
                    for (int j = 0; j < CPL; ++j)
#pragma unroll
                        for (int p = 0; p < RPW; ++p) H[j][x][p] = 0.0f;
            }
        };

        // Pipeline over the units in (chunk, row) order: the loads of units u+1 ..
        // u+D are in flight while unit u is reduced.  The loop is unrolled by
        // the ring size so every buffer index is a constant.
        constexpr int NBUF = D + 1;
        RawPix<T, CPL> v[NBUF][CX];
        const int units = ny * nch;
        int ic = 0, iy = 0;      // next unit to issue
        int cc = 0, cy = 0;      // next unit to consume
        auto step = [&](int &ch, int &y) {
            if (++y == ny) {
                y = 0;
                ++ch;
            }
        };
#pragma unroll
        for (int d = 0; d < D; ++d) {
            if (d < units) {
                issue(ic, iy, v[d]);
                step(ic, iy);
            }
        }
        for (int u0 = 0; u0 < units; u0 += NBUF) {
#pragma unroll
            for (int jj = 0; jj < NBUF; ++jj) {
                if (u0 + jj >= units) break;
                if (u0 + jj + D < units) {
                    issue(ic, iy, v[(jj + D) % NBUF]);
                    step(ic, iy);
                }
                __builtin_amdgcn_sched_barrier(0);
                consume(cc, cy, v[jj]);
                step(cc, cy);
                __builtin_amdgcn_sched_barrier(0);
            }
        }

        // Every value the wave loaded reaches every one of its outputs through the
        // dense products above, so a non-finite feature anywhere in the footprint shows
        // up as a non-finite output.
        uint32_t bad = 0;
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int p = 0; p < RPW; ++p)
#pragma unroll
                for (int q = 0; q < PW; ++q) bad |= __builtin_isfinite(acc[j][p][q]) ? 0u : 1u;

        // Then a zero weight times an infinity may have reached bins whose samples never
        // touch that pixel, so this wave's bins are recomputed sample by sample, every
        // product taken only where the definition takes it.
        if (__builtin_amdgcn_ballot_w64(bad != 0) != 0) {
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const uint32_t vb = vbase + static_cast<uint32_t>(j) * uint32_t(sizeof(T));
#pragma unroll
                for (int p = 0; p < RPW; ++p) {
                    if (p0 + p >= p1) continue;
#pragma unroll 1
                    for (int q = 0; q < PW; ++q) {
                        float sum = 0.0f;
                        for (int iy2 = 0; iy2 < S; ++iy2) {
                            const SampleTap ty = srow[(p0 + p) * S + iy2];
                            if (ty.lo < 0) continue;
                            const uint32_t r0 = vb + static_cast<uint32_t>(ty.lo) * sh_b;
                            const uint32_t r1 = vb + static_cast<uint32_t>(ty.hi) * sh_b;
                            for (int ix = 0; ix < S; ++ix) {
                                const SampleTap tx = scol[q * S + ix];
                                if (tx.lo < 0) continue;
                                const uint32_t cl = static_cast<uint32_t>(tx.lo) * sw_b;
                                const uint32_t chh = static_cast<uint32_t>(tx.hi) * sw_b;
                                const float v00 = raw_to_f32<T>(buf_load_raw<T>(res, r0 + cl));
                                const float v01 = raw_to_f32<T>(buf_load_raw<T>(res, r0 + chh));
                                const float v10 = raw_to_f32<T>(buf_load_raw<T>(res, r1 + cl));
                                const float v11 = raw_to_f32<T>(buf_load_raw<T>(res, r1 + chh));
                                const float xl = fmaf(tx.w_hi, v01, tx.w_lo * v00);
                                const float xh = fmaf(tx.w_hi, v11, tx.w_lo * v10);
                                sum += fmaf(ty.w_hi, xh, ty.w_lo * xl);
                            }
                        }
                        sum = sum / static_cast<float>(S * S);
#pragma unroll
                        for (int qq = 0; qq < PW; ++qq) acc[j][p][qq] = (qq == q) ? sum : acc[j][p][qq];
                    }
                }
            }
        }

        // a5: the slice's [SLICE][PH][PW] block is contiguous in the output at RoI k;
        // transposed through LDS in rounds of CHK channels.
        const int nchan = min(SLICE, lv.C - slice * SLICE);
        const gptr<TO> out_blk = as_global_mut<TO>(a.out) +
                                 (static_cast<int64_t>(k) * lv.C + static_cast<int64_t>(slice) * SLICE) * NB;
#pragma unroll
        for (int c0 = 0; c0 < SLICE; c0 += CHK) {
            if (lane * CPL >= c0 && lane * CPL < c0 + CHK) {
#pragma unroll
                for (int j = 0; j < CPL; ++j)
#pragma unroll
                    for (int p = 0; p < RPW; ++p) {
                        if (p0 + p >= p1) continue;
#pragma unroll
                        for (int q = 0; q < PW; ++q)
                            stile[(lane * CPL + j - c0) * NB + (p0 + p) * PW + q] = acc[j][p][q];
                    }
            }
            __syncthreads();
            const int ne = max(0, min(CHK, nchan - c0)) * NB;
            if (kvalid)
                store_run_f32<TO>(out_blk + c0 * NB, stile, ne, t, 256);
            if (c0 + CHK < SLICE) __syncthreads();
        }
    }   // slices
}

template <typename T, typename TO, int PH, int PW, int S, int CX, int CHK, int CPL, int D>
__global__ __launch_bounds__(256) void fwd_cl_kernel(FwdArgs a) {
    __shared__ FwdSmem<PH, PW, S, CX, CHK> sm;
    // The arguments are read in place from the kernel-argument segment (a reference to
    // the by-value parameter would make the compiler copy the level table to private
    // memory to index it by the RoI's level).
    const FwdArgs &ka = *(const FwdArgs *)__builtin_amdgcn_kernarg_segment_ptr();
    // XCD-aware block order: consecutive logical ids (neighbouring RoIs of the plan
    // order) land on one XCD
    fwd_cl_body<T, TO, PH, PW, S, CX, CHK, CPL, FwdArgs, D>(ka, ka.lv, xcd_remap(blockIdx.x, gridDim.x),
                                                          sm);
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------

bool fwd_fast_available(int PH, int PW, int S) {
    return S == 2 && ((PH == 7 && PW == 7) || (PH == 14 && PW == 14));
}

template <typename T, typename TO, int PH, int PW, int CX, int CHK, int CPL, int D = kFwdDepth>
static hipError_t launch_fwd_cl(FwdArgs a, hipStream_t stream) {
    a.nslices = (a.lv.C + 64 * CPL - 1) / (64 * CPL);
    // Slices per workgroup: the RoI's geometry (two IEEE divisions, the distinct-tap
    // reductions) is built once per workgroup, so a workgroup takes up to 4 slices
    // while the grid keeps at least 32 workgroups per CU; below that the longest
    // workgroups would set the kernel's tail (measured, 1024 RoIs x 256 channels:
    // 53 us with one slice, 56 with two; 8192 RoIs: 361 us with one, 328 with four).
    a.spw = 1;
    for (int spw = 4; spw > 1; spw /= 2)
        if (static_cast<int64_t>(a.K) * ((a.nslices + spw - 1) / spw) >= 8192) {
            a.spw = spw;
            break;
        }
    a.wg_per_roi = (a.nslices + a.spw - 1) / a.spw;
    const int64_t grid = static_cast<int64_t>(a.K) * a.wg_per_roi;
    if (grid >= (int64_t(1) << 24)) return hipErrorInvalidConfiguration;
    fwd_cl_kernel<T, TO, PH, PW, 2, CX, CHK, CPL, D><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
    return hipGetLastError();
}

template <typename T, typename TO>
static hipError_t launch_fwd_typed(FwdArgs a, bool fast, hipStream_t stream) {
    // a dispatch holds fewer than 2^32 work-items; beyond that, the strided kernel
    if (fast && static_cast<int64_t>(a.K) * ((a.lv.C + 63) / 64) >= (int64_t(1) << 24)) fast = false;
    if (fast) {
        if (a.PH == 7) {
            // bf16 features: two adjacent channels per lane (one 32-bit load per pixel)
            // when the channel count is even -- half the load and address instructions of
            // one channel per lane, and twice the bytes in flight per load (batch-1
            // inference, 1000 RoIs: 49.3 -> 41.9 us; batch 16: 316 -> 268 us).  For
            // binary32 (64-bit loads) the same layout is slower (1024 RoIs: 51.0 -> 54.6
            // us): the grid halves and occupancy drops from six to four waves, so fewer
            // bytes are in flight per SIMD; so is sharing one geometry between two slices
            // taken at once by an 8-wave workgroup (53.5 -> 59.8 us).
            // With two channels per lane, units of 4 columns and 4 units in flight (batch
            // 16, 8192 RoIs: 241 -> 227 us; batch 1, 1000 RoIs: 38.2 -> 38.0 us); one
            // channel per lane keeps 8 columns and 2 units (1024 RoIs: 47.2 vs 49.0 us).
            if constexpr (sizeof(T) == 2)
                if (a.lv.C % 2 == 0)
                    return launch_fwd_cl<T, TO, 7, 7, REX_FWD_CX2_BF16, 64, 2, REX_FWD_DEPTH2_BF16>(
                        a, stream);
            return launch_fwd_cl<T, TO, 7, 7, kFwdCX, 64, 1>(a, stream);
        }
        // 4 columns per unit keep the 14x14 kernel at 124 registers, four workgroups
        // per CU (8 columns: 164 registers, three; mask head batch 2: 44 vs 51 us);
        // the 7x7 kernel with one channel per lane is fastest with 8 (4: 60 registers,
        // 336 vs 321 us batch 16)
        return launch_fwd_cl<T, TO, 14, 14, 4, 16, 1>(a, stream);
    }
    // other layouts (channels in separate planes): the staged kernel on the same grids
    if (fwd_fast_available(a.PH, a.PW, a.S) && static_cast<int64_t>(a.K) * a.lv.C < (int64_t(1) << 30)) {
        if (a.PH == 7) return launch_fwd_nchw<T, TO, 7, 7, REX_NCHW_CC7>(a, stream);
        return launch_fwd_nchw<T, TO, 14, 14, REX_NCHW_CC14>(a, stream);
    }
    const int64_t total = static_cast<int64_t>(a.K) * a.lv.C * a.PH * a.PW;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 16384);
    fwd_generic_kernel<T, TO><<<static_cast<uint32_t>(blocks), 256, 0, stream>>>(a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Channels in separate planes (NCHW): staged footprint, lanes along x
// ---------------------------------------------------------------------------
//
// One workgroup per (RoI, CC channels).  The sample positions of an axis grow with
// the sample index, so the tap rows (columns) form runs of equal `lo`, each adding
// `lo` and, unless it is the next run's `lo` or the map edge, `lo + 1` to the
// distinct set: one wave lists the distinct rows and gives every sample the indices
// of its two taps in the list (a scan over the run ends).  The workgroup then loads
// every channel's distinct rows x distinct columns into LDS with consecutive lanes
// on consecutive columns (a RoI's columns are a contiguous run unless its bins are
// wider than a pixel), reduces each tap row along x per bin column, and the tap
// rows along y per bin.  Any other grid, or a RoI whose taps are not monotone, takes
// the per-output path.
template <int N>
struct NchwAxis {
    int idx_lo[N], idx_hi[N];   // per sample: its taps' positions in the distinct list
    float w_lo[N], w_hi[N];     // bilinear weights (0 for a sample off the map)
    int list[2 * N];            // distinct tap rows (columns)
    int n;                      // their count
    int bad;                    // taps not monotone in the sample index
};

// Lanes 0..N-1 of one wave: sample u of axis `ax` on a map of `size` pixels.
template <int N, int S>
__device__ __forceinline__ void nchw_axis(const Axis &ax, int size, bool active,
                                          NchwAxis<N> &o) {
    const int lane = threadIdx.x & 63;
    Tap tp{-1, -1, 0.0f, 0.0f};
    if (lane < N && active) tp = axis_tap(ax, lane / S, lane % S, size);
    const bool valid = tp.lo >= 0;
    const int nlo = __shfl_down(tp.lo, 1);      // the next sample's lo (-1 past the last)
    const bool next_valid = lane + 1 < N && nlo >= 0;
    const bool run_end = valid && (!next_valid || nlo != tp.lo);
    const bool extra = run_end && tp.hi != tp.lo && !(next_valid && nlo == tp.lo + 1);
    const int contrib = run_end ? 1 + (extra ? 1 : 0) : 0;
    const int incl = wave_inclusive_scan(contrib, lane);
    const int pos = incl - contrib;             // the run's position (every sample of it)
    const uint64_t bad = __ballot(valid && next_valid && nlo < tp.lo);
    if (lane < N) {
        o.idx_lo[lane] = valid ? pos : -1;   // -1: the sample is off the map
        o.idx_hi[lane] = valid ? (tp.hi == tp.lo ? pos : pos + 1) : -1;
        o.w_lo[lane] = tp.wlo;
        o.w_hi[lane] = tp.whi;
    }
    if (run_end) {
        o.list[pos] = tp.lo;
        if (extra) o.list[pos + 1] = tp.lo + 1;
    }
    if (lane == 63) {
        o.n = incl;
        o.bad = bad != 0;
    }
}

template <int PH, int PW, int CC>
struct NchwSmem {
    static constexpr int S = 2;
    static constexpr int NR = PH * S, NCOL = PW * S;
    NchwAxis<NR> y;
    NchwAxis<NCOL> x;
    float fw[CC * 2 * NR * 2 * NCOL];   // [channel][distinct row][distinct column]
    float rw[CC * 2 * NR * PW];         // [channel][distinct row][bin column]
};

template <typename T, typename TO, int PH, int PW, int CC>
__global__ __launch_bounds__(256) void fwd_nchw_kernel(FwdArgs a) {
    constexpr int S = 2;
    using SM = NchwSmem<PH, PW, CC>;
    constexpr int NR = SM::NR, NCOL = SM::NCOL;
    __shared__ SM sm;
    const FwdArgs &ka = *(const FwdArgs *)__builtin_amdgcn_kernarg_segment_ptr();
    const LevelTable &lv = ka.lv;
    // channel chunk outer, plan order inner: neighbouring workgroups read the same
    // planes around neighbouring RoIs
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    const int chunk = static_cast<int>(lid / static_cast<uint32_t>(ka.K));
    const int slot = static_cast<int>(lid) - chunk * ka.K;
    const int c0 = chunk * CC;
    int k = uniform_i(ka.perm ? ka.perm[slot] : slot);
    const bool kvalid = k >= 0 && k < ka.K;
    if (!kvalid) k = 0;
    const float *r = ka.rois + 5 * static_cast<int64_t>(k);
    const float rb = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
    const int lvl = uniform_i(ka.roi_levels ? ka.roi_levels[k] : 0);
    const bool lvalid = lvl >= 0 && lvl < lv.num;
    const LevelArg L = level_at(lv, lvalid ? lvl : 0);
    const int b = roi_batch(rb, lv.N);
    const bool active = kvalid && lvalid && b >= 0;
    const int t = threadIdx.x;
    const int wave = t >> 6;
    const Axis ax = axis_setup(x1, x2, L.scale, ka.aligned, PW, S);
    const Axis ay = axis_setup(y1, y2, L.scale, ka.aligned, PH, S);
    if (wave == 0) nchw_axis<NR, S>(ay, L.H, active, sm.y);
    else if (wave == 1) nchw_axis<NCOL, S>(ax, L.W, active, sm.x);
    __syncthreads();
    const int nr = sm.y.n, nc = sm.x.n;
    const int nch = min(CC, lv.C - c0);
    const int64_t kout = static_cast<int64_t>(k) * lv.C * PH * PW;
    constexpr float inv_count = 1.0f / static_cast<float>(S * S);
    if (!kvalid) return;   // a plan slot past the RoIs (never with a valid plan)

    if (sm.y.bad || sm.x.bad) {
        // taps out of order (binary32 ties): each output from its own samples
        for (int e = t; e < nch * PH * PW; e += 256) {
            const int c = e / (PH * PW), j = e - c * (PH * PW);
            const int ph = j / PW, pw = j - ph * PW;
            float sum = 0.0f;
            if (active) {
                const gcptr<T> base = as_global<T>(L.data) + b * L.sn + (c0 + c) * L.sc;
                for (int iy = 0; iy < S; ++iy) {
                    const Tap ty = axis_tap(ay, ph, iy, L.H);
                    if (ty.lo < 0) continue;
                    for (int ix = 0; ix < S; ++ix) {
                        const Tap tx = axis_tap(ax, pw, ix, L.W);
                        if (tx.lo < 0) continue;
                        sum = fmaf(ty.wlo * tx.wlo, load_f32(base + ty.lo * L.sh + tx.lo * L.sw), sum);
                        sum = fmaf(ty.wlo * tx.whi, load_f32(base + ty.lo * L.sh + tx.hi * L.sw), sum);
                        sum = fmaf(ty.whi * tx.wlo, load_f32(base + ty.hi * L.sh + tx.lo * L.sw), sum);
                        sum = fmaf(ty.whi * tx.whi, load_f32(base + ty.hi * L.sh + tx.hi * L.sw), sum);
                    }
                }
            }
            store_f32(as_global_mut<TO>(ka.out) + kout + static_cast<int64_t>(c0) * PH * PW + e,
                      sum * inv_count);
        }
        return;
    }

    // a4: the footprint of every channel of the chunk, eight loads in flight per lane
    const int per_c = nr * nc;
    const int nload = nch * per_c;
    const gcptr<T> img = as_global<T>(L.data) + b * L.sn + static_cast<int64_t>(c0) * L.sc;
    for (int e0 = t; e0 < nload; e0 += 8 * 256) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = e0 + u * 256;
            v[u] = 0.0f;
            if (e < nload) {
                const int c = small_div_exact(e, per_c);
                const int rem = e - c * per_c;
                const int j = small_div_exact(rem, nc);
                const int i = rem - j * nc;
                v[u] = load_f32(img + c * L.sc + sm.y.list[j] * L.sh + sm.x.list[i] * L.sw);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (e0 + u * 256 < nload) sm.fw[e0 + u * 256] = v[u];
    }
    __syncthreads();
    // along x: every distinct tap row of every channel, per bin column
    const int nx = nch * nr * PW;
    for (int e = t; e < nx; e += 256) {
        const int cj = small_div_exact(e, PW);          // channel * nr + row
        const int pw = e - cj * PW;
        const float *row = sm.fw + cj * nc;
        float acc = 0.0f;
#pragma unroll
        for (int ix = 0; ix < S; ++ix) {
            const int u = pw * S + ix;
            const int il = sm.x.idx_lo[u];
            if (il < 0) continue;   // off the map: no contribution
            acc = fmaf(sm.x.w_lo[u], row[il], acc);
            acc = fmaf(sm.x.w_hi[u], row[sm.x.idx_hi[u]], acc);
        }
        sm.rw[e] = acc;
    }
    __syncthreads();
    // along y: every bin, then the output (written in order, one channel's bins
    // contiguous)
    for (int e = t; e < nch * PH * PW; e += 256) {
        const int c = small_div_exact(e, PH * PW);
        const int jj = e - c * (PH * PW);
        const int ph = small_div_exact(jj, PW);
        const int pw = jj - ph * PW;
        const float *col = sm.rw + c * nr * PW + pw;
        float acc = 0.0f;
#pragma unroll
        for (int iy = 0; iy < S; ++iy) {
            const int u = ph * S + iy;
            const int il = sm.y.idx_lo[u];
            if (il < 0) continue;
            acc = fmaf(sm.y.w_lo[u], col[il * PW], acc);
            acc = fmaf(sm.y.w_hi[u], col[sm.y.idx_hi[u] * PW], acc);
        }
        store_f32(as_global_mut<TO>(ka.out) + kout + static_cast<int64_t>(c0) * PH * PW + e,
                  acc * inv_count);
    }
}

template <typename T, typename TO, int PH, int PW, int CC>
static hipError_t launch_fwd_nchw(const FwdArgs &a, hipStream_t stream) {
    const int64_t grid = static_cast<int64_t>(a.K) * ((a.lv.C + CC - 1) / CC);
    if (grid >= (int64_t(1) << 31)) return hipErrorInvalidConfiguration;
    fwd_nchw_kernel<T, TO, PH, PW, CC><<<static_cast<uint32_t>(grid), 256, 0, stream>>>(a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Several heads in one launch
// ---------------------------------------------------------------------------
//
// The workgroups of every head form one grid: logical block ids [first_h, first_{h+1})
// belong to head h (each head's blocks in its own plan order), and the XCD-aware
// remapping runs over the whole grid.  A head takes the 7x7 or the 14x14 body; the
// kernel holds the LDS of both as a union and the registers of the larger, so a launch
// that mixes the two grids runs the 7x7 heads at the 14x14 occupancy.
template <typename T, typename TO, bool H7, bool H14, int CPL7>
__global__ __launch_bounds__(256, 4) void fwd_multi_kernel(FwdMultiArgs m) {
    using S7 = FwdSmem<7, 7, 2, kFwdCX, 64>;
    using S14 = FwdSmem<14, 14, 2, 4, 16>;
    union Smem {
        S7 s7;
        S14 s14;
    };
    __shared__ Smem sm;
    const FwdMultiArgs &ka = *(const FwdMultiArgs *)__builtin_amdgcn_kernarg_segment_ptr();
    const uint32_t lid = xcd_remap(blockIdx.x, gridDim.x);
    int h = 0;
#pragma unroll
    for (int i = 1; i < kMaxFwdHeads; ++i)
        if (i < ka.nheads && lid >= static_cast<uint32_t>(ka.head[i].first)) h = i;
    const FwdHeadArgs &a = ka.head[h];
    const uint32_t local = lid - static_cast<uint32_t>(a.first);
    if constexpr (H7 && H14) {
        if (a.PH == 7)
            fwd_cl_body<T, TO, 7, 7, 2, kFwdCX, 64, CPL7>(a, ka.lv, local, sm.s7);
        else
            fwd_cl_body<T, TO, 14, 14, 2, 4, 16, 1>(a, ka.lv, local, sm.s14);
    } else if constexpr (H7) {
        fwd_cl_body<T, TO, 7, 7, 2, kFwdCX, 64, CPL7>(a, ka.lv, local, sm.s7);
    } else {
        fwd_cl_body<T, TO, 14, 14, 2, 4, 16, 1>(a, ka.lv, local, sm.s14);
    }
}

#ifndef REX_FWD_MULTI_ORDER
#define REX_FWD_MULTI_ORDER 1
#endif
// One channel per lane (fp32 features, or an odd channel count): the 7x7 body needs 78
// registers and the 14x14 one 124, so a kernel holding both runs the 7x7 heads at four
// workgroups per CU instead of six; there the two grids go in two launches, 14x14 first
// (batch 2, box 1024 + mask 256 RoIs, fp32: 100 us, against 145 in one mixed launch
// and 110 as two roi_align_fwd calls).  Two bf16 channels per lane already take 116
// registers on the 7x7 grid, and one mixed launch is fastest (batch 16, box 8192 +
// mask 2048 RoIs: 503 us, against 536 as two calls).
#ifndef REX_FWD_MULTI_MIX1
#define REX_FWD_MULTI_MIX1 0
#endif

template <typename T, typename TO>
static hipError_t launch_fwd_multi_typed(FwdMultiArgs m, hipStream_t stream) {
    // two bf16 channels per lane on the 7x7 grid, as in the single-head launch
    const int cpl7 = (sizeof(T) == 2 && m.lv.C % 2 == 0) ? 2 : 1;
    if (REX_FWD_MULTI_ORDER) {
        // 14x14 heads first: their workgroups are the longest, and the short 7x7 ones
        // then fill the tail of the grid
        FwdMultiArgs o = m;
        int n = 0;
        for (int pass = 0; pass < 2; ++pass)
            for (int i = 0; i < m.nheads; ++i)
                if ((m.head[i].PH == 14) == (pass == 0)) o.head[n++] = m.head[i];
        m = o;
    }
    if (!REX_FWD_MULTI_MIX1 && cpl7 == 1) {
        int n14 = 0;
        while (n14 < m.nheads && m.head[n14].PH == 14) ++n14;
        if (REX_FWD_MULTI_ORDER && n14 > 0 && n14 < m.nheads) {
            FwdMultiArgs a = m, b = m;
            a.nheads = n14;
            b.nheads = m.nheads - n14;
            for (int i = 0; i < b.nheads; ++i) b.head[i] = m.head[n14 + i];
            hipError_t e = launch_fwd_multi_typed<T, TO>(a, stream);
            return e != hipSuccess ? e : launch_fwd_multi_typed<T, TO>(b, stream);
        }
    }
    bool h7 = false, h14 = false;
    int64_t first = 0;
    for (int i = 0; i < m.nheads; ++i) {
        FwdHeadArgs &a = m.head[i];
        const int cpl = a.PH == 7 ? cpl7 : 1;
        (a.PH == 7 ? h7 : h14) = true;
        a.nslices = (m.lv.C + 64 * cpl - 1) / (64 * cpl);
        a.spw = 1;
        for (int spw = 4; spw > 1; spw /= 2)
            if (static_cast<int64_t>(a.K) * ((a.nslices + spw - 1) / spw) >= 8192) {
                a.spw = spw;
                break;
            }
        a.wg_per_roi = (a.nslices + a.spw - 1) / a.spw;
        a.first = static_cast<int32_t>(first);
        first += static_cast<int64_t>(a.K) * a.wg_per_roi;
        if (first >= (int64_t(1) << 24)) return hipErrorInvalidConfiguration;
    }
    if (first == 0) return hipSuccess;
    const uint32_t g = static_cast<uint32_t>(first);
    if (cpl7 == 2) {
        if constexpr (sizeof(T) == 2) {
            if (h7 && h14) fwd_multi_kernel<T, TO, true, true, 2><<<g, 256, 0, stream>>>(m);
            else if (h7) fwd_multi_kernel<T, TO, true, false, 2><<<g, 256, 0, stream>>>(m);
            else fwd_multi_kernel<T, TO, false, true, 2><<<g, 256, 0, stream>>>(m);
        }
    } else {
        if (h7 && h14) fwd_multi_kernel<T, TO, true, true, 1><<<g, 256, 0, stream>>>(m);
        else if (h7) fwd_multi_kernel<T, TO, true, false, 1><<<g, 256, 0, stream>>>(m);
        else fwd_multi_kernel<T, TO, false, true, 1><<<g, 256, 0, stream>>>(m);
    }
    return hipGetLastError();
}

hipError_t launch_fwd_multi(FwdMultiArgs m, int feat_dtype, int out_dtype, hipStream_t stream) {
    if (feat_dtype == kF32 && out_dtype == kF32) return launch_fwd_multi_typed<float, float>(m, stream);
    if (feat_dtype == kF32 && out_dtype == kBF16)
        return launch_fwd_multi_typed<float, uint16_t>(m, stream);
    if (feat_dtype == kBF16 && out_dtype == kF32)
        return launch_fwd_multi_typed<uint16_t, float>(m, stream);
    return launch_fwd_multi_typed<uint16_t, uint16_t>(m, stream);
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
