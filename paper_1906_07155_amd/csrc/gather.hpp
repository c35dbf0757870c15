// gather.hpp -- the tile-gather machinery shared by the backward kernels that write
// every gradient element once: the RoIAlign gather (bwd.hip) and the RoI max pooling
// gather (pool.hip).
//
// The plan bins RoIs to square tiles of one (level, image) and orders the tiles by
// decreasing list length.  A workgroup of such a kernel owns one tile (or a block of
// four 8x8 quadrants of it) and one group of 64 channels: each of its four waves keeps
// an 8x8 quadrant of pixels in registers, one channel per lane, and stores it once at
// the end.
#pragma once

#include <algorithm>

#include "internal.hpp"

namespace rex {

// Where a workgroup of the quadrant-form gather sits: the tile's level and image,
// its wave's quadrant and the bounding box of the workgroup's quadrants.
struct GatherTile {
    LevelArg L;
    int l, b;
    int R0, Q0;                 // this wave's quadrant
    int WR0, WR1, WC0, WC1;     // the workgroup's region
    int cg, nch;
    bool wave_on;
};

// Decodes a quadrant-form workgroup: blocks in dispatch order walk the tiles in
// `order` (longest list first); the channel groups and quadrant blocks of one tile
// are adjacent.
__device__ __forceinline__ int gather_tile(const GatherArgs &a, const int32_t *order,
                                           GatherTile &x) {
    const int tid = threadIdx.x;
    const int wave = uniform_i(tid >> 6);
    const uint32_t lid = blockIdx.x;
    const int per_tile = a.ncg * a.wg_per_tile;
    const int rank = static_cast<int>(fdiv(lid, a.div_tile));
    const int rem = static_cast<int>(lid) - rank * per_tile;
    const int cg = rem >> a.wgpt_shift;   // wg_per_tile is a power of two
    int t = order[rank];
    t = max(0, min(t, a.ntiles - 1));
    const int quad0 = (rem & (a.wg_per_tile - 1)) * 4;
    const int quad = quad0 + wave;

    int l = 0;
#pragma unroll
    for (int i = 1; i < kMaxLevels; ++i)
        if (i < a.lv.num && t >= a.tbase[i]) l = i;
    x.L = level_at(a.lv, l);
    x.l = l;
    const int ntx = pick(a.ntx, l);
    const int per_img = pick(a.nty, l) * ntx;
    const int local = t - pick(a.tbase, l);
    x.b = static_cast<int>(fdiv(static_cast<uint32_t>(local), pick(a.img_m, l), pick(a.img_sh, l)));
    const int rt = local - x.b * per_img;
    const int ty = static_cast<int>(fdiv(static_cast<uint32_t>(rt), pick(a.row_m, l), pick(a.row_sh, l)));
    const int tx = rt - ty * ntx;
    const int qs = a.qside, qsh = a.qs_shift;   // qside is a power of two
    x.R0 = (ty << a.tile_shift) + (quad >> qsh) * 8;
    x.Q0 = (tx << a.tile_shift) + (quad & (qs - 1)) * 8;
    // Waves whose quadrant is off the map still take part in staging and barriers.
    x.wave_on = quad < qs * qs && x.R0 < x.L.H && x.Q0 < x.L.W;
    // The workgroup's region: the bounding box of its (up to 4) quadrants.
    const int qlast = min(quad0 + 3, qs * qs - 1);
    x.WR0 = (ty << a.tile_shift) + (quad0 >> qsh) * 8;
    x.WR1 = (ty << a.tile_shift) + (qlast >> qsh) * 8 + 8;
    x.WC0 = (tx << a.tile_shift) + ((qlast >> qsh > quad0 >> qsh) ? 0 : (quad0 & (qs - 1))) * 8;
    x.WC1 = (tx << a.tile_shift) + ((qlast >> qsh > quad0 >> qsh) ? qs : (qlast & (qs - 1)) + 1) * 8;
    x.cg = cg;
    x.nch = min(64, a.lv.C - cg * 64);
    return t;
}

// Every pixel of this wave's quadrant is written once (the clearing is fused).  The
// pixel offset is the same for the whole wave (scalar), the channel offset is the
// lane's; lanes past the last channel write out of range, which is dropped.  The
// gradient pyramid is far larger than the L2 and read only by a later pass, so the
// stores are non-temporal: they stream to memory instead of evicting cached data.
__device__ __forceinline__ void gather_store(const GatherTile &x, int zero_init,
                                             const float (&acc)[8][8], float *scratch) {
    if (!x.wave_on) return;
    const int lane = threadIdx.x & 63;
    const int c = x.cg * 64 + lane;
    const bool lane_on = lane < x.nch;
    const LevelArg &L = x.L;
    const char *img = static_cast<const char *>(L.data) + static_cast<int64_t>(x.b) * L.sn * 4;
    const __amdgpu_buffer_rsrc_t dst = make_rsrc(img, L.img_bytes);
    // the lane's channel: stride_c elements apart (1 for channels-last levels)
    const uint32_t vo = lane_on ? static_cast<uint32_t>(c) * static_cast<uint32_t>(L.sc) * 4u
                                : kBufOOB;
    const uint32_t sh4 = static_cast<uint32_t>(L.sh) * 4u;
    const uint32_t sw4 = static_cast<uint32_t>(L.sw) * 4u;
    const uint32_t base = static_cast<uint32_t>(x.R0) * sh4 + static_cast<uint32_t>(x.Q0) * sw4;
    if (L.sc != 1 && L.sw == 1 && zero_init && x.R0 + 8 <= L.H && x.Q0 + 8 <= L.W) {
        // Channels in separate planes (NCHW): a lane's row of 8 pixels is 32 contiguous
        // bytes, written as two 16-byte stores, and the neighbouring quadrant's wave
        // writes the other half of the 64-byte run; ordinary stores, so the L2 merges
        // the halves before they go to memory.
#pragma unroll
        for (int rr = 0; rr < 8; ++rr) {
            const uint32_t o = base + rr * sh4;
            const u32x4 lo = {__float_as_uint(acc[rr][0]), __float_as_uint(acc[rr][1]),
                              __float_as_uint(acc[rr][2]), __float_as_uint(acc[rr][3])};
            const u32x4 hi = {__float_as_uint(acc[rr][4]), __float_as_uint(acc[rr][5]),
                              __float_as_uint(acc[rr][6]), __float_as_uint(acc[rr][7])};
            __builtin_amdgcn_raw_buffer_store_b128(lo, dst, vo, o, 0);
            __builtin_amdgcn_raw_buffer_store_b128(hi, dst, vo, o + 16u, 0);
        }
        return;
    }
    if (L.sc == 1 && zero_init && x.nch == 64 && x.R0 + 8 <= L.H && x.Q0 + 8 <= L.W) {
        // Channels-last, a whole quadrant inside the map and a full channel group: each
        // row of 8 pixels is turned around in this wave's 2 KiB of LDS so a lane holds 4
        // adjacent channels of one pixel, and leaves as two 16-byte stores per lane (1
        // KiB per instruction instead of 256 bytes: 16 store instructions per wave
        // instead of 64).
        const int lq = lane >> 4;           // pixel of a group of 4
        const int lc = (lane & 15) * 4;     // its first channel in the group
        const uint32_t cvo = static_cast<uint32_t>(x.cg * 64 + lc) * 4u;
#pragma unroll
        for (int rr = 0; rr < 8; ++rr) {
#pragma unroll
            for (int q = 0; q < 8; ++q) scratch[q * 64 + lane] = acc[rr][q];
            wave_sync();
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float4 v = *reinterpret_cast<const float4 *>(scratch + (h * 4 + lq) * 64 + lc);
                const u32x4 w = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                                 __float_as_uint(v.w)};
                const uint32_t vo4 = static_cast<uint32_t>(h * 4 + lq) * sw4 + cvo;
                __builtin_amdgcn_raw_buffer_store_b128(w, dst, vo4, base + rr * sh4, kStoreNT);
            }
            wave_sync();   // the row's values are read before the next row overwrites them
        }
        return;
    }
    // channel-contiguous lanes stream past the L2; strided channels go through it
    const bool nt = L.sc == 1;
    auto st32 = [&](float v, uint32_t lane_off, uint32_t off) {
        if (nt) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), dst, lane_off, off, kStoreNT);
        else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), dst, lane_off, off, 0);
    };
    if (zero_init && x.R0 + 8 <= L.H && x.Q0 + 8 <= L.W) {
        // a whole quadrant inside the map: 64 plain stores, no per-pixel checks
#pragma unroll
        for (int rr = 0; rr < 8; ++rr)
#pragma unroll
            for (int q = 0; q < 8; ++q)
                st32(acc[rr][q], vo, base + rr * sh4 + q * sw4);
        return;
    }
    // Quadrants cut by the map edge, or accumulation: pixels off the map take an
    // out-of-range offset (loads read 0, stores are dropped), so there are no branches.
    // When accumulating, a row's old values are loaded together before it is stored,
    // one row at a time (the empty asm keeps the compiler from hoisting every row's
    // loads, which would cost registers).
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) {
        const bool row_on = x.R0 + rr < L.H;
        uint32_t vq[8];
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            vq[q] = (row_on && x.Q0 + q < L.W) ? vo : kBufOOB;
            v[q] = acc[rr][q];
        }
        if (!zero_init) {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                v[q] += __uint_as_float(
                    __builtin_amdgcn_raw_buffer_load_b32(dst, vq[q], base + rr * sh4 + q * sw4, 0));
        }
#pragma unroll
        for (int q = 0; q < 8; ++q)
            st32(v[q], vq[q], base + rr * sh4 + q * sw4);
        asm volatile("" ::: "memory");
    }
}

// Launch-time fields of a gather (block-id decoding without integer division); false
// when the tile geometry is not one the decoding covers.
inline bool gather_prepare(GatherArgs &a) {
    a.ncg = (a.lv.C + 63) / 64;
    a.wg_per_tile = (a.qside * a.qside + 3) / 4;
    // qside = 2^(tile_shift - 3) with tile_shift >= 4, so qside and wg_per_tile are
    // powers of two
    a.qs_shift = a.tile_shift - 3;
    a.wgpt_shift = 2 * a.qs_shift - 2;
    if (a.qs_shift < 1 || a.qside != (1 << a.qs_shift) || a.wg_per_tile != (1 << a.wgpt_shift))
        return false;
    a.div_tile = make_fastdiv(static_cast<uint32_t>(a.ncg * a.wg_per_tile));
    for (int l = 0; l < kMaxLevels; ++l) {
        const FastDiv di = make_fastdiv(static_cast<uint32_t>(std::max(1, a.ntx[l] * a.nty[l])));
        const FastDiv dr = make_fastdiv(static_cast<uint32_t>(std::max(1, a.ntx[l])));
        a.img_m[l] = di.m;
        a.img_sh[l] = di.sh;
        a.row_m[l] = dr.m;
        a.row_sh[l] = dr.sh;
        const FastDiv dw = make_fastdiv(static_cast<uint32_t>(l < a.lv.num ? std::max<int64_t>(1, a.lv.l[l].W) : 1));
        a.wid_m[l] = dw.m;
        a.wid_sh[l] = dw.sh;
    }
    return true;
}

}  // namespace rex
