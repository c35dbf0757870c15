// common.hpp -- device-side building blocks shared by the RoIAlign kernels.
//
// Geometry follows the definition stated in include/roi_extract.h: the sample
// coordinates are computed in binary32 with one rounding per operation, in the
// written order, with no contraction into fused multiply-adds (the whole library
// is compiled with -ffp-contract=off; accumulations that should fuse call fmaf
// explicitly).  Division is the correctly rounded IEEE division (hipcc's default).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rex {

constexpr int kMaxLevels = 8;
constexpr int kGridCap = 64;   // adaptive sampling grid cap (RE_MAX_SAMPLING)

enum : int { kF32 = 0, kBF16 = 1 };

// One pyramid level as the kernels see it.  Strides are in elements.
struct LevelArg {
    const void *data;
    int64_t sn, sc, sh, sw;
    int32_t H, W;
    float scale;
    uint32_t img_bytes;   // bytes spanned by one image (0: too large for buffer addressing)
};

struct LevelTable {
    LevelArg l[kMaxLevels];
    int32_t num;
    int32_t N;
    int32_t C;
    int32_t pad;
};

// Level `l` of the table.  Every access uses a constant index so the kernel
// argument block is read straight from the kernarg segment (no scratch copy).
__device__ __forceinline__ LevelArg level_at(const LevelTable &t, int l) {
    switch (l) {
        case 1: return t.l[1];
        case 2: return t.l[2];
        case 3: return t.l[3];
        case 4: return t.l[4];
        case 5: return t.l[5];
        case 6: return t.l[6];
        case 7: return t.l[7];
        default: return t.l[0];
    }
}

// Element `l` (0 <= l < 8) of a small per-level array in the kernel arguments,
// written with constant indices only, for the same reason as level_at.
template <typename T, int N>
__device__ __forceinline__ T pick(const T (&arr)[N], int l) {
    static_assert(N >= kMaxLevels, "per-level array");
    switch (l) {
        case 1: return arr[1];
        case 2: return arr[2];
        case 3: return arr[3];
        case 4: return arr[4];
        case 5: return arr[5];
        case 6: return arr[6];
        case 7: return arr[7];
        default: return arr[0];
    }
}

// ---------------------------------------------------------------------------
// bfloat16 <-> binary32
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even, on the 16 discarded bits; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Pointers into global memory.  Data pointers that arrive inside an argument
// struct lose their address space, which would turn every access into a flat
// instruction; these casts restore it.
#define REX_GLOBAL __attribute__((address_space(1)))
template <typename T> using gptr = REX_GLOBAL T *;
template <typename T> using gcptr = const REX_GLOBAL T *;
template <typename T> __device__ __forceinline__ gcptr<T> as_global(const void *p) {
    return (gcptr<T>)(p);
}
template <typename T> __device__ __forceinline__ gptr<T> as_global_mut(void *p) {
    return (gptr<T>)(p);
}

template <typename T> __device__ __forceinline__ float load_f32(gcptr<T> p);
template <> __device__ __forceinline__ float load_f32<float>(gcptr<float> p) { return *p; }
template <> __device__ __forceinline__ float load_f32<uint16_t>(gcptr<uint16_t> p) {
    return bf16_to_f32(*p);
}

template <typename T> __device__ __forceinline__ void store_f32(gptr<T> p, float v);
template <> __device__ __forceinline__ void store_f32<float>(gptr<float> p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_f32<uint16_t>(gptr<uint16_t> p, float v) {
    *p = f32_to_bf16(v);
}


// ---------------------------------------------------------------------------
// Buffer-resource loads
// ---------------------------------------------------------------------------
// A raw buffer resource (stride 0) holds a base address and a byte range in
// scalar registers; each lane then supplies one 32-bit byte offset, and the
// hardware's range check makes an offset at or past the range read 0 without a
// memory access.  Offsets inside one image of a level stay below 2^30 (checked on
// the host), so adding kBufOOB to any term of a lane-offset sum pushes it out of
// range without wrapping, even when all three terms carry it.  The check covers the
// lane offset only: a scalar offset added by the instruction is not checked.
constexpr uint32_t kBufOOB = 0x40000000u;
constexpr uint32_t kBufMaxBytes = 0x40000000u;
constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, no swizzle (gfx9 family)
constexpr int kStoreNT = 2;              // buffer store cache policy: non-temporal
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // a 16-byte buffer store
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// n contiguous values from src (16-byte aligned) to dst, 4 per store where dst is
// aligned to 4 elements (one 16-byte or 8-byte store), the rest one at a time; every
// thread i of `nt` takes groups i, i + nt, ...  The vector stores are non-temporal: the
// kernel never reads what it writes here, so it streams past the caches and leaves
// them to the data that is read (batch-2 box head forward: 46.8 -> 45.5 us).
template <typename T>
__device__ __forceinline__ void store_run_f32(gptr<T> dst, const float *src, int n, int i, int nt) {
    int done = 0;
    if ((reinterpret_cast<uintptr_t>(dst) & (4 * sizeof(T) - 1)) == 0) {
        const int nv = n >> 2;
        for (int v = i; v < nv; v += nt) {
            const float4 f = *reinterpret_cast<const float4 *>(src + 4 * v);
            if constexpr (sizeof(T) == 4) {
                const u32x4 w = {__float_as_uint(f.x), __float_as_uint(f.y), __float_as_uint(f.z),
                                 __float_as_uint(f.w)};
                __builtin_nontemporal_store(w, reinterpret_cast<REX_GLOBAL u32x4 *>(dst + 4 * v));
            } else {
                const u32x2 w = {
                    static_cast<uint32_t>(f32_to_bf16(f.x)) | (static_cast<uint32_t>(f32_to_bf16(f.y)) << 16),
                    static_cast<uint32_t>(f32_to_bf16(f.z)) | (static_cast<uint32_t>(f32_to_bf16(f.w)) << 16)};
                __builtin_nontemporal_store(w, reinterpret_cast<REX_GLOBAL u32x2 *>(dst + 4 * v));
            }
        }
        done = nv << 2;
    }
    for (int e = done + i; e < n; e += nt) store_f32<T>(dst + e, src[e]);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0,
                                             static_cast<int>(bytes), kBufDword3);
}

// Raw element bits (fp32 bits, or bf16 bits zero-extended); the conversion is a
// separate step so a batch of loads can be issued before any of them is waited on.
template <typename T> __device__ __forceinline__ uint32_t buf_load_raw(__amdgpu_buffer_rsrc_t r,
                                                                       uint32_t off);
template <> __device__ __forceinline__ uint32_t buf_load_raw<float>(__amdgpu_buffer_rsrc_t r,
                                                                    uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
template <> __device__ __forceinline__ uint32_t buf_load_raw<uint16_t>(__amdgpu_buffer_rsrc_t r,
                                                                       uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
// Same, with a scalar byte offset added to every lane's offset.  The range check
// sees the lane offset only: the scalar offset must itself keep the access inside
// the range (mark an access out of range through the lane offset, never through
// the scalar one).
template <typename T> __device__ __forceinline__ uint32_t buf_load_raw_s(__amdgpu_buffer_rsrc_t r,
                                                                         uint32_t off, uint32_t soff);
template <> __device__ __forceinline__ uint32_t buf_load_raw_s<float>(__amdgpu_buffer_rsrc_t r,
                                                                      uint32_t off, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, soff, 0);
}
template <> __device__ __forceinline__ uint32_t buf_load_raw_s<uint16_t>(__amdgpu_buffer_rsrc_t r,
                                                                         uint32_t off, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, soff, 0);
}
template <typename T> __device__ __forceinline__ float raw_to_f32(uint32_t v);
template <> __device__ __forceinline__ float raw_to_f32<float>(uint32_t v) {
    return __uint_as_float(v);
}
template <> __device__ __forceinline__ float raw_to_f32<uint16_t>(uint32_t v) {
    return __uint_as_float(v << 16);
}

// ---------------------------------------------------------------------------
// FPN level (threshold form), binary32
// ---------------------------------------------------------------------------

// box_plus1: boxes are inclusive pixel ranges, each side (x2 - x1) + 1.
__device__ __forceinline__ int fpn_level(float x1, float y1, float x2, float y2, int num_levels,
                                         float finest_scale, int box_plus1) {
    float w = x2 - x1;
    float h = y2 - y1;
    if (box_plus1) {
        w = w + 1.0f;
        h = h + 1.0f;
    }
    const float area = w * h;
    int lvl = 0;
    for (int j = 1; j < num_levels; ++j) {
        const float side = finest_scale * static_cast<float>(1 << j);
        const float thr = side * side;
        lvl += (area >= thr) ? 1 : 0;
    }
    return lvl;
}

// Column 0 of a RoI: truncated toward zero; -1 if it names no image of the batch.
__device__ __forceinline__ int roi_batch(float v, int n) {
    const float t = truncf(v);
    if (!(t >= 0.0f) || !(t < static_cast<float>(n))) return -1;
    return static_cast<int>(t);
}

// ---------------------------------------------------------------------------
// Sampling geometry along one axis
// ---------------------------------------------------------------------------

struct Axis {
    float start;
    float bin;
    int grid;
    float len;   // box length on the level (after the minimum size)
};

// Bin-tiles met by a conservative box around the footprint of a RoI on its level (scale
// s, W x H map, tiles of 2^shift pixels, ntx x nty of them): every sample of the RoI
// lies between the (shifted) box edges for any output size, sampling ratio and
// alignment; taps add one pixel, and a 1.5-pixel margin absorbs rounding.  Non-finite
// boxes cover the whole map.  The plan bins RoIs to tiles with it, and the backward of
// deformable pooling uses it to tell which taps the tile lists reach.
__device__ __forceinline__ void roi_tile_range(float x1, float y1, float x2, float y2, float s,
                                               int Wi, int Hi, int shift, int ntx, int nty,
                                               int &tx0, int &tx1, int &ty0, int &ty1) {
    const float W = static_cast<float>(Wi - 1);
    const float H = static_cast<float>(Hi - 1);
    float lx = 0.0f, hx = W, ly = 0.0f, hy = H;
    if (isfinite(x1) && isfinite(x2) && isfinite(y1) && isfinite(y2)) {
        lx = fminf(fmaxf(fminf(x1, x2) * s - 1.5f, 0.0f), W);
        hx = fminf(fmaxf(fmaxf(fmaxf(x1, x2) * s, x1 * s + 1.0f) + 2.5f, 0.0f), W);
        ly = fminf(fmaxf(fminf(y1, y2) * s - 1.5f, 0.0f), H);
        hy = fminf(fmaxf(fmaxf(fmaxf(y1, y2) * s, y1 * s + 1.0f) + 2.5f, 0.0f), H);
    }
    tx0 = static_cast<int>(lx) >> shift;
    tx1 = max(static_cast<int>(hx) >> shift, tx0);
    ty0 = static_cast<int>(ly) >> shift;
    ty1 = max(static_cast<int>(hy) >> shift, ty0);
    tx1 = min(tx1, ntx - 1);
    ty1 = min(ty1, nty - 1);
}

__device__ __forceinline__ Axis axis_setup(float c1, float c2, float scale, int aligned, int P,
                                           int S) {
    const float off = aligned ? 0.5f : 0.0f;
    float s = c1 * scale;
    s = s - off;
    float e = c2 * scale;
    e = e - off;
    float len = e - s;
    if (!aligned) len = fmaxf(len, 1.0f);
    const float bin = len / static_cast<float>(P);
    int g;
    if (S > 0) {
        g = S;
    } else if (!(bin > 0.0f)) {
        g = 0;
    } else {
        const float cg = ceilf(bin);
        g = cg > static_cast<float>(kGridCap) ? kGridCap : static_cast<int>(cg);
    }
    Axis a;
    a.start = s;
    a.bin = bin;
    a.grid = g;
    a.len = len;
    return a;
}

// Bilinear neighbours of one sample.  lo < 0 marks a sample outside [-1, size].
struct Tap {
    int lo;
    int hi;
    float wlo;
    float whi;
};

__device__ __forceinline__ Tap axis_tap(const Axis &a, int p, int i, int size) {
    const float t1 = static_cast<float>(p) * a.bin;
    const float t2 = a.start + t1;
    const float t3 = static_cast<float>(i) + 0.5f;
    const float t4 = t3 * a.bin;
    const float t5 = t4 / static_cast<float>(a.grid);
    float v = t2 + t5;
    Tap t;
    if (v < -1.0f || v > static_cast<float>(size)) {
        t.lo = -1;
        t.hi = -1;
        t.wlo = 0.0f;
        t.whi = 0.0f;
        return t;
    }
    v = fmaxf(v, 0.0f);
    int lo = static_cast<int>(v);
    int hi;
    if (lo >= size - 1) {
        lo = size - 1;
        hi = size - 1;
        v = static_cast<float>(lo);
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

// ---------------------------------------------------------------------------
// Launch-order helpers
// ---------------------------------------------------------------------------

// Consecutive workgroup ids are dispatched round-robin over the 8 XCDs of an
// MI355X.  Map them so XCD x receives one contiguous slice of the logical order,
// which keeps neighbouring (plan-sorted) RoIs inside one XCD's L2.  Bijective on
// [0, n) for any n.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t n) {
    constexpr uint32_t X = 8;
    const uint32_t q = n / X, r = n % X;
    const uint32_t x = bid % X, i = bid / X;
    return (x < r) ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

// Orders LDS writes and later LDS reads of other lanes within one wavefront.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// n / d for 0 <= n < 2^21 - 1 and d >= 1, exactly: (n + 1/2) times the hardware
// reciprocal of d (1 ulp) is within (n + 1/2) 2^-22 / d < 1 / (2d) of (n + 1/2) / d,
// closer than the nearest integer.
__device__ __forceinline__ int small_div_exact(int n, int d) {
    return static_cast<int>((static_cast<float>(n) + 0.5f) *
                            __builtin_amdgcn_rcpf(static_cast<float>(d)));
}

__device__ __forceinline__ int uniform_i(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float uniform_f(float v) {
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

}  // namespace rex
