// Host stand-in for the HIP runtime header, for running the plan kernels' source on the
// CPU: one workgroup at a time, one fiber per work-item, a real workgroup barrier,
// and wave-level exchanges for ballot and DPP (defined in emu_main.cpp).
#pragma once
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>
using std::max; using std::min;
struct EmuDim { unsigned x = 0, y = 0, z = 0; };
extern thread_local EmuDim threadIdx;
extern EmuDim blockIdx, blockDim, gridDim;
#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static
typedef int hipError_t;
typedef void *hipStream_t;
#define hipSuccess 0
#define __align__(n) __attribute__((aligned(n)))
enum hipMemcpyKind { hipMemcpyHostToDevice = 1, hipMemcpyDeviceToHost = 2, hipMemcpyDeviceToDevice = 3 };
#define HIP_SYMBOL(x) (&(x))
hipError_t hipGetDevice(int *d);
hipError_t hipGetSymbolAddress(void **p, const void *sym);
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t n, hipMemcpyKind k, hipStream_t s);
void __syncthreads();
inline int atomicAdd(int *p, int v) { return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST); }
inline unsigned atomicAdd(unsigned *p, unsigned v) { return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST); }
unsigned long long __ballot(int pred);
inline int __popcll(unsigned long long v) { return __builtin_popcountll(v); }
int emu_update_dpp(int old, int src, int ctrl, int row_mask, int bank_mask, bool bound);
#define __builtin_amdgcn_update_dpp(o, s, c, r, b, bc) emu_update_dpp(o, s, c, r, b, bc)
inline float __builtin_amdgcn_rcpf(float x) { return 1.0f / x; }
inline int __builtin_amdgcn_readfirstlane(int v) { return v; }
typedef struct { int w[4]; } __amdgpu_buffer_rsrc_t;
#define __builtin_amdgcn_make_buffer_rsrc(...) __amdgpu_buffer_rsrc_t{}
#define __builtin_amdgcn_raw_buffer_load_b32(...) 0u
#define __builtin_amdgcn_raw_buffer_load_b16(...) 0u
#define __builtin_amdgcn_fence(...)
#define __builtin_amdgcn_wave_barrier()
#define __builtin_amdgcn_ballot_w64(p) __ballot(p)
#define __builtin_amdgcn_mbcnt_lo(a, b) 0
#define __builtin_amdgcn_mbcnt_hi(a, b) 0
inline float __uint_as_float(unsigned v) { float f; std::memcpy(&f, &v, 4); return f; }
inline unsigned __float_as_uint(float f) { unsigned v; std::memcpy(&v, &f, 4); return v; }
inline int __float_as_int(float f) { int v; std::memcpy(&v, &f, 4); return v; }
inline float __int_as_float(int v) { float f; std::memcpy(&f, &v, 4); return f; }
inline unsigned __umulhi(unsigned a, unsigned b) { return (unsigned)(((unsigned long long)a * b) >> 32); }
struct float4 { float x, y, z, w; };
struct float2 { float x, y; };
struct int4 { int x, y, z, w; };
struct uint2 { unsigned x, y; };
struct uint4 { unsigned x, y, z, w; };
inline float4 make_float4(float a, float b, float c, float d) { return {a, b, c, d}; }
using std::isfinite;
// clang builtin of the device code: a plain store here
template <typename V, typename P> inline void __builtin_nontemporal_store(V v, P p) { *p = v; }
