// Host-only stand-in for the HIP runtime header, for building the library's host code
// (argument validation, workspace layout, dispatch) for the CPU under AddressSanitizer
// and UndefinedBehaviorSanitizer.  Device builtins have inert definitions (the device
// helpers in the shared headers are compiled but never called); the runtime calls and
// the kernel launchers are stubs that do nothing and report success.
#pragma once
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
using std::isfinite;
using std::max;
using std::min;
#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static
#define __align__(n) __attribute__((aligned(n)))
typedef int hipError_t;
typedef void *hipStream_t;
enum { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorInvalidConfiguration = 9 };
enum hipMemcpyKind { hipMemcpyHostToDevice = 1, hipMemcpyDeviceToHost = 2, hipMemcpyDeviceToDevice = 3 };
#define HIP_SYMBOL(x) (&(x))
struct dim3 { unsigned x = 1, y = 1, z = 1; };
extern thread_local dim3 threadIdx, blockIdx, blockDim, gridDim;
hipError_t hipGetDevice(int *d);
hipError_t hipGetSymbolAddress(void **p, const void *sym);
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t n, hipMemcpyKind k, hipStream_t s);
hipError_t hipGetLastError();
inline void __syncthreads() {}
inline unsigned long long __ballot(int p) { return p ? 1ull : 0ull; }
inline int __popcll(unsigned long long v) { return __builtin_popcountll(v); }
template <typename T> inline T __shfl(T v, int) { return v; }
template <typename T> inline T __shfl_up(T v, unsigned) { return v; }
template <typename T> inline T __shfl_down(T v, unsigned) { return v; }
inline int atomicAdd(int *p, int v) { int o = *p; *p += v; return o; }
inline unsigned atomicAdd(unsigned *p, unsigned v) { unsigned o = *p; *p += v; return o; }
inline float atomicAdd(float *p, float v) { float o = *p; *p += v; return o; }
inline float __uint_as_float(unsigned v) { float f; std::memcpy(&f, &v, 4); return f; }
inline unsigned __float_as_uint(float f) { unsigned v; std::memcpy(&v, &f, 4); return v; }
inline int __float_as_int(float f) { int v; std::memcpy(&v, &f, 4); return v; }
inline float __int_as_float(int v) { float f; std::memcpy(&f, &v, 4); return f; }
inline unsigned __umulhi(unsigned a, unsigned b) { return (unsigned)(((unsigned long long)a * b) >> 32); }
struct float2 { float x, y; };
struct float4 { float x, y, z, w; };
struct uint2 { unsigned x, y; };
struct uint4 { unsigned x, y, z, w; };
struct int4 { int x, y, z, w; };
typedef struct { int w[4]; } __amdgpu_buffer_rsrc_t;
inline int __builtin_amdgcn_readfirstlane(int v) { return v; }
inline float __builtin_amdgcn_rcpf(float x) { return 1.0f / x; }
inline int __builtin_amdgcn_update_dpp(int o, int, int, int, int, bool) { return o; }
#define __builtin_amdgcn_make_buffer_rsrc(...) __amdgpu_buffer_rsrc_t{}
#define __builtin_amdgcn_raw_buffer_load_b32(...) 0u
#define __builtin_amdgcn_raw_buffer_load_b16(...) 0u
#define __builtin_amdgcn_fence(...)
#define __builtin_amdgcn_wave_barrier()
#define __builtin_amdgcn_ballot_w64(p) __ballot(p)
#define __builtin_amdgcn_mbcnt_lo(a, b) 0u
#define __builtin_amdgcn_mbcnt_hi(a, b) 0u
#define __builtin_amdgcn_kernarg_segment_ptr() nullptr
// clang builtin of the device code: a plain store here
template <typename V, typename P> inline void __builtin_nontemporal_store(V v, P p) { *p = v; }
