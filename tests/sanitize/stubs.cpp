// Stubs for the host build of api.hip (see hip/hip_runtime.h): the kernel launchers
// and the runtime calls do nothing and report success; the launch-eligibility
// predicates are the library's own rules, restated.
#include "hip/hip_runtime.h"
#include "internal.hpp"

thread_local dim3 threadIdx, blockIdx, blockDim, gridDim;
static unsigned char g_symbol[1 << 20];
hipError_t hipGetDevice(int *d) { *d = 0; return hipSuccess; }
hipError_t hipGetSymbolAddress(void **p, const void *) { *p = g_symbol; return hipSuccess; }
hipError_t hipMemcpyAsync(void *, const void *, size_t, hipMemcpyKind, hipStream_t) { return hipSuccess; }
hipError_t hipGetLastError() { return hipSuccess; }

namespace rex {
bool fwd_fast_available(int PH, int PW, int S) {
    return S == 2 && ((PH == 7 && PW == 7) || (PH == 14 && PW == 14));
}
bool bwd_fast_available(int PH, int PW, int S) { return fwd_fast_available(PH, PW, S); }
bool gather_available(int PH, int PW, int S) { return fwd_fast_available(PH, PW, S); }
bool pool_fwd_fast_available(int PH, int PW) { return PH * PW <= kPoolFastBins; }
bool pool_gather_available(int PH, int PW) { return PH == 7 && PW == 7; }
hipError_t launch_level_map(const float *, int32_t, int32_t, float, int32_t, int32_t *, hipStream_t) { return hipSuccess; }
hipError_t launch_plan(const PlanArgs &, hipStream_t) { return hipSuccess; }
hipError_t launch_fwd(FwdArgs, int, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_fwd_multi(FwdMultiArgs, int, int, hipStream_t) { return hipSuccess; }
hipError_t launch_bwd(BwdArgs, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_gather(GatherArgs, int, hipStream_t) { return hipSuccess; }
hipError_t launch_pool_fwd(PoolArgs, int, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_pool_bwd(PoolArgs, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_pool_gather(GatherArgs, int, hipStream_t) { return hipSuccess; }
hipError_t launch_deform_fwd(DeformArgs, int, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_deform_bwd(DeformArgs, int, int, bool, hipStream_t) { return hipSuccess; }
hipError_t launch_deform_gather(GatherArgs, const DeformArgs &, int, hipStream_t) { return hipSuccess; }
bool deform_gather_available(int PH, int PW, int S) { return PH == 7 && PW == 7 && S >= 1 && S <= 2; }
hipError_t launch_nms(NmsArgs, hipStream_t) { return hipSuccess; }
hipError_t launch_nms_batched(const NmsBatchArgs &, hipStream_t) { return hipSuccess; }
hipError_t launch_zero(const LevelTable &, const int64_t *, const int *, hipStream_t) { return hipSuccess; }
}  // namespace rex
