// host_stubs.cpp -- stand-ins for the device side of libsom.so, so that the host layer
// (paper_2608_24067_amd/csrc/som_api.cpp) can be built for the CPU alone with the
// sanitizers. The host checks under test must reject every bad call before anything
// would reach a device: any call that gets here is reported and aborts the run.
#include <cstdio>
#include <cstdlib>

#include "../../paper_2608_24067_amd/csrc/som_internal.h"

namespace {
[[noreturn]] void reached(const char *what)
{
    std::fprintf(stderr, "host check let a call through to the device side: %s\n", what);
    std::abort();
}
}  // namespace

namespace som {
hipError_t launch_norms(const float *, int64_t, int64_t, double *, hipStream_t) { reached("launch_norms"); }
hipError_t launch_norms_f16(const uint16_t *, int64_t, int64_t, double *, hipStream_t) { reached("launch_norms_f16"); }
hipError_t launch_clear_flags(uint32_t *, hipStream_t) { reached("launch_clear_flags"); }
hipError_t launch_check_rows(const int32_t *, int64_t, int64_t, uint32_t *, hipStream_t) { reached("launch_check_rows"); }
hipError_t launch_plan(int, const int32_t *, const int32_t *, const float *, int64_t, int64_t, int64_t,
                       const OrderBuffers *, uint2 *, int2 *, float *, double *, uint32_t *, hipStream_t)
{
    reached("launch_plan");
}
hipError_t launch_sweep(int, bool, bool, const void *, const double *, int64_t, int64_t, int64_t, int64_t,
                        const uint2 *, const int2 *, const float *, const SweepOut &, hipStream_t)
{
    reached("launch_sweep");
}
hipError_t launch_finalize(int, const double *, int64_t, const int32_t *, int64_t, int64_t, const OrderBuffers *,
                           const double *, const SweepOut &, int32_t *, double *, int32_t *, double *, hipStream_t)
{
    reached("launch_finalize");
}
hipError_t launch_order(const int32_t *, const int32_t *, int64_t, int64_t, int64_t, const OrderBuffers &, uint32_t *,
                        hipStream_t)
{
    reached("launch_order");
}
hipError_t launch_update(bool, void *, int64_t, int64_t, const int32_t *, const int32_t *, int64_t, int64_t,
                         const int32_t *, int64_t, int64_t, const UpdateBuffers &, hipStream_t)
{
    reached("launch_update");
}
}  // namespace som

extern "C" {
const char *hipGetErrorString(hipError_t) { reached("hipGetErrorString"); }
hipError_t hipStreamSynchronize(hipStream_t) { reached("hipStreamSynchronize"); }
hipError_t hipMemcpy(void *, const void *, size_t, hipMemcpyKind) { reached("hipMemcpy"); }
}
