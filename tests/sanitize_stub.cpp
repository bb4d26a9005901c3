// Stand-ins for the device side of the library, for a host-only build of the C ABI
// (gemm_api.cpp) and the selector (selector.cpp) under AddressSanitizer and
// UndefinedBehaviorSanitizer on a machine without a GPU.  The CPU tests that run
// against that build never reach a launch: every call they make is rejected or
// answered on the host first.  Any launch that did get here reports a HIP error.
#include <stdint.h>

#include "../include/gemm_mi355x.h"
#include "../paper_2512_13282_amd/csrc/launch.h"

namespace gemm {
int launch_gemm(const KernelArgs &, int32_t, int64_t, void *, bool) { return LAUNCH_HIP_ERROR; }
int release_workspaces() { return LAUNCH_OK; }
}  // namespace gemm

extern "C" int gemm_probe_mfma(int, int, int32_t, int64_t *, unsigned *, gemm_probe_info *, void *) {
    return GEMM_ERR_HIP;
}
extern "C" int gemm_probe_read(const void *, int64_t, unsigned *, int64_t, void *) { return GEMM_ERR_HIP; }
