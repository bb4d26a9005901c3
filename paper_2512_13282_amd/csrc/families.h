// families.h -- per-family launch functions.  Each kernel family is compiled in
// its own translation unit (launch_*.hip) so that the library builds in
// parallel; gemm_launch.hip routes a plan's configuration to its family.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace gemm {

// Each queues the kernel of configuration `cfg` (an index into kConfigs) on
// `s` with `grid` workgroups, and returns hipErrorInvalidValue for a
// configuration (or B layout) the family does not compile.
template <int DT> hipError_t launch_tile_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s);
template <int DT> hipError_t launch_direct_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s);
template <int DT, bool BT>
hipError_t launch_ring_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s);
template <int DT> hipError_t launch_small_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s);
// The separate split-K reduction over the partial planes of a.workspace.
template <int DT> hipError_t launch_splitk_reduce(const KernelArgs &a, int64_t blocks, hipStream_t s);

}  // namespace gemm
