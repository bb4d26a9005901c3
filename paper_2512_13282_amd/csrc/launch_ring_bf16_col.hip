// launch_ring_bf16_col.hip -- the RING instances for bf16 inputs, B col-major.
#include "launch_ring.h"

namespace gemm {
template hipError_t launch_ring_family<DT_BF16, true>(int32_t, const KernelArgs &, int64_t, hipStream_t);
}  // namespace gemm
