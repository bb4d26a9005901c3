// launch_ring_bf16_row.hip -- the RING instances for bf16 inputs, B row-major.
#include "launch_ring.h"

namespace gemm {
template hipError_t launch_ring_family<DT_BF16, false>(int32_t, const KernelArgs &, int64_t, hipStream_t);
}  // namespace gemm
