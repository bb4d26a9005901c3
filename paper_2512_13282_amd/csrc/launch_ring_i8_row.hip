// launch_ring_i8_row.hip -- the RING instances for int8 inputs, B row-major.
#include "launch_ring.h"

namespace gemm {
template hipError_t launch_ring_family<DT_I8, false>(int32_t, const KernelArgs &, int64_t, hipStream_t);
}  // namespace gemm
