// launch_small.hip -- instances of the narrow-M streaming kernels, the
// matrix-vector kernels and the separate split-K reduction.
#include "families.h"
#include "kern_small.h"

namespace gemm {

template <int DT>
hipError_t launch_small_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    switch (cfg) {
        case 14:
            if (a.b_trans) return hipErrorInvalidValue;
            hipLaunchKernelGGL((gemm_stream_kernel<DT, 32, 4>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        case 15:
            if (a.b_trans) return hipErrorInvalidValue;
            hipLaunchKernelGGL((gemm_stream_kernel<DT, 64, 3>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        case 26:
            if (a.b_trans) return hipErrorInvalidValue;
            hipLaunchKernelGGL((gemv_kernel<DT>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        case 27:
            if (!a.b_trans) return hipErrorInvalidValue;
            hipLaunchKernelGGL((gemv_bt_kernel<DT>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        default: return hipErrorInvalidValue;
    }
}

template <int DT>
hipError_t launch_splitk_reduce(const KernelArgs &a, int64_t blocks, hipStream_t s) {
    hipLaunchKernelGGL(splitk_reduce_kernel<DT>, dim3(unsigned(blocks)), dim3(256), 0, s, a);
    return hipGetLastError();
}

template hipError_t launch_small_family<DT_I8>(int32_t, const KernelArgs &, int64_t, hipStream_t);
template hipError_t launch_small_family<DT_BF16>(int32_t, const KernelArgs &, int64_t, hipStream_t);
template hipError_t launch_splitk_reduce<DT_I8>(const KernelArgs &, int64_t, hipStream_t);
template hipError_t launch_splitk_reduce<DT_BF16>(const KernelArgs &, int64_t, hipStream_t);

}  // namespace gemm
