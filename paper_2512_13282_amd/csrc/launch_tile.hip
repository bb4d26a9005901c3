// launch_tile.hip -- instances of the GENERIC, MACRO and register-staged
// SKINNY configurations.
#include "families.h"
#include "kern_tile.h"

namespace gemm {

template <int DT, int BM, int BN, int WM, int WN, bool VEC, int WPE>
static hipError_t launch_tile(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    if constexpr (VEC)
        hipLaunchKernelGGL((gemm_vec_kernel<DT, BM, BN, WM, WN, WPE>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_tile_kernel<DT, BM, BN, WM, WN, false, WPE>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_tile_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    if (a.b_trans) {
        // Column-major B (stored N x K): the element-wise generic kernels only.
        switch (cfg) {
            case 0:
                hipLaunchKernelGGL((gemm_tile_kernel<DT, 64, 64, 2, 2, false, 2, true>), dim3(unsigned(grid)),
                                   dim3(256), 0, s, a);
                return hipGetLastError();
            case 1:
                hipLaunchKernelGGL((gemm_tile_kernel<DT, 128, 128, 2, 2, false, 1, true>), dim3(unsigned(grid)),
                                   dim3(256), 0, s, a);
                return hipGetLastError();
            default: return hipErrorInvalidValue;
        }
    }
    switch (cfg) {
        case 0: return launch_tile<DT, 64, 64, 2, 2, false, 2>(a, grid, s);
        case 1: return launch_tile<DT, 128, 128, 2, 2, false, 1>(a, grid, s);
        case 2: return launch_tile<DT, 256, 256, 2, 2, true, 1>(a, grid, s);
        case 3: return launch_tile<DT, 128, 256, 2, 2, true, 1>(a, grid, s);
        case 4: return launch_tile<DT, 256, 128, 2, 2, true, 1>(a, grid, s);
        case 5: return launch_tile<DT, 128, 128, 2, 2, true, 2>(a, grid, s);
        case 6: return launch_tile<DT, 32, 256, 1, 4, true, 2>(a, grid, s);
        case 7: return launch_tile<DT, 64, 256, 1, 4, true, 2>(a, grid, s);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_tile_family<DT_I8>(int32_t, const KernelArgs &, int64_t, hipStream_t);
template hipError_t launch_tile_family<DT_BF16>(int32_t, const KernelArgs &, int64_t, hipStream_t);

}  // namespace gemm
