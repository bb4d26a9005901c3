// gemm_launch.hip -- routes a plan to its kernel family and owns the split-K
// workspaces.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdlib.h>

#include <map>
#include <mutex>
#include <utility>

#include "configs.h"
#include "families.h"
#include "launch.h"

namespace gemm {

// Configuration index -> the translation unit that compiles it.  The streaming
// narrow-M kernels (configurations 14 and 15) are SKINNY by purpose but live
// with the other small-shape kernels.
template <int DT>
static hipError_t launch_config(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    if (cfg < 0 || cfg >= kNumConfigs) return hipErrorInvalidValue;
    switch (kConfigs[cfg].family) {
        case FAM_GENERIC:
        case FAM_MACRO: return launch_tile_family<DT>(cfg, a, grid, s);
        case FAM_SKINNY:
            return (cfg == 14 || cfg == 15) ? launch_small_family<DT>(cfg, a, grid, s)
                                            : launch_tile_family<DT>(cfg, a, grid, s);
        case FAM_DIRECT: return launch_direct_family<DT>(cfg, a, grid, s);
        case FAM_RING:
            return a.b_trans ? launch_ring_family<DT, true>(cfg, a, grid, s)
                             : launch_ring_family<DT, false>(cfg, a, grid, s);
        case FAM_GEMV: return launch_small_family<DT>(cfg, a, grid, s);
        default: return hipErrorInvalidValue;
    }
}

__global__ __launch_bounds__(256) void zero_u32_kernel(uint32_t *__restrict__ p, int64_t n) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0u;
}

// Split-K workspace, one per (device, stream): the partial planes and the
// per-tile arrival counters.  Kept for the life of the process and grown on
// demand, so a split-K call costs no allocation and no extra launch.  Every
// buffer is allocated, zeroed (counters) and released in stream order on the
// stream that uses it, so work still queued with an old buffer is unaffected
// by its replacement.  Launches on one stream run in order and each launch
// leaves every counter it touched at zero, which is what makes the counters
// reusable; separate streams get separate workspaces.
namespace {
struct Workspace {
    void *partials = nullptr;
    size_t partial_bytes = 0;
    uint32_t *counters = nullptr;
    int64_t counter_cap = 0;
};
std::mutex g_ws_mu;
std::map<std::pair<int, uintptr_t>, Workspace> g_ws;

size_t grow(size_t need, size_t have, size_t quantum) {
    size_t n = need > 2 * have ? need : 2 * have;
    return (n + quantum - 1) / quantum * quantum;
}
}  // namespace

// Test hook: with GEMM_MI355X_TEST_FAIL_WORKSPACE=1 in the environment, every workspace
// allocation the library would make fails as if the device were out of memory (the
// caller then gets GEMM_ERR_NO_MEMORY and nothing is queued).  Read at each allocation,
// so a process can switch it on and off.
static bool fail_workspace_for_test() {
    const char *e = getenv("GEMM_MI355X_TEST_FAIL_WORKSPACE");
    return e != nullptr && e[0] == '1';
}

static int acquire_workspace(hipStream_t stream, size_t partial_bytes, int64_t counter_words, void **partials,
                             uint32_t **counters) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return LAUNCH_HIP_ERROR;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    Workspace &w = g_ws[{dev, reinterpret_cast<uintptr_t>(stream)}];
    if ((w.partial_bytes < partial_bytes || w.counter_cap < counter_words) && fail_workspace_for_test())
        return LAUNCH_NO_MEMORY;
    if (w.partial_bytes < partial_bytes) {
        if (w.partials != nullptr && hipFreeAsync(w.partials, stream) != hipSuccess) return LAUNCH_HIP_ERROR;
        w.partials = nullptr;
        const size_t bytes = grow(partial_bytes, w.partial_bytes, size_t(1) << 20);
        w.partial_bytes = 0;
        if (hipMallocAsync(&w.partials, bytes, stream) != hipSuccess || w.partials == nullptr) {
            (void)hipGetLastError();
            w.partials = nullptr;
            return LAUNCH_NO_MEMORY;
        }
        w.partial_bytes = bytes;
    }
    if (w.counter_cap < counter_words) {
        if (w.counters != nullptr && hipFreeAsync(w.counters, stream) != hipSuccess) return LAUNCH_HIP_ERROR;
        w.counters = nullptr;
        const int64_t cap = int64_t(grow(size_t(counter_words), size_t(w.counter_cap), 4096));
        w.counter_cap = 0;
        void *p = nullptr;
        if (hipMallocAsync(&p, size_t(cap) * 4, stream) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return LAUNCH_NO_MEMORY;
        }
        int64_t blocks = (cap + 255) / 256;
        if (blocks > 1024) blocks = 1024;
        hipLaunchKernelGGL(zero_u32_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream,
                           static_cast<uint32_t *>(p), cap);
        if (hipGetLastError() != hipSuccess) {
            (void)hipFreeAsync(p, stream);
            return LAUNCH_HIP_ERROR;
        }
        w.counters = static_cast<uint32_t *>(p);
        w.counter_cap = cap;
    }
    *partials = w.partials;
    *counters = w.counters;
    return LAUNCH_OK;
}

int release_workspaces() {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return LAUNCH_HIP_ERROR;
    int rc = LAUNCH_OK;
    for (auto &kv : g_ws) {
        Workspace &w = kv.second;
        if (w.partials == nullptr && w.counters == nullptr) continue;
        if (hipSetDevice(kv.first.first) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
            rc = LAUNCH_HIP_ERROR;
            continue;
        }
        if (w.partials != nullptr && hipFree(w.partials) != hipSuccess) rc = LAUNCH_HIP_ERROR;
        if (w.counters != nullptr && hipFree(w.counters) != hipSuccess) rc = LAUNCH_HIP_ERROR;
        w = Workspace{};
    }
    g_ws.clear();
    if (hipSetDevice(cur) != hipSuccess) rc = LAUNCH_HIP_ERROR;
    return rc;
}

// Split-K scratch of the entry point that allocates nothing (gemm_bf16_f32_noalloc):
// a fixed array in device memory, one copy per GPU the library runs on, held until
// the process ends.  Host code never uses the array's name as an address (on the
// host it only stands for the symbol): the device address of each GPU's copy comes
// from hipGetSymbolAddress, taken once per device with that device current, and is
// the only form of it that kernels and fills receive.  Every call on a GPU shares
// that GPU's copy, so calls that overlap in time on one GPU race on it.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
std::map<int, uint8_t *> g_scratch_ptr;   // device -> device address of its copy of `scratch`
}  // namespace

static int static_scratch_address(uint8_t **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return LAUNCH_HIP_ERROR;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it == g_scratch_ptr.end()) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return LAUNCH_HIP_ERROR;
        }
        it = g_scratch_ptr.emplace(dev, static_cast<uint8_t *>(p)).first;
    }
    *out = it->second;
    return LAUNCH_OK;
}

// Zeroes the M x N outputs of an int32 C with row pitch ldc (the atomic split-K
// reduction's starting point); the row padding is not touched.
__global__ __launch_bounds__(256) void zero_c_kernel(uint32_t *__restrict__ c, int64_t M, int64_t N, int64_t ldc) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x, total = M * N;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / N;
        c[r * ldc + (i - r * N)] = 0u;
    }
}

int launch_gemm(const KernelArgs &a, int32_t cfg, int64_t grid, void *stream_ptr, bool static_scratch) {
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    KernelArgs args = a;
    args.workspace = nullptr;
    args.counters = nullptr;
    if (args.split_k > 1 && args.reduce_in_kernel == REDUCE_ATOMIC) {
        if (args.dtype != DT_I8 || args.epilogue != EPI_NONE) return LAUNCH_HIP_ERROR;
        int64_t blocks = (args.M * args.N + 255) / 256;
        if (blocks > 2048) blocks = 2048;
        hipLaunchKernelGGL(zero_c_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, static_cast<uint32_t *>(args.C),
                           args.M, args.N, args.ldc);
        if (hipGetLastError() != hipSuccess) return LAUNCH_HIP_ERROR;
    } else if (args.split_k > 1) {
        const bool flag = args.reduce_in_kernel == REDUCE_ATOMIC_FLAG;
        if (flag && (args.dtype != DT_I8 || args.epilogue != EPI_NONE ||
                     (kConfigs[cfg].family != FAM_RING && kConfigs[cfg].family != FAM_GEMV)))
            return LAUNCH_HIP_ERROR;
        // REDUCE_ATOMIC_FLAG needs the counters only, one 128-byte line per tile.
        const size_t bytes = flag ? 0 : size_t(args.split_k) * size_t(args.M) * size_t(args.N) * 4;
        const int64_t counter_words = args.reduce_in_kernel == REDUCE_LAST_SLICE ? int64_t(args.tiles_m) * args.tiles_n
                              : flag ? int64_t(args.tiles_m) * args.tiles_n * kFlagCounterStride : 0;
        if (static_scratch) {
            if (bytes > size_t(kStaticScratchBytes - kScratchCounterBytes) || counter_words * 4 > kScratchCounterBytes)
                return LAUNCH_SCRATCH_LIMIT;
            uint8_t *base = nullptr;
            const int rc = static_scratch_address(&base);
            if (rc != LAUNCH_OK) return rc;
            args.counters = reinterpret_cast<uint32_t *>(base);
            args.workspace = base + kScratchCounterBytes;
            // The array keeps the previous call's contents: the arrival counters must start
            // at zero (a fill kernel, which a stream capture records like any launch).
            if (counter_words > 0) {
                int64_t blocks = (counter_words + 255) / 256;
                hipLaunchKernelGGL(zero_u32_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, args.counters,
                                   counter_words);
                if (hipGetLastError() != hipSuccess) return LAUNCH_HIP_ERROR;
            }
        } else {
            const int rc = acquire_workspace(stream, bytes, counter_words, &args.workspace, &args.counters);
            if (rc != LAUNCH_OK) return rc;
        }
    }
    hipError_t e = args.dtype == DT_I8 ? launch_config<DT_I8>(cfg, args, grid, stream)
                                       : launch_config<DT_BF16>(cfg, args, grid, stream);
    if (e == hipSuccess && args.split_k > 1 && args.reduce_in_kernel == REDUCE_SEPARATE) {
        const int64_t total = args.M * args.N;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        // unsigned adds: int32 partials wrap modulo 2^32, defined
        e = args.dtype == DT_I8 ? launch_splitk_reduce<DT_I8>(args, blocks, stream)
                                : launch_splitk_reduce<DT_BF16>(args, blocks, stream);
    }
    return e == hipSuccess ? LAUNCH_OK : LAUNCH_HIP_ERROR;
}

}  // namespace gemm
