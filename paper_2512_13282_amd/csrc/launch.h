// launch.h -- interface between the host API (gemm_api.cpp) and the kernels.
// Pure C++: no HIP types, so the API file builds without HIP headers.
#pragma once

#include <stdint.h>

namespace gemm {

struct KernelArgs {
    int32_t dtype;                 // DT_I8 or DT_BF16
    const void *A;
    const void *B;
    void *C;
    void *workspace;               // split-K partials [split][M][N], set by launch_gemm
    uint32_t *counters;            // split-K arrival counter per output tile (zero between launches)
    int64_t M, N, K;
    int64_t lda, ldb, ldc;         // row strides in elements
    int64_t k_chunk;               // K elements per slice
    int32_t split_k;
    int32_t tiles_m, tiles_n;      // output tiles along M and N
    int32_t group_m;               // tile-rows per group in the launch order
    int32_t reduce_in_kernel;      // split-K reduction, REDUCE_* below
    int32_t b_trans;               // 1: B is stored column-major (N x K, row stride ldb >= K)
    int32_t epilogue;              // output conversion, EPI_* below
    int32_t shift;                 // EPI_I8 / EPI_I16: results are divided by 2^shift
};

// Output conversions.  EPI_NONE writes the accumulator type (int32 / fp32).
// EPI_I8 / EPI_I16: int32 result / 2^shift rounded to the nearest integer, ties
// to even, saturated to the int8 / int16 range.  EPI_BF16: fp32 result rounded
// to the nearest bf16, ties to even.
enum { EPI_NONE = 0, EPI_I8 = 1, EPI_I16 = 2, EPI_BF16 = 3 };

// Split-K reductions.  REDUCE_SEPARATE: every slice writes its partial plane and a
// second kernel sums the planes.  REDUCE_LAST_SLICE: the slice of each tile that
// finishes last sums the tile's partials.  REDUCE_ATOMIC (int8 with int32 output
// only): C is zeroed first and every slice adds its partial tile into C with device
// atomics; int32 addition modulo 2^32 is exact and order-free, so the result is the
// same bits as the other two give, and no workspace is needed.  REDUCE_ATOMIC_FLAG
// (the same outputs; RING and GEMV kernels): as REDUCE_ATOMIC, but slice 0 of each
// tile zeroes the tile inside the GEMM and hands the other slices a credit on the
// tile's counter, so no fill kernel runs ahead of the GEMM (counters only, no
// partial planes).
enum { REDUCE_SEPARATE = 0, REDUCE_LAST_SLICE = 1, REDUCE_ATOMIC = 2, REDUCE_ATOMIC_FLAG = 3 };

// REDUCE_ATOMIC_FLAG keeps each tile's counter in a 128-byte line of its own (tile t
// at word t * kFlagCounterStride): every slice of a tile polls and returns credits on
// it, and counters of neighbouring tiles sharing a line queued those same-line
// atomics behind each other (a GEMV with 32 slices per tile ran 1.9x slower).
constexpr int kFlagCounterStride = 32;

enum { LAUNCH_OK = 0, LAUNCH_HIP_ERROR = 1, LAUNCH_NO_MEMORY = 2, LAUNCH_SCRATCH_LIMIT = 3 };

// The fixed split-K scratch of the entry point that allocates nothing: per device,
// kScratchCounterBytes of per-tile arrival counters followed by the partial planes.
constexpr int64_t kStaticScratchBytes = int64_t(16) << 20;
constexpr int64_t kScratchCounterBytes = int64_t(64) << 10;

// Queues the plan's kernels on `stream` (a hipStream_t).  Never synchronizes.  With
// static_scratch a split-K plan takes its partials and counters from the library's
// fixed per-device scratch instead of the per-stream workspace (no allocation), or
// returns LAUNCH_SCRATCH_LIMIT, before queueing anything, when they do not fit.
int launch_gemm(const KernelArgs &a, int32_t config, int64_t grid, void *stream, bool static_scratch = false);

// Frees every cached split-K workspace (all devices and streams) after
// synchronising each device that holds one.
int release_workspaces();

}  // namespace gemm
