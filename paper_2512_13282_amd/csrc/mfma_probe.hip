// mfma_probe.hip -- measurement aids: the sustained MFMA rate of this GPU on random
// operands (gemm_probe_mfma), and the time of a plain read (gemm_probe_read).
//
// A measurement aid, not part of the GEMM: one workgroup of 8 waves per CU
// (forced by its LDS request) issues only 32x32 MFMAs of the GEMM's own
// instruction shapes, eight independent accumulators per wave, cycling
// through four operand register sets filled with random data shaped like the
// GEMM inputs (int8: uniform bytes; bf16: approximately N(0,1)).  No memory
// traffic happens inside the timed loop, so the rate it reaches is the MFMA
// ceiling at whatever clock the chip sustains under that load -- on MI355X
// the clock drops well below its 2.4 GHz maximum when the multipliers see
// random data, which is what bounds a GEMM on random inputs.
//
// Every workgroup records its shader-clock cycles (s_memtime) and constant
// 100 MHz-class ticks (s_memrealtime) around the loop, from which the caller
// derives the clock the loop ran at.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gemm_mi355x.h"

namespace {

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kProbeWaves = 8;
constexpr int kProbeLds = 96 * 1024;      // more than half the CU's LDS: one workgroup per CU

// 32-bit integer hash: Chris Wellons' "lowbias32" xor-shift-multiply mixer (constants
// from his hash-prospector search), used only to draw probe operands.
__device__ __forceinline__ unsigned mix32(unsigned x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// bf16 bits of an approximately standard-normal value: the centred sum of four
// uniforms (variance 4/12) scaled to unit variance, truncated to bf16.
__device__ __forceinline__ unsigned normal_bf16(unsigned seed) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) s += float(mix32(seed * 4u + unsigned(i)) >> 8) * (1.0f / 16777216.0f);
    const float v = (s - 2.0f) * 1.7320508f;
    return __float_as_uint(v) >> 16;
}

template <int DT>
__global__ __launch_bounds__(64 * kProbeWaves) void mfma_probe_kernel(int random_operands, int iters,
                                                                      int64_t *clocks, unsigned *sink) {
    extern __shared__ unsigned char probe_lds[];
    const unsigned tid = threadIdx.x;
    if (tid == 0) probe_lds[0] = 1;
    u32x4_t a[4], b[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const unsigned base = ((blockIdx.x * blockDim.x + tid) * 4u + unsigned(s)) * 8u;
        unsigned w[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (!random_operands) w[e] = DT == 0 ? 0x01010101u : 0x3f803f80u;
            else if (DT == 0) w[e] = mix32(base + unsigned(e));
            else w[e] = normal_bf16(2u * (base + unsigned(e))) | (normal_bf16(2u * (base + unsigned(e)) + 1u) << 16);
        }
        a[s] = u32x4_t{w[0], w[1], w[2], w[3]};
        b[s] = u32x4_t{w[4], w[5], w[6], w[7]};
    }
    i32x16_t ai[8];
    f32x16_t af[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        ai[c] = i32x16_t{};
        af[c] = f32x16_t{};
    }
    const int64_t c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                if constexpr (DT == 0)
                    ai[c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(i32x4_t, a[s]),
                                                                  __builtin_bit_cast(i32x4_t, b[(s + c) & 3]),
                                                                  ai[c], 0, 0, 0);
                else
                    af[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a[s]),
                                                                    __builtin_bit_cast(bf16x8_t, b[(s + c) & 3]),
                                                                    af[c], 0, 0, 0);
            }
    }
    const int64_t c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
    unsigned acc = probe_lds[0];
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc += DT == 0 ? unsigned(ai[c][e]) : __float_as_uint(af[c][e]);
    sink[blockIdx.x * blockDim.x + tid] = acc;
    if (tid == 0) {
        clocks[2 * blockIdx.x] = c1 - c0;
        clocks[2 * blockIdx.x + 1] = r1 - r0;
    }
}

// Streams `n16` 16-byte pieces of `src` once (grid-stride, four loads in flight per
// lane), folding them into one value per thread so that nothing is skipped: the time
// a plain read of those bytes takes, the reference for the memory-bound GEMMs.
__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4_t *__restrict__ src, int64_t n16,
                                                         unsigned *sink) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4_t a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        acc ^= a ^ b ^ c ^ d;
    }
    for (; i < n16; i += stride) acc ^= src[i];
    sink[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

constexpr int kReadProbeBlocksPerCu = 8;

}  // namespace

extern "C" int gemm_probe_read(const void *src, int64_t bytes, unsigned *sink, int64_t sink_elems, void *stream) {
    if (bytes < 0 || (bytes > 0 && src == nullptr) || (reinterpret_cast<uintptr_t>(src) & 15) != 0 || (bytes & 15) != 0)
        return GEMM_ERR_INVALID_VALUE;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return GEMM_ERR_HIP;
    const int64_t threads = int64_t(cus) * kReadProbeBlocksPerCu * 256;
    if (sink == nullptr || sink_elems < threads) return GEMM_ERR_INVALID_VALUE;
    hipLaunchKernelGGL(read_probe_kernel, dim3(unsigned(cus * kReadProbeBlocksPerCu)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const u32x4_t *>(src), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? GEMM_OK : GEMM_ERR_HIP;
}

extern "C" int gemm_probe_mfma(int dtype, int random_operands, int32_t iters, int64_t *clocks,
                               unsigned *sink, gemm_probe_info *info, void *stream) {
    if ((dtype != GEMM_DTYPE_I8_I32 && dtype != GEMM_DTYPE_BF16_F32) || iters < 1 || info == nullptr)
        return GEMM_ERR_INVALID_VALUE;
    int dev = 0, cus = 0, wall_khz = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
        return GEMM_ERR_HIP;
    info->workgroups = cus;
    info->threads_per_workgroup = 64 * kProbeWaves;
    info->ops_per_launch = double(cus) * kProbeWaves * double(iters) * 32.0 * (dtype == 0 ? 65536.0 : 32768.0);
    info->wall_clock_hz = double(wall_khz) * 1e3;
    if (clocks == nullptr && sink == nullptr) return GEMM_OK;      // query only
    if (clocks == nullptr || sink == nullptr) return GEMM_ERR_INVALID_VALUE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const void *fn = dtype == 0 ? reinterpret_cast<const void *>(&mfma_probe_kernel<0>)
                                : reinterpret_cast<const void *>(&mfma_probe_kernel<1>);
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kProbeLds) != hipSuccess)
        return GEMM_ERR_HIP;
    if (dtype == 0)
        hipLaunchKernelGGL(mfma_probe_kernel<0>, dim3(unsigned(cus)), dim3(64 * kProbeWaves), kProbeLds, s,
                           random_operands, iters, clocks, sink);
    else
        hipLaunchKernelGGL(mfma_probe_kernel<1>, dim3(unsigned(cus)), dim3(64 * kProbeWaves), kProbeLds, s,
                           random_operands, iters, clocks, sink);
    return hipGetLastError() == hipSuccess ? GEMM_OK : GEMM_ERR_HIP;
}
