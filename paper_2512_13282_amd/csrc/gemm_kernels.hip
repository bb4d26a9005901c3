// gemm_kernels.hip -- gfx950 (CDNA4) MFMA GEMM kernels and their launcher.
//
// One kernel template serves both dtypes and every tile configuration of
// configs.h.  Per workgroup (one output tile BM x BN, one K slice):
//
//   * output-stationary: the accumulators of the whole tile stay in registers
//     for every K stage (paper, Sec. 4.2.1); they start at zero, which replaces
//     the paper's separate zeroing kernel;
//   * K is walked in 128-byte stages (64 bf16 or 128 int8 elements).  Stage
//     k+1 is fetched from global memory into registers while the MFMAs consume
//     stage k from LDS, then written to the other LDS buffer: the double
//     buffering of inputs (Sec. 4.2.1) with one barrier per stage;
//   * LDS holds A as BM rows of 128 K-bytes and B transposed, BN rows of 128
//     K-bytes, so that every MFMA operand fragment is one 16-byte LDS read.
//     This is the on-the-fly layout transformation of Sec. 4.3: matrices stay
//     row-major in memory and are re-tiled on the way into local memory.  B is
//     row-major (K x N), so its K-contiguous fragments are produced by an
//     in-register transpose of 8 x 8 (bf16) or 16 x 8 (int8) element blocks --
//     the mirror image of the paper's in-core shuffle for column-major B
//     (Sec. 4.3);
//   * 16-byte chunks are XOR-swizzled within each 128-byte LDS row so that
//     fragment reads and transposed writes spread over all banks;
//   * workgroup ids are remapped so that each XCD (workgroups are dealt
//     round-robin to the 8 XCDs) runs a compact block of output tiles that
//     shares A row-panels and B column-panels in its L2 -- the GPU analog of
//     broadcasting A tiles along array rows and B tiles along columns
//     (Sec. 4.2.1).
//
// MFMA fragment layout used (32 x 32 output, 64 lanes): lane l supplies row
// (l mod 32) of the A tile and column (l mod 32) of the B tile, each with 16
// bytes of K; lanes 0-31 and 32-63 hold two different 16-byte K halves.  Any
// assignment of K positions is valid as long as A and B use the same one, and
// both are read with the same (chunk, lane) mapping below.  Output register r
// of lane l holds C[8*(r/4) + 4*(l/32) + (r mod 4)][l mod 32].
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "configs.h"
#include "launch.h"

namespace gemm {

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef int i32x16_t __attribute__((ext_vector_type(16)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));

template <int DT> struct Types;
template <> struct Types<DT_I8> {
    using acc_vec = i32x16_t;
    using out_t = int32_t;
    static constexpr int E = 1;
};
template <> struct Types<DT_BF16> {
    using acc_vec = f32x16_t;
    using out_t = float;
    static constexpr int E = 2;
};

template <int DT>
__device__ __forceinline__ typename Types<DT>::acc_vec mfma32(u32x4_t a, u32x4_t b,
                                                             typename Types<DT>::acc_vec c);
template <>
__device__ __forceinline__ i32x16_t mfma32<DT_I8>(u32x4_t a, u32x4_t b, i32x16_t c) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(i32x4_t, a),
                                                 __builtin_bit_cast(i32x4_t, b), c, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x16_t mfma32<DT_BF16>(u32x4_t a, u32x4_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Physical 16-byte chunk of logical chunk `c` in LDS row `row`.  Eight
// consecutive rows (fragment reads) and rows eight apart (transposed B
// writes) both land on eight distinct chunks.
__device__ __forceinline__ int swz(int c, int row) { return c ^ ((row ^ (row >> 3)) & 7); }

// Workgroup id -> (tile_m, tile_n, slice).  Consecutive hardware ids go to
// different XCDs; the remap gives XCD x a contiguous range of logical ids, and
// logical ids walk GROUP_M tile-rows column by column.
__device__ __forceinline__ void map_tile(const KernelArgs &a, int &tm, int &tn, int &slice) {
    const int total = int(gridDim.x);
    const int hw = int(blockIdx.x);
    const int per = total / 8, rem = total % 8;
    const int xcd = hw % 8, local = hw / 8;
    const int id = xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
    const int tiles = a.tiles_m * a.tiles_n;
    slice = id / tiles;
    const int t = id % tiles;
    const int width = a.group_m * a.tiles_n;
    const int group = t / width;
    const int first_m = group * a.group_m;
    const int gsize = (a.tiles_m - first_m) < a.group_m ? (a.tiles_m - first_m) : a.group_m;
    const int in_group = t % width;
    tm = first_m + in_group % gsize;
    tn = in_group / gsize;
}

template <int DT, int BM, int BN, int WM, int WN, bool VEC>
struct TileKernel {
    static constexpr int THREADS = 64 * WM * WN;
    static constexpr int E = Types<DT>::E;
    static constexpr int VECE = 16 / E;          // elements per 16-byte chunk
    static constexpr int BK = kStageKBytes / E;  // elements per stage
    static constexpr int TM = BM / WM / 32;      // 32x32 MFMA tiles per wave along M
    static constexpr int TN = BN / WN / 32;
    static constexpr int A_CHUNKS = BM * 8 / THREADS;
    // Vector B loader: one block = 8 columns x KPB k-rows, transposed into 8
    // column pieces of KPB*E bytes (16 = whole chunk, 8 = half chunk).
    static constexpr bool B_FULL = BN >= THREADS;
    static constexpr int KPB = (B_FULL ? 16 : 8) / E;
    static constexpr int OUTB = KPB * E;
    static constexpr int B_BLOCKS = (BK / KPB) * (BN / 8) / THREADS;
    static constexpr int ROWW = 16 / E == 8 ? 4 : 2;  // dwords per loaded B row piece
    // Element-wise B loader: BN*8 chunks.
    static constexpr int B_CHUNKS = BN * 8 / THREADS;

    static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "wave tile must hold 32x32 MFMAs");
    static_assert(A_CHUNKS >= 1 && A_CHUNKS * THREADS == BM * 8, "A stage must split evenly");
    static_assert(!VEC || (B_BLOCKS >= 1 && B_BLOCKS * THREADS == (BK / KPB) * (BN / 8)),
                  "B stage must split evenly");
    static_assert(VEC || (B_CHUNKS >= 1 && B_CHUNKS * THREADS == BN * 8), "B chunks split evenly");
};

// ---------------------------------------------------------------------------
// In-register transposes of a B block (row-major pieces -> K-contiguous
// column pieces).  bf16: row piece = 8 columns (4 dwords, column c in dword
// c/2, half c%2); int8: row piece = 8 columns (2 dwords, column c in dword
// c/4, byte c%4).
// ---------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ unsigned bf16_col_dword(const u32x4_t (&rows)[N], int base, int c, int j) {
    const unsigned lo = rows[base + 2 * j][c >> 1], hi = rows[base + 2 * j + 1][c >> 1];
    return (c & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
}

template <int N>
__device__ __forceinline__ unsigned i8_col_dword(const u32x2_t (&rows)[N], int base, int c, int j) {
    const int sh = 8 * (c & 3);
    const unsigned b0 = (rows[base + 4 * j + 0][c >> 2] >> sh) & 0xFFu;
    const unsigned b1 = (rows[base + 4 * j + 1][c >> 2] >> sh) & 0xFFu;
    const unsigned b2 = (rows[base + 4 * j + 2][c >> 2] >> sh) & 0xFFu;
    const unsigned b3 = (rows[base + 4 * j + 3][c >> 2] >> sh) & 0xFFu;
    return b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
}

template <int DT, int BM, int BN, int WM, int WN, bool VEC, int WAVES_PER_EU>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_tile_kernel(KernelArgs args) {
    using T = TileKernel<DT, BM, BN, WM, WN, VEC>;
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int E = T::E, BK = T::BK, VECE = T::VECE;
    constexpr int TM = T::TM, TN = T::TN;

    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (BM + BN) * kStageKBytes];
    uint8_t *const a_lds = smem;                               // [2][BM][128]
    uint8_t *const b_lds = smem + 2 * BM * kStageKBytes;       // [2][BN][128]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wave_m = wave / WN, wave_n = wave % WN;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int64_t nk = k_end > k_begin ? (k_end - k_begin + BK - 1) / BK : 0;

    const uint8_t *const A = static_cast<const uint8_t *>(args.A);
    const uint8_t *const B = static_cast<const uint8_t *>(args.B);
    const int64_t lda = args.lda, ldb = args.ldb;

    // ---------------- staging registers ----------------
    u32x4_t ra[T::A_CHUNKS];
    constexpr int RB_N = VEC ? T::B_BLOCKS * T::KPB : 1;
    constexpr int RB_CH = VEC ? 1 : T::B_CHUNKS;
    u32x4_t rb4[DT == DT_BF16 ? RB_N : 1];
    u32x2_t rb2[DT == DT_I8 ? RB_N : 1];
    u32x4_t rbc[RB_CH];
    (void)rb4; (void)rb2; (void)rbc;

    auto load_stage = [&](int64_t kt) {
        const int64_t k0 = k_begin + kt * BK;
#pragma unroll
        for (int i = 0; i < T::A_CHUNKS; ++i) {
            const int q = i * T::THREADS + tid;
            const int row = q >> 3, c = q & 7;
            const int64_t gm = m0 + row, gk = k0 + int64_t(c) * VECE;
            if (VEC) {
                u32x4_t v = {0u, 0u, 0u, 0u};
                if (gm < M && gk < k_end)
                    v = *reinterpret_cast<const u32x4_t *>(A + (gm * lda + gk) * E);
                ra[i] = v;
            } else {
                unsigned w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int e = 0; e < VECE; ++e) {
                    unsigned x = 0;
                    if (gm < M && gk + e < k_end) {
                        if (E == 1) x = A[gm * lda + gk + e];
                        else x = reinterpret_cast<const uint16_t *>(A)[gm * lda + gk + e];
                    }
                    w[(e * E) >> 2] |= x << (8 * ((e * E) & 3));
                }
                ra[i] = u32x4_t{w[0], w[1], w[2], w[3]};
            }
        }
        if (VEC) {
#pragma unroll
            for (int bI = 0; bI < T::B_BLOCKS; ++bI) {
                const int b = bI * T::THREADS + tid;
                const int nb = b % (BN / 8), kb = b / (BN / 8);
                const int64_t gn = n0 + int64_t(nb) * 8;
#pragma unroll
                for (int r = 0; r < T::KPB; ++r) {
                    const int64_t gk = k0 + int64_t(kb) * T::KPB + r;
                    const bool ok = gk < k_end && gn < N;
                    if (DT == DT_BF16) {
                        u32x4_t v = {0u, 0u, 0u, 0u};
                        if (ok) v = *reinterpret_cast<const u32x4_t *>(B + (gk * ldb + gn) * 2);
                        rb4[bI * T::KPB + r] = v;
                    } else {
                        u32x2_t v = {0u, 0u};
                        if (ok) v = *reinterpret_cast<const u32x2_t *>(B + gk * ldb + gn);
                        rb2[bI * T::KPB + r] = v;
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < T::B_CHUNKS; ++i) {
                const int q = i * T::THREADS + tid;
                const int n = q % BN, c = q / BN;
                const int64_t gn = n0 + n, gk = k0 + int64_t(c) * VECE;
                unsigned w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int e = 0; e < VECE; ++e) {
                    unsigned x = 0;
                    if (gn < N && gk + e < k_end) {
                        if (E == 1) x = B[(gk + e) * ldb + gn];
                        else x = reinterpret_cast<const uint16_t *>(B)[(gk + e) * ldb + gn];
                    }
                    w[(e * E) >> 2] |= x << (8 * ((e * E) & 3));
                }
                rbc[i] = u32x4_t{w[0], w[1], w[2], w[3]};
            }
        }
    };

    auto store_stage = [&](int buf) {
        uint8_t *const as = a_lds + buf * BM * kStageKBytes;
        uint8_t *const bs = b_lds + buf * BN * kStageKBytes;
#pragma unroll
        for (int i = 0; i < T::A_CHUNKS; ++i) {
            const int q = i * T::THREADS + tid;
            const int row = q >> 3, c = q & 7;
            *reinterpret_cast<u32x4_t *>(as + row * kStageKBytes + swz(c, row) * 16) = ra[i];
        }
        if (VEC) {
#pragma unroll
            for (int bI = 0; bI < T::B_BLOCKS; ++bI) {
                const int b = bI * T::THREADS + tid;
                const int nb = b % (BN / 8), kb = b / (BN / 8);
                const int byte = kb * T::OUTB;
                const int chunk = byte >> 4, half = (byte >> 3) & 1;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const int n = nb * 8 + c;
                    uint8_t *dst = bs + n * kStageKBytes + swz(chunk, n) * 16 + half * 8;
                    const int base = bI * T::KPB;
                    if (DT == DT_BF16) {
                        if (T::OUTB == 16) {
                            *reinterpret_cast<u32x4_t *>(dst) =
                                u32x4_t{bf16_col_dword(rb4, base, c, 0), bf16_col_dword(rb4, base, c, 1),
                                        bf16_col_dword(rb4, base, c, 2), bf16_col_dword(rb4, base, c, 3)};
                        } else {
                            *reinterpret_cast<u32x2_t *>(dst) =
                                u32x2_t{bf16_col_dword(rb4, base, c, 0), bf16_col_dword(rb4, base, c, 1)};
                        }
                    } else {
                        if (T::OUTB == 16) {
                            *reinterpret_cast<u32x4_t *>(dst) =
                                u32x4_t{i8_col_dword(rb2, base, c, 0), i8_col_dword(rb2, base, c, 1),
                                        i8_col_dword(rb2, base, c, 2), i8_col_dword(rb2, base, c, 3)};
                        } else {
                            *reinterpret_cast<u32x2_t *>(dst) =
                                u32x2_t{i8_col_dword(rb2, base, c, 0), i8_col_dword(rb2, base, c, 1)};
                        }
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < T::B_CHUNKS; ++i) {
                const int q = i * T::THREADS + tid;
                const int n = q % BN, c = q / BN;
                *reinterpret_cast<u32x4_t *>(bs + n * kStageKBytes + swz(c, n) * 16) = rbc[i];
            }
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);

    if (nk > 0) {
        load_stage(0);
        store_stage(0);
        __syncthreads();
    }
    for (int64_t kt = 0; kt < nk; ++kt) {
        const int buf = int(kt & 1);
        if (kt + 1 < nk) load_stage(kt + 1);
        const uint8_t *const as = a_lds + buf * BM * kStageKBytes;
        const uint8_t *const bs = b_lds + buf * BN * kStageKBytes;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int chunk = 2 * s + frag_half;
            u32x4_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wrow0 + i * 32 + frag_row;
                af[i] = *reinterpret_cast<const u32x4_t *>(as + row * kStageKBytes + swz(chunk, row) * 16);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = wcol0 + j * 32 + frag_row;
                bfr[j] = *reinterpret_cast<const u32x4_t *>(bs + col * kStageKBytes + swz(chunk, col) * 16);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(af[i], bfr[j], acc[i][j]);
        }
        if (kt + 1 < nk) store_stage(buf ^ 1);
        __syncthreads();
    }

    // ---------------- epilogue ----------------
    out_t *out;
    int64_t ldo;
    if (args.split_k > 1) {
        out = static_cast<out_t *>(args.workspace) + int64_t(slice) * M * N;
        ldo = N;
    } else {
        out = static_cast<out_t *>(args.C);
        ldo = args.ldc;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t col = n0 + wcol0 + j * 32 + frag_row;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wrow0 + i * 32 + 8 * (r >> 2) + 4 * frag_half + (r & 3);
                if (row < M && col < N) out[row * ldo + col] = acc[i][j][r];
            }
        }
    }
}

// Sums split-K partials [split][M][N] into C in slice order 0, 1, ... (a fixed
// order, so fp32 results are reproducible run to run).
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const T *__restrict__ ws, int32_t split,
                                                            int64_t M, int64_t N,
                                                            T *__restrict__ C, int64_t ldc) {
    const int64_t total = M * N;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        T s = ws[idx];
        for (int32_t p = 1; p < split; ++p) s += ws[int64_t(p) * total + idx];
        const int64_t row = idx / N, col = idx % N;
        C[row * ldc + col] = s;
    }
}

// ---------------------------------------------------------------------------
// Launch: config index -> template instance.
// ---------------------------------------------------------------------------
template <int DT, int BM, int BN, int WM, int WN, bool VEC, int WPE>
static hipError_t launch_tile(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    hipLaunchKernelGGL((gemm_tile_kernel<DT, BM, BN, WM, WN, VEC, WPE>), dim3(unsigned(grid)),
                       dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_config(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
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

int launch_gemm(const KernelArgs &a, int32_t cfg, int64_t grid, void *stream_ptr) {
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    KernelArgs args = a;
    void *ws = nullptr;
    if (args.split_k > 1) {
        const size_t bytes = size_t(args.split_k) * size_t(args.M) * size_t(args.N) * 4;
        if (hipMallocAsync(&ws, bytes, stream) != hipSuccess || ws == nullptr) {
            (void)hipGetLastError();
            return LAUNCH_NO_MEMORY;
        }
        args.workspace = ws;
    }
    hipError_t e = args.dtype == DT_I8 ? launch_config<DT_I8>(cfg, args, grid, stream)
                                       : launch_config<DT_BF16>(cfg, args, grid, stream);
    if (e == hipSuccess && args.split_k > 1) {
        const int64_t total = args.M * args.N;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        if (args.dtype == DT_I8)   // unsigned adds: int32 partials wrap modulo 2^32, defined
            hipLaunchKernelGGL(splitk_reduce_kernel<uint32_t>, dim3(unsigned(blocks)), dim3(256), 0, stream,
                               static_cast<const uint32_t *>(ws), args.split_k, args.M, args.N,
                               static_cast<uint32_t *>(args.C), args.ldc);
        else
            hipLaunchKernelGGL(splitk_reduce_kernel<float>, dim3(unsigned(blocks)), dim3(256), 0, stream,
                               static_cast<const float *>(ws), args.split_k, args.M, args.N,
                               static_cast<float *>(args.C), args.ldc);
        e = hipGetLastError();
    }
    if (ws) {
        if (hipFreeAsync(ws, stream) != hipSuccess && e == hipSuccess) e = hipErrorUnknown;
    }
    return e == hipSuccess ? LAUNCH_OK : LAUNCH_HIP_ERROR;
}

}  // namespace gemm
