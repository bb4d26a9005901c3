// gemm_common.h -- device helpers shared by every GEMM kernel family.
//
// Kernel templates serve both dtypes and every tile configuration of configs.h.
// Common to the tile kernels (one output tile BM x BN and one K slice per
// workgroup):
//
//   * output-stationary: the accumulators of the whole tile stay in registers
//     for the whole K slice (paper, Sec. 4.2.1); they start at zero, which
//     replaces the paper's separate zeroing kernel;
//   * K is walked in stages of 128 K-bytes (64 bf16 or 128 int8 elements), or
//     in 64-byte slots for the ring kernels, with the next stage's operands in
//     flight while the MFMAs consume the current one: the double buffering of
//     inputs (Sec. 4.2.1), generalised to deeper rings;
//   * LDS holds A as BM rows of K-bytes and B either as BN rows of K-bytes
//     (column-major B, and the register-staged kernels, which transpose B in
//     registers) or as K rows of BN elements read back with the LDS transpose
//     reads, so every MFMA operand fragment is one 16-byte or two 8-byte LDS
//     reads.  Matrices stay in their standard order in memory and are re-tiled
//     on the way into local memory, as in Sec. 4.3;
//   * 16-byte chunks are XOR-swizzled within LDS rows so that fragment reads
//     and writes spread over all banks;
//   * workgroup ids are remapped so that each XCD (workgroups are dealt
//     round-robin to the 8 XCDs) runs a compact block of output tiles that
//     shares A row-panels and B column-panels in its L2 -- the GPU analog of
//     broadcasting A tiles along array rows and B tiles along columns
//     (Sec. 4.2.1).
//
// Families: gemm_lds_kernel (DIRECT: global -> LDS buffer loads into two
// stages), gemm_ring_kernel (RING: the same loads into a ring of 64-byte
// slots), gemm_vec_kernel / gemm_tile_kernel (MACRO / GENERIC: loads through
// registers), gemm_stream_kernel (narrow-M streaming), gemv_kernel and
// gemv_bt_kernel (M = 1 on the vector ALUs), plus the split-K reduction.
//
// MFMA fragment layout used (32 x 32 output, 64 lanes): lane l supplies row
// (l mod 32) of the A tile and column (l mod 32) of the B tile, each with 16
// bytes of K; lanes 0-31 and 32-63 hold two different 16-byte K halves.  Any
// assignment of K positions is valid as long as A and B use the same one, and
// both are read with the same (chunk, lane) mapping below.  Output register r
// of lane l holds C[8*(r/4) + 4*(l/32) + (r mod 4)][l mod 32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

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

// Epilogue shared by every kernel: writes the accumulators of one wave (TM x
// TN 32x32 MFMA tiles whose top-left output element is (r0, c0)) of the
// BM x BN output tile (tm, tn) to C.
//
// With split-K each K slice stores its partial tile in the workspace
// ([split][M][N]).  Then either a separate kernel sums the planes
// (REDUCE_SEPARATE, splitk_reduce_kernel), or (REDUCE_LAST_SLICE) every slice
// takes a ticket from the tile's arrival counter and the workgroup that arrives
// last sums the slices of the tile and writes C, then resets the counter to zero
// for the next launch on the stream.  Both sum in the fixed slice order
// 0, 1, ..., so fp32 results are identical run to run whichever slice finishes
// last and whichever reduction runs.  int8 with int32 output may instead add
// every slice's partial tile straight into C with device atomics, C zeroed by a
// fill kernel beforehand (REDUCE_ATOMIC) or by each tile's first slice inside the
// GEMM (REDUCE_ATOMIC_FLAG, below): integer addition is exact and order-free, so
// the bits are the same, with no partial planes and no second pass over them.
//
// The slices of a tile run on different XCDs, whose L2 caches are not kept
// coherent with each other for ordinary accesses.  Instead of device-scope
// fences (which write back and invalidate the whole L2 of the XCD), the
// partials are stored and loaded with device-scope (sc1) accesses, which go
// to the device coherence point: each thread waits until its partial stores
// are complete, the workgroup synchronises, and only then takes its ticket
// (an atomic, itself coherent device-wide); the partial loads of the last
// workgroup depend on the ticket and are issued after it.  The HIP memory model
// would ask for a release/acquire ticket to order these relaxed accesses; on
// gfx950 that adds an L2 write-back and invalidate around every ticket (measured
// 7-22 % slower on the skinny shapes that reduce in-kernel), while the hardware
// order above (completed sc1 stores, barrier, atomic, then in-order loads that
// read the coherence point) already delivers every partial to the last slice.
template <typename T>
__device__ __forceinline__ void store_coherent(T *p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T load_coherent(const T *p) {
    return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// REDUCE_ATOMIC_FLAG.  Slice 0 of a tile zeroes the tile's part of C with
// device-coherent stores before it loads anything, waits until every thread's zeros
// are complete, and then adds split_k - 1 credits to the tile's counter.  Every other
// slice reads the counter some K steps before its end (early, so that the read's
// latency hides under the last steps), polls only if no credit had arrived by then,
// gives one credit back and then adds its partial tile into C.  So a slice adds only
// after the zeros of its tile are complete at the coherence point, where the atomics
// are performed, and the counter is zero again when the launch ends.  A waiting
// slice depends only on slice 0 of its tile, which waits for nothing; on every XCD
// the slice-0 workgroups have the lowest numbers (map_tile) and start first.  The
// polling is bounded all the same (about a second), so a slice 0 that never runs
// cannot hang the kernel; its tile's result is then wrong, and a credit it hands
// out later stays on the counter for a later call on the stream to take too early
// (a GPU on which slice-0 workgroups cannot start for that long is out of scope).
constexpr unsigned kCreditPollLimit = 1u << 20;

__device__ __forceinline__ uint32_t *flag_counter(const KernelArgs &args, int tile) {
    return args.counters + int64_t(tile) * kFlagCounterStride;
}

// Slice 0's part, by all NT threads of the workgroup: the BM x BN tile at (m0, n0),
// clipped to M x N.  `tile` numbers the tile (its counter: flag_counter).
template <int BM, int BN, int NT>
__device__ __forceinline__ void flag_zero_tile(const KernelArgs &args, int64_t m0, int64_t n0, int tile) {
    uint32_t *const cc = static_cast<uint32_t *>(args.C);
    const int rows = int((args.M - m0) < BM ? (args.M - m0) : BM);
    const int cols = int((args.N - n0) < BN ? (args.N - n0) : BN);
    for (int e = int(threadIdx.x); e < rows * BN; e += NT) {
        const int r = e / BN, c = e % BN;
        if (c < cols) store_coherent(&cc[(m0 + r) * args.ldc + n0 + c], 0u);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's zeros are complete
    __syncthreads();                                   // ... and every thread's
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(flag_counter(args, tile), uint32_t(args.split_k - 1), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
}

// Another slice's part, by every thread before its atomics; `seen` is the counter as
// thread 0 read it earlier (0 if it did not).
__device__ __forceinline__ void flag_take_credit(const KernelArgs &args, int tile, uint32_t seen) {
    if (threadIdx.x == 0) {
        uint32_t v = seen;
        for (unsigned i = 0; v == 0u && i < kCreditPollLimit; ++i) {
            __builtin_amdgcn_s_sleep(8);
            v = load_coherent(flag_counter(args, tile));
        }
        if (v != 0u) __hip_atomic_fetch_sub(flag_counter(args, tile), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
}

// Output element idx (row * ldc + col, in output elements) of C from a result v of
// the accumulator type, converted as the call's epilogue asks (launch.h).  int32
// partial sums arrive as uint32 (they wrap modulo 2^32) and are read back as int32.
__device__ __forceinline__ int32_t requant_nearest_even(int32_t v, int shift, int32_t lo, int32_t hi) {
    const int64_t x = v;
    int64_t q = x >> shift;                              // floor(x / 2^shift)
    if (shift > 0) {
        const int64_t r = x - (q << shift), half = int64_t(1) << (shift - 1);
        if (r > half || (r == half && (q & 1))) ++q;
    }
    return int32_t(q < lo ? lo : (q > hi ? hi : q));
}

// fp32 -> bf16, round to nearest with ties to even.  A NaN keeps its upper half with
// the quiet bit set (adding the rounding bias to a NaN could carry it into an
// infinity, a zero or the sign); an infinity and a finite value past the largest
// bf16 both land on the infinity.
__device__ __forceinline__ uint16_t bf16_nearest_even(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return uint16_t((u >> 16) | 0x40u);
    return uint16_t((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Element type of C under epilogue EPI.
template <int DT, int EPI> struct OutElem { using type = typename Types<DT>::out_t; };
template <> struct OutElem<DT_I8, EPI_I8> { using type = int8_t; };
template <> struct OutElem<DT_I8, EPI_I16> { using type = int16_t; };
template <> struct OutElem<DT_BF16, EPI_BF16> { using type = uint16_t; };

template <int DT, int EPI>
__device__ __forceinline__ typename OutElem<DT, EPI>::type convert_out(const KernelArgs &a,
                                                                         typename Types<DT>::out_t v) {
    if constexpr (DT == DT_I8 && EPI == EPI_I8) return int8_t(requant_nearest_even(int32_t(v), a.shift, -128, 127));
    else if constexpr (DT == DT_I8 && EPI == EPI_I16)
        return int16_t(requant_nearest_even(int32_t(v), a.shift, -32768, 32767));
    else if constexpr (DT == DT_BF16 && EPI == EPI_BF16) return bf16_nearest_even(float(v));
    else return v;
}

template <int DT, int EPI, typename V>
__device__ __forceinline__ void write_c_as(const KernelArgs &a, int64_t idx, V v) {
    __builtin_nontemporal_store(convert_out<DT, EPI>(a, typename Types<DT>::out_t(v)),
                                &static_cast<typename OutElem<DT, EPI>::type *>(a.C)[idx]);
}

template <int DT, typename V>
__device__ __forceinline__ void write_c(const KernelArgs &a, int64_t idx, V v) {
    if constexpr (DT == DT_I8) {
        if (a.epilogue == EPI_I8) write_c_as<DT, EPI_I8>(a, idx, v);
        else if (a.epilogue == EPI_I16) write_c_as<DT, EPI_I16>(a, idx, v);
        else write_c_as<DT, EPI_NONE>(a, idx, v);
    } else {
        if (a.epilogue == EPI_BF16) write_c_as<DT, EPI_BF16>(a, idx, v);
        else write_c_as<DT, EPI_NONE>(a, idx, v);
    }
}

// 4 x 4 transpose inside each group of four lanes: on entry lane q (= lane % 4)
// holds x[k] = X[k][q], on exit x[k] = X[q][k].  Two butterfly stages, the first
// exchanging 2 x 2 blocks with lane q ^ 2, the second single values with lane q ^ 1;
// each stage sends two values through one DPP quad permutation apiece.  Every lane
// of the wave must be active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_quad(uint32_t v) {
    return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ void quad_transpose(uint32_t (&x)[4], int lane) {
    constexpr int XOR2 = 2 | (3 << 2) | (0 << 4) | (1 << 6);   // lane q reads lane q ^ 2
    constexpr int XOR1 = 1 | (0 << 2) | (3 << 4) | (2 << 6);   // lane q reads lane q ^ 1
    const bool hi = (lane & 2) != 0, odd = (lane & 1) != 0;
    const uint32_t r0 = dpp_quad<XOR2>(hi ? x[0] : x[2]), r1 = dpp_quad<XOR2>(hi ? x[1] : x[3]);
    const uint32_t z0 = hi ? r0 : x[0], z1 = hi ? r1 : x[1], z2 = hi ? x[2] : r0, z3 = hi ? x[3] : r1;
    const uint32_t u0 = dpp_quad<XOR1>(odd ? z0 : z1), u1 = dpp_quad<XOR1>(odd ? z2 : z3);
    x[0] = odd ? u0 : z0;
    x[1] = odd ? z1 : u0;
    x[2] = odd ? u1 : z2;
    x[3] = odd ? z3 : u1;
}

// Four consecutive outputs of one row as one non-temporal store (16, 8 or 4 bytes).
template <typename O>
__device__ __forceinline__ void store4_nt(O *dst, const O (&c)[4]) {
    if constexpr (sizeof(O) == 4) {
        const u32x4_t v{__builtin_bit_cast(uint32_t, c[0]), __builtin_bit_cast(uint32_t, c[1]),
                        __builtin_bit_cast(uint32_t, c[2]), __builtin_bit_cast(uint32_t, c[3])};
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(dst));
    } else if constexpr (sizeof(O) == 2) {
        const u32x2_t v{uint32_t(__builtin_bit_cast(uint16_t, c[0])) | (uint32_t(__builtin_bit_cast(uint16_t, c[1])) << 16),
                        uint32_t(__builtin_bit_cast(uint16_t, c[2])) | (uint32_t(__builtin_bit_cast(uint16_t, c[3])) << 16)};
        __builtin_nontemporal_store(v, reinterpret_cast<u32x2_t *>(dst));
    } else {
        const uint32_t v = uint32_t(uint8_t(c[0])) | (uint32_t(uint8_t(c[1])) << 8) |
                           (uint32_t(uint8_t(c[2])) << 16) | (uint32_t(uint8_t(c[3])) << 24);
        __builtin_nontemporal_store(v, reinterpret_cast<uint32_t *>(dst));
    }
}

// A wave's output fragments straight into C with the epilogue EPI, four
// consecutive outputs of a row per store.  Lane l holds,
// for fragment (i, j) and register r, row r0 + 4 (l / 32) + 32 i + 8 (r / 4) + r % 4
// and column c0 + l % 32 + 32 j.  Each group of four registers (four consecutive
// rows of one column) is transposed across the four lanes of a quad
// (quad_transpose), after which lane l holds four consecutive columns,
// c0 + 32 j + 4 ((l % 32) / 4) .. + 3, of row r0 + 4 (l / 32) + l % 4 + 32 i + 8 g,
// and writes them with one store: a quarter of the store instructions of one
// element per lane, which is what bounds the epilogue (each wave retires about one
// store instruction per 80 clocks, whatever its width).  Where the four columns run
// past N, or C's pitch or address does not allow the wide store, the four values go
// out one by one.  Row offsets are constants times ldc, which the scalar unit forms.
// The epilogue is a template argument so that the loop bodies stay small enough to
// unroll fully: the accumulators are then only indexed by constants and stay in
// registers (with a run-time choice per element, the 256-register tiles of the
// 4-wave 256 x 256 int8 kernels went to scratch).  The stores are non-temporal: C
// is written once and not read back by the kernel, and streaming it past the caches
// keeps the A and B panels that other workgroups are still reading resident in L2
// and in the last-level cache (measured at 8192^3: 6 % faster for int8, 3 % for
// bf16).
template <int DT, int EPI, int TM, int TN>
__device__ __forceinline__ void store_c_wide(const KernelArgs &args,
                                               const typename Types<DT>::acc_vec (&acc)[TM][TN],
                                               int64_t r0, int64_t c0, int lane) {
    using o_t = typename OutElem<DT, EPI>::type;
    using out_t = typename Types<DT>::out_t;
    const int64_t row0 = r0 + 4 * (lane >> 5) + (lane & 3);
    const int64_t col = c0 + (lane & 28);
    const int64_t rows_left = args.M - row0;
    const int64_t ldc = args.ldc;
    const bool wide = (ldc % 4) == 0 && (reinterpret_cast<uintptr_t>(args.C) % (4 * sizeof(o_t))) == 0;
    o_t *const base = static_cast<o_t *>(args.C) + row0 * ldc + col;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int64_t cols_left = args.N - (col + 32 * j);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                uint32_t x[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // Copied out before the cast: clang's bit cast of a vector-element
                    // expression reads the vector's first element, whatever the index.
                    const auto e = acc[i][j][4 * g + k];
                    x[k] = __builtin_bit_cast(uint32_t, e);
                }
                quad_transpose(x, lane);
                o_t c[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) c[k] = convert_out<DT, EPI>(args, __builtin_bit_cast(out_t, x[k]));
                const int dr = 32 * i + 8 * g;
                if (dr < rows_left && cols_left > 0) {
                    o_t *const dst = base + dr * ldc + 32 * j;
                    if (wide && cols_left >= 4) {
                        store4_nt(dst, c);
                    } else {
#pragma unroll
                        for (int k = 0; k < 4; ++k)
                            if (k < cols_left) __builtin_nontemporal_store(c[k], dst + k);
                    }
                }
            }
            // One fragment at a time: keeps the scheduler from reading every accumulator
            // out ahead of its stores.
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// The same, one output per store: lane l writes its registers as they are (column
// c0 + l % 32 + 32 j, two rows per store instruction).  Kept for the 4-wave
// 256 x 256 tiles, whose waves each hold a 128 x 128 block (256 accumulator
// registers): the transposes' extra live values would push them into scratch.
template <int DT, int EPI, int TM, int TN>
__device__ __forceinline__ void store_c_elementwise(const KernelArgs &args,
                                                    const typename Types<DT>::acc_vec (&acc)[TM][TN],
                                                    int64_t r0, int64_t c0, int lane) {
    using o_t = typename OutElem<DT, EPI>::type;
    const int64_t row0 = r0 + 4 * (lane >> 5);
    const int64_t col = c0 + (lane & 31);
    const int64_t rows_left = args.M - row0;
    const int64_t ldc = args.ldc;
    o_t *const base = static_cast<o_t *>(args.C) + row0 * ldc + col;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        if (col + 32 * j >= args.N) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int dr = 32 * i + 8 * (r >> 2) + (r & 3);
                if (dr < rows_left)
                    __builtin_nontemporal_store(convert_out<DT, EPI>(args, acc[i][j][r]), &base[dr * ldc + 32 * j]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// Which form a tile uses, as measured (same-process A/B against element-wise
// stores): four-wave tiles of at most 64 x 64 per wave write a quarter of the
// store instructions and gain (128 x 128 at 2048^3: 3.5 %); tiles of eight waves
// lose 1-7 %, their epilogue being bound by the chip's aggregate write rate rather
// than by store instructions, so the transposes only add VALU work.
template <int DT, int EPI, int WAVES, int TM, int TN>
__device__ __forceinline__ void store_c_direct(const KernelArgs &args,
                                               const typename Types<DT>::acc_vec (&acc)[TM][TN],
                                               int64_t r0, int64_t c0, int lane) {
    if constexpr (WAVES <= 4 && TM * TN <= 4) store_c_wide<DT, EPI, TM, TN>(args, acc, r0, c0, lane);
    else store_c_elementwise<DT, EPI, TM, TN>(args, acc, r0, c0, lane);
}

// s_last: one int of LDS for the in-kernel split-K reduction's "last slice"
// broadcast; a kernel whose LDS is otherwise free at this point may lend it a word
// of its operand buffers (all of its global -> LDS loads complete, all of its
// fragment reads done).
template <int DT, int BM, int BN, int TM, int TN>
__device__ __forceinline__ void store_tile(const KernelArgs &args,
                                           const typename Types<DT>::acc_vec (&acc)[TM][TN],
                                           int tm, int tn, int slice, int64_t r0, int64_t c0, int lane,
                                           int &s_last, uint32_t seen = 0u) {
    using out_t = typename Types<DT>::out_t;
    using sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;  // int32 wraps mod 2^32
    constexpr int WAVES = (BM / (32 * TM)) * (BN / (32 * TN));
    const int frag_row = lane & 31, frag_half = lane >> 5;
    const int64_t M = args.M, N = args.N;
    const int64_t plane = M * N;
    if (args.split_k == 1) {
        // C itself, through the call's output conversion.
        if constexpr (DT == DT_I8) {
            if (args.epilogue == EPI_I8) store_c_direct<DT, EPI_I8, WAVES>(args, acc, r0, c0, lane);
            else if (args.epilogue == EPI_I16) store_c_direct<DT, EPI_I16, WAVES>(args, acc, r0, c0, lane);
            else store_c_direct<DT, EPI_NONE, WAVES>(args, acc, r0, c0, lane);
        } else {
            if (args.epilogue == EPI_BF16) store_c_direct<DT, EPI_BF16, WAVES>(args, acc, r0, c0, lane);
            else store_c_direct<DT, EPI_NONE, WAVES>(args, acc, r0, c0, lane);
        }
        return;
    }
    if constexpr (DT == DT_I8) {
        if (args.reduce_in_kernel == REDUCE_ATOMIC || args.reduce_in_kernel == REDUCE_ATOMIC_FLAG) {
            if (args.reduce_in_kernel == REDUCE_ATOMIC_FLAG && slice != 0)
                flag_take_credit(args, tm * args.tiles_n + tn, seen);
            // Relaxed device-scope adds, no return value: the kernel's end orders them
            // before anything that reads C.
            uint32_t *const cc = static_cast<uint32_t *>(args.C);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int64_t col = c0 + j * 32 + frag_row;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int64_t row = r0 + i * 32 + 8 * (r >> 2) + 4 * frag_half + (r & 3);
                        if (row < M && col < N)
                            __hip_atomic_fetch_add(&cc[row * args.ldc + col], uint32_t(acc[i][j][r]),
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            return;
        }
    }
    if (args.reduce_in_kernel == REDUCE_SEPARATE) {
        // This slice's partial plane for the separate reduction.
        out_t *out = static_cast<out_t *>(args.workspace) + int64_t(slice) * plane;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t col = c0 + j * 32 + frag_row;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = r0 + i * 32 + 8 * (r >> 2) + 4 * frag_half + (r & 3);
                    if (row < M && col < N) out[row * N + col] = acc[i][j][r];
                }
            }
        return;
    }

    sum_t *ws = static_cast<sum_t *>(args.workspace);
    {
        sum_t *out = ws + int64_t(slice) * plane;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t col = c0 + j * 32 + frag_row;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = r0 + i * 32 + 8 * (r >> 2) + 4 * frag_half + (r & 3);
                    if (row < M && col < N) store_coherent(&out[row * N + col], sum_t(acc[i][j][r]));
                }
            }
    }
    const int tile = tm * args.tiles_n + tn;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's partial stores are complete
    __syncthreads();                                   // ... and every thread's
    if (threadIdx.x == 0) {
        const unsigned ticket = __hip_atomic_fetch_add(&args.counters[tile], 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
        s_last = ticket == unsigned(args.split_k - 1);
    }
    __syncthreads();
    if (!s_last) return;

    // Last slice of this tile: C = ((ws[0] + ws[1]) + ws[2]) + ... over the valid part of the
    // tile, by all threads, consecutive columns per thread, with up to sixteen slices in flight.
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int rows = int(M - m0 < BM ? M - m0 : BM);
    const int cols = int(N - n0 < BN ? N - n0 : BN);
    const int split = args.split_k;
    constexpr int V = 2;                               // columns per thread and pass
    const int groups = (cols + V - 1) / V;
    for (int q = int(threadIdx.x); q < rows * groups; q += int(blockDim.x)) {
        const int rr = q / groups, cv = (q % groups) * V;
        const int64_t base = (m0 + rr) * N + n0 + cv;
        const int nv = cols - cv < V ? cols - cv : V;
        sum_t s[V];
        for (int p0 = 0; p0 < split; p0 += 16) {
            sum_t v[16][V];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const sum_t *src = ws + int64_t(p0 + u < split ? p0 + u : 0) * plane + base;
#pragma unroll
                for (int e = 0; e < V; ++e) v[u][e] = e < nv ? load_coherent(src + e) : sum_t(0);
            }
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (p0 + u < split) {
#pragma unroll
                    for (int e = 0; e < V; ++e) s[e] = (p0 + u == 0) ? v[u][e] : s[e] + v[u][e];
                }
        }
        const int64_t dst = (m0 + rr) * args.ldc + n0 + cv;
#pragma unroll
        for (int e = 0; e < V; ++e)
            if (e < nv) write_c<DT>(args, dst + e, s[e]);
    }
    if (threadIdx.x == 0)
        __hip_atomic_store(&args.counters[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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


// v_perm_b32 byte select: selector byte values 0-3 pick bytes of the SECOND
// operand, 4-7 bytes of the FIRST.
__device__ __forceinline__ unsigned perm(unsigned hi, unsigned lo, unsigned sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// bf16 block: rows[base .. base+KPB) are row pieces of 8 columns (column c in
// dword c/2, half c%2).  col[c][j] = (row 2j, row 2j+1) of column c.
template <int KPB, int N>
__device__ __forceinline__ void bf16_transpose(const u32x4_t (&rows)[N], int base, unsigned (&col)[8][KPB / 2]) {
#pragma unroll
    for (int j = 0; j < KPB / 2; ++j)
#pragma unroll
        for (int c = 0; c < 8; ++c)
            col[c][j] = perm(rows[base + 2 * j + 1][c >> 1], rows[base + 2 * j][c >> 1],
                             (c & 1) ? 0x07060302u : 0x05040100u);
}

// int8 block: row pieces of 8 columns (column c in dword c/4, byte c%4).
// col[c][j] = bytes (row 4j, 4j+1, 4j+2, 4j+3) of column c: pairs of rows are
// interleaved bytewise first, then pairs of pairs halfword-wise.
template <int KPB, int N>
__device__ __forceinline__ void i8_transpose(const u32x2_t (&rows)[N], int base, unsigned (&col)[8][KPB / 4]) {
#pragma unroll
    for (int j = 0; j < KPB / 4; ++j)
#pragma unroll
        for (int d = 0; d < 2; ++d) {
            const unsigned r0 = rows[base + 4 * j + 0][d], r1 = rows[base + 4 * j + 1][d];
            const unsigned r2 = rows[base + 4 * j + 2][d], r3 = rows[base + 4 * j + 3][d];
            const unsigned lo01 = perm(r1, r0, 0x05010400u), hi01 = perm(r1, r0, 0x07030602u);
            const unsigned lo23 = perm(r3, r2, 0x05010400u), hi23 = perm(r3, r2, 0x07030602u);
            col[4 * d + 0][j] = perm(lo23, lo01, 0x05040100u);
            col[4 * d + 1][j] = perm(lo23, lo01, 0x07060302u);
            col[4 * d + 2][j] = perm(hi23, hi01, 0x05040100u);
            col[4 * d + 3][j] = perm(hi23, hi01, 0x07060302u);
        }
}

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

constexpr int kBufferFlags = 0x00020000;   // raw untyped dword access (gfx9 family descriptor word 3)
constexpr uint32_t kOOB = 0x80000000u;     // offset past any resource used here -> load returns 0

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const uint8_t *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(base), (short)0, (int)bytes, kBufferFlags);
}

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

template <int DT> __device__ __forceinline__ int bswz(int k);
template <> __device__ __forceinline__ int bswz<DT_BF16>(int k) {
    const int m = k & 3;
    return (m << 2) ^ ((m >> 1) << 1);          // 0, 4, 10, 14
}
template <> __device__ __forceinline__ int bswz<DT_I8>(int k) {
    const int m = k & 7;
    return (m << 1) | (m >> 2);                 // 0, 2, 4, 6, 9, 11, 13, 15
}

template <int DT> __device__ __forceinline__ u32x2_t lds_read_tr(const uint8_t *p);
template <> __device__ __forceinline__ u32x2_t lds_read_tr<DT_BF16>(const uint8_t *p) {
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                                           (LDS_AS bf16x4_t *)(const_cast<uint8_t *>(p))));
}
template <> __device__ __forceinline__ u32x2_t lds_read_tr<DT_I8>(const uint8_t *p) {
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                                           (LDS_AS i32x2_t *)(const_cast<uint8_t *>(p))));
}

__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rsrc, uint8_t *lds_wave_base, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (LDS_AS void *)lds_wave_base, 16, int(voff), 0, 0, 0);
}

// Swizzle of the ring's 64-byte rows (A, and column-major B): chunk c of row r sits at
// chunk c ^ ((r >> 2) & 3).  Measured on gfx950 with a read-throughput probe (16 waves
// issuing the fragment reads of a 32-row block): 4 cycles per 16-byte-per-lane read,
// the conflict-free rate, where ((r >> 1) ^ (r >> 3)) & 3 took 8 and no swizzle 16.
// Period 16 in r, so the tiles 32 rows apart read at fixed offsets.
__device__ __forceinline__ int ring_swz(int row) { return (row >> 2) & 3; }

// Swizzle of row-major B rows (k) for the transpose reads, by row width: chunk c of
// row k sits at chunk c ^ ring_bswz(k).  Rows of 16 or more chunks use bswz; the
// narrow rows of the small-N ring tiles use functions found by measuring every
// GF(2)-linear map of k's low row bits onto the chunk bits with the same probe
// (each at 2.5 cycles per 8-byte-per-lane read; unswizzled rows took 4.2-8.2):
//   int8, 8 chunks (N tile 128):  k & 7
//   int8, 4 chunks (N tile 64):   (k & 4) >> 1
//   bf16, 8 chunks (N tile 64):   k1 | k0 << 1 | k1 << 2   (k0, k1: the low bits of k)
// Each depends only on the row within one transpose read's 4- or 8-row block.
template <int DT, int CPR>
__device__ __forceinline__ int ring_bswz(int k) {
    if constexpr (CPR >= 16) return bswz<DT>(k);
    else if constexpr (DT == DT_I8 && CPR == 8) return k & 7;
    else if constexpr (DT == DT_I8 && CPR == 4) return (k & 4) >> 1;
    else if constexpr (DT == DT_BF16 && CPR == 8) return ((k >> 1) & 1) | ((k & 1) << 1) | (((k >> 1) & 1) << 2);
    else return 0;
}

// Buffer resource as four dwords (base, stride 0, size in bytes, raw-access flags)
// for the inline-assembly load below.
__device__ __forceinline__ i32x4_t ring_rsrc(const uint8_t *base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return i32x4_t{int(uint32_t(a)), int(uint32_t(a >> 32) & 0xffffu), int(bytes), kBufferFlags};
}

// One wave-wide 16-byte-per-lane global -> LDS load: lane l's 16 bytes from
// rsrc + voff land at LDS byte lds + 16 l.  Written as inline assembly so that
// the compiler does not tie the LDS reads that follow to these writes (it cannot
// tell the ring buffers apart and would wait for every load in flight before each
// read); completion is tracked by the explicit vmcnt waits of the ring instead,
// and nothing else in the kernel accesses the ring.
// The LDS address goes in M0, which the "{m0}" operand has the compiler load.
__device__ __forceinline__ void ring_load16(i32x4_t rsrc, uint32_t lds, uint32_t voff) {
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" :: "v"(voff), "s"(rsrc), "{m0}"(lds) : "memory");
}

// The same with 4 bytes per lane: lane l's dword lands at LDS byte lds + 4 l.
__device__ __forceinline__ void ring_load4(i32x4_t rsrc, uint32_t lds, uint32_t voff) {
    asm volatile("buffer_load_dword %0, %1, 0 offen lds" :: "v"(voff), "s"(rsrc), "{m0}"(lds) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p) {
    return uint32_t(reinterpret_cast<uintptr_t>((LDS_AS const void *)p));
}

template <int VMCNT>
__device__ __forceinline__ void ring_barrier() {
    static_assert(VMCNT >= 0 && VMCNT < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(VMCNT) : "memory");
}

__device__ __forceinline__ void phase_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
__device__ __forceinline__ void stage_barrier() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace gemm
