// gemm_kernels.hip -- gfx950 (CDNA4) MFMA GEMM kernels and their launcher.
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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>
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
// (splitk_reduce_kernel), or, with args.reduce_in_kernel, every slice takes a
// ticket from the tile's arrival counter and the workgroup that arrives last
// sums the slices of the tile and writes C, then resets the counter to zero
// for the next launch on the stream.  Both sum in the fixed slice order
// 0, 1, ..., so fp32 results are identical run to run whichever slice finishes
// last and whichever reduction runs.
//
// The slices of a tile run on different XCDs, whose L2 caches are not kept
// coherent with each other for ordinary accesses.  Instead of device-scope
// fences (which write back and invalidate the whole L2 of the XCD), the
// partials are stored and loaded with device-scope (sc1) accesses, which go
// to the device coherence point: each thread waits until its partial stores
// are complete, the workgroup synchronises, and only then takes its ticket
// (an atomic, itself coherent device-wide); the partial loads of the last
// workgroup depend on the ticket and are issued after it.
template <typename T>
__device__ __forceinline__ void store_coherent(T *p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T load_coherent(const T *p) {
    return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

__device__ __forceinline__ uint16_t bf16_nearest_even(float f) {
    const uint32_t u = __float_as_uint(f);
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
    static_cast<typename OutElem<DT, EPI>::type *>(a.C)[idx] =
        convert_out<DT, EPI>(a, typename Types<DT>::out_t(v));
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

// A wave's output fragments straight into C with the epilogue EPI.  Lane l holds,
// for fragment (i, j) and register r, row r0 + 4 (l / 32) + 32 i + 8 (r / 4) + r % 4
// and column c0 + l % 32 + 32 j: one base pointer per lane plus a row offset that
// is a constant times ldc, which the scalar unit forms.  The epilogue is a template
// argument so that the loop bodies stay small enough to unroll fully: the
// accumulators are then only indexed by constants and stay in registers (with a
// run-time choice per element, the 256-register tiles of the 4-wave 256 x 256
// int8 kernels went to scratch).
template <int DT, int EPI, int TM, int TN>
__device__ __forceinline__ void store_c_direct(const KernelArgs &args,
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
                if (dr < rows_left) base[dr * ldc + 32 * j] = convert_out<DT, EPI>(args, acc[i][j][r]);
            }
            // One fragment at a time: keeps the scheduler from reading every accumulator
            // out ahead of its stores.
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// s_last: one int of LDS for the in-kernel split-K reduction's "last slice"
// broadcast; a kernel whose LDS is otherwise free at this point may lend it a word
// of its operand buffers (all of its global -> LDS loads complete, all of its
// fragment reads done).
template <int DT, int BM, int BN, int TM, int TN>
__device__ __forceinline__ void store_tile(const KernelArgs &args,
                                           const typename Types<DT>::acc_vec (&acc)[TM][TN],
                                           int tm, int tn, int slice, int64_t r0, int64_t c0, int lane,
                                           int &s_last) {
    using out_t = typename Types<DT>::out_t;
    using sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;  // int32 wraps mod 2^32
    const int frag_row = lane & 31, frag_half = lane >> 5;
    const int64_t M = args.M, N = args.N;
    const int64_t plane = M * N;
    if (args.split_k == 1) {
        // C itself, through the call's output conversion.
        if constexpr (DT == DT_I8) {
            if (args.epilogue == EPI_I8) store_c_direct<DT, EPI_I8>(args, acc, r0, c0, lane);
            else if (args.epilogue == EPI_I16) store_c_direct<DT, EPI_I16>(args, acc, r0, c0, lane);
            else store_c_direct<DT, EPI_NONE>(args, acc, r0, c0, lane);
        } else {
            if (args.epilogue == EPI_BF16) store_c_direct<DT, EPI_BF16>(args, acc, r0, c0, lane);
            else store_c_direct<DT, EPI_NONE>(args, acc, r0, c0, lane);
        }
        return;
    }
    if (!args.reduce_in_kernel) {
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

template <int DT, int BM, int BN, int WM, int WN, bool VEC, int WAVES_PER_EU, bool BT = false>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_tile_kernel(KernelArgs args) {
    static_assert(!(VEC && BT), "the vector B loader reads row-major B only");
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
                // Row-major B: neighbouring threads take neighbouring columns.  Column-major
                // B (stored N x K): neighbouring threads take neighbouring K chunks of a column.
                const int q = i * T::THREADS + tid;
                const int n = BT ? q >> 3 : q % BN, c = BT ? q & 7 : q / BN;
                const int64_t gn = n0 + n, gk = k0 + int64_t(c) * VECE;
                unsigned w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int e = 0; e < VECE; ++e) {
                    unsigned x = 0;
                    if (gn < N && gk + e < k_end) {
                        const int64_t idx = BT ? gn * ldb + gk + e : (gk + e) * ldb + gn;
                        if (E == 1) x = B[idx];
                        else x = reinterpret_cast<const uint16_t *>(B)[idx];
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
                const int n = BT ? q >> 3 : q % BN, c = BT ? q & 7 : q / BN;
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
    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Vectorised kernel: 16-byte (A, bf16 B) and 8-byte (int8 B) buffer loads.
//
// Every global load goes through a buffer resource.  A load whose offset is
// at or past the resource's size returns zero without touching memory, which
// replaces all bounds branches: rows past M and columns past N get an offset
// that is out of range by construction, the K tail of A is masked per chunk,
// and the K tail of B (and every stage past the end of the slice) is masked
// by shrinking the resource's size to the valid rows of the stage.  The loop
// body is therefore branch-free, so loads, LDS traffic and MFMAs of one stage
// live in one scheduling region.
// ---------------------------------------------------------------------------

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

template <int DT, int BM, int BN, int WM, int WN, int WAVES_PER_EU>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_vec_kernel(KernelArgs args) {
    using T = TileKernel<DT, BM, BN, WM, WN, true>;
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int E = T::E, BK = T::BK, VECE = T::VECE;
    constexpr int TM = T::TM, TN = T::TN;
    constexpr int THREADS = T::THREADS;
    constexpr int KPB = T::KPB, OUTB = T::OUTB, B_BLOCKS = T::B_BLOCKS;
    constexpr int A_CHUNKS = T::A_CHUNKS;

    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (BM + BN) * kStageKBytes];
    uint8_t *const a_lds = smem;
    uint8_t *const b_lds = smem + 2 * BM * kStageKBytes;

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
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;   // row strides in bytes

    // ---- per-thread global offsets (constant over the K loop) ----
    // A: chunk i of this thread is row (i * THREADS + tid) / 8, logical chunk tid % 8.
    // The per-chunk row step is uniform; rows at or past M are masked by the
    // resource size (rows are contiguous with stride lda from the tile's first row).
    const int a_c = tid & 7;
    const uint32_t a_voff0 = uint32_t((tid >> 3) * lda_b + a_c * 16);
    constexpr int A_ROW_STEP = THREADS / 8;
    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    // B: block bI of this thread covers k-rows kb*KPB .. +KPB and 8 columns from nb*8.
    // Row r of the block is the uniform offset r * ldb_b.  Columns at or past N get an
    // out-of-range base; K rows past the slice end are masked by the resource size
    // (whole blocks, since the slice length is a multiple of KPB).
    uint32_t b_voff[B_BLOCKS];
#pragma unroll
    for (int bI = 0; bI < B_BLOCKS; ++bI) {
        const int b = bI * THREADS + tid;
        const int nb = b % (BN / 8), kb = b / (BN / 8);
        b_voff[bI] = (n0 + nb * 8 < N) ? uint32_t(kb * KPB * ldb_b + nb * 8 * E) : kOOB;
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) + (k_begin * args.ldb + n0) * E;

    // One stage of staged global data.
    struct Stage {
        u32x4_t a[A_CHUNKS];
        u32x4_t b4[DT == DT_BF16 ? B_BLOCKS * KPB : 1];
        u32x2_t b2[DT == DT_I8 ? B_BLOCKS * KPB : 1];
    };

    // Loads stage kt into st (kt may be past the last stage: every load then returns 0).
    auto load_stage = [&](Stage &st, int kt) {
        const int64_t rem = (k_end - k_begin) - int64_t(kt) * BK;   // valid K elements left
        const __amdgpu_buffer_rsrc_t ra_rsrc = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const uint32_t a0 = int64_t(a_c) * VECE < rem ? a_voff0 : kOOB;
#pragma unroll
        for (int i = 0; i < A_CHUNKS; ++i)
            st.a[i] = __builtin_amdgcn_raw_buffer_load_b128(ra_rsrc, a0 + uint32_t(i * A_ROW_STEP * lda_b), 0, 0);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const __amdgpu_buffer_rsrc_t rb_rsrc =
            make_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
#pragma unroll
        for (int bI = 0; bI < B_BLOCKS; ++bI)
#pragma unroll
            for (int r = 0; r < KPB; ++r) {
                const int soff = int(r * ldb_b);
                if (DT == DT_BF16)
                    st.b4[bI * KPB + r] = __builtin_amdgcn_raw_buffer_load_b128(rb_rsrc, b_voff[bI], soff, 0);
                else
                    st.b2[bI * KPB + r] = __builtin_amdgcn_raw_buffer_load_b64(rb_rsrc, b_voff[bI], soff, 0);
            }
    };

    auto store_stage = [&](const Stage &st, int buf) {
        uint8_t *const as = a_lds + buf * BM * kStageKBytes;
        uint8_t *const bs = b_lds + buf * BN * kStageKBytes;
#pragma unroll
        for (int i = 0; i < A_CHUNKS; ++i) {
            const int row = (i * THREADS + tid) >> 3;
            *reinterpret_cast<u32x4_t *>(as + row * kStageKBytes + swz(a_c, row) * 16) = st.a[i];
        }
#pragma unroll
        for (int bI = 0; bI < B_BLOCKS; ++bI) {
            const int b = bI * THREADS + tid;
            const int nb = b % (BN / 8), kb = b / (BN / 8);
            const int byte = kb * OUTB;
            const int chunk = byte >> 4, half = (byte >> 3) & 1;
            const int base = bI * KPB;
            constexpr int DW = OUTB / 4;                 // dwords per column piece
            unsigned col[8][DW];
            if (DT == DT_BF16) bf16_transpose<KPB>(st.b4, base, *reinterpret_cast<unsigned(*)[8][KPB / 2]>(&col));
            else i8_transpose<KPB>(st.b2, base, *reinterpret_cast<unsigned(*)[8][KPB / 4]>(&col));
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int n = nb * 8 + c;
                uint8_t *dst = bs + n * kStageKBytes + swz(chunk, n) * 16 + half * 8;
                if (DW == 4)
                    *reinterpret_cast<u32x4_t *>(dst) = u32x4_t{col[c][0], col[c][DW > 1 ? 1 : 0],
                                                                col[c][DW > 2 ? 2 : 0], col[c][DW > 3 ? 3 : 0]};
                else
                    *reinterpret_cast<u32x2_t *>(dst) = u32x2_t{col[c][0], col[c][DW > 1 ? 1 : 0]};
            }
        }
    };

    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);
    u32x4_t fa[2][TM], fb[2][TN];
    auto load_frags = [&](int buf, int s, int slot) {
        const uint8_t *const as = a_lds + buf * BM * kStageKBytes;
        const uint8_t *const bs = b_lds + buf * BN * kStageKBytes;
        const int chunk = 2 * s + frag_half;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = wrow0 + i * 32 + frag_row;
            fa[slot][i] = *reinterpret_cast<const u32x4_t *>(as + row * kStageKBytes + swz(chunk, row) * 16);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wcol0 + j * 32 + frag_row;
            fb[slot][j] = *reinterpret_cast<const u32x4_t *>(bs + col * kStageKBytes + swz(chunk, col) * 16);
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    // MFMAs over the stage in LDS buffer `buf`; fragments of k-step s+1 are read
    // while the MFMAs of k-step s run.  Expects k-step 0's fragments in slot 0.
    auto compute = [&](int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s < 3) load_frags(buf, s + 1, (s + 1) & 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[s & 1][i], fb[s & 1][j], acc[i][j]);
        }
    };

    // Software pipeline, two stages of global loads in flight:
    //   loop top (kt even): LDS[0] = stage kt, s1 = stage kt+1, s0 = stage kt+2 (in flight).
    Stage s0, s1;
    if (nk > 0) {
        load_stage(s0, 0);
        load_stage(s1, 1);
        store_stage(s0, 0);
        __syncthreads();
        load_stage(s0, 2);
        load_frags(0, 0, 0);
    }
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        compute(0);
        store_stage(s1, 1);
        __syncthreads();
        load_stage(s1, kt + 3);
        load_frags(1, 0, 0);
        compute(1);
        store_stage(s0, 0);
        __syncthreads();
        load_stage(s0, kt + 4);
        load_frags(0, 0, 0);
    }
    if (kt < nk) compute(0);

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS kernel (gfx950): both operands go from global memory straight
// into LDS with buffer_load ... lds, and B's K-contiguous MFMA fragments are
// produced by LDS transpose reads (ds_read_b64_tr_b16 / _b8) instead of an
// in-register transpose.  The K loop then holds only loads, LDS reads, MFMAs
// and one barrier per stage.
//
// LDS, per stage: A as BM rows of 128 K-bytes (16-byte chunks XOR-swizzled by
// swz(c, row)), B untransposed as BK rows (k) of BN*E bytes (chunks swizzled by
// a function of k mod 4 (bf16) or k mod 8 (int8), matched to the row sets the
// transpose reads touch together).
//
// Transpose read, per 16-lane group (lane g within the group): every lane
// supplies the address of one 8-byte piece; lane g receives column g of the
// block formed by the group's pieces -- b16: 4 rows x 16 columns, lane g
// addresses row g/4, columns 4(g%4)..+3; b8: 8 rows x 16 columns, lane g
// addresses row g/2, columns 8(g%2)..+7.
// ---------------------------------------------------------------------------
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

template <int DT, int BM, int BN, int WM, int WN, int WAVES_PER_EU, bool BT = false>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_lds_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;                  // K elements per stage
    constexpr int THREADS = 64 * WM * WN;
    constexpr int WAVES = WM * WN;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int A_STAGE = BM * kStageKBytes;            // bytes
    // Row-major B sits in LDS as BK rows (k) of BN*E bytes; column-major B (BT)
    // as BN rows (n) of 128 K-bytes, exactly like A.
    constexpr int B_PITCH = BT ? kStageKBytes : BN * E;   // bytes per B row in LDS
    constexpr int B_STAGE = BN * kStageKBytes;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;       // 1 KiB per wave-wide load
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;         // B rows covered by one wave-wide load
    static_assert(A_INSTR >= 1 && A_INSTR * 1024 * WAVES == A_STAGE, "A stage split");
    static_assert(B_INSTR >= 1 && B_INSTR * 1024 * WAVES == B_STAGE, "B stage split");
    static_assert(B_PITCH <= 1024 && 1024 % B_PITCH == 0, "B row pitch");

    // One LDS array per stage buffer and operand: with every access naming a
    // fixed array, the compiler can tell the direct-to-LDS writes of one stage
    // from the fragment reads of the other and does not serialise them.
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds0[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds1[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds0[B_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds1[B_STAGE];

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
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // ---- global source offsets of this lane's 16-byte pieces (constant over K) ----
    // A load i of this wave fills LDS bytes [(i*WAVES + wave) KiB, +1 KiB): lane L
    // writes physical chunk L%8 of row (i*WAVES + wave)*8 + L/8, which holds the
    // logical chunk c = (L%8) ^ f(row).  Rows at or past M are masked by the
    // resource size (rows_valid * lda bytes from the tile's first row).
    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        const int row = (i * WAVES + wave) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16);
    }
    // B load i fills LDS bytes [(i*WAVES + wave) KiB, +1 KiB) of the B stage: lane L
    // writes physical chunk p = L % B_CPR of row (i*WAVES+wave)*B_ROWS_PER_KB + L / B_CPR,
    // holding logical chunk p ^ bswz(row).  Columns at or past N get an out-of-range
    // offset; K rows past the slice end are masked by the resource size.
    // Column-major B (BT): the same scheme as A over BN rows (n) of the N x K
    // matrix; rows at or past N are masked by the resource size.
    constexpr int B_CPR = B_PITCH / 16;                   // chunks per B row
    static_assert(BT || B_CPR >= 16, "transpose-read swizzle needs rows of at least 16 chunks");
    const int64_t b_rows_valid = (N - n0) < BN ? (N - n0) : BN;
    const uint32_t bt_bytes = uint32_t(b_rows_valid * ldb_b);
    uint32_t b_voff[B_INSTR];
    int b_chunk[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        if constexpr (BT) {
            const int row = (i * WAVES + wave) * 8 + (lane >> 3);
            const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
            b_chunk[i] = c;
            b_voff[i] = uint32_t(row * ldb_b + c * 16);
        } else {
            const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
            const int c = (lane % B_CPR) ^ bswz<DT>(row);
            b_chunk[i] = 0;
            b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
        }
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) +
                                  (BT ? n0 * args.ldb + k_begin : k_begin * args.ldb + n0) * E;
    // B resource of stage kt; `rows` valid K rows bound row-major B only.
    auto b_rsrc = [&](int kt, int64_t rows) {
        if constexpr (BT) return make_rsrc(b_base + int64_t(kt) * kStageKBytes, bt_bytes);
        else return make_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
    };
    const int64_t k_len = k_end - k_begin;

    // Issues the loads of stage kt into LDS buffer BUF.  Full stages use the
    // precomputed offsets as they are; only a partial last stage (and stages past
    // the end, which load nothing) pays for the per-chunk K mask.
    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const __amdgpu_buffer_rsrc_t rb = b_rsrc(kt, rows);
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
        if (rem >= BK) {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
                if (i < B_INSTR) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
#pragma unroll
            for (int i = A_INSTR; i < B_INSTR; ++i) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
        } else {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
                load_lds16(ra, as + (i * WAVES + wave) * 1024, off);
            }
#pragma unroll
            for (int i = 0; i < B_INSTR; ++i) {
                // Column-major B masks its K tail per chunk, as A does; row-major B by rows.
                const uint32_t off = (!BT || int64_t(b_chunk[i]) * VECE < rem) ? b_voff[i] : kOOB;
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, off);
            }
        }
    };

    // A full stage's loads issued in two halves, at the start of k-steps 0 and 1:
    // issuing all of them in one burst backs up the vector memory path and
    // stalls the issuing waves (and their MFMAs) for longer than the spread
    // costs in latency.  A partial last stage is loaded whole with part 0.
    auto load_stage_part = [&](int kt, auto buf_c, int part) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        if (rem < BK) {
            if (part == 0) load_stage(kt, buf_c);
            return;
        }
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const __amdgpu_buffer_rsrc_t rb = b_rsrc(kt, BK);
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int i = 0; i < (A_INSTR > B_INSTR ? A_INSTR : B_INSTR); ++i) {
            if ((i & 1) != part) continue;
            if (i < A_INSTR) load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
            if (i < B_INSTR) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
        }
    };

    // ---- fragment offsets (lane constants; the k-step and tile index only add immediates) ----
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);
    // A tile i, k-step s: row r_i = wrow0 + 32 i + frag_row, chunk 2s + half, swizzled by
    // f(r_i) = f(r_0) ^ 4 (i & 1).  Offset = r_0*128 + 4096 i + 16 ((2s + half) ^ f(r_0) ^ 4(i&1)).
    const int r0 = wrow0 + frag_row;
    const int f0 = (r0 ^ (r0 >> 3)) & 7;
    int a_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) a_fo[p][st] = r0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ f0 ^ (4 * p));
    // B transpose reads: group = lane/16, g = lane%16.
    // bf16: rows 4*h + g/4 (+8 for the upper K half), byte columns 8*(g%4) (+32 for odd groups)
    // int8: rows 8*h + g/2 (+16 for the upper K half), byte columns 8*(g%2) (+16 for odd groups)
    // The row's swizzle depends only on g (k mod 4 or 8), so tile j, read h, k-step s
    // is b_fo[j] + (s*KSTEP + h*TR_ROWS) * B_PITCH.
    const int grp = lane >> 4, g16 = lane & 15;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;        // rows per transpose read
    constexpr int KSTEP = 32 / E;                         // K elements per MFMA
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (grp & 1) * 16 * E;
    const int tr_khalf = (grp >> 1) * (KSTEP / 2);
    const int bz = bswz<DT>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }
    // Column-major B: fragments are 16-byte reads of K-contiguous rows, as for A.
    const int rb0 = wcol0 + frag_row;
    const int fb0 = (rb0 ^ (rb0 >> 3)) & 7;
    int bt_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) bt_fo[p][st] = rb0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ fb0 ^ (4 * p));

    u32x4_t fa[2][TM], fb[2][TN];
    auto load_frags = [&](auto buf_c, auto s_c, auto slot_c) {
        constexpr int BUF = decltype(buf_c)::value;
        constexpr int S = decltype(s_c)::value;
        constexpr int SLOT = decltype(slot_c)::value;
        const uint8_t *const as = BUF ? a_lds1 : a_lds0;
        const uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            fa[SLOT][i] = *reinterpret_cast<const u32x4_t *>(as + a_fo[i & 1][S] + 4096 * i);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            if constexpr (BT) {
                fb[SLOT][j] = *reinterpret_cast<const u32x4_t *>(bs + bt_fo[j & 1][S] + 4096 * j);
            } else {
                const u32x2_t lo = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP) * B_PITCH);
                const u32x2_t hi = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH);
                fb[SLOT][j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[1][i] = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[1][j] = u32x4_t{0u, 0u, 0u, 0u};

    auto mfma_slot = [&](auto slot_c) {
        constexpr int SLOT = decltype(slot_c)::value;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[SLOT][i], fb[SLOT][j], acc[i][j]);
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;

    // One stage (buffer BUF holds stage kt, visible).  On entry slot 1 holds the
    // fragments of the previous stage's last k-step, whose MFMAs run here, under
    // the latency of this stage's first LDS reads; on exit slot 1 holds this
    // stage's last k-step and every wave has finished reading buffer BUF.
    auto stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        using OTHER = std::integral_constant<int, 1 - BUF>;
        load_stage_part(kt + 1, OTHER{}, 0);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I0{}, I0{});
        mfma_slot(I1{});
        __builtin_amdgcn_sched_barrier(0);
        load_stage_part(kt + 1, OTHER{}, 1);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I1{}, I1{});
        mfma_slot(I0{});
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I2{}, I0{});
        mfma_slot(I1{});
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I3{}, I1{});
        mfma_slot(I0{});
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    };

    if (nk > 0) {
        load_stage(0, I0{});
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        stage(kt, I0{});
        stage(kt + 1, I1{});
    }
    if (kt < nk) stage(kt, I0{});
    mfma_slot(I1{});

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Ring kernel (gfx950): the direct-to-LDS data path of gemm_lds_kernel with a
// deeper prefetch.  K is walked in 64-byte slots (32 bf16 or 64 int8 elements,
// two MFMA k-steps) held in an NB-deep ring of LDS buffers, so that a slot's
// global -> LDS loads are issued NB - 1 slots before the slot is consumed
// instead of one 128-byte stage before; the double buffering of inputs
// (paper, Sec. 4.2.1) generalised to NB buffers.  Measured on the 8192^3 GEMM,
// the one-stage lead of the two-buffer kernel leaves the MFMAs waiting on the
// L2 for about a quarter of the time.
//
// Per slot s (buffer s % NB):
//   phase A: read the k-step 1 fragments of slot s, run the k-step 0 MFMAs
//            (fragments read during slot s - 1);
//   wait until this wave's loads of slot s + 1 have landed, barrier: slot s + 1
//            is visible, and every wave holds all of slot s in registers, so
//            buffer s % NB is free;
//   phase B: run the k-step 1 MFMAs of slot s, read the k-step 0 fragments of
//            slot s + 1, and issue the first half of the loads of slot s + NB into
//            buffer s % NB (phase A of slot s + 1 issues the other half).
// The barrier sits between two runs of MFMAs whose operands are already in
// registers, so the matrix pipes stay fed across it.  Within a phase, the MFMAs,
// LDS reads and global loads are issued in a fixed interleaved order.
//
// LDS, per slot: A as BM rows of 64 K-bytes, the 16-byte chunk c of row r at
// chunk c ^ ga(r), ga(r) = ((r >> 1) ^ (r >> 3)) & 3, which keeps the fragment
// reads of any 8 (and any 16) consecutive rows on distinct banks; B row-major
// as 64 / E rows (k) of BN * E bytes with gemm_lds_kernel's swizzle (rows of
// at least 256 bytes; narrower rows unswizzled), or column-major (BT) like A.  Every slot of every iteration issues the same
// number of loads (slots past the end of the K range get an empty resource and
// load zeros without touching memory), so the wait before each barrier is a
// fixed count of this wave's loads still allowed in flight.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int ring_swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

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

template <int DT, int BM, int BN, int WM, int WN, int WAVES_PER_EU, bool BT, int NB>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_ring_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BKS = kSlotKBytes / E;                  // K elements per slot
    constexpr int WAVES = WM * WN;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int A_SLOT = BM * kSlotKBytes;              // bytes
    constexpr int B_PITCH = BT ? kSlotKBytes : BN * E;    // bytes per B row in LDS
    constexpr int B_SLOT = BN * kSlotKBytes;
    // A moves in 16-byte pieces per lane (1 KiB per wave-wide load) when its slot
    // splits evenly into such loads over the waves, else in 4-byte pieces (256 B per
    // load); B always moves in 16-byte pieces.
    constexpr int A_W = (A_SLOT % (1024 * WAVES) == 0) ? 16 : 4;
    constexpr int A_LOAD = 64 * A_W;                      // bytes per wave-wide A load
    constexpr int A_INSTR = A_SLOT / A_LOAD / WAVES;
    constexpr int A_ROWS_PER_LOAD = A_LOAD / kSlotKBytes;
    constexpr int B_INSTR = B_SLOT / 1024 / WAVES;
    constexpr int LPS = A_INSTR + B_INSTR;                // loads per wave per slot
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;                   // 16-byte chunks per B row
    // Row-major B rows of 16 or more chunks are swizzled for conflict-free transpose
    // reads; narrower rows (small BN) are stored as they are.
    constexpr bool B_SWZ = !BT && B_CPR >= 16;
    constexpr int NREAD = TM + (BT ? TN : 2 * TN);        // LDS reads per k-step
    static_assert(NB >= 3 && NB <= 8, "ring depth");
    static_assert(TM >= 1 && TN >= 1, "wave tile of at least one 32 x 32 MFMA tile");
    static_assert(A_INSTR >= 1 && A_INSTR * A_LOAD * WAVES == A_SLOT, "A slot split");
    static_assert(B_INSTR >= 1 && B_INSTR * 1024 * WAVES == B_SLOT, "B slot split");
    static_assert(B_PITCH <= 1024 && 1024 % B_PITCH == 0, "B row pitch");
    static_assert((NB - 1) * LPS < 64, "loads in flight must fit vmcnt");

    // The ring: NB buffers, each an A part then a B part.
    __shared__ __attribute__((aligned(1024))) uint8_t ring_lds[NB][A_SLOT + B_SLOT];
    auto abuf = [&](auto j_c) -> uint8_t * { return ring_lds[decltype(j_c)::value]; };
    auto bbuf = [&](auto j_c) -> uint8_t * { return abuf(j_c) + A_SLOT; };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wave_m = wave / WN, wave_n = wave % WN;
    const uint32_t wave_u = uint32_t(__builtin_amdgcn_readfirstlane(wave));   // uniform copy for LDS addresses

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int ns = k_end > k_begin ? int((k_end - k_begin + BKS - 1) / BKS) : 0;
    const int64_t k_len = k_end - k_begin;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // ---- global source offsets of this lane's 16-byte pieces (constant over K) ----
    // A load i of this wave fills bytes [(i*WAVES + wave) KiB, +1 KiB) of the A slot:
    // lane L writes physical chunk L%4 of row (i*WAVES + wave)*16 + L/4, which holds
    // logical chunk (L%4) ^ ga(row).  Rows at or past M are masked by the resource size.
    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        // Lane L writes A_W bytes at byte L * A_W of the load's block of A_ROWS_PER_LOAD rows.
        const int row = (i * WAVES + wave) * A_ROWS_PER_LOAD + (lane * A_W) / kSlotKBytes;
        const int byte = (lane * A_W) % kSlotKBytes;
        const int c = (byte >> 4) ^ ring_swz(row);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16 + (byte & 15));
    }
    // Row-major B: load i fills B-slot bytes [(i*WAVES + wave) KiB, +1 KiB): lane L writes
    // physical chunk p = L % B_CPR of row (i*WAVES + wave)*B_ROWS_PER_KB + L / B_CPR, holding
    // logical chunk p ^ bswz(row); columns at or past N get an out-of-range offset, K rows
    // past the slice end are masked by the resource size.  Column-major B: as A, over BN
    // rows (n) of the N x K matrix.
    const int64_t b_rows_valid = (N - n0) < BN ? (N - n0) : BN;
    const uint32_t bt_bytes = uint32_t(b_rows_valid * ldb_b);
    uint32_t b_voff[B_INSTR];
    int b_chunk[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        if constexpr (BT) {
            const int row = (i * WAVES + wave) * 16 + (lane >> 2);
            const int c = (lane & 3) ^ ring_swz(row);
            b_chunk[i] = c;
            b_voff[i] = uint32_t(row * ldb_b + c * 16);
        } else {
            const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
            const int c = (lane % B_CPR) ^ (B_SWZ ? bswz<DT>(row) : 0);
            b_chunk[i] = 0;
            b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
        }
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) +
                                  (BT ? n0 * args.ldb + k_begin : k_begin * args.ldb + n0) * E;

    // Issues load L (A loads first, then B loads) of slot kt into ring buffer J.  A
    // partial last slot masks its K tail per chunk (A, and column-major B) or by rows
    // (row-major B, through the resource size); slots past the end load nothing.
    auto load_one = [&](int kt, auto j_c, auto l_c) {
        constexpr int L = decltype(l_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BKS;
        if constexpr (L < A_INSTR) {
            const i32x4_t ra = ring_rsrc(a_base + int64_t(kt) * kSlotKBytes, rem > 0 ? a_bytes : 0u);
            const uint32_t off = (rem >= BKS || int64_t(a_chunk[L]) * VECE < rem) ? a_voff[L] : kOOB;
            const uint32_t dst = lds_addr(abuf(j_c)) + (L * WAVES + wave_u) * A_LOAD;
            if constexpr (A_W == 16) ring_load16(ra, dst, off);
            else ring_load4(ra, dst, off);
        } else {
            constexpr int I = L - A_INSTR;
            i32x4_t rb;
            uint32_t off = b_voff[I];
            if constexpr (BT) {
                rb = ring_rsrc(b_base + int64_t(kt) * kSlotKBytes, rem > 0 ? bt_bytes : 0u);
                off = (rem >= BKS || int64_t(b_chunk[I]) * VECE < rem) ? off : kOOB;
            } else {
                const int64_t rows = rem <= 0 ? 0 : (rem < BKS ? rem : BKS);
                rb = ring_rsrc(b_base + int64_t(kt) * BKS * ldb_b, uint32_t(rows * ldb_b));
            }
            ring_load16(rb, lds_addr(bbuf(j_c)) + (I * WAVES + wave_u) * 1024, off);
        }
    };
    auto load_slot = [&](int kt, auto j_c) {
        static_for<0, LPS>([&](auto l_c) { load_one(kt, j_c, l_c); });
    };

    // ---- fragment offsets (lane constants; the k-step and tile index only add immediates) ----
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);
    // A tile i, k-step S: row r_i = wrow0 + 32 i + frag_row, logical chunk 2S + half;
    // ga(r_i) = ga(r_0) (ga has period 32), so the offset is a_fo[S] + 2048 i.
    const int r0 = wrow0 + frag_row;
    int a_fo[2];
#pragma unroll
    for (int S = 0; S < 2; ++S) a_fo[S] = r0 * kSlotKBytes + 16 * ((2 * S + frag_half) ^ ring_swz(r0));
    const int rb0 = wcol0 + frag_row;
    int bt_fo[2];
#pragma unroll
    for (int S = 0; S < 2; ++S) bt_fo[S] = rb0 * kSlotKBytes + 16 * ((2 * S + frag_half) ^ ring_swz(rb0));
    // Row-major B transpose reads: as in gemm_lds_kernel.
    const int grp = lane >> 4, g16 = lane & 15;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;        // rows per transpose read
    constexpr int KSTEP = 32 / E;                         // K elements per MFMA
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (grp & 1) * 16 * E;
    const int tr_khalf = (grp >> 1) * (KSTEP / 2);
    const int bz = B_SWZ ? bswz<DT>(tr_row) : 0;
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }

    u32x4_t fa[2][TM], fb[2][TN];
    // LDS read R of k-step S of ring buffer J into register set SET: reads 0 .. TM-1
    // are A's fragments; then B's, one 16-byte read per fragment (column-major B) or
    // two 8-byte transpose reads (row-major B).
    auto read_one = [&](auto j_c, auto s_c, auto set_c, auto r_c) {
        constexpr int S = decltype(s_c)::value;
        constexpr int SET = decltype(set_c)::value;
        constexpr int R = decltype(r_c)::value;
        const uint8_t *const as = abuf(j_c);
        const uint8_t *const bs = bbuf(j_c);
        if constexpr (R < TM) {
            fa[SET][R] = *reinterpret_cast<const u32x4_t *>(as + a_fo[S] + 2048 * R);
        } else if constexpr (BT) {
            constexpr int J = R - TM;
            fb[SET][J] = *reinterpret_cast<const u32x4_t *>(bs + bt_fo[S] + 2048 * J);
        } else {
            constexpr int J = (R - TM) / 2, H = (R - TM) % 2;
            const u32x2_t v = lds_read_tr<DT>(bs + b_fo[J] + (S * KSTEP + H * TR_ROWS) * B_PITCH);
            fb[SET][J][2 * H] = v[0];
            fb[SET][J][2 * H + 1] = v[1];
        }
    };
    auto load_frags = [&](auto j_c, auto s_c, auto set_c) {
        static_for<0, NREAD>([&](auto r_c) { read_one(j_c, s_c, set_c, r_c); });
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    // One phase, in a fixed order: MFMA q of register set MS (q = 0 .. TM*TN-1), then,
    // after even q, the next of this phase's global loads [L0, L1) of slot lkt into
    // buffer LJ, then LDS reads 2q and 2q+1 of k-step RS of buffer RJ into set RSET.
    // The loads leave one at a time between MFMAs rather than in a burst that backs
    // up the vector memory path and stalls the issuing waves, and the reads go out
    // early enough for their latency to hide under the MFMAs that follow.
    constexpr int NQ = TM * TN;
    auto phase = [&](auto ms_c, auto rj_c, auto rs_c, auto rset_c, int lkt, auto lj_c, auto l0_c, auto l1_c) {
        constexpr int MS = decltype(ms_c)::value;
        constexpr int L0 = decltype(l0_c)::value, L1 = decltype(l1_c)::value;
        static_for<0, NQ>([&](auto q_c) {
            constexpr int Q = decltype(q_c)::value;
            acc[Q / TN][Q % TN] = mfma32<DT>(fa[MS][Q / TN], fb[MS][Q % TN], acc[Q / TN][Q % TN]);
            constexpr int L = L0 + Q / 2;
            if constexpr (Q % 2 == 0 && L < L1) load_one(lkt, lj_c, std::integral_constant<int, L>{});
            if constexpr (2 * Q < NREAD) read_one(rj_c, rs_c, rset_c, std::integral_constant<int, 2 * Q>{});
            if constexpr (2 * Q + 1 < NREAD) read_one(rj_c, rs_c, rset_c, std::integral_constant<int, 2 * Q + 1>{});
            __builtin_amdgcn_sched_barrier(0);
        });
        // Reads beyond two per MFMA (none for the configurations compiled here).
        static_for<2 * NQ, NREAD>([&](auto r_c) { read_one(rj_c, rs_c, rset_c, r_c); });
        static_for<L0 + (NQ + 1) / 2, L1>([&](auto l_c) { load_one(lkt, lj_c, l_c); });
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // The loads of slot s + NB (into buffer s % NB, free after the barrier of slot s) are
    // split between phase B of slot s (loads 0 .. LB-1) and phase A of slot s + 1 (the
    // rest); both come before the barrier of slot s + 1, which waits for slot s + 2.
    constexpr int LB = (LPS + 1) / 2;
    using LBC = std::integral_constant<int, LB>;
    using LPSC = std::integral_constant<int, LPS>;

    auto slot = [&](int kt, auto j_c) {
        constexpr int J = decltype(j_c)::value;
        using NEXT = std::integral_constant<int, (J + 1) % NB>;
        using PREV = std::integral_constant<int, (J + NB - 1) % NB>;
        // phase A: MFMAs of k-step 0 (set 0); read k-step 1 of this slot into set 1;
        // finish the loads of slot kt - 1 + NB into buffer J - 1.
        phase(I0{}, j_c, I1{}, I1{}, kt - 1 + NB, PREV{}, LBC{}, LPSC{});
        ring_barrier<(NB - 2) * LPS>();
        __builtin_amdgcn_sched_barrier(0);
        // phase B: MFMAs of k-step 1 (set 1); start the loads of slot kt + NB into
        // buffer J; read k-step 0 of the next slot into set 0.
        phase(I1{}, NEXT{}, I0{}, I0{}, kt + NB, j_c, I0{}, LBC{});
    };

    if (ns > 0) {
        // Prologue: slots 0 .. NB-2 whole and the first LB loads of slot NB-1 (phase A
        // of slot 0 issues the rest, as every phase A does), then slot 0 is waited for.
        static_for<0, NB - 1>([&](auto u) { load_slot(decltype(u)::value, u); });
        static_for<0, LB>([&](auto l_c) { load_one(NB - 1, std::integral_constant<int, NB - 1>{}, l_c); });
        ring_barrier<(NB - 2) * LPS + LB>();
        load_frags(I0{}, I0{}, I0{});
        for (int kt = 0; kt < ns; kt += NB) {
            static_for<0, NB>([&](auto u) {
                if (kt + decltype(u)::value < ns) slot(kt + decltype(u)::value, u);
            });
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // drain ring loads past the end before exit

    // The ring is drained and every wave is past its last fragment read when
    // store_tile first synchronises, so it lends the last-slice flag a word.
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane,
                                   *reinterpret_cast<int *>(ring_lds[0]));
}

// ---------------------------------------------------------------------------
// Ping-pong direct-to-LDS kernel: 256 x 256 macro-tile, 8 waves, two wave
// groups that alternate between a compute phase and a memory phase.
//
// Waves w and w + 4 share a SIMD.  Group 0 (waves 0-3) owns output rows 0-127
// of the tile, group 1 rows 128-255; each wave a 128 x 64 sub-tile.  A "unit"
// is half a stage (two MFMA k-steps).  Group 1 runs one phase behind group 0,
// so in every phase one wave per SIMD issues a dense run of 16 MFMAs from
// fragments already in registers while the other reads its next unit's
// fragments from LDS and issues its share of the next stage's global -> LDS
// loads.  Phases are separated by workgroup barriers.  Stage s sits in LDS
// buffer s % 2 and is read in phases 4s .. 4s+3; the loads of stage s+1 are
// issued in phases 4s (group 0) and 4s+1 (group 1) and waited for at the end
// of phase 4s+3, so a load has three phases to land.  Every wave executes
// the same barrier sequence; only the work between barriers depends on the
// group.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void phase_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
__device__ __forceinline__ void stage_barrier() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void gemm_pingpong_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int BM = 256, BN = 256, WAVES = 8;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;
    constexpr int TM = 4, TN = 2;                          // 128 x 64 per wave
    constexpr int A_STAGE = BM * kStageKBytes;
    constexpr int B_PITCH = BN * E;
    constexpr int B_STAGE = BK * B_PITCH;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;        // 4
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;        // 4
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;

    __shared__ __attribute__((aligned(1024))) uint8_t a_lds0[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds1[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds0[B_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds1[B_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = wave >> 2;
    const int wave_m = grp, wave_n = wave & 3;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // global -> LDS source offsets (see gemm_lds_kernel)
    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        const int row = (i * WAVES + wave) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16);
    }
    uint32_t b_voff[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
        const int c = (lane % B_CPR) ^ bswz<DT>(row);
        b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) + (k_begin * args.ldb + n0) * E;
    const int64_t k_len = k_end - k_begin;

    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const __amdgpu_buffer_rsrc_t rb = make_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
        if (rem >= BK) {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
                load_lds16(ra, as + (i * WAVES + wave) * 1024, off);
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
        }
    };

    // fragment offsets (see gemm_lds_kernel)
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / 2);
    const int wcol0 = wave_n * (BN / 4);
    const int r0 = wrow0 + frag_row;
    const int f0 = (r0 ^ (r0 >> 3)) & 7;
    int a_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) a_fo[p][st] = r0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ f0 ^ (4 * p));
    const int g16 = lane & 15, lgrp = lane >> 4;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;
    constexpr int KSTEP = 32 / E;
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (lgrp & 1) * 16 * E;
    const int tr_khalf = (lgrp >> 1) * (KSTEP / 2);
    const int bz = bswz<DT>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }

    u32x4_t fa[2][TM], fb[2][TN];                          // one unit: two k-steps
    auto load_unit = [&](auto buf_c, auto h_c) {
        constexpr int BUF = decltype(buf_c)::value;
        constexpr int H = decltype(h_c)::value;
        const uint8_t *const as = BUF ? a_lds1 : a_lds0;
        const uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            constexpr int dummy = 0; (void)dummy;
            const int S = 2 * H + ks;
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[ks][i] = *reinterpret_cast<const u32x4_t *>(as + a_fo[i & 1][S] + 4096 * i);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32x2_t lo = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP) * B_PITCH);
                const u32x2_t hi = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH);
                fb[ks][j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    auto compute_unit = [&]() {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[ks][i], fb[ks][j], acc[i][j]);
        __builtin_amdgcn_s_setprio(0);
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;

    // Four phases of stage s (LDS buffer BUF = s % 2).
    auto stage_phases = [&](int s, auto buf_c) {
        using OTHER = std::integral_constant<int, 1 - decltype(buf_c)::value>;
        // phase 4s
        if (grp == 0) {
            if (s + 1 < nk) load_stage(s + 1, OTHER{});
            load_unit(buf_c, I0{});
        } else if (s > 0) {
            compute_unit();
        }
        phase_barrier();
        // phase 4s+1
        if (grp == 0) {
            compute_unit();
        } else {
            if (s + 1 < nk) load_stage(s + 1, OTHER{});
            load_unit(buf_c, I0{});
        }
        phase_barrier();
        // phase 4s+2
        if (grp == 0) load_unit(buf_c, I1{});
        else compute_unit();
        phase_barrier();
        // phase 4s+3
        if (grp == 0) compute_unit();
        else load_unit(buf_c, I1{});
        stage_barrier();
    };

    if (nk > 0) {
        load_stage(0, I0{});
        stage_barrier();
        for (int s = 0; s < nk; s += 2) {
            stage_phases(s, I0{});
            if (s + 1 < nk) stage_phases(s + 1, I1{});
        }
        if (grp == 1) compute_unit();                       // group 1's last unit
    }

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Streaming kernel for small M (memory-bound shapes): BM = 32 or 64 rows, BN =
// 256 columns, 4 waves (each a BM x 64 sub-tile), and an NS-deep ring of LDS
// stages so that NS - 1 stages of B stream in while one is consumed.  Same
// LDS layouts, swizzles and fragment reads as gemm_lds_kernel.  Each
// iteration waits only until its own stage has landed (vmcnt counts the loads
// of the younger stages still in flight), then one barrier publishes it and
// retires the buffer the next load overwrites.  Loads of stages past the end
// of the slice are still issued (zero-size resource: they return zero without
// touching memory) so that every iteration counts the same loads.
// ---------------------------------------------------------------------------

template <int DT, int BM, int NS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_stream_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int BN = 256, WAVES = 4;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;
    constexpr int TM = BM / 32, TN = 2;                    // wave tile BM x 64
    constexpr int A_STAGE = BM * kStageKBytes;
    constexpr int B_PITCH = BN * E;
    constexpr int B_STAGE = BK * B_PITCH;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;        // 1 (BM 32) or 2 (BM 64)
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;        // 8
    constexpr int LPS = A_INSTR + B_INSTR;                 // loads per wave per stage
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;
    static_assert(A_INSTR >= 1 && A_INSTR * 1024 * WAVES == A_STAGE, "A stage split");
    static_assert((NS - 2) * LPS < 64, "outstanding loads must fit vmcnt");

    __shared__ __attribute__((aligned(1024))) uint8_t a_lds[NS][A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds[NS][B_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        const int row = (i * WAVES + wave) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16);
    }
    uint32_t b_voff[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
        const int c = (lane % B_CPR) ^ bswz<DT>(row);
        b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) + (k_begin * args.ldb + n0) * E;
    const int64_t k_len = k_end - k_begin;

    // The loads are the ring kernel's inline-assembly form, invisible to the compiler's
    // wait-count tracking (which cannot tell the stage buffers apart and would make every
    // fragment read wait for all loads in flight); the explicit vmcnt wait before each
    // barrier accounts for them.
    const uint32_t wave_u = uint32_t(__builtin_amdgcn_readfirstlane(wave));
    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const i32x4_t ra = ring_rsrc(a_base + int64_t(kt) * kStageKBytes, rem > 0 ? a_bytes : 0u);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const i32x4_t rb = ring_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
#pragma unroll
        for (int i = 0; i < A_INSTR; ++i) {
            const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
            ring_load16(ra, lds_addr(&a_lds[BUF][0]) + (i * WAVES + wave_u) * 1024, off);
        }
#pragma unroll
        for (int i = 0; i < B_INSTR; ++i)
            ring_load16(rb, lds_addr(&b_lds[BUF][0]) + (i * WAVES + wave_u) * 1024, b_voff[i]);
    };

    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wcol0 = wave * 64;
    const int r0 = frag_row;
    const int f0 = (r0 ^ (r0 >> 3)) & 7;
    int a_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) a_fo[p][st] = r0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ f0 ^ (4 * p));
    const int g16 = lane & 15, lgrp = lane >> 4;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;
    constexpr int KSTEP = 32 / E;
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (lgrp & 1) * 16 * E;
    const int tr_khalf = (lgrp >> 1) * (KSTEP / 2);
    const int bz = bswz<DT>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    auto compute = [&](auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
#pragma unroll
        for (int S = 0; S < 4; ++S) {
            u32x4_t fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *reinterpret_cast<const u32x4_t *>(&a_lds[BUF][a_fo[i & 1][S] + 4096 * i]);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32x2_t lo = lds_read_tr<DT>(&b_lds[BUF][b_fo[j] + (S * KSTEP) * B_PITCH]);
                const u32x2_t hi = lds_read_tr<DT>(&b_lds[BUF][b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH]);
                fb[j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[i], fb[j], acc[i][j]);
        }
    };

    // One iteration: stage kt is in buffer BUF; buffer (BUF + NS - 1) % NS receives stage kt + NS - 1.
    auto iteration = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        ring_barrier<(NS - 2) * LPS>();                    // own loads of stage kt have landed, then
                                                           // everyone's; buffer BUF-1 retired
        load_stage(kt + NS - 1, std::integral_constant<int, (BUF + NS - 1) % NS>{});
        compute(buf_c);
    };

    if (nk > 0) {
        static_for<0, NS - 1>([&](auto u) { load_stage(decltype(u)::value, u); });
        for (int kt = 0; kt < nk; kt += NS) {
            static_for<0, NS>([&](auto u) {
                if (kt + decltype(u)::value < nk) iteration(kt + decltype(u)::value, u);
            });
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // drain ring loads past the end before exit

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Matrix-vector kernels for M = 1 (the paper's stated future work: GEMV).  With
// one row of A there is no reuse to stage through LDS or to feed MFMAs with: the
// work is a single pass over B, bound by HBM bandwidth, so these kernels only
// keep enough 16-byte loads in flight and do the few multiply-adds per byte on
// the vector ALUs.
//
// Row-major B (gemv_kernel): a workgroup owns 1024 columns of one K slice; lane l
// of each wave holds 16 consecutive columns (16 int8 or 2 x 8 bf16 per row), the
// four waves take every fourth row of the slice, and their partial sums meet in
// LDS at the end.
//
// Column-major B (gemv_bt_kernel, B stored N x K): a workgroup owns 16 columns
// (rows of the stored matrix), four per wave; the lanes of a wave split K in
// 16-byte pieces and accumulate with the 4-way int8 dot-product instruction
// (bf16: widened to fp32, fused multiply-adds), then a butterfly over the wave
// sums the lanes.
//
// Split-K uses the partial planes and arrival counters of the tile kernels,
// with the same fixed slice order.
// ---------------------------------------------------------------------------
template <int DT>
using gemv_acc_t = typename std::conditional<DT == DT_I8, int32_t, float>::type;
template <int DT>
using gemv_sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;   // int32 wraps mod 2^32

// Writes `cols` results v[c] of columns n0 + c (one output row) for K slice
// `slice`: straight into C without split-K, else into the slice's partial plane;
// with the in-kernel reduction the workgroup arriving last for this column block
// sums the planes in slice order.  Thread t handles c = t, t + 256, ...
template <int DT, int COLS>
__device__ __forceinline__ void gemv_store(const KernelArgs &args, const gemv_acc_t<DT> *v, int64_t n0,
                                           int tile, int slice) {
    using sum_t = gemv_sum_t<DT>;
    const int64_t N = args.N;
    sum_t *ws = static_cast<sum_t *>(args.workspace);
    const int t = int(threadIdx.x);
    if (args.split_k == 1) {
        for (int c = t; c < COLS; c += 256)
            if (n0 + c < N) write_c<DT>(args, n0 + c, v[c]);
        return;
    }
    if (!args.reduce_in_kernel) {
        for (int c = t; c < COLS; c += 256)
            if (n0 + c < N) ws[int64_t(slice) * N + n0 + c] = sum_t(v[c]);
        return;
    }
    for (int c = t; c < COLS; c += 256)
        if (n0 + c < N) store_coherent(&ws[int64_t(slice) * N + n0 + c], sum_t(v[c]));
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's partial stores are complete
    __syncthreads();                                   // ... and every thread's
    if (t == 0) {
        const unsigned ticket = __hip_atomic_fetch_add(&args.counters[tile], 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
        s_last = ticket == unsigned(args.split_k - 1);
    }
    __syncthreads();
    if (!s_last) return;
    // Sixteen slices per round trip: the loads of a batch are all issued before any is
    // used, then added in slice order.
    for (int c = t; c < COLS; c += 256) {
        if (n0 + c >= N) continue;
        sum_t s = sum_t(0);
        for (int p0 = 0; p0 < args.split_k; p0 += 16) {
            sum_t v16[16];
#pragma unroll
            for (int u = 0; u < 16; ++u)
                v16[u] = load_coherent(&ws[int64_t(p0 + u < args.split_k ? p0 + u : 0) * N + n0 + c]);
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (p0 + u < args.split_k) s = (p0 + u == 0) ? v16[u] : s + v16[u];
        }
        write_c<DT>(args, n0 + c, s);
    }
    if (t == 0) __hip_atomic_store(&args.counters[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int DT>
__global__ __launch_bounds__(256) void gemv_kernel(KernelArgs args) {
    using acc_t = gemv_acc_t<DT>;
    constexpr int E = Types<DT>::E;
    constexpr int CB = 1024;                   // columns per workgroup
    constexpr int CPL = 16;                    // columns per lane
    constexpr int PIECES = CPL * E / 16;       // 16-byte pieces per lane and row (1 int8, 2 bf16)
    constexpr int U = 8 / PIECES;              // rows in flight per lane and iteration
    const int lane = int(threadIdx.x) & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    (void)tm;
    const int64_t N = args.N;
    const int64_t n0 = int64_t(tn) * CB;
    const int64_t col = n0 + int64_t(lane) * CPL;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    // N * E is a multiple of 16 bytes, so a 16-byte piece is either wholly inside a row or past its end.
    bool piece_ok[PIECES];
#pragma unroll
    for (int h = 0; h < PIECES; ++h) piece_ok[h] = col + h * (16 / E) < N;

    const uint8_t *const Ab = static_cast<const uint8_t *>(args.A);
    const uint8_t *const Bb = static_cast<const uint8_t *>(args.B);
    const int64_t ldb_b = args.ldb * E;

    acc_t acc[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) acc[j] = acc_t(0);

    // Batches of U rows (this wave's rows k0, k0 + 4, ..., k0 + 4(U-1)); the loads of
    // the next batch are issued before the current one is consumed, so two batches
    // are in flight per lane.
    struct Batch {
        u32x4_t v[U][PIECES];
        acc_t a[U];
    };
    auto load_batch = [&](Batch &bt, int64_t k0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t k = k0 + 4 * u;
            const bool row_ok = k < k_end;
            const uint8_t *const row = Bb + k * ldb_b + col * E;
#pragma unroll
            for (int h = 0; h < PIECES; ++h)
                bt.v[u][h] = (row_ok && piece_ok[h]) ? *reinterpret_cast<const u32x4_t *>(row + 16 * h)
                                                     : u32x4_t{0u, 0u, 0u, 0u};
            if constexpr (DT == DT_I8) {
                bt.a[u] = row_ok ? acc_t(reinterpret_cast<const int8_t *>(Ab)[k]) : acc_t(0);
            } else {
                const uint32_t bits = row_ok ? uint32_t(reinterpret_cast<const uint16_t *>(Ab)[k]) : 0u;
                bt.a[u] = __uint_as_float(bits << 16);
            }
        }
    };
    auto use_batch = [&](const Batch &bt) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int h = 0; h < PIECES; ++h)
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const unsigned x = bt.v[u][h][w];
                    if constexpr (DT == DT_I8) {
#pragma unroll
                        for (int b = 0; b < 4; ++b)
                            acc[4 * w + b] += int32_t(int8_t(uint8_t(x >> (8 * b)))) * bt.a[u];
                    } else {
                        acc[8 * h + 2 * w] = fmaf(__uint_as_float(x << 16), bt.a[u], acc[8 * h + 2 * w]);
                        acc[8 * h + 2 * w + 1] =
                            fmaf(__uint_as_float(x & 0xffff0000u), bt.a[u], acc[8 * h + 2 * w + 1]);
                    }
                }
    };
    constexpr int64_t STEP = 4 * U;            // rows advanced per batch (four waves interleaved)
    Batch b0, b1;
    int64_t k0 = k_begin + wave;
    if (k0 < k_end) load_batch(b0, k0);
    for (; k0 < k_end; k0 += 2 * STEP) {
        if (k0 + STEP < k_end) load_batch(b1, k0 + STEP);
        use_batch(b0);
        if (k0 + STEP >= k_end) break;
        if (k0 + 2 * STEP < k_end) load_batch(b0, k0 + 2 * STEP);
        use_batch(b1);
    }

    // The four waves' partial sums of the same columns, added in wave order.
    __shared__ acc_t red[4][CB];
#pragma unroll
    for (int j = 0; j < CPL; ++j) red[wave][lane * CPL + j] = acc[j];
    __syncthreads();
    acc_t tot[CB / 256];
#pragma unroll
    for (int i = 0; i < CB / 256; ++i) {
        const int c = int(threadIdx.x) + 256 * i;
        tot[i] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < CB / 256; ++i) red[0][int(threadIdx.x) + 256 * i] = tot[i];
    __syncthreads();
    gemv_store<DT, CB>(args, red[0], n0, tn, slice);
}

template <int DT>
__global__ __launch_bounds__(256) void gemv_bt_kernel(KernelArgs args) {
    using acc_t = gemv_acc_t<DT>;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;               // K elements per 16-byte piece
    constexpr int R = 4;                       // columns (stored rows) per wave
    constexpr int CB = 4 * R;                  // columns per workgroup
    const int lane = int(threadIdx.x) & 63;
    const int wave = int(threadIdx.x) >> 6;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    (void)tm;
    const int64_t N = args.N;
    const int64_t n0 = int64_t(tn) * CB;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const uint8_t *const Ab = static_cast<const uint8_t *>(args.A);
    const uint8_t *const Bb = static_cast<const uint8_t *>(args.B);
    const int64_t ldb_b = args.ldb * E;
    bool row_ok[R];
    const uint8_t *brow[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t n = n0 + wave * R + r;
        row_ok[r] = n < N;
        brow[r] = Bb + (row_ok[r] ? n : 0) * ldb_b;
    }

    acc_t acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = acc_t(0);
    // K * E is a multiple of 16 bytes and so are the slice bounds: a piece is wholly in or out.
    for (int64_t k = k_begin + int64_t(lane) * VECE; k < k_end; k += 64 * VECE) {
        const u32x4_t a = *reinterpret_cast<const u32x4_t *>(Ab + k * E);
        u32x4_t b[R];
#pragma unroll
        for (int r = 0; r < R; ++r)
            b[r] = row_ok[r] ? *reinterpret_cast<const u32x4_t *>(brow[r] + k * E) : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if constexpr (DT == DT_I8) {
                    acc[r] = __builtin_amdgcn_sdot4(int(a[w]), int(b[r][w]), acc[r], false);
                } else {
                    // Both bf16 halves widened exactly to fp32, then two fused multiply-adds.
                    acc[r] = fmaf(__uint_as_float(a[w] << 16), __uint_as_float(b[r][w] << 16), acc[r]);
                    acc[r] = fmaf(__uint_as_float(a[w] & 0xffff0000u), __uint_as_float(b[r][w] & 0xffff0000u), acc[r]);
                }
            }
    }
    // Butterfly over the 64 lanes: every lane ends with the wave's sums.
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) acc[r] += __shfl_xor(acc[r], m, 64);
    __shared__ acc_t res[CB];
    if (lane < R) {
        acc_t v = acc[0];
#pragma unroll
        for (int r = 1; r < R; ++r) v = lane == r ? acc[r] : v;
        res[wave * R + lane] = v;
    }
    __syncthreads();
    gemv_store<DT, CB>(args, res, n0, tn, slice);
}

// Sums split-K partials [split][M][N] into C in slice order 0, 1, ... (the
// same fixed order as the in-kernel reduction).
template <int DT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(KernelArgs a) {
    using sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;   // int32 wraps mod 2^32
    const sum_t *__restrict__ ws = static_cast<const sum_t *>(a.workspace);
    const int64_t total = a.M * a.N;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        sum_t s = ws[idx];
        for (int32_t p = 1; p < a.split_k; ++p) s += ws[int64_t(p) * total + idx];
        const int64_t row = idx / a.N, col = idx % a.N;
        write_c<DT>(a, row * a.ldc + col, s);
    }
}

// ---------------------------------------------------------------------------
// Launch: config index -> template instance.
// ---------------------------------------------------------------------------
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

template <int DT, int BM, int BN, int WM, int WN, int WPE>
static hipError_t launch_direct(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    if (a.b_trans)
        hipLaunchKernelGGL((gemm_lds_kernel<DT, BM, BN, WM, WN, WPE, true>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_lds_kernel<DT, BM, BN, WM, WN, WPE, false>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

template <int DT, int BM, int BN, int WM, int WN, int WPE, int NB>
static hipError_t launch_ring(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    if (a.b_trans)
        hipLaunchKernelGGL((gemm_ring_kernel<DT, BM, BN, WM, WN, WPE, true, NB>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_ring_kernel<DT, BM, BN, WM, WN, WPE, false, NB>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

// Column-major B (stored N x K): the element-wise generic kernel and the
// direct-to-LDS kernel, whose B tile then has A's layout.
template <int DT>
static hipError_t launch_config_bt(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    switch (cfg) {
        case 0:
            hipLaunchKernelGGL((gemm_tile_kernel<DT, 64, 64, 2, 2, false, 2, true>), dim3(unsigned(grid)),
                               dim3(256), 0, s, a);
            return hipGetLastError();
        case 1:
            hipLaunchKernelGGL((gemm_tile_kernel<DT, 128, 128, 2, 2, false, 1, true>), dim3(unsigned(grid)),
                               dim3(256), 0, s, a);
            return hipGetLastError();
        case 8: return launch_direct<DT, 256, 256, 2, 2, 1>(a, grid, s);
        case 9: return launch_direct<DT, 128, 256, 2, 2, 1>(a, grid, s);
        case 10: return launch_direct<DT, 256, 256, 2, 4, 2>(a, grid, s);
        case 11: return launch_direct<DT, 256, 256, 4, 2, 2>(a, grid, s);
        case 12: return launch_direct<DT, 128, 256, 2, 4, 2>(a, grid, s);
        case 16: return launch_ring<DT, 256, 256, 2, 4, 2, 4>(a, grid, s);
        case 17: return launch_ring<DT, 256, 256, 4, 2, 2, 4>(a, grid, s);
        case 18: return launch_ring<DT, 128, 256, 2, 4, 2, 5>(a, grid, s);
        case 19: return launch_ring<DT, 256, 256, 2, 2, 1, 4>(a, grid, s);
        case 20: return launch_ring<DT, 32, 64, 1, 2, 2, 8>(a, grid, s);
        case 21: return launch_ring<DT, 64, 64, 1, 2, 2, 8>(a, grid, s);
        case 22: return launch_ring<DT, 32, 128, 1, 4, 2, 8>(a, grid, s);
        case 23: return launch_ring<DT, 64, 128, 1, 4, 2, 8>(a, grid, s);
        case 24: return launch_ring<DT, 32, 256, 1, 4, 1, 6>(a, grid, s);
        case 25: return launch_ring<DT, 64, 256, 1, 4, 1, 6>(a, grid, s);
        case 28: return launch_ring<DT, 32, 256, 1, 4, 2, 4>(a, grid, s);
        case 29: return launch_ring<DT, 32, 128, 1, 4, 2, 6>(a, grid, s);
        case 30: return launch_ring<DT, 64, 128, 1, 4, 2, 5>(a, grid, s);
        case 31: return launch_ring<DT, 128, 128, 2, 2, 2, 4>(a, grid, s);
        case 32: return launch_ring<DT, 128, 128, 2, 2, 2, 8>(a, grid, s);
        case 33: return launch_ring<DT, 128, 128, 2, 4, 2, 8>(a, grid, s);
        case 34: return launch_ring<DT, 256, 256, 4, 2, 2, 5>(a, grid, s);
        case 35: return launch_ring<DT, 256, 256, 2, 4, 2, 5>(a, grid, s);
        case 36: return launch_ring<DT, 256, 256, 2, 2, 1, 5>(a, grid, s);
        case 37: return launch_ring<DT, 128, 256, 2, 2, 2, 3>(a, grid, s);
        case 38: return launch_ring<DT, 256, 128, 2, 2, 2, 3>(a, grid, s);
        case 39: return launch_ring<DT, 128, 256, 1, 4, 2, 3>(a, grid, s);
        case 40: return launch_ring<DT, 128, 256, 2, 4, 4, 3>(a, grid, s);
        case 27:
            hipLaunchKernelGGL((gemv_bt_kernel<DT>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        default: return hipErrorInvalidValue;
    }
}

template <int DT>
static hipError_t launch_config(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    if (a.b_trans) return launch_config_bt<DT>(cfg, a, grid, s);
    switch (cfg) {
        case 0: return launch_tile<DT, 64, 64, 2, 2, false, 2>(a, grid, s);
        case 1: return launch_tile<DT, 128, 128, 2, 2, false, 1>(a, grid, s);
        case 2: return launch_tile<DT, 256, 256, 2, 2, true, 1>(a, grid, s);
        case 3: return launch_tile<DT, 128, 256, 2, 2, true, 1>(a, grid, s);
        case 4: return launch_tile<DT, 256, 128, 2, 2, true, 1>(a, grid, s);
        case 5: return launch_tile<DT, 128, 128, 2, 2, true, 2>(a, grid, s);
        case 6: return launch_tile<DT, 32, 256, 1, 4, true, 2>(a, grid, s);
        case 7: return launch_tile<DT, 64, 256, 1, 4, true, 2>(a, grid, s);
        case 8: return launch_direct<DT, 256, 256, 2, 2, 1>(a, grid, s);
        case 9: return launch_direct<DT, 128, 256, 2, 2, 1>(a, grid, s);
        case 10: return launch_direct<DT, 256, 256, 2, 4, 2>(a, grid, s);
        case 11: return launch_direct<DT, 256, 256, 4, 2, 2>(a, grid, s);
        case 12: return launch_direct<DT, 128, 256, 2, 4, 2>(a, grid, s);
        case 13:
            hipLaunchKernelGGL((gemm_pingpong_kernel<DT>), dim3(unsigned(grid)), dim3(512), 0, s, a);
            return hipGetLastError();
        case 14:
            hipLaunchKernelGGL((gemm_stream_kernel<DT, 32, 4>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        case 15:
            hipLaunchKernelGGL((gemm_stream_kernel<DT, 64, 3>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
        case 16: case 17: case 18: case 19: case 20: case 21: case 22: case 23: case 24: case 25:
        case 28: case 29: case 30: case 31: case 32: case 33: case 34: case 35: case 36: case 37: case 38:
        case 39: case 40:
            return launch_config_bt<DT>(cfg, a, grid, s);   // the ring kernels take either B layout
        case 26:
            hipLaunchKernelGGL((gemv_kernel<DT>), dim3(unsigned(grid)), dim3(256), 0, s, a);
            return hipGetLastError();
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

static int acquire_workspace(hipStream_t stream, size_t partial_bytes, int64_t tiles, void **partials,
                             uint32_t **counters) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return LAUNCH_HIP_ERROR;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    Workspace &w = g_ws[{dev, reinterpret_cast<uintptr_t>(stream)}];
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
    if (w.counter_cap < tiles) {
        if (w.counters != nullptr && hipFreeAsync(w.counters, stream) != hipSuccess) return LAUNCH_HIP_ERROR;
        w.counters = nullptr;
        const int64_t cap = int64_t(grow(size_t(tiles), size_t(w.counter_cap), 4096));
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

int launch_gemm(const KernelArgs &a, int32_t cfg, int64_t grid, void *stream_ptr) {
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    KernelArgs args = a;
    args.workspace = nullptr;
    args.counters = nullptr;
    if (args.split_k > 1) {
        const size_t bytes = size_t(args.split_k) * size_t(args.M) * size_t(args.N) * 4;
        const int64_t tiles = args.reduce_in_kernel ? int64_t(args.tiles_m) * args.tiles_n : 0;
        const int rc = acquire_workspace(stream, bytes, tiles, &args.workspace, &args.counters);
        if (rc != LAUNCH_OK) return rc;
    }
    hipError_t e = args.dtype == DT_I8 ? launch_config<DT_I8>(cfg, args, grid, stream)
                                       : launch_config<DT_BF16>(cfg, args, grid, stream);
    if (e == hipSuccess && args.split_k > 1 && !args.reduce_in_kernel) {
        const int64_t total = args.M * args.N;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        if (args.dtype == DT_I8)   // unsigned adds: int32 partials wrap modulo 2^32, defined
            hipLaunchKernelGGL(splitk_reduce_kernel<DT_I8>, dim3(unsigned(blocks)), dim3(256), 0, stream, args);
        else
            hipLaunchKernelGGL(splitk_reduce_kernel<DT_BF16>, dim3(unsigned(blocks)), dim3(256), 0, stream, args);
        e = hipGetLastError();
    }
    return e == hipSuccess ? LAUNCH_OK : LAUNCH_HIP_ERROR;
}

}  // namespace gemm
