// kern_tile.h -- register-staged tile kernels: GENERIC (element-wise loads,
// any alignment) and MACRO / SKINNY (16-byte buffer loads, B transposed in
// registers).
#pragma once

#include "gemm_common.h"

namespace gemm {

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

    // Every wave is past its last fragment read when store_tile first synchronises, so
    // the last-slice flag borrows a word of the operand buffers (a separate __shared__
    // word would take the 64 x 256 tile past half of the CU's LDS).
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane,
                                   *reinterpret_cast<int *>(smem));
}

}  // namespace gemm
