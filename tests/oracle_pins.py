"""Pins of the CPU oracle against facts the mathematics fixes (not against itself).

Each ``pin_*`` function takes a loaded ``oracle.Oracle`` and raises
AssertionError when the oracle disagrees with:

* exact big-integer / rational brute force on tiny inputs,
* closed forms (all-ones, extreme int8 values, an index-structured sum),
* textbook identities (identity and permutation matrices),
* the transpose invariant C^T = B^T A^T (bit-identical),
* split-K linearity, thread-count invariance, the int32 range check,
* numpy's int64 matmul as an independent library GEMM.

The same functions run against deliberately broken oracle builds in
``test_oracle_mutants.py``: each plausible mistake must trip at least one pin.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

from paper_2512_13282_amd import inputs

RNG = np.random.default_rng


def _strided(x: np.ndarray, pad: int) -> np.ndarray:
    """Same values, row stride cols + pad (a view into a wider buffer)."""
    buf = np.zeros((x.shape[0], x.shape[1] + pad), dtype=x.dtype)
    buf[:, : x.shape[1]] = x
    return buf[:, : x.shape[1]]


# ----------------------------------------------------------------------------- int8
def pin_i8_bruteforce_tiny(o):
    """All (M, N, K) in {0..4}^3 against Python big-int sums, mixed strides/threads."""
    rng = RNG(11)
    for M in range(5):
        for N in range(5):
            for K in range(5):
                A = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
                B = rng.integers(-128, 128, size=(K, N), dtype=np.int8)
                pad = (M + N + K) % 3
                Av, Bv = _strided(A, pad), _strided(B, 2 - pad % 2)
                C, ovf = o.gemm_i8_i32(Av, Bv, nthreads=1 + (M % 3), ldc_pad=pad)
                assert ovf == 0
                for i in range(M):
                    for j in range(N):
                        exact = sum(int(A[i, k]) * int(B[k, j]) for k in range(K))
                        assert int(C[i, j]) == exact, (M, N, K, i, j)


def pin_i8_extremes_bruteforce(o):
    """Operands drawn only from {-128, -1, 0, 1, 127} on a ragged shape."""
    rng = RNG(12)
    vals = np.array([-128, -1, 0, 1, 127], dtype=np.int8)
    M, N, K = 7, 9, 13
    A = vals[rng.integers(0, 5, size=(M, K))]
    B = vals[rng.integers(0, 5, size=(K, N))]
    C, _ = o.gemm_i8_i32(A, B, nthreads=3)
    for i in range(M):
        for j in range(N):
            assert int(C[i, j]) == sum(int(A[i, k]) * int(B[k, j]) for k in range(K))


def pin_i8_closed_forms(o):
    """ones.ones = K; (-128)(-128)K = 16384K; (-128)(127)K = -16256K."""
    for K in (1, 5, 64, 1000):
        C, _ = o.gemm_i8_i32(np.ones((3, K), np.int8), np.ones((K, 4), np.int8))
        assert (C == K).all()
        C, _ = o.gemm_i8_i32(np.full((2, K), -128, np.int8), np.full((K, 3), -128, np.int8))
        assert (C == 16384 * K).all()
        C, _ = o.gemm_i8_i32(np.full((2, K), -128, np.int8), np.full((K, 3), 127, np.int8))
        assert (C == -16256 * K).all()
    # the largest K of the workload sweep: 16384 * 14336 = 234,881,024 still fits int32
    C, ovf = o.gemm_i8_i32(np.full((1, 14336), -128, np.int8), np.full((14336, 2), -128, np.int8))
    assert ovf == 0 and (C == 234881024).all()


def pin_i8_index_structured(o):
    """A[i][k] = i - k, B[k][j] = k + 3j (asymmetric in every index), closed form:
    sum_k (i-k)(k+3j) = i*S1 + 3ijK - S2 - 3j*S1, S1 = K(K-1)/2, S2 = (K-1)K(2K-1)/6."""
    M, N, K = 23, 29, 37
    i = np.arange(M)[:, None]
    k = np.arange(K)
    A = (i - k[None, :]).astype(np.int8)
    j = np.arange(N)[None, :]
    B = (k[:, None] + 3 * j).astype(np.int8)
    assert A.min() >= -128 and B.max() <= 127
    C, _ = o.gemm_i8_i32(_strided(A, 5), B, nthreads=4, ldc_pad=3)
    S1, S2 = K * (K - 1) // 2, (K - 1) * K * (2 * K - 1) // 6
    expect = i * S1 + 3 * i * j * K - S2 - 3 * j * S1
    assert (C == expect).all()


def pin_i8_identity_permutation(o):
    """A.I = A, I.B = B, P.B permutes rows of B, A.Q permutes columns of A."""
    rng = RNG(13)
    M, K, N = 17, 19, 11
    A = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
    B = rng.integers(-128, 128, size=(K, N), dtype=np.int8)
    C, _ = o.gemm_i8_i32(A, np.eye(K, dtype=np.int8))
    assert (C == A).all()
    C, _ = o.gemm_i8_i32(np.eye(K, dtype=np.int8), B)
    assert (C == B).all()
    perm = rng.permutation(K)
    P = np.zeros((K, K), np.int8)
    P[np.arange(K), perm] = 1            # (P.B)[r] = B[perm[r]]
    C, _ = o.gemm_i8_i32(P, B)
    assert (C == B[perm]).all()
    Q = np.zeros((K, K), np.int8)
    Q[perm, np.arange(K)] = 1            # (A.Q)[:, c] = A[:, perm[c]]
    C, _ = o.gemm_i8_i32(A, Q)
    assert (C == A[:, perm]).all()


def pin_i8_transpose_invariant(o):
    """C^T == oracle(B^T, A^T), element for element."""
    M, N, K = 31, 45, 53
    A, B = inputs.make_inputs("int8", M, N, K, seed=21)
    C, _ = o.gemm_i8_i32(A, B, nthreads=3)
    Ct, _ = o.gemm_i8_i32(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T), nthreads=5)
    assert (C.T == Ct).all()


def pin_i8_numpy_library(o):
    """Against numpy's int64 matmul on a multi-row, strided, ragged problem."""
    M, N, K = 67, 131, 259
    A, B = inputs.make_inputs("int8", M, N, K, seed=22)
    C, ovf = o.gemm_i8_i32(_strided(A, 9), _strided(B, 3), nthreads=7, ldc_pad=5)
    ref = A.astype(np.int64) @ B.astype(np.int64)
    assert ovf == 0 and (C == ref).all()
    C64 = o.gemm_i8_i64(A, B, nthreads=2, ldc_pad=1)
    assert (C64 == ref).all()


def pin_i8_split_k_linearity(o):
    """oracle(A, B) == oracle(A[:, :s], B[:s]) + oracle(A[:, s:], B[s:])."""
    M, N, K = 12, 14, 100
    A, B = inputs.make_inputs("int8", M, N, K, seed=23)
    C, _ = o.gemm_i8_i32(A, B)
    s = 37
    C1, _ = o.gemm_i8_i32(np.ascontiguousarray(A[:, :s]), np.ascontiguousarray(B[:s]))
    C2, _ = o.gemm_i8_i32(np.ascontiguousarray(A[:, s:]), np.ascontiguousarray(B[s:]))
    assert (C == C1.astype(np.int64) + C2).all()


def pin_i8_thread_invariance(o):
    M, N, K = 29, 33, 41
    A, B = inputs.make_inputs("int8", M, N, K, seed=24)
    ref, _ = o.gemm_i8_i32(A, B, nthreads=1)
    for t in (2, 3, 8, 29, 64):
        C, _ = o.gemm_i8_i32(A, B, nthreads=t)
        assert (C == ref).all(), t


def pin_i8_overflow_detection(o):
    """K = 131072 of (-128)(-128) sums to 2^31 (one past INT32_MAX); K = 131071 fits;
    140000 of (-128)(127) is below INT32_MIN."""
    K = 131072
    C, ovf = o.gemm_i8_i32(np.full((2, K), -128, np.int8), np.full((K, 3), -128, np.int8))
    assert ovf == 6
    assert (C == np.int32(-(2 ** 31))).all()          # 2^31 wrapped modulo 2^32
    C, ovf = o.gemm_i8_i32(np.full((1, K - 1), -128, np.int8), np.full((K - 1, 1), -128, np.int8))
    assert ovf == 0 and int(C[0, 0]) == 16384 * (K - 1) == 2147467264
    K = 140000
    C, ovf = o.gemm_i8_i32(np.full((1, K), -128, np.int8), np.full((K, 2), 127, np.int8))
    assert ovf == 2
    assert int(C[0, 0]) == ((-16256 * K + 2 ** 31) % 2 ** 32) - 2 ** 31
    C64 = o.gemm_i8_i64(np.full((1, K), -128, np.int8), np.full((K, 2), 127, np.int8))
    assert (C64 == -16256 * K).all()


def pin_freivalds(o):
    """Freivalds accepts the exact product and rejects any single wrong element."""
    M, N, K = 40, 50, 60
    A, B = inputs.make_inputs("int8", M, N, K, seed=25)
    ref = (A.astype(np.int64) @ B.astype(np.int64)).astype(np.int32)
    assert o.freivalds_i8_i32(A, B, ref, trials=3) == 0
    for (i, j) in ((0, 0), (M - 1, N - 1), (17, 3)):
        bad = ref.copy()
        bad[i, j] += 1
        assert o.freivalds_i8_i32(A, B, bad, trials=2) > 0, (i, j)
    # a strided C view is read with its own stride
    wide = np.zeros((M, N + 7), np.int32)
    wide[:, :N] = ref
    assert o.freivalds_i8_i32(A, B, wide[:, :N], trials=2) == 0


# ----------------------------------------------------------------------------- bf16
def _frac_bf16(bits: int) -> Fraction:
    return Fraction(float(inputs.f32_from_bf16_bits(np.array([bits], np.uint16))[0]))


def pin_bf16_widening(o):
    """Known bf16 encodings: sign, exponent bias 127, 7 fraction bits."""
    cases = {0x3F80: 1.0, 0xC000: -2.0, 0x3FC0: 1.5, 0x4049: 3.140625, 0x0000: 0.0,
             0x7F7F: (2 - 2 ** -7) * 2.0 ** 127, 0x0080: 2.0 ** -126, 0x0001: 2.0 ** -133,
             0x3B80: 2.0 ** -8, 0xBF81: -(1 + 2 ** -7)}
    for bits, val in cases.items():
        assert o.bf16_to_double(bits) == val, hex(bits)
    assert math.copysign(1.0, o.bf16_to_double(0x8000)) == -1.0


def pin_bf16_exact_rational_tiny(o):
    """All (M, N, K) in {0..4}^3: |oracle - exact| <= (K-1) u sum|ab|, u = 2^-53
    (recursive-summation bound; products are exact), exact sums by Fraction."""
    rng = RNG(31)
    for M in range(5):
        for N in range(5):
            for K in range(5):
                A = inputs.bf16_bits_from_f32(rng.standard_normal((M, K), dtype=np.float32) * 3)
                B = inputs.bf16_bits_from_f32(rng.standard_normal((K, N), dtype=np.float32) * 3)
                C = o.gemm_bf16_f64(_strided(A, 1), B, nthreads=2, ldc_pad=K % 2)
                for i in range(M):
                    for j in range(N):
                        terms = [_frac_bf16(int(A[i, k])) * _frac_bf16(int(B[k, j])) for k in range(K)]
                        exact = sum(terms, Fraction(0))
                        bound = max(K - 1, 0) * Fraction(1, 2 ** 53) * sum(abs(t) for t in terms)
                        assert abs(Fraction(float(C[i, j])) - exact) <= bound, (M, N, K, i, j)


def pin_bf16_exact_rational_wide_range(o):
    """Products spanning ~2^60 of dynamic range, where an fp32 accumulator would lose
    terms: fp64 must stay within its bound of the exact rational sum."""
    rng = RNG(32)
    M, N, K = 5, 6, 24
    A32 = (rng.standard_normal((M, K)) * np.exp2(rng.integers(-30, 30, size=(M, K)))).astype(np.float32)
    B32 = (rng.standard_normal((K, N)) * np.exp2(rng.integers(-30, 30, size=(K, N)))).astype(np.float32)
    A, B = inputs.bf16_bits_from_f32(A32), inputs.bf16_bits_from_f32(B32)
    C = o.gemm_bf16_f64(A, B)
    for i in range(M):
        for j in range(N):
            terms = [_frac_bf16(int(A[i, k])) * _frac_bf16(int(B[k, j])) for k in range(K)]
            exact = sum(terms, Fraction(0))
            bound = (K - 1) * Fraction(1, 2 ** 53) * sum(abs(t) for t in terms)
            assert abs(Fraction(float(C[i, j])) - exact) <= bound, (i, j)


def pin_bf16_integer_exact(o):
    """Integer-valued bf16 operands: every sum is an exact integer, equal to the int64 GEMM."""
    M, N, K = 19, 23, 301
    A = inputs.small_int_bf16_matrix(M, K, seed=33)
    B = inputs.small_int_bf16_matrix(K, N, seed=34)
    C = o.gemm_bf16_f64(A, B, nthreads=3)
    Ai = inputs.f32_from_bf16_bits(A).astype(np.int64)
    Bi = inputs.f32_from_bf16_bits(B).astype(np.int64)
    assert (C == (Ai @ Bi).astype(np.float64)).all()


def pin_bf16_closed_forms(o):
    one = int(inputs.bf16_bits_from_f32(np.array([1.0], np.float32))[0])
    mhalf = int(inputs.bf16_bits_from_f32(np.array([-0.5], np.float32))[0])
    for K in (1, 7, 256, 4097):
        C = o.gemm_bf16_f64(np.full((2, K), one, np.uint16), np.full((K, 3), one, np.uint16))
        assert (C == K).all()
        C = o.gemm_bf16_f64(np.full((2, K), mhalf, np.uint16), np.full((K, 3), one, np.uint16))
        assert (C == -0.5 * K).all()


def pin_bf16_identity_permutation(o):
    M, K, N = 9, 12, 10
    A, B = inputs.make_inputs("bf16", M, N, K, seed=35)
    one = int(inputs.bf16_bits_from_f32(np.array([1.0], np.float32))[0])
    eye = np.where(np.eye(K, dtype=bool), one, 0).astype(np.uint16)
    C = o.gemm_bf16_f64(A, eye)
    assert (C == inputs.f32_from_bf16_bits(A).astype(np.float64)).all()
    C = o.gemm_bf16_f64(eye, B)
    assert (C == inputs.f32_from_bf16_bits(B).astype(np.float64)).all()
    perm = RNG(36).permutation(K)
    P = np.zeros((K, K), np.uint16)
    P[np.arange(K), perm] = one
    C = o.gemm_bf16_f64(P, B)
    assert (C == inputs.f32_from_bf16_bits(B[perm]).astype(np.float64)).all()


def pin_bf16_transpose_invariant(o):
    """Same products (multiplication commutes), same k order: bit-identical."""
    M, N, K = 21, 34, 77
    A, B = inputs.make_inputs("bf16", M, N, K, seed=37)
    C = o.gemm_bf16_f64(A, B, nthreads=2)
    Ct = o.gemm_bf16_f64(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T), nthreads=3)
    assert np.array_equal(C.T.view(np.uint64), Ct.view(np.uint64))


def pin_bf16_sequential_order(o):
    """The fp64 sum runs k ascending: reversing k changes some results, and the
    oracle matches the ascending left-to-right sum bit for bit."""
    M, N, K = 3, 4, 50
    A, B = inputs.make_inputs("bf16", M, N, K, seed=38)
    C = o.gemm_bf16_f64(A, B)
    Af = inputs.f32_from_bf16_bits(A).astype(np.float64)
    Bf = inputs.f32_from_bf16_bits(B).astype(np.float64)
    for i in range(M):
        for j in range(N):
            s = 0.0
            for k in range(K):
                s += Af[i, k] * Bf[k, j]
            assert C[i, j] == s


# ----------------------------------------------------------------------------- column-major B
def pin_i8_bt_bruteforce_tiny(o):
    """C = A Bt^T with Bt stored N x K: all (M, N, K) in {0..3}^3 (square shapes included,
    where a missing transpose would still type-check) against Python big-int sums."""
    rng = RNG(61)
    for M in range(4):
        for N in range(4):
            for K in range(4):
                A = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
                Bt = rng.integers(-128, 128, size=(N, K), dtype=np.int8)
                C, ovf = o.gemm_i8_i32_bt(A, Bt)
                assert ovf == 0 and C.shape == (M, N)
                for i in range(M):
                    for j in range(N):
                        exact = sum(int(A[i, k]) * int(Bt[j, k]) for k in range(K))
                        assert int(C[i, j]) == exact, (M, N, K, i, j)
    A = rng.integers(-128, 128, size=(6, 9), dtype=np.int8)
    Bt = rng.integers(-128, 128, size=(5, 9), dtype=np.int8)
    C = o.gemm_i8_i32_bt(A, Bt)[0]
    assert o.freivalds_i8_i32_bt(A, Bt, C) == 0
    C[2, 3] += 1
    assert o.freivalds_i8_i32_bt(A, Bt, C) > 0


def pin_bf16_bt_exact_rational_tiny(o):
    """bf16 C = A Bt^T on small shapes within the fp64 summation bound of the exact sum."""
    rng = RNG(62)
    for (M, N, K) in ((1, 1, 1), (3, 3, 3), (2, 5, 4), (4, 2, 7)):
        A = inputs.bf16_bits_from_f32(rng.standard_normal((M, K), dtype=np.float32) * 3)
        Bt = inputs.bf16_bits_from_f32(rng.standard_normal((N, K), dtype=np.float32) * 3)
        C = o.gemm_bf16_f64_bt(A, Bt)
        for i in range(M):
            for j in range(N):
                terms = [_frac_bf16(int(A[i, k])) * _frac_bf16(int(Bt[j, k])) for k in range(K)]
                exact = sum(terms, Fraction(0))
                bound = max(K - 1, 0) * Fraction(1, 2 ** 53) * sum(abs(t) for t in terms)
                assert abs(Fraction(float(C[i, j])) - exact) <= bound, (M, N, K, i, j)


# ----------------------------------------------------------------------------- reduced-precision outputs
def _i32_values(s: int, rng) -> list[int]:
    """int32 values around the rounding and saturation boundaries of shift s."""
    d = 2 ** s
    cand = [0, 1, -1, 2, -2, 127, 128, -128, -129, 32767, 32768, -32768, -32769, 2 ** 31 - 1, -2 ** 31]
    for m in range(-5, 6):
        for off in (-1, 0, 1):
            cand += [m * d + d // 2 + off, m * d + off, 127 * d + off, -128 * d + off,
                     32767 * d + d // 2 + off, -32768 * d - d // 2 + off]
    cand += [int(x) for x in rng.integers(-2 ** 31, 2 ** 31, size=200)]
    return [v for v in cand if -2 ** 31 <= v < 2 ** 31]


def pin_requant_exact_rational(o):
    """int32 -> int8 / int16 for every shift 0..31 against exact rational rounding to the
    nearest integer, ties to even (Python's round of a Fraction), then saturation."""
    rng = RNG(31)
    for s in range(32):
        vals = _i32_values(s, rng)
        arr = np.array(vals, dtype=np.int32)
        for bits in (8, 16):
            lo, hi = -(2 ** (bits - 1)), 2 ** (bits - 1) - 1
            got = o.requant_i32(arr, s, bits)
            assert got.dtype == (np.int8 if bits == 8 else np.int16)
            for v, g in zip(vals, got.tolist()):
                ref = min(hi, max(lo, round(Fraction(v, 2 ** s))))
                assert g == ref, (v, s, bits, g, ref)


def pin_requant_closed_forms(o):
    """Hand-checked cases: halves go to the even neighbour, both signs; saturation at both ends."""
    cases = [  # (value, shift, bits, expected)
        (1, 1, 8, 0), (3, 1, 8, 2), (5, 1, 8, 2), (7, 1, 8, 4), (-1, 1, 8, 0), (-3, 1, 8, -2),
        (-5, 1, 8, -2), (6, 2, 8, 2), (10, 2, 8, 2), (14, 2, 8, 4), (-6, 2, 8, -2), (9, 2, 8, 2),
        (255, 1, 8, 127), (-257, 1, 8, -128), (256, 1, 8, 127), (-256, 1, 8, -128), (-255, 1, 8, -128),
        (2 ** 31 - 1, 0, 16, 32767), (-2 ** 31, 0, 16, -32768), (-2 ** 31, 31, 8, -1),
        (2 ** 31 - 1, 31, 8, 1), (2 ** 30, 31, 8, 0), (3 * 2 ** 29, 31, 8, 1), (234881024, 20, 8, 127),
        (234881024, 20, 16, 224), (-234881024, 22, 16, -56), (100, 0, 8, 100), (-100, 0, 16, -100),
    ]
    for v, s, bits, want in cases:
        got = int(o.requant_i32(np.array([v], dtype=np.int32), s, bits)[0])
        assert got == want, (v, s, bits, got, want)


def _bf16_rne_from_f32_bits(f: np.ndarray) -> np.ndarray:
    """Round finite binary32 values to bf16, ties to even, on their bit patterns."""
    u = f.astype(np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def pin_bf16_round_fp32_values(o):
    """For values that are binary32 numbers, rounding the double equals rounding the binary32
    bit pattern (an independent formulation), across normal and subnormal magnitudes."""
    rng = RNG(32)
    f = np.concatenate([
        rng.standard_normal(4000).astype(np.float32) * np.float32(1000),
        (rng.standard_normal(1000) * 2.0 ** rng.integers(-140, 120, size=1000)).astype(np.float32),
        np.array([1.0, -1.0, 3.0, 0.1, 1e30, -1e-40, 1e-45], dtype=np.float32),
    ])
    f = f[np.isfinite(f)]
    got = o.round_bf16(f.astype(np.float64))
    assert np.array_equal(got, _bf16_rne_from_f32_bits(f))


def pin_bf16_round_exact_rational(o):
    """Doubles that are not binary32 numbers (sums of bf16 products) against exact rational
    rounding to 8 significant bits, ties to even."""
    rng = RNG(33)
    xs = list(rng.standard_normal(2000) * 300.0) + [1 + 2 ** -8 + 2 ** -40, 1 + 2 ** -8 - 2 ** -40,
                                                     -(3 + 2 ** -6 + 2 ** -50), 2 ** -130 * 1.75]
    for x in xs:
        bits = o.bf16_from_double(float(x))
        fr = Fraction(float(x))
        sign = -1 if fr < 0 else 1
        a = abs(fr)
        e = a.numerator.bit_length() - a.denominator.bit_length()
        if Fraction(2) ** e > a:
            e -= 1
        ulp = Fraction(2) ** max(e - 7, -133)
        ref = sign * round(a / ulp) * ulp
        got = Fraction(o.bf16_to_double(bits))
        assert got == ref, (x, hex(bits), float(ref))


def pin_bf16_round_specials(o):
    """Ties, signed zero, the largest finite value, overflow, and the subnormal range."""
    cases = [
        (1.0, 0x3F80), (1 + 2 ** -8, 0x3F80), (1 + 3 * 2 ** -8, 0x3F82), (-(1 + 2 ** -8), 0xBF80),
        (1 + 2 ** -7, 0x3F81), (2 - 2 ** -8, 0x4000), (0.0, 0x0000), (-0.0, 0x8000),
        (float.fromhex("0x1.fcp127"), 0x7F7E), (float.fromhex("0x1.fep127"), 0x7F7F),
        (float.fromhex("0x1.fefffp127"), 0x7F7F), (float.fromhex("0x1.ffp127"), 0x7F80),
        (-float.fromhex("0x1.ffp127"), 0xFF80), (float.fromhex("0x1.fdp127"), 0x7F7E),
        (2.0 ** -133, 0x0001), (2.0 ** -134, 0x0000), (3 * 2.0 ** -134, 0x0002),
        (2.0 ** -126, 0x0080), (-(2.0 ** -133), 0x8001),
    ]
    for x, want in cases:
        got = o.bf16_from_double(x)
        assert got == want, (x, hex(got), hex(want))


def pin_bf16_round_nan_inf(o):
    """Infinities keep their sign; a NaN (either sign) rounds to a NaN: all-ones exponent,
    non-zero significand (IEEE 754 rounding never turns a NaN into a number)."""
    assert o.bf16_from_double(math.inf) == 0x7F80
    assert o.bf16_from_double(-math.inf) == 0xFF80
    for x in (math.nan, -math.nan, float(np.float32(np.nan))):
        b = o.bf16_from_double(x)
        assert (b & 0x7F80) == 0x7F80 and (b & 0x007F) != 0, hex(b)


PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
