"""Pins for the CPU oracle: printed tables, Eq. 5, brute force, closed forms and exact-rounding checks.

Every check here compares the oracle with something other than itself: the values the paper prints
(Table 5, Table 6), the mathematics (brute-force dot products with Python integers, exact rationals,
closed forms, invariances) or hand-computed positions from the written layout definitions.
"""
import itertools
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import bitnet_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return [line.split() for line in fh if line.strip() and not line.startswith("#")]


def _nearest_f32(exact: Fraction, got: np.float32) -> bool:
    """True when got is the round-to-nearest-even float32 of the exact rational."""
    g = Fraction(float(got))
    up = Fraction(float(np.nextafter(got, np.float32(np.inf))))
    dn = Fraction(float(np.nextafter(got, np.float32(-np.inf)))) if got > 0 else Fraction(0)
    d = abs(g - exact)
    for nb in (up, dn):
        dn_ = abs(nb - exact)
        if dn_ < d:
            return False
        if dn_ == d and nb != g:
            # tie: the chosen value must have an even significand
            bits = int(np.float32(got).view(np.uint32))
            if bits & 1:
                return False
    return True


# ---------------------------------------------------------------------------------------------
# Table 5 and Table 6
# ---------------------------------------------------------------------------------------------
def test_tl1_codes_match_table5():
    rows = _rows("tl1_table5.txt")
    assert len(rows) == 9
    for w0, w1, bits in rows:
        code = int(O.tl1_code(int(w0), int(w1)))
        assert code == int(bits, 2), (w0, w1, bits)
        # the TL1 table entry enumerated for this code multiplies the pair by exactly (w0, w1)
        assert (code // 3 - 1, code % 3 - 1) == (int(w0), int(w1))


def test_tl2_codes_match_table6_printed_rows():
    rows = _rows("tl2_table6.txt")
    assert len(rows) == 9
    for w0, w1, w2, sbit, bits in rows:
        idx, sign = O.tl2_codes(int(w0), int(w1), int(w2))
        assert int(idx) == int(bits, 2), (w0, w1, w2)
        assert int(sign) == int(sbit), (w0, w1, w2)


def test_tl2_mirror_consolidation_all_27():
    seen = set()
    for t in itertools.product((-1, 0, 1), repeat=3):
        idx, sign = (int(v) for v in O.tl2_codes(*t))
        assert 0 <= idx <= 13
        seen.add((idx, sign))
        nidx, nsign = (int(v) for v in O.tl2_codes(*(-v for v in t)))
        assert nidx == idx
        if any(t):
            assert nsign == 1 - sign
        else:
            assert (idx, sign, nsign) == (0, 0, 0)
        # the digits of the index times the sign give back the triple
        d = O.balanced_ternary_digits(idx)
        assert tuple(-v if sign else v for v in d) == t
    assert len(seen) == 27          # a bijection onto the 27 used (index, sign) pairs
    # ceil(3^3 / 2) = 14 table entries fit a 4-bit index (Sec. 3.1.1)
    assert max(i for i, _ in seen) == 13


def test_balanced_ternary_representatives():
    for i in range(14):
        d0, d1, d2 = O.balanced_ternary_digits(i)
        assert 9 * d0 + 3 * d1 + d2 == i
        lead = next((v for v in (d0, d1, d2) if v), 0)
        assert lead >= 0              # mirror representative: leading digit non-negative
    with pytest.raises(ValueError):
        O.balanced_ternary_digits(14)


# ---------------------------------------------------------------------------------------------
# Eq. 5 sign operation
# ---------------------------------------------------------------------------------------------
def test_sign_op_exhaustive_int16():
    x = np.arange(-32767, 32768, dtype=np.int64)
    assert np.array_equal(O.sign_op(x, np.zeros_like(x)), x)
    assert np.array_equal(O.sign_op(x, np.ones_like(x)), -x)


# ---------------------------------------------------------------------------------------------
# MAD accumulation: brute force and closed forms
# ---------------------------------------------------------------------------------------------
@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 6])
def test_mad_brute_force_all_ternary_rows(K):
    rng = np.random.default_rng(100 + K)
    t = np.array(list(itertools.product((-1, 0, 1), repeat=K)), dtype=np.int8)
    xq = rng.integers(-128, 128, size=(3, K), dtype=np.int64).astype(np.int8)
    acc = O.mad_gemm(xq, t)
    for m in range(3):
        a = [int(v) for v in xq[m]]
        for n in range(t.shape[0]):
            ref = sum(a[k] * int(t[n, k]) for k in range(K))
            assert int(acc[m, n]) == ref


def test_mad_largest_k_against_python_integers():
    # the longest rows the library accepts, with the extreme codes -128 and 127: exact sums of Python integers
    rng = np.random.default_rng(11)
    K = 132096
    xq = rng.choice(np.array([-128, 127, -1, 0, 1], dtype=np.int8), size=(2, K))
    t = np.stack([np.ones(K, np.int8), -np.ones(K, np.int8), rng.integers(-1, 2, size=K).astype(np.int8),
                  np.sign(xq[0]).astype(np.int8)])
    acc = O.mad_gemm(xq, t)
    for m in range(2):
        a = [int(v) for v in xq[m]]
        for n in range(t.shape[0]):
            w = [int(v) for v in t[n]]
            assert int(acc[m, n]) == sum(p * q for p, q in zip(a, w))
    assert int(acc[0, 3]) == sum(abs(int(v)) for v in xq[0])


def test_mad_closed_forms():
    rng = np.random.default_rng(7)
    M, N, K = 4, 32, 320
    xq = rng.integers(-127, 128, size=(M, K)).astype(np.int8)
    ones = np.ones((N, K), dtype=np.int8)
    assert np.array_equal(O.mad_gemm(xq, ones), np.repeat(xq.astype(np.int64).sum(1)[:, None], N, 1))
    assert not O.mad_gemm(xq, np.zeros((N, K), np.int8)).any()
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    acc = O.mad_gemm(xq, t)
    assert np.array_equal(O.mad_gemm(xq, -t), -acc)
    split = 128
    assert np.array_equal(O.mad_gemm(xq[:, :split], t[:, :split]).astype(np.int64)
                          + O.mad_gemm(xq[:, split:], t[:, split:]), acc)
    assert np.abs(acc).max() <= 127 * K
    # zero-weight padding changes nothing
    tp = np.concatenate([t, np.zeros((N, 64), np.int8)], 1)
    xp = np.concatenate([xq, rng.integers(-127, 128, size=(M, 64)).astype(np.int8)], 1)
    assert np.array_equal(O.mad_gemm(xp, tp), acc)


# ---------------------------------------------------------------------------------------------
# Packing: hand-computed positions, round trips, sizes
# ---------------------------------------------------------------------------------------------
def test_i2s_positions_hand_computed():
    N, K = 32, 320      # one full 256-k block and a 64-k block
    cases = {           # (n, k): (byte, shift), worked out by hand from the layout definition
        (0, 0): (0, 0), (0, 5): (1, 2), (1, 0): (16, 0), (0, 16): (256, 0), (0, 64): (4, 0),
        (0, 256): (1024, 0), (3, 300): (1164, 6), (16, 0): (1280, 0), (17, 0): (1296, 0), (0, 255): (4 * 4 * 48 + 12 + 3, 6),
    }
    for (n, k), (byte, shift) in cases.items():
        b, s = O.i2s_position(n, k, N, K)
        assert (int(b), int(s)) == (byte, shift), (n, k)


def test_tl2_positions_hand_computed():
    N, K = 16, 448      # ThreeK = 384, TwoK = 64
    assert O.tl2_split(K) == (384, 64)
    cases = {(0, 0): (0, 0, 1024, 0), (0, 1): (0, 4, 1024, 1), (2, 33): (288, 4, 1096, 1)}
    for (n, g), exp in cases.items():
        got = tuple(int(v) for v in O.tl2_idx_position(n, g, N, K))
        assert got == exp, (n, g)
    assert tuple(int(v) for v in O.tl1_tail_position(0, 0, N, K)) == (1280, 0)
    assert tuple(int(v) for v in O.tl1_tail_position(1, 9, N, K)) == (1348, 4)


def test_tl1_positions_hand_computed():
    N, K = 32, 320      # one full 256-k block and a 64-k block
    cases = {           # (n, pair): (byte, shift), worked out by hand from the layout definition
        (0, 0): (0, 0), (0, 1): (1, 0), (0, 4): (0, 4), (0, 7): (3, 4), (1, 0): (16, 0), (0, 8): (256, 0),
        (0, 32): (4, 0), (0, 128): (1024, 0), (3, 150): (1166, 4), (16, 0): (1280, 0), (17, 0): (1296, 0),
    }
    for (n, pr), (byte, shift) in cases.items():
        b, sh = O.tl1_pair_position(n, pr, N, K)
        assert (int(b), int(sh)) == (byte, shift), (n, pr)


@pytest.mark.parametrize("N,K", [(16, 64), (32, 320), (16, 1600)])
def test_tl1_round_trip_every_nibble_once(N, K):
    rng = np.random.default_rng(N + 13 * K)
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    p = O.pack_tl1(t)
    assert p.size * 8 == 2 * N * K                    # 4 bits per pair: 2 bits per weight (Table 1, TL1)
    assert np.array_equal(O.unpack_tl1(p, N, K), t)
    nn, pp = np.meshgrid(np.arange(N), np.arange(K // 2), indexing="ij")
    b, sh = O.tl1_pair_position(nn, pp, N, K)
    nib = b.ravel() * 2 + sh.ravel() // 4
    assert np.unique(nib).size == N * K // 2 and nib.max() == N * K // 2 - 1
    codes = O.tl1_decode_codes(p, N, K)
    assert np.array_equal(codes, O.tl1_code(t[:, 0::2], t[:, 1::2]))   # Table 5 code of every pair


@pytest.mark.parametrize("N,K", [(16, 64), (16, 128), (32, 192), (16, 256), (48, 320), (16, 384),
                                 (32, 448), (16, 832), (32, 1600)])
def test_pack_round_trips_and_sizes(N, K):
    rng = np.random.default_rng(N * 10007 + K)
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    p = O.pack_i2s(t)
    assert p.size == N * K // 4                       # 2 bits per weight (Table 1)
    assert np.array_equal(O.unpack_i2s(p, N, K), t)
    assert not np.any((p[:, None] >> np.array([0, 2, 4, 6], np.uint8)) & 3 == 3)
    q = O.pack_tl2(t)
    three, two = O.tl2_split(K)
    assert three % 384 == 0 and three + two == K and 0 <= two < 384
    # 5 bits per 3 weights for the TL2 part (Sec. 3.1.1), 4 bits per 2 weights for the TL1 tail
    assert q.size * 8 == N * (three * 5 // 3 + two * 2)
    assert np.array_equal(O.unpack_tl2(q, N, K), t)


def test_pack_writes_every_position_once():
    N, K = 32, 448
    nn, kk = np.meshgrid(np.arange(N), np.arange(K), indexing="ij")
    b, s = O.i2s_position(nn, kk, N, K)
    slots = b.ravel() * 4 + s.ravel() // 2
    assert np.unique(slots).size == N * K and slots.max() == N * K - 1
    three, two = O.tl2_split(K)
    nn, gg = np.meshgrid(np.arange(N), np.arange(three // 3), indexing="ij")
    ib, ish, sb, sbit = O.tl2_idx_position(nn, gg, N, K)
    nib = ib.ravel() * 2 + ish.ravel() // 4
    bits = sb.ravel() * 8 + sbit.ravel()
    nn, pp = np.meshgrid(np.arange(N), np.arange(two // 2), indexing="ij")
    tb, tsh = O.tl1_tail_position(nn, pp, N, K)
    tnib = tb.ravel() * 2 + tsh.ravel() // 4
    assert np.unique(nib).size == nib.size and nib.max() < 2 * N * three // 6
    assert np.unique(bits).size == bits.size
    assert bits.min() == 8 * N * three // 6 and bits.max() < 8 * (N * three // 6 + N * three // 24)
    assert np.unique(tnib).size == tnib.size and tnib.max() == 2 * O.tl2_packed_bytes(N, K) - 1


def test_table3_bits_per_weight():
    # element-wise bpw with mirror consolidation: (ceil(log2(ceil(C^g / 2))) + 1) / g
    def bpw_mirror(C, g):
        return (math.ceil(math.log2(math.ceil(C ** g / 2))) + 1) / g

    def bpw_plain(C, g):
        return math.ceil(math.log2(C ** g)) / g

    assert round(bpw_mirror(3, 3), 2) == 1.67      # TL2
    assert bpw_plain(3, 2) == 2.0                  # TL1
    assert bpw_plain(4, 2) == 2.0
    assert bpw_mirror(5, 2) == 2.5


# ---------------------------------------------------------------------------------------------
# ELUT route equals MAD (Eq. 1 == Eq. 3)
# ---------------------------------------------------------------------------------------------
@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (3, 16, 384), (2, 32, 448), (1, 16, 832), (4, 48, 1600),
                                   (2, 16, 4096)])
def test_elut_equals_mad(M, N, K):
    rng = np.random.default_rng(M * 31 + N * 7 + K)
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    xq = rng.integers(-127, 128, size=(M, K)).astype(np.int8)
    packed = O.pack_tl2(t)
    assert np.array_equal(O.elut_gemm(xq, packed, N, K), O.mad_gemm(xq, t))


@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (3, 32, 320), (2, 16, 1600)])
def test_elut_tl1_equals_mad(M, N, K):
    rng = np.random.default_rng(M * 17 + N * 5 + K)
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    xq = rng.integers(-128, 128, size=(M, K)).astype(np.int8)
    assert np.array_equal(O.elut_gemm_tl1(xq, O.pack_tl1(t), N, K), O.mad_gemm(xq, t))


def test_tl1_tables_are_enumerations():
    rng = np.random.default_rng(5)
    xq = rng.integers(-128, 128, size=(2, 64)).astype(np.int8)
    lut = O.tl1_tables(xq)
    assert lut.shape == (2, 32, 9)
    for m in range(2):
        for p in (0, 17, 31):
            b = [int(v) for v in xq[m, 2 * p:2 * p + 2]]
            for t in itertools.product((-1, 0, 1), repeat=2):
                assert int(lut[m, p, int(O.tl1_code(*t))]) == b[0] * t[0] + b[1] * t[1]


def test_elut_tables_are_enumerations():
    rng = np.random.default_rng(3)
    xq = rng.integers(-127, 128, size=(2, 448)).astype(np.int8)
    lut, lut1 = O.elut_tables(xq)
    assert lut.shape == (2, 128, 14) and lut1.shape == (2, 32, 9)
    for m in range(2):
        for g in (0, 5, 127):
            a = [int(v) for v in xq[m, 3 * g:3 * g + 3]]
            for t in itertools.product((-1, 0, 1), repeat=3):
                idx, sign = (int(v) for v in O.tl2_codes(*t))
                val = int(O.sign_op(lut[m, g, idx], sign))
                assert val == sum(x * w for x, w in zip(a, t))
        for p in (0, 31):
            b = [int(v) for v in xq[m, 384 + 2 * p:384 + 2 * p + 2]]
            for t in itertools.product((-1, 0, 1), repeat=2):
                assert int(lut1[m, p, int(O.tl1_code(*t))]) == b[0] * t[0] + b[1] * t[1]
    assert np.abs(lut).max() <= 3 * 127


# ---------------------------------------------------------------------------------------------
# Exact rational rounding, beta and ternarisation
# ---------------------------------------------------------------------------------------------
def test_f32_from_rational_exact_and_ties():
    rng = np.random.default_rng(11)
    vals = np.concatenate([rng.standard_normal(200).astype(np.float32) ** 2,
                           np.array([1e-45, 3e-39, 1.1754944e-38, 1.0, 3.4e38], np.float32)])
    for v in vals:
        fr = Fraction(float(v))
        assert O.f32_from_rational(fr.numerator, fr.denominator) == v
        up = np.nextafter(v, np.float32(np.inf))
        mid = (fr + Fraction(float(up))) / 2
        got = O.f32_from_rational(mid.numerator, mid.denominator)
        assert _nearest_f32(mid, got)
        even = v if (int(v.view(np.uint32)) & 1) == 0 else up
        assert got == even
    for _ in range(200):
        num, den = int(rng.integers(1, 2**62)), int(rng.integers(1, 2**62))
        got = O.f32_from_rational(num, den)
        assert _nearest_f32(Fraction(num, den), got)


@pytest.mark.parametrize("shape", [(1, 7), (16, 64), (33, 65), (64, 320)])
def test_beta_is_nearest_f32_of_exact_mean(shape):
    rng = np.random.default_rng(sum(shape))
    W = (rng.standard_normal(shape) * 0.02).astype(np.float32)
    exact = sum(Fraction(float(abs(w))) for w in W.ravel()) / W.size
    beta = O.absmean_beta(W)
    assert _nearest_f32(exact, beta)


def test_beta_constructed_cases():
    one = np.float32(1.0)
    e = np.float32(2.0 ** -23)
    assert O.absmean_beta(np.array([[1.0, -1.0, 1.0, -1.0]], np.float32)) == 1.0
    # exact mean 1 + 2^-24: a tie between 1 and 1 + 2^-23, resolved to the even 1.0
    assert O.absmean_beta(np.array([[one, one + e]], np.float32)) == one
    # exact mean 1 + 1.5 * 2^-23: a tie resolved upward to the even 1 + 2^-22
    assert O.absmean_beta(np.array([[one + e, one + 2 * e]], np.float32)) == one + 2 * e
    # subnormal: half of the smallest subnormal ties to zero
    assert O.absmean_beta(np.array([[1e-45, 0.0]], np.float32)) == 0.0
    # a large value next to many small ones: a sequential fp32 sum loses the small ones, the exact mean does not
    W = np.full((1, 1 << 16), np.float32(2.0 ** -30))
    W[0, 0] = np.float32(1.0)
    exact = (Fraction(1) + Fraction((1 << 16) - 1, 2**30)) / (1 << 16)
    assert _nearest_f32(exact, O.absmean_beta(W))


def test_ternarize_ties_and_scaling():
    W = np.array([[0.5, -0.5, 1.5, -1.5]], np.float32)      # beta = 1 exactly
    t, beta = O.ternarize(W)
    assert beta == 1.0
    assert t.tolist() == [[0, 0, 1, -1]]                    # half-even: 0.5 -> 0, 1.5 -> 2 -> clamp 1
    rng = np.random.default_rng(5)
    W = (rng.standard_normal((32, 256)) * 0.02).astype(np.float32)
    t, beta = O.ternarize(W)
    for k in (-3, 4):
        t2, b2 = O.ternarize(W * np.float32(2.0 ** k))
        assert b2 == beta * np.float32(2.0 ** k)
        assert np.array_equal(t2, t)
    # each ratio is the correctly rounded fp32 quotient
    r = W / beta
    for w, rv in zip(W.ravel()[:64], r.ravel()[:64]):
        assert _nearest_f32(abs(Fraction(float(w))) / Fraction(float(beta)), np.float32(abs(rv)))
    z, bz = O.ternarize(np.zeros((4, 8), np.float32))
    assert bz == 0 and not z.any()


def test_ternarize_zero_fraction_matches_gaussian():
    # t = 0 iff |w| < beta/2 with beta ~ sigma*sqrt(2/pi): P = 2*Phi(sqrt(2/pi)/2) - 1 = 0.3101
    rng = np.random.default_rng(9)
    W = (rng.standard_normal((512, 2048)) * 0.02).astype(np.float32)
    t, _ = O.ternarize(W)
    p = 2 * 0.5 * (1 + math.erf(math.sqrt(2 / math.pi) / 2 / math.sqrt(2))) - 1
    assert abs(p - 0.3101) < 1e-4
    assert abs(float((t == 0).mean()) - p) < 3e-3
    assert abs(float((t == 1).mean()) - float((t == -1).mean())) < 3e-3


# ---------------------------------------------------------------------------------------------
# Activation quantisation
# ---------------------------------------------------------------------------------------------
def test_quantize_constructed():
    x = np.array([[127.0, 63.5, -0.5, 1.5, 2.5, -127.0],
                  [1.0, 0.5, -0.25, 0.0, 0.0, 0.0],
                  [0.0, 0.0, 0.0, 0.0, 0.0, 0.0]], np.float32)
    xq, s = O.quantize_act(x)
    assert s[0] == 1.0
    assert xq[0].tolist() == [127, 64, 0, 2, 2, -127]           # ties to even
    assert s[1] == 127.0
    assert xq[1].tolist() == [127, 64, -32, 0, 0, 0]            # 63.5 -> 64, -31.75 -> -32
    assert not xq[2].any()
    assert s[2] == np.float32(127.0) / np.float32(1e-5)
    assert _nearest_f32(Fraction(127) / Fraction(float(np.float32(1e-5))), s[2])


def test_quantize_properties():
    rng = np.random.default_rng(21)
    x = rng.standard_normal((5, 1000)).astype(np.float32)
    xq, s = O.quantize_act(x)
    assert np.abs(xq.astype(np.int64)).max() <= 127
    am = np.argmax(np.abs(x), axis=1)
    assert np.all(np.abs(xq[np.arange(5), am].astype(np.int64)) == 127)
    for m in range(5):
        gamma = Fraction(float(np.abs(x[m]).max()))
        assert _nearest_f32(Fraction(127) / gamma, s[m])
    for k in (-2, 3):
        xq2, s2 = O.quantize_act(x * np.float32(2.0 ** k))
        assert np.array_equal(xq2, xq)
        assert np.array_equal(s2, s / np.float32(2.0 ** k))
    # each code is the nearest integer to the fp32 product (ties to even)
    prod = x * s[:, None]
    assert np.all(np.abs(prod - xq) <= 0.5)


def test_epilogue_closed_form():
    acc = np.array([[3, -4, 0]], np.int32)
    y = O.epilogue(acc, np.float32(0.5), np.array([2.0], np.float32))
    assert y.tolist() == [[0.75, -1.0, 0.0]]


def test_reference_path_small():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 128)).astype(np.float32)
    W = (rng.standard_normal((16, 128)) * 0.02).astype(np.float32)
    y, acc, xq, s, t, beta = O.mpgemm_reference(x, W)
    # y approximates x @ W.T up to the quantisation error of both operands
    dense = x.astype(np.float64) @ (t.astype(np.float64) * float(beta)).T
    assert np.allclose(y, dense, rtol=0.05, atol=0.05 * np.abs(dense).max())


# ---------------------------------------------------------------------------------------------
# ELUT for other weight cardinalities (Appendix "Insight", Table 3)
# ---------------------------------------------------------------------------------------------
def test_elut_formats_bits_per_weight_match_table3():
    # Table 3 rows: (C, g, bpw_b, bpw_e) = (3, 3, 2, 1.67), (4, 2, 2, 2), (5, 2, 3, 2.5)
    for C, g, mirror, bpw_b, bpw_e in [(3, 3, True, 2, 1.67), (4, 2, False, 2, 2.0), (5, 2, True, 3, 2.5)]:
        assert math.ceil(math.log2(C)) == bpw_b
        assert round(O.elut_bits(C, g, mirror) / g, 2) == bpw_e
    # the formats built beyond Table 3's rows: C = 3 with g = 5 fits a byte per group (1.6 bits per weight)
    assert O.elut_bits(3, 5, True) / 5 == 1.6 and O.elut_entries(3, 5, True) == 122
    assert O.elut_entries(4, 2, False) == 16 and O.elut_entries(5, 2, True) == 13
    for fmt, (C, g, mirror) in O.ELUT_FORMATS.items():
        N, K = 16, 640
        assert O.elut_packed_bytes(fmt, N, K) * 8 == N * K * O.elut_bits(C, g, mirror) // g


def test_elut_generic_reduces_to_tl1_and_tl2_codes():
    # C = 3: g = 3 mirrored is Table 6 (TL2), g = 2 plain is Table 5 (TL1)
    d3 = O.elut_entry_weights(3, 3, True)
    assert [tuple(int(v) for v in r) for r in d3] == [O.balanced_ternary_digits(i) for i in range(14)]
    for t in itertools.product((-1, 0, 1), repeat=3):
        idx, sign = O.elut_group_codes(np.array([t]), 3, 3, True)
        ref = O.tl2_codes(*t)
        assert (int(idx[0, 0]), int(sign[0, 0])) == (int(ref[0]), int(ref[1]))
    for row in _rows("tl1_table5.txt"):
        t0, t1, code = int(row[0]), int(row[1]), int(row[2], 2)
        idx, sign = O.elut_group_codes(np.array([[t0, t1]]), 3, 2, False)
        assert int(idx[0, 0]) == code and int(sign[0, 0]) == 0
        assert tuple(int(v) for v in O.elut_entry_weights(3, 2, False)[code]) == (t0, t1)


@pytest.mark.parametrize("fmt", list(O.ELUT_FORMATS))
def test_elut_tables_enumerate_every_group(fmt):
    C, g, mirror = O.ELUT_FORMATS[fmt]
    rng = np.random.default_rng(len(fmt) + C)
    a = rng.integers(-128, 128, size=g)
    xq = np.tile(a, (1, 4)).astype(np.int8)                        # one token, four groups of the same codes
    lut = O.elut_generic_tables(xq, C, g, mirror)
    vals = [int(v) for v in O.elut_values(C)]
    seen = set()
    for grp in itertools.product(vals, repeat=g):
        idx, sign = O.elut_group_codes(np.array([grp]), C, g, mirror)
        i, sg = int(idx[0, 0]), int(sign[0, 0])
        seen.add((i, sg))
        assert int(O.sign_op(lut[0, 0, i], sg)) == sum(int(x) * w for x, w in zip(a, grp))
        if mirror and any(grp):
            neg = O.elut_group_codes(np.array([[-w for w in grp]]), C, g, mirror)
            assert (int(neg[0][0, 0]), int(neg[1][0, 0])) == (i, 1 - sg)
    assert len(seen) == C ** g                                      # every group has its own code


@pytest.mark.parametrize("fmt", list(O.ELUT_FORMATS))
@pytest.mark.parametrize("M,N,K", [(1, 16, 640), (3, 32, 1280)])
def test_elut_generic_equals_mad_and_round_trips(fmt, M, N, K):
    C, g, mirror = O.ELUT_FORMATS[fmt]
    rng = np.random.default_rng(M * 7 + N + K + C)
    w = rng.choice(O.elut_values(C), size=(N, K)).astype(np.int8)
    w[0] = O.elut_values(C)[0]                                      # extreme rows: every weight the smallest value
    w[1] = O.elut_values(C)[-1]
    xq = rng.integers(-128, 128, size=(M, K)).astype(np.int8)
    xq[0, :] = -128
    p = O.pack_elut(w, fmt)
    assert np.array_equal(O.unpack_elut(p, fmt, N, K), w)
    idx, sign = O.elut_decode_codes(p, fmt, N, K)
    assert np.array_equal(O.elut_generic_gemm(xq, idx, sign, C, g, mirror), O.mad_gemm(xq, w))


def test_elut_positions_hand_computed_and_every_field_once():
    N, K = 32, 640
    # c4g2 / c5g2: group j of row n in byte n*K/4 + j//2 (low nibble first); c5g2 signs after N*K/4 bytes, one bit
    # per group; c3g5: one byte per group at n*K/5 + j
    assert tuple(int(v) for v in O.elut_group_position("c4g2", 1, 3, N, K)[:2]) == (161, 4)
    assert tuple(int(v) for v in O.elut_group_position("c5g2", 2, 9, N, K)) == (324, 4, 5120 + 80 + 1, 1)
    assert int(O.elut_group_position("c3g5", 3, 7, N, K)[0]) == 3 * 128 + 7
    for fmt, (C, g, mirror) in O.ELUT_FORMATS.items():
        nn, jj = np.meshgrid(np.arange(N), np.arange(K // g), indexing="ij")
        ib, ish, sb, sbit = O.elut_group_position(fmt, nn, jj, N, K)
        width = 8 if fmt == "c3g5" else 4
        slots = ib.ravel() * (8 // width) + ish.ravel() // width
        assert np.unique(slots).size == slots.size
        if fmt == "c5g2":
            bits = sb.ravel() * 8 + sbit.ravel()
            assert np.unique(bits).size == bits.size and bits.max() == 8 * O.elut_packed_bytes(fmt, N, K) - 1


# ---------------------------------------------------------------------------------------------
# Lossy TL2_0 / TL1_0 (Sec. 3.2.1, Table 1): int8 tables with a power-of-two scale per token and block
# ---------------------------------------------------------------------------------------------
def test_lossy_shift_is_the_smallest_that_fits_int8():
    assert [int(v) for v in O.lossy_shift([0, 127, 128, 254, 255, 381, 508, 509])] == [0, 0, 1, 1, 2, 2, 2, 3]


def test_lossy_tl2_worked_example():
    # one 384-k block, every activation code 127 and every weight +1: the largest entry (+++) is 381, so s = 2 and
    # that entry becomes round(381 / 4) = round(95.25) = 95; each of the 128 triples gives 95 * 4 = 380 instead
    # of 381, so the sum is 128 * 380 = 48640 (the exact sum is 127 * 384 = 48768)
    N, K = 16, 384
    t = np.ones((N, K), np.int8)
    xq = np.full((1, K), 127, np.int8)
    acc = O.elut_gemm_lossy(xq, O.pack_tl2(t), N, K)
    assert np.all(acc == 48640) and int(O.mad_gemm(xq, t)[0, 0]) == 48768
    # TL1_0 on the same weights: pair (+,+) = 254, s = 1, round(127) = 127: exact
    assert np.all(O.elut_gemm_tl1_lossy(xq, O.pack_tl1(t), N, K) == 48768)
    # codes (127, 0, 0) with weights (+, 0, 0): entry 127 at s = 2 (one triple of all 127 makes the block's largest
    # entry 381) -> round(31.75) = 32, scaled back to 128 per triple
    xq2 = np.tile(np.array([[127, 0, 0]], np.int8), (1, 128))
    xq2[0, :3] = 127                                        # one triple of all 127 sets the block's shift to 2
    t2 = np.zeros((N, K), np.int8)
    t2[:, 3::3] = 1                                         # every triple but the first: (+, 0, 0)
    assert np.all(O.elut_gemm_lossy(xq2, O.pack_tl2(t2), N, K) == 127 * 32 * 4)


@pytest.mark.parametrize("M,N,K", [(1, 16, 448), (3, 32, 832), (2, 16, 1600)])
def test_lossy_exact_when_tables_fit_int8_and_error_bounded(M, N, K):
    rng = np.random.default_rng(M + N + K)
    t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    small = rng.integers(-42, 43, size=(M, K)).astype(np.int8)            # every TL2 entry within 3 * 42 = 126
    assert np.array_equal(O.elut_gemm_lossy(small, O.pack_tl2(t), N, K), O.mad_gemm(small, t))
    assert np.array_equal(O.elut_gemm_tl1_lossy(small, O.pack_tl1(t), N, K), O.mad_gemm(small, t))
    xq = rng.integers(-128, 128, size=(M, K)).astype(np.int8)
    exact = O.mad_gemm(xq, t).astype(np.int64)
    sym = xq.astype(np.int16).clip(-127, 127).astype(np.int8)
    for route, packed in [(O.elut_gemm_lossy, O.pack_tl2(t)), (O.elut_gemm_tl1_lossy, O.pack_tl1(t))]:
        lossy = route(xq, packed, N, K)
        # rounding half to even is odd-symmetric, so negating the codes negates the result
        assert np.array_equal(route(-sym, packed, N, K), -route(sym, packed, N, K))
        # every group's entry is off by at most half its block's step 2^s, and s <= 2 for these tables
        groups = K // 3 + K // 2
        assert np.all(np.abs(lossy - exact) <= groups * 2)
        assert not np.array_equal(lossy, exact)                              # these codes do lose precision
