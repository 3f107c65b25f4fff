"""Plain, slow CPU oracle for the ternary-weight x int8-activation mpGEMM of Bitnet.cpp (arXiv 2502.11880).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library: no kernels, headers, tables or helpers.  It reads
numpy arrays and returns numpy arrays.

What it computes, with the part of the paper each step follows:

* ``absmean_beta`` / ``ternarize`` -- ternary weights (Sec. 2.1, "Ternary Weights"): one fp32 scale per
  tensor, beta = mean(|W|), t = clamp(round(W / beta), -1, 1).  The paper only says the weights are
  ternarised the way BitNet b1.58 trains them (Sec. 2.1 "Lossless Inference"; Sec. 3.2.2); the formula is
  the one this library's workloads fix.  beta is the correctly rounded fp32 value of the *exact* rational
  mean, so it does not depend on any summation order.
* ``quantize_act`` -- int8 activations, absmax with one scale per token row (Sec. 2.1, Sec. 3.2.2).
* ``pack_i2s`` / ``unpack_i2s`` -- the I2_S format: 2 bits per weight plus one tensor scale (Table 1,
  Sec. 3.2.2).  The bit layout is not given by the paper; the one defined here is tiled for 16-row,
  64-k MFMA operands (see ``i2s_position``).
* ``tl2_codes`` / ``tl1_code`` / ``pack_tl2`` / ``unpack_tl2`` -- the TL2 format (Sec. 3.1, Table 6):
  each weight triple becomes a 4-bit index plus a 1-bit sign held in separate planes (signed-unsigned
  weight splitting, Sec. 3.1.2); the K remainder that does not fill a TL2 block uses TL1 pair codes
  (Table 5), as block-fitting weight splitting prescribes (Sec. 3.1.2).
* ``pack_tl1`` / ``unpack_tl1`` -- the TL1 format on its own (Table 1 "TL1_1", Algorithm TL1, Table 5): every
  weight pair is its 4-bit Table 5 code, 2 bits per weight, tiled like I2_S (see ``tl1_pair_position``).
* ``mad_gemm`` -- Eq. 1 / Algorithm "MAD-based mpGEMM": acc[m, n] = sum_k xq[m, k] * t[n, k], exact.
* ``elut_tables`` / ``elut_gemm`` -- Eq. 3 / Algorithm "ELUT mpGEMM" with mirror consolidation
  (Sec. 3.1.1) and the 1-bit sign operation of Eq. 5: an independent second route to the same integers;
  ``tl1_tables`` / ``elut_gemm_tl1`` the same for the TL1 format (Algorithm TL1: 9-entry pair tables).
* ``elut_gemm_lossy`` / ``elut_gemm_tl1_lossy`` -- the lossy TL2_0 and TL1_0 kernels of Table 1 (Sec. 3.2.1): the
  same lookups on tables quantised to int8, with one power-of-two scale per token and table block.
* ``elut_*`` / ``pack_elut`` -- the ELUT method for integer weights of other cardinalities (Appendix "Insight",
  Table 3, Algorithm "ELUT mpGEMM"): group codes, tables of the C^g sums (mirrored for symmetric sets) and the
  packed formats c4g2, c5g2 and c3g5.
* ``epilogue`` -- y = acc * beta / s_m in float64 (the dequantisation the quantisers above imply).

All floating-point decisions that produce integers (the weight divide and round, the activation multiply
and round) are taken in IEEE fp32 with round-to-nearest-even, the precision the GPU kernels use.
"""
from __future__ import annotations

import math

import numpy as np

# ----------------------------------------------------------------------------------------------
# Layout constants (definitions of the packed formats; see the position functions below)
# ----------------------------------------------------------------------------------------------
ROWS_PER_GROUP = 16       # both formats tile 16 weight rows together
I2S_SUBTILE_K = 64        # I2_S: one 16-row x 64-k sub-tile = 256 bytes
I2S_BLOCK_K = 256         # I2_S: up to 4 sub-tiles per block (1 KiB for 16 rows)
TL2_BLOCK_K = 384         # TL2 block length BK3 (128 triples per row per block)
TL2_GROUPS_PER_BLOCK = TL2_BLOCK_K // 3
TAIL_UNIT_K = 64          # TL1 tail: one 16-row x 64-k unit = 16 bytes per row

ACT_GAMMA_FLOOR = np.float32(1e-5)
ACT_QMAX = np.float32(127.0)


# ----------------------------------------------------------------------------------------------
# Exact rational -> fp32 (round to nearest, ties to even)
# ----------------------------------------------------------------------------------------------
def f32_from_rational(num: int, den: int) -> np.float32:
    """Correctly rounded (nearest-even) float32 of the non-negative rational num/den."""
    if num < 0 or den <= 0:
        raise ValueError("f32_from_rational expects num >= 0 and den > 0")
    if num == 0:
        return np.float32(0.0)
    # e = floor(log2(num/den))
    e = num.bit_length() - den.bit_length()
    if e >= 0:
        if num < (den << e):
            e -= 1
    else:
        if (num << -e) < den:
            e -= 1
    # quantum 2^q: 24 significant bits for normals, 2^-149 for subnormals
    q = e - 23 if e >= -126 else -149
    if q >= 0:
        d = den << q
        n0, rem = divmod(num, d)
    else:
        d = den
        n0, rem = divmod(num << -q, d)
    twice = 2 * rem
    if twice > d or (twice == d and (n0 & 1)):
        n0 += 1
    val = math.ldexp(float(n0), q)   # exact in float64: n0 <= 2^24 and q >= -149
    out = np.float32(val)
    if not np.isfinite(out):
        raise OverflowError("rational exceeds the float32 range")
    return out


# ----------------------------------------------------------------------------------------------
# a1: absmean ternarisation (Sec. 2.1; one fp32 scale per tensor)
# ----------------------------------------------------------------------------------------------
def absmean_beta(W: np.ndarray, chunk: int = 1 << 24) -> np.float32:
    """beta = mean(|W|) over the whole tensor, as the correctly rounded fp32 of the exact mean.

    Each |w| is m * 2^(e-150) with an integer significand m < 2^24 and biased exponent e (subnormals use
    e = 1 and no hidden bit).  Significands are summed exactly per exponent: bincount adds integers below
    2^12 in float64, which stays exact for fewer than 2^41 elements.
    """
    flat = np.ascontiguousarray(W, dtype=np.float32).ravel()
    n = flat.size
    if n == 0:
        raise ValueError("empty weight tensor")
    hi_tot = np.zeros(256, dtype=np.float64)
    lo_tot = np.zeros(256, dtype=np.float64)
    for start in range(0, n, chunk):
        bits = flat[start:start + chunk].view(np.uint32) & np.uint32(0x7FFFFFFF)
        e = (bits >> np.uint32(23)).astype(np.int64)
        if np.any(e == 255):
            raise ValueError("weights must be finite")
        f = (bits & np.uint32(0x7FFFFF)).astype(np.int64)
        m = np.where(e > 0, f | (1 << 23), f)
        e = np.maximum(e, 1)
        hi_tot += np.bincount(e, weights=(m >> 12).astype(np.float64), minlength=256)
        lo_tot += np.bincount(e, weights=(m & 0xFFF).astype(np.float64), minlength=256)
    total = 0   # sum |w| = total * 2^-149
    for b in range(1, 256):
        s_b = int(hi_tot[b]) * 4096 + int(lo_tot[b])
        if s_b:
            total += s_b << (b - 1)
    return f32_from_rational(total, n << 149)


def ternarize(W: np.ndarray) -> tuple[np.ndarray, np.float32]:
    """t = clamp(round_half_even(fp32(W / beta)), -1, 1) with beta = absmean_beta(W); beta == 0 gives t = 0."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    beta = absmean_beta(W)
    if beta == 0:
        return np.zeros(W.shape, dtype=np.int8), beta
    r = W / beta                      # IEEE fp32 divide, correctly rounded
    t = np.clip(np.rint(r), -1, 1).astype(np.int8)
    return t, beta


# ----------------------------------------------------------------------------------------------
# a3: per-token absmax int8 activation quantisation (Sec. 2.1, Sec. 3.2.2)
# ----------------------------------------------------------------------------------------------
def quantize_act(x: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """gamma_m = max_k |x[m,k]| (floored at 1e-5), s_m = fp32(127 / gamma_m), xq = clamp(rint(fp32(x*s_m)))."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim != 2 or x.shape[1] == 0:
        raise ValueError("x must be [M, K] with K >= 1")
    if not np.all(np.isfinite(x)):
        raise ValueError("activations must be finite")
    gamma = np.max(np.abs(x), axis=1)
    gamma = np.maximum(gamma, ACT_GAMMA_FLOOR)
    s = (ACT_QMAX / gamma).astype(np.float32)
    prod = x * s[:, None]             # fp32 multiply, correctly rounded
    xq = np.clip(np.rint(prod), -128, 127).astype(np.int8)
    return xq, s


# ----------------------------------------------------------------------------------------------
# a2: I2_S packing (Table 1, Sec. 3.2.2).  Layout definition.
# ----------------------------------------------------------------------------------------------
def check_shape(N: int, K: int) -> None:
    if N <= 0 or K <= 0 or N % ROWS_PER_GROUP or K % I2S_SUBTILE_K:
        raise ValueError("packed formats need N % 16 == 0 and K % 64 == 0")


def i2s_packed_bytes(N: int, K: int) -> int:
    check_shape(N, K)
    return N * K // 4


def i2s_position(n, k, N: int, K: int):
    """Byte offset and bit shift of weight (n, k) in the I2_S buffer.

    Code = t + 1 in two bits (00 -> -1, 01 -> 0, 10 -> +1).  Rows are tiled in groups of 16; K is cut into
    blocks of up to 256 (4 sub-tiles of 64).  Within a block of T sub-tiles, the 16 rows own 64 "lanes"
    l = 16*q + r (r = row in the group, q = which 16-k quarter of a sub-tile), and lane l owns 4*T contiguous
    bytes: one 32-bit word per sub-tile j.  Word j of lane (r, q) holds the 16 weights
    k = 64*(4*s + j) + 16*q + 4*f + b in byte b, bits [2f, 2f+1].
    """
    n = np.asarray(n, dtype=np.int64)
    k = np.asarray(k, dtype=np.int64)
    R, r = n // 16, n % 16
    u = k // 64
    s, j = u // 4, u % 4
    kk = k % 64
    q = kk // 16
    w = kk % 16
    f, b = w // 4, w % 4
    T = np.minimum(4, K // 64 - 4 * s)
    lane = 16 * q + r
    byte = R * (4 * K) + s * 1024 + 4 * T * lane + 4 * j + b
    return byte, 2 * f


def pack_i2s(t: np.ndarray) -> np.ndarray:
    t = np.asarray(t)
    N, K = t.shape
    check_shape(N, K)
    if t.min(initial=0) < -1 or t.max(initial=0) > 1:
        raise ValueError("weights must be ternary")
    out = np.zeros(N * K // 4, dtype=np.uint8)
    rows_per_chunk = max(16, (1 << 22) // K // 16 * 16)
    for n0 in range(0, N, rows_per_chunk):
        n1 = min(N, n0 + rows_per_chunk)
        nn, kk = np.meshgrid(np.arange(n0, n1), np.arange(K), indexing="ij")
        byte, shift = i2s_position(nn, kk, N, K)
        code = (t[n0:n1].astype(np.int64) + 1) << shift
        np.bitwise_or.at(out, byte.ravel(), code.ravel().astype(np.uint8))
    return out


def unpack_i2s(packed: np.ndarray, N: int, K: int) -> np.ndarray:
    check_shape(N, K)
    packed = np.asarray(packed, dtype=np.uint8)
    if packed.size != N * K // 4:
        raise ValueError("I2_S buffer has the wrong size")
    nn, kk = np.meshgrid(np.arange(N), np.arange(K), indexing="ij")
    byte, shift = i2s_position(nn, kk, N, K)
    code = (packed[byte].astype(np.int64) >> shift) & 3
    if np.any(code == 3):
        raise ValueError("I2_S code 3 never occurs in a valid buffer")
    return (code - 1).astype(np.int8)


# ----------------------------------------------------------------------------------------------
# a2: TL2 packing (Sec. 3.1, Table 5, Table 6).  Layout definition.
# ----------------------------------------------------------------------------------------------
def tl2_split(K: int) -> tuple[int, int]:
    """Block-fitting weight splitting (Sec. 3.1.2): ThreeK = floor(K/BK3)*BK3 through TL2, the rest through TL1."""
    three = (K // TL2_BLOCK_K) * TL2_BLOCK_K
    return three, K - three


def tl2_packed_bytes(N: int, K: int) -> int:
    check_shape(N, K)
    three, two = tl2_split(K)
    groups = three // 3
    return N * groups // 2 + N * groups // 8 + N * two // 4


def tl2_codes(t0, t1, t2):
    """TL2 code of one weight triple (Table 6): v = 9*t0 + 3*t1 + t2, index = |v| (0..13), sign = [v < 0]."""
    v = 9 * np.asarray(t0, dtype=np.int64) + 3 * np.asarray(t1, dtype=np.int64) + np.asarray(t2, dtype=np.int64)
    return np.abs(v), (v < 0).astype(np.int64)


def tl1_code(t0, t1):
    """TL1 code of one weight pair (Table 5): 3*(t0+1) + (t1+1), 0..8."""
    return 3 * (np.asarray(t0, dtype=np.int64) + 1) + (np.asarray(t1, dtype=np.int64) + 1)


def tl2_idx_position(n, g, N: int, K: int):
    """(index-plane byte, nibble shift) and (sign-plane byte, bit) of triple g of row n.

    Triple g covers k = 3g, 3g+1, 3g+2 (g < ThreeK/3).  Rows are tiled in 16; each block of 128 triples
    gives lane l = 16*q + r (q = g_in_block // 32) 16 index bytes (triple i = g_in_block % 32 in byte i//2,
    low nibble when i is even) and 4 sign bytes (triple i in byte i//8, bit i%8).  The index plane is
    followed by the sign plane, then by the TL1 tail plane.
    """
    n = np.asarray(n, dtype=np.int64)
    g = np.asarray(g, dtype=np.int64)
    three, _ = tl2_split(K)
    nblk = three // TL2_BLOCK_K
    R, r = n // 16, n % 16
    blk, gg = g // TL2_GROUPS_PER_BLOCK, g % TL2_GROUPS_PER_BLOCK
    q, i = gg // 32, gg % 32
    lane = 16 * q + r
    idx_byte = R * (nblk * 1024) + blk * 1024 + 16 * lane + i // 2
    sign_byte = N * (three // 6) + R * (nblk * 256) + blk * 256 + 4 * lane + i // 8
    return idx_byte, 4 * (i % 2), sign_byte, i % 8


def tl1_tail_position(n, p, N: int, K: int):
    """(byte, nibble shift) of tail pair p of row n (k = ThreeK + 2p, ThreeK + 2p + 1).

    The tail is cut into units of 64 k; lane l = 16*q + r owns one 32-bit word per unit, word u holding
    pairs 32*u + 8*q + i (i = 0..7) in byte i//2, low nibble when i is even.  Lane words are contiguous.
    """
    n = np.asarray(n, dtype=np.int64)
    p = np.asarray(p, dtype=np.int64)
    three, two = tl2_split(K)
    units = two // TAIL_UNIT_K
    base = N * (three // 6) + N * (three // 24)
    R, r = n // 16, n % 16
    u, pp = p // 32, p % 32
    q, i = pp // 8, pp % 8
    lane = 16 * q + r
    byte = base + R * (16 * two // 4) + 4 * units * lane + 4 * u + i // 2
    return byte, 4 * (i % 2)


def pack_tl2(t: np.ndarray) -> np.ndarray:
    t = np.asarray(t)
    N, K = t.shape
    check_shape(N, K)
    if t.min(initial=0) < -1 or t.max(initial=0) > 1:
        raise ValueError("weights must be ternary")
    three, two = tl2_split(K)
    out = np.zeros(tl2_packed_bytes(N, K), dtype=np.uint8)
    G = three // 3
    if G:
        nn, gg = np.meshgrid(np.arange(N), np.arange(G), indexing="ij")
        tt = t[:, :three].astype(np.int64).reshape(N, G, 3)
        idx, sign = tl2_codes(tt[..., 0], tt[..., 1], tt[..., 2])
        ib, ish, sb, sbit = tl2_idx_position(nn, gg, N, K)
        np.bitwise_or.at(out, ib.ravel(), (idx << ish).ravel().astype(np.uint8))
        np.bitwise_or.at(out, sb.ravel(), (sign << sbit).ravel().astype(np.uint8))
    P = two // 2
    if P:
        nn, pp = np.meshgrid(np.arange(N), np.arange(P), indexing="ij")
        tp = t[:, three:].astype(np.int64).reshape(N, P, 2)
        code = tl1_code(tp[..., 0], tp[..., 1])
        b, sh = tl1_tail_position(nn, pp, N, K)
        np.bitwise_or.at(out, b.ravel(), (code << sh).ravel().astype(np.uint8))
    return out


def tl2_decode_fields(packed: np.ndarray, N: int, K: int):
    """Read back (index, sign) per triple [N, G] and the TL1 code per tail pair [N, P]."""
    packed = np.asarray(packed, dtype=np.uint8)
    if packed.size != tl2_packed_bytes(N, K):
        raise ValueError("TL2 buffer has the wrong size")
    three, two = tl2_split(K)
    G, P = three // 3, two // 2
    nn, gg = np.meshgrid(np.arange(N), np.arange(G), indexing="ij")
    ib, ish, sb, sbit = tl2_idx_position(nn, gg, N, K)
    idx = (packed[ib].astype(np.int64) >> ish) & 0xF
    sign = (packed[sb].astype(np.int64) >> sbit) & 1
    nn, pp = np.meshgrid(np.arange(N), np.arange(P), indexing="ij")
    b, sh = tl1_tail_position(nn, pp, N, K)
    tail = (packed[b].astype(np.int64) >> sh) & 0xF
    return idx, sign, tail


def balanced_ternary_digits(i: int) -> tuple[int, int, int]:
    """Digits (d0, d1, d2) in {-1, 0, 1} with i = 9*d0 + 3*d1 + d2, for 0 <= i <= 13."""
    d = []
    v = i
    for _ in range(3):
        r = v % 3
        if r == 2:
            r = -1
        d.append(r)
        v = (v - r) // 3
    if v != 0:
        raise ValueError("index outside the balanced-ternary range of three digits")
    return d[2], d[1], d[0]


def unpack_tl2(packed: np.ndarray, N: int, K: int) -> np.ndarray:
    idx, sign, tail = tl2_decode_fields(packed, N, K)
    three, two = tl2_split(K)
    if np.any(idx > 13) or np.any((idx == 0) & (sign == 1)) or np.any(tail > 8):
        raise ValueError("invalid TL2 code")
    t = np.zeros((N, K), dtype=np.int8)
    digits = np.array([balanced_ternary_digits(i) for i in range(14)], dtype=np.int64)  # [14, 3]
    trip = digits[idx] * np.where(sign == 1, -1, 1)[..., None]
    t[:, :three] = trip.reshape(N, three)
    pair = np.stack([tail // 3 - 1, tail % 3 - 1], axis=-1)
    t[:, three:] = pair.reshape(N, two)
    return t


# ----------------------------------------------------------------------------------------------
# a2: TL1 packing on its own (Table 1 "TL1_1", Algorithm TL1, Table 5).  Layout definition.
# ----------------------------------------------------------------------------------------------
def tl1_packed_bytes(N: int, K: int) -> int:
    """4 bits per pair of weights: 2 bits per weight, like I2_S."""
    check_shape(N, K)
    return N * K // 4


def tl1_pair_position(n, p, N: int, K: int):
    """(byte, nibble shift) of pair p of row n, the weights k = 2p and 2p + 1.

    The tiling is that of I2_S (``i2s_position``): 16-row groups, 256-k blocks, lane l = 16*q + r owning one
    32-bit word per 64-k sub-tile j of a block, and that word holding the 16 weights k = 64*(4*s + j) + 16*q + e
    (e = 0..15) of row 16R + r.  Inside the word the 8 pair codes sit as: pair e // 2 = i of the 16 in byte
    i % 4, low nibble for i < 4 and high nibble for i >= 4.
    """
    n = np.asarray(n, dtype=np.int64)
    p = np.asarray(p, dtype=np.int64)
    k = 2 * p
    R, r = n // 16, n % 16
    u = k // 64
    s, j = u // 4, u % 4
    kk = k % 64
    q = kk // 16
    i = (kk % 16) // 2
    T = np.minimum(4, K // 64 - 4 * s)
    lane = 16 * q + r
    byte = R * (4 * K) + s * 1024 + 4 * T * lane + 4 * j + i % 4
    return byte, 4 * (i // 4)


def pack_tl1(t: np.ndarray) -> np.ndarray:
    t = np.asarray(t)
    N, K = t.shape
    check_shape(N, K)
    if t.min(initial=0) < -1 or t.max(initial=0) > 1:
        raise ValueError("weights must be ternary")
    out = np.zeros(tl1_packed_bytes(N, K), dtype=np.uint8)
    P = K // 2
    nn, pp = np.meshgrid(np.arange(N), np.arange(P), indexing="ij")
    tp = t.astype(np.int64).reshape(N, P, 2)
    code = tl1_code(tp[..., 0], tp[..., 1])
    byte, shift = tl1_pair_position(nn, pp, N, K)
    np.bitwise_or.at(out, byte.ravel(), (code << shift).ravel().astype(np.uint8))
    return out


def tl1_decode_codes(packed: np.ndarray, N: int, K: int) -> np.ndarray:
    """The Table 5 code of every pair, [N, K/2]."""
    check_shape(N, K)
    packed = np.asarray(packed, dtype=np.uint8)
    if packed.size != tl1_packed_bytes(N, K):
        raise ValueError("TL1 buffer has the wrong size")
    nn, pp = np.meshgrid(np.arange(N), np.arange(K // 2), indexing="ij")
    byte, shift = tl1_pair_position(nn, pp, N, K)
    return (packed[byte].astype(np.int64) >> shift) & 0xF


def unpack_tl1(packed: np.ndarray, N: int, K: int) -> np.ndarray:
    code = tl1_decode_codes(packed, N, K)
    if np.any(code > 8):
        raise ValueError("TL1 codes above 8 never occur in a valid buffer")
    pair = np.stack([code // 3 - 1, code % 3 - 1], axis=-1)
    return pair.reshape(N, K).astype(np.int8)


# ----------------------------------------------------------------------------------------------
# a5/a6: MAD accumulation (Eq. 1, Algorithm "MAD-based mpGEMM")
# ----------------------------------------------------------------------------------------------
F64_EXACT = 1 << 53       # every integer of magnitude up to 2^53 is a float64


def mad_gemm(xq: np.ndarray, t: np.ndarray) -> np.ndarray:
    """acc[m, n] = sum_k xq[m, k] * t[n, k] in exact integer arithmetic (checked to fit int32).

    Every term is an integer of magnitude at most 128, so every partial sum of a row is an integer of
    magnitude at most 128 K.  While 128 K < 2^53 each of them is a float64, so a float64 matrix product gives
    the exact sum whatever order it adds in; beyond that bound the product is taken in int64.
    """
    a = np.asarray(xq)
    w = np.asarray(t)
    if a.ndim != 2 or w.ndim != 2 or a.shape[1] != w.shape[1]:
        raise ValueError("K mismatch")
    if 128 * max(1, a.shape[1]) < F64_EXACT:
        acc = np.rint(a.astype(np.float64) @ w.astype(np.float64).T).astype(np.int64)
    else:
        acc = a.astype(np.int64) @ w.astype(np.int64).T
    if acc.size and (acc.max() > np.iinfo(np.int32).max or acc.min() < np.iinfo(np.int32).min):
        raise OverflowError("accumulator exceeds int32")
    return acc.astype(np.int32)


# ----------------------------------------------------------------------------------------------
# a4 + a5 (LUT route): ELUT with mirror consolidation (Eq. 3, Sec. 3.1.1, Eq. 5, Algorithm "ELUT mpGEMM")
# ----------------------------------------------------------------------------------------------
def sign_op(x, sign):
    """Eq. 5 with the sign bit widened to a mask m in {0, -1}: (x + m) XOR m is x for m = 0 and -x for m = -1."""
    m = -np.asarray(sign, dtype=np.int64)
    return (np.asarray(x, dtype=np.int64) + m) ^ m


def elut_tables(xq: np.ndarray, K: int | None = None):
    """Per token, the 14-entry mirror-consolidated table of every triple and the 9-entry TL1 table of every
    tail pair (Table-setup step of the ELUT algorithm; PreCompute of the TL1/TL2 algorithms).

    lut[m, g, i] = d0(i)*a0 + d1(i)*a1 + d2(i)*a2 where (a0, a1, a2) = xq[m, 3g:3g+3] and (d0, d1, d2) are
    the balanced-ternary digits of i; lut1[m, p, i] = (i//3 - 1)*b0 + (i%3 - 1)*b1 with (b0, b1) the pair.
    """
    a = np.asarray(xq, dtype=np.int64)
    M, Kx = a.shape
    K = Kx if K is None else K
    three, two = tl2_split(K)
    G, P = three // 3, two // 2
    trip = a[:, :three].reshape(M, G, 3)
    lut = np.zeros((M, G, 14), dtype=np.int64)
    for i in range(14):
        d0, d1, d2 = balanced_ternary_digits(i)
        lut[:, :, i] = d0 * trip[..., 0] + d1 * trip[..., 1] + d2 * trip[..., 2]
    pair = a[:, three:].reshape(M, P, 2)
    lut1 = np.zeros((M, P, 9), dtype=np.int64)
    for i in range(9):
        lut1[:, :, i] = (i // 3 - 1) * pair[..., 0] + (i % 3 - 1) * pair[..., 1]
    return lut, lut1


def elut_gemm(xq: np.ndarray, packed_tl2: np.ndarray, N: int, K: int) -> np.ndarray:
    """acc via table lookups on the packed TL2 buffer: sum over triples of sign_op(lut[idx], sign) plus the
    TL1 lookups of the tail pairs.  Shares nothing with ``mad_gemm``."""
    idx, sign, tail = tl2_decode_fields(packed_tl2, N, K)
    lut, lut1 = elut_tables(xq, K)
    M = lut.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for m in range(M):
        if lut.shape[1]:
            vals = np.take_along_axis(lut[m][None, :, :], idx[:, :, None], axis=2)[..., 0]   # [N, G]
            acc[m] += sign_op(vals, sign).sum(axis=1)
        if lut1.shape[1]:
            vals1 = np.take_along_axis(lut1[m][None, :, :], tail[:, :, None], axis=2)[..., 0]
            acc[m] += vals1.sum(axis=1)
    return acc.astype(np.int32)


def tl1_tables(xq: np.ndarray) -> np.ndarray:
    """Per token, the 9-entry table of every weight pair (PreCompute of Algorithm TL1):
    lut[m, p, i] = (i//3 - 1)*a0 + (i%3 - 1)*a1 with (a0, a1) = xq[m, 2p:2p+2], i the Table 5 code."""
    a = np.asarray(xq, dtype=np.int64)
    M, K = a.shape
    pair = a.reshape(M, K // 2, 2)
    lut = np.zeros((M, K // 2, 9), dtype=np.int64)
    for i in range(9):
        lut[:, :, i] = (i // 3 - 1) * pair[..., 0] + (i % 3 - 1) * pair[..., 1]
    return lut


def elut_gemm_tl1(xq: np.ndarray, packed_tl1: np.ndarray, N: int, K: int) -> np.ndarray:
    """acc via one table lookup per weight pair on the packed TL1 buffer (Algorithm TL1, Eq. 3 with g = 2).
    Shares nothing with ``mad_gemm``."""
    code = tl1_decode_codes(packed_tl1, N, K)            # [N, K/2]
    lut = tl1_tables(xq)                                  # [M, K/2, 9]
    M = lut.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for m in range(M):
        vals = np.take_along_axis(lut[m][None, :, :], code[:, :, None], axis=2)[..., 0]   # [N, K/2]
        acc[m] = vals.sum(axis=1)
    return acc.astype(np.int32)


# ----------------------------------------------------------------------------------------------
# Lossy TL2_0 / TL1_0 (Sec. 3.2.1, Table 1): the table sums quantised to int8 before the lookups
# ----------------------------------------------------------------------------------------------
LOSSY_TRIPLES_PER_BLOCK = TL2_BLOCK_K // 3      # one scale per token for the 128 triples of a 384-k block
LOSSY_PAIRS_PER_UNIT = TAIL_UNIT_K // 2         # one scale per token for the 32 pairs of a 64-k unit


def lossy_shift(max_abs) -> np.ndarray:
    """The smallest s >= 0 with max_abs <= 127 * 2^s: the table block's int8 scale is 2^-s."""
    m = np.asarray(max_abs, dtype=np.int64)
    s = np.zeros_like(m)
    while np.any(m > 127 * (1 << s)):
        s = np.where(m > 127 * (1 << s), s + 1, s)
    return s


def quantize_table(lut: np.ndarray, blocks: np.ndarray):
    """int8 tables of one kind: lut [M, G, E] int sums; blocks [G] the block of every group.  Per token and block
    the entries are divided by 2^s (s from the block's largest |entry|) and rounded half to even.  Returns the
    quantised entries [M, G, E] and the shift of every token and group [M, G]."""
    lut = np.asarray(lut, dtype=np.int64)
    M, G, _ = lut.shape
    shift = np.zeros((M, G), dtype=np.int64)
    for b in np.unique(blocks):
        sel = blocks == b
        mx = np.abs(lut[:, sel, :]).reshape(M, -1).max(axis=1)                 # [M]
        shift[:, sel] = lossy_shift(mx)[:, None]
    q = np.rint(lut / (2.0 ** shift)[..., None]).astype(np.int64)             # exact: |lut| < 2^10, powers of two
    return q, shift


def elut_gemm_lossy(xq: np.ndarray, packed_tl2: np.ndarray, N: int, K: int) -> np.ndarray:
    """TL2_0: Eq. 3 lookups on int8-quantised tables.  Each triple (and each TL1 tail pair) contributes its
    quantised entry with the Eq. 5 sign operation; a block's sum is scaled back by 2^s, exactly."""
    idx, sign, tail = tl2_decode_fields(packed_tl2, N, K)
    lut, lut1 = elut_tables(xq, K)
    q, sh = quantize_table(lut, np.arange(lut.shape[1]) // LOSSY_TRIPLES_PER_BLOCK)
    q1, sh1 = quantize_table(lut1, np.arange(lut1.shape[1]) // LOSSY_PAIRS_PER_UNIT)
    M = lut.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for m in range(M):
        if lut.shape[1]:
            vals = np.take_along_axis(q[m][None, :, :], idx[:, :, None], axis=2)[..., 0]      # [N, G]
            acc[m] += (sign_op(vals, sign) << sh[m][None, :]).sum(axis=1)
        if lut1.shape[1]:
            vals1 = np.take_along_axis(q1[m][None, :, :], tail[:, :, None], axis=2)[..., 0]
            acc[m] += (vals1 << sh1[m][None, :]).sum(axis=1)
    return acc


def elut_gemm_tl1_lossy(xq: np.ndarray, packed_tl1: np.ndarray, N: int, K: int) -> np.ndarray:
    """TL1_0: Algorithm TL1's lookups on int8-quantised pair tables (one scale per token and 64-k unit)."""
    code = tl1_decode_codes(packed_tl1, N, K)
    q, sh = quantize_table(tl1_tables(xq), np.arange(K // 2) // LOSSY_PAIRS_PER_UNIT)
    M = q.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for m in range(M):
        vals = np.take_along_axis(q[m][None, :, :], code[:, :, None], axis=2)[..., 0]
        acc[m] = (vals << sh[m][None, :]).sum(axis=1)
    return acc


# ----------------------------------------------------------------------------------------------
# ELUT beyond ternary weights (Appendix "Insight", Table 3, Algorithm "ELUT mpGEMM", Eq. 3 and Eq. 4):
# integer weights from a set of C values, one table of the C^g sums per group of g weights
# ----------------------------------------------------------------------------------------------
# Formats: name -> (C, g, mirror).  C = 4 with g = 2 and C = 5 with g = 2 are rows of Table 3; C = 3 with g = 5 is
# a group too long for a 16-entry register table (the register-length analysis of the appendix) whose 122-entry
# mirrored table lives in GPU LDS.
ELUT_FORMATS = {"c4g2": (4, 2, False), "c5g2": (5, 2, True), "c3g5": (3, 5, True)}


def elut_values(C: int) -> np.ndarray:
    """The weight set of cardinality C: the C consecutive integers -floor(C/2) .. C - 1 - floor(C/2)
    ({-1, 0, 1} for C = 3, the two's-complement {-2, -1, 0, 1} for C = 4, {-2, .., 2} for C = 5)."""
    return np.arange(-(C // 2), C - C // 2, dtype=np.int64)


def elut_entries(C: int, g: int, mirror: bool) -> int:
    """Table length: C^g, or the non-negative half (C^g + 1) / 2 with mirror consolidation (odd C only)."""
    if mirror and C % 2 == 0:
        raise ValueError("mirror consolidation needs a weight set symmetric about 0 (odd C)")
    return (C ** g + 1) // 2 if mirror else C ** g


def elut_bits(C: int, g: int, mirror: bool) -> int:
    """Bits per group: the index of an entry, plus the sign bit with mirror consolidation."""
    return math.ceil(math.log2(elut_entries(C, g, mirror))) + (1 if mirror else 0)


def elut_entry_weights(C: int, g: int, mirror: bool) -> np.ndarray:
    """[E, g] weights of table entry e: without mirroring the base-C digits of e (first weight most significant)
    offset by the set's minimum; with mirroring the balanced base-C digits of e (so entry e is the group whose value
    sum_j w_j C^(g-1-j) equals e)."""
    E = elut_entries(C, g, mirror)
    out = np.zeros((E, g), dtype=np.int64)
    lo = int(elut_values(C)[0])
    for e in range(E):
        v = e
        for j in range(g - 1, -1, -1):
            if mirror:
                r = v % C
                if r > C // 2:
                    r -= C
                out[e, j] = r
                v = (v - r) // C
            else:
                out[e, j] = v % C + lo
                v //= C
        if v != 0:
            raise ValueError("entry outside the group's range")
    return out


def elut_group_codes(w: np.ndarray, C: int, g: int, mirror: bool):
    """(index, sign) of every group of g weights along the rows of w [N, K] (K % g == 0); sign is 0 without
    mirroring.  Plain: the base-C number of the digits w_j - min.  Mirrored: v = sum_j w_j C^(g-1-j),
    index |v|, sign [v < 0] (the rule of Table 6 for any odd C)."""
    w = np.asarray(w, dtype=np.int64)
    N, K = w.shape
    if K % g:
        raise ValueError("K must be a multiple of the group size")
    vals = elut_values(C)
    if w.min(initial=0) < vals[0] or w.max(initial=0) > vals[-1]:
        raise ValueError("weights outside the set")
    grp = w.reshape(N, K // g, g)
    if mirror:
        v = np.zeros(grp.shape[:2], dtype=np.int64)
        for j in range(g):
            v = v * C + grp[..., j]
        return np.abs(v), (v < 0).astype(np.int64)
    code = np.zeros(grp.shape[:2], dtype=np.int64)
    for j in range(g):
        code = code * C + (grp[..., j] - vals[0])
    return code, np.zeros_like(code)


def elut_generic_tables(xq: np.ndarray, C: int, g: int, mirror: bool) -> np.ndarray:
    """Table-setup step: lut[m, j, e] = sum_i d_i(e) * xq[m, g j + i] over the entry weights d(e)."""
    a = np.asarray(xq, dtype=np.int64)
    M, K = a.shape
    d = elut_entry_weights(C, g, mirror)                 # [E, g]
    grp = a.reshape(M, K // g, g)
    return np.einsum("mjg,eg->mje", grp, d)


def elut_generic_gemm(xq: np.ndarray, idx: np.ndarray, sign: np.ndarray, C: int, g: int, mirror: bool) -> np.ndarray:
    """acc[m, n] = sum over the groups of row n of the looked-up entry, negated where the group's sign is set
    (Eq. 5 with the sign widened to a mask).  Shares nothing with ``mad_gemm``."""
    lut = elut_generic_tables(xq, C, g, mirror)          # [M, G, E]
    M = lut.shape[0]
    N = idx.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for m in range(M):
        vals = np.take_along_axis(lut[m][None, :, :], idx[:, :, None], axis=2)[..., 0]   # [N, G]
        acc[m] = sign_op(vals, sign).sum(axis=1)
    return acc


def elut_layout_check(fmt: str, N: int, K: int) -> None:
    C, g, _ = ELUT_FORMATS[fmt]
    step = 320 if g == 5 else 64
    if N <= 0 or K <= 0 or N % 16 or K % step:
        raise ValueError(f"{fmt} needs N % 16 == 0 and K % {step} == 0")


def elut_packed_bytes(fmt: str, N: int, K: int) -> int:
    """c4g2: a 4-bit code per pair (N K / 4 bytes); c5g2: a 4-bit index plane (N K / 4) then a sign plane of one
    bit per pair (N K / 16); c3g5: one byte per group of five (index in bits 0-6, sign in bit 7; N K / 5)."""
    elut_layout_check(fmt, N, K)
    return {"c4g2": N * K // 4, "c5g2": N * K // 4 + N * K // 16, "c3g5": N * K // 5}[fmt]


def elut_group_position(fmt: str, n, j, N: int, K: int):
    """(byte, shift) of the index field of group j of row n, and (byte, bit) of its sign (-1 where the sign
    shares the index byte or does not exist).  Rows are row-major in each plane; in the 4-bit planes group j
    sits in byte j // 2, low nibble first."""
    n = np.asarray(n, dtype=np.int64)
    j = np.asarray(j, dtype=np.int64)
    C, g, mirror = ELUT_FORMATS[fmt]
    none = np.full(np.broadcast(n, j).shape, -1, dtype=np.int64)
    if fmt == "c3g5":
        return n * (K // 5) + j, np.zeros_like(none), none, none
    ib, ish = n * (K // 4) + j // 2, 4 * (j % 2)
    if fmt == "c5g2":
        return ib, ish, N * K // 4 + n * (K // 16) + j // 8, j % 8
    return ib, ish, none, none


def pack_elut(w: np.ndarray, fmt: str) -> np.ndarray:
    w = np.asarray(w)
    N, K = w.shape
    elut_layout_check(fmt, N, K)
    C, g, mirror = ELUT_FORMATS[fmt]
    idx, sign = elut_group_codes(w, C, g, mirror)
    out = np.zeros(elut_packed_bytes(fmt, N, K), dtype=np.uint8)
    nn, jj = np.meshgrid(np.arange(N), np.arange(K // g), indexing="ij")
    ib, ish, sb, sbit = elut_group_position(fmt, nn, jj, N, K)
    field = idx | (sign << 7) if fmt == "c3g5" else idx
    np.bitwise_or.at(out, ib.ravel(), (field << ish).ravel().astype(np.uint8))
    if fmt == "c5g2":
        np.bitwise_or.at(out, sb.ravel(), (sign << sbit).ravel().astype(np.uint8))
    return out


def elut_decode_codes(packed: np.ndarray, fmt: str, N: int, K: int):
    """(index, sign) of every group, [N, K / g] each, read back from a packed buffer."""
    packed = np.asarray(packed, dtype=np.uint8)
    if packed.size != elut_packed_bytes(fmt, N, K):
        raise ValueError("buffer has the wrong size")
    C, g, mirror = ELUT_FORMATS[fmt]
    nn, jj = np.meshgrid(np.arange(N), np.arange(K // g), indexing="ij")
    ib, ish, sb, sbit = elut_group_position(fmt, nn, jj, N, K)
    if fmt == "c3g5":
        byte = packed[ib].astype(np.int64)
        return byte & 0x7F, byte >> 7
    idx = (packed[ib].astype(np.int64) >> ish) & 0xF
    sign = (packed[sb].astype(np.int64) >> sbit) & 1 if fmt == "c5g2" else np.zeros_like(idx)
    return idx, sign


def unpack_elut(packed: np.ndarray, fmt: str, N: int, K: int) -> np.ndarray:
    C, g, mirror = ELUT_FORMATS[fmt]
    idx, sign = elut_decode_codes(packed, fmt, N, K)
    E = elut_entries(C, g, mirror)
    if np.any(idx >= E) or (mirror and np.any((idx == 0) & (sign == 1))):
        raise ValueError("invalid group code")
    d = elut_entry_weights(C, g, mirror)
    grp = d[idx] * np.where(sign == 1, -1, 1)[..., None]
    return grp.reshape(N, K).astype(np.int8)


# ----------------------------------------------------------------------------------------------
# a7: dequantisation epilogue
# ----------------------------------------------------------------------------------------------
def epilogue(acc: np.ndarray, beta, s: np.ndarray) -> np.ndarray:
    """y[m, n] = acc[m, n] * beta / s_m, in float64."""
    return np.asarray(acc, dtype=np.float64) * float(beta) / np.asarray(s, dtype=np.float64)[:, None]


def mpgemm_reference(x: np.ndarray, W: np.ndarray):
    """Whole path on one linear: quantise x, ternarise W, accumulate, dequantise."""
    xq, s = quantize_act(x)
    t, beta = ternarize(W)
    acc = mad_gemm(xq, t)
    return epilogue(acc, beta, s), acc, xq, s, t, beta
