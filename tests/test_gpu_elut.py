"""GPU parity of the integer-weight ELUT layouts (Appendix "Insight", Table 3, Algorithm "ELUT mpGEMM"): packing
bit-exact against the oracle's formats, and the table-lookup accumulation and epilogue against the oracle's MAD sum,
for C = 4 and C = 5 with g = 2 and ternary groups of g = 5."""
import numpy as np
import pytest
import torch

import paper_2502_11880_amd as B
from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu

FMTS = list(O.ELUT_FORMATS)


def _announce(*what):
    print("case:", *what, flush=True)


def _pack(fmt, w):
    N, K = w.shape
    packed = torch.empty(B.bitnet_packed_bytes(fmt, N, K), dtype=torch.uint8, device=H.DEV)
    B.bitnet_pack_int_weights(fmt, w.to(H.DEV).contiguous(), packed)
    return packed


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("N,K", [(16, 640), (48, 1280), (208, 3200), (64, 8640)])
def test_pack_int_bit_exact(fmt, N, K):
    _announce("pack", fmt, N, K)
    C, g, mirror = O.ELUT_FORMATS[fmt]
    w = inputs.int_weights(N, K, C, seed=inputs.seed_for(13, N + K + C))
    assert np.array_equal(H.to_np(_pack(fmt, w)), O.pack_elut(w.numpy(), fmt))


@pytest.mark.parametrize("fmt", FMTS)
def test_pack_int_clamps_values_outside_the_set(fmt):
    _announce("pack clamp", fmt)
    C, g, mirror = O.ELUT_FORMATS[fmt]
    vals = O.elut_values(C)
    w = torch.randint(-6, 7, (32, 640), generator=torch.Generator().manual_seed(3)).to(torch.int8)
    ref = O.pack_elut(np.clip(w.numpy(), vals[0], vals[-1]), fmt)
    assert np.array_equal(H.to_np(_pack(fmt, w)), ref)


def _vs_oracle(fmt, M, N, K, seed, extreme=False):
    C, g, mirror = O.ELUT_FORMATS[fmt]
    w = inputs.int_weights(N, K, C, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 1)
    if extreme:
        vals = O.elut_values(C)
        w[0::2] = int(vals[0])
        w[1::2] = int(vals[-1])
        x = torch.full((M, K), 3.0)
        x[1::2] = -3.0                                       # every code +127 or -127
    packed = _pack(fmt, w)
    beta = torch.tensor([0.0173], dtype=torch.float32)
    xq, s = H.quantize(x)
    y, acc = H.mpgemm(fmt, packed, beta.to(H.DEV), N, K, xq, s)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    acc_ref = O.mad_gemm(xq_ref, w.numpy())
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), O.epilogue(acc_ref, beta.numpy()[0], s_ref), acc_ref)
    return acc_ref


# 1 to 17 tokens (slices of 4, or 2 for c3g5), partial last blocks (K = 640, 3200, 8640), the 3B-class shapes, and
# every rows-per-wave count the launcher picks (1 to 8: the fewest rows per wave that keep one work group per CU;
# N = 12288 .. 30720 take 3, 4, 5, 6, 7 and 8 on 256 CUs).
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K", [(1, 16, 640), (2, 48, 1280), (3, 208, 3200), (5, 64, 8640), (8, 3200, 3200),
                                   (17, 96, 640), (1, 9600, 640), (1, 8640, 3200), (3, 12288, 640), (1, 16384, 640),
                                   (1, 17280, 640), (2, 20496, 640), (1, 28672, 640), (1, 30720, 640)])
def test_elut_mpgemm_parity(fmt, M, N, K):
    _announce("elut mpgemm", fmt, M, N, K)
    _vs_oracle(fmt, M, N, K, seed=inputs.seed_for(13, 100 + M * 31 + N + K))


@pytest.mark.parametrize("fmt", FMTS)
def test_elut_extreme_values(fmt):
    _announce("elut extremes", fmt)
    C, g, mirror = O.ELUT_FORMATS[fmt]
    acc_ref = _vs_oracle(fmt, 3, 32, 1280, seed=inputs.seed_for(13, 7), extreme=True)
    assert np.abs(acc_ref).max() == 127 * 1280 * max(abs(int(v)) for v in O.elut_values(C))


@pytest.mark.parametrize("fmt", FMTS)
def test_elut_fused_and_noalloc(fmt):
    _announce("elut fused", fmt)
    C, g, mirror = O.ELUT_FORMATS[fmt]
    M, K, Ns = 3, 3200, [3200, 640]
    ws_ = [inputs.int_weights(N, K, C, seed=inputs.seed_for(13, 300 + i)) for i, N in enumerate(Ns)]
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(13, 399))
    packs = [_pack(fmt, w) for w in ws_]
    betas = [torch.tensor([0.01 * (i + 1)], dtype=torch.float32, device=H.DEV) for i in range(len(Ns))]
    xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.empty(M, dtype=torch.float32, device=H.DEV)
    rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
    ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    B.bitnet_mpgemm_fused(fmt, packs, betas, x.to(H.DEV), xq, s, rs, ys)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    for w, b, y, p, N in zip(ws_, betas, ys, packs, Ns):
        acc_ref = O.mad_gemm(xq_ref, w.numpy())
        H.check_y(H.to_np(y), O.epilogue(acc_ref, float(H.to_np(b)[0]), s_ref), acc_ref)
        y2 = torch.empty((M, N), dtype=torch.float32, device=H.DEV)
        B.bitnet_mpgemm_noalloc(fmt, p, b, N, K, xq, s, y2)
        assert np.array_equal(H.to_np(y2), H.to_np(y))


# The fused call: every weight of the group in one table-lookup launch (rows of several weights in one work group,
# ragged row counts); at one token the launch also quantises the row (codes, scale and code sum bit-exact against
# the oracle's quantiser), otherwise the quantiser runs first.  Outputs against the oracle and bit-identical to the
# separate calls.
@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,K,Ns", [(1, 3200, [3200, 3200, 3200]), (1, 640, [16, 48, 208]), (1, 8640, [3200]),
                                    (1, 1280, [9600, 16]), (6, 640, [48, 16]), (1, 640, [8640, 8640]),
                                    (1, 640, [14336, 14336])])
def test_elut_fused_groups(fmt, M, K, Ns):
    _announce("elut fused groups", fmt, M, K, Ns)
    _elut_fused(fmt, M, K, Ns)


def _elut_fused(fmt, M, K, Ns):
    C, g, mirror = O.ELUT_FORMATS[fmt]
    ws_ = [inputs.int_weights(N, K, C, seed=inputs.seed_for(13, 500 + 7 * i + K)) for i, N in enumerate(Ns)]
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(13, 599 + K + M))
    packs = [_pack(fmt, w) for w in ws_]
    betas = [torch.tensor([0.013 * (i + 1)], dtype=torch.float32, device=H.DEV) for i in range(len(Ns))]
    xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.empty(M, dtype=torch.float32, device=H.DEV)
    rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
    ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    B.bitnet_mpgemm_fused(fmt, packs, betas, x.to(H.DEV), xq, s, rs, ys)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(xq), xq_ref)
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))
    for w, b, y, p, N in zip(ws_, betas, ys, packs, Ns):
        acc_ref = O.mad_gemm(xq_ref, w.numpy())
        H.check_y(H.to_np(y), O.epilogue(acc_ref, float(H.to_np(b)[0]), s_ref), acc_ref)
        y_sep, acc = H.mpgemm(fmt, p, b, N, K, xq, s)
        assert np.array_equal(H.to_np(acc), acc_ref)
        assert np.array_equal(H.to_np(y_sep), H.to_np(y))


# The exact groups the benchmark times on the integer-weight layouts: the 3B-class layer set at one token (every
# format) and the 8B-class layer set at one and eight tokens (C4G2 and C5G2; C3G5 needs K % 320 == 0).
ELUT_WORKLOAD_GROUPS = (
    [(fmt, 1, K, Ns) for fmt in FMTS
     for K, Ns in [(3200, [3200, 3200, 3200]), (3200, [3200]), (3200, [8640, 8640]), (8640, [3200])]] +
    [(fmt, M, K, Ns) for fmt in ("c4g2", "c5g2") for M in (1, 8)
     for K, Ns in [(4096, [4096, 1024, 1024]), (4096, [4096]), (4096, [14336, 14336]), (14336, [4096])]])


@pytest.mark.parametrize("fmt,M,K,Ns", ELUT_WORKLOAD_GROUPS)
def test_elut_fused_workload_groups(fmt, M, K, Ns):
    _announce("elut fused workload group", fmt, M, K, Ns)
    _elut_fused(fmt, M, K, Ns)
