"""GPU parity of the I2_S path against the CPU oracle, through the C ABI.

Integers (beta bits, packed bytes, int8 codes, activation scales, int32 accumulators) must match the
oracle bit for bit; fp32 outputs within 1e-5 relative of the float64 reference.
"""
import numpy as np
import pytest
import torch

from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _announce(*what):
    print("case:", *what, flush=True)


# ------------------------------------------------------------------------------------------------
# a3: activation quantisation
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("M,K", [(1, 64), (1, 1536), (3, 1001), (8, 4096), (17, 3200), (1, 33024), (96, 14336),
                                 (2, 1)])
def test_quantize_act_bit_exact(M, K):
    _announce("quantize", M, K)
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(9, M * 7 + K))
    xq, s, rs = H.quantize(x, with_rowsum=True)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(xq), xq_ref)
    assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))


# More than 64 rows: one wave per row up to K = 4096, one work group per row above; constructed ties and an
# all-zero row placed among random rows.
@pytest.mark.parametrize("K", [64, 1024, 1600, 4096, 4160, 14336])
def test_quantize_act_many_rows(K):
    _announce("quantize many rows", 130, K)
    x = inputs.activation_f32(130, K, seed=inputs.seed_for(9, 5000 + K))
    x[7] = 0.0
    x[8, :6] = torch.tensor([127.0, 63.5, -0.5, 1.5, 2.5, -127.0])
    x[8, 6:] = 0.25
    xq, s, rs = H.quantize(x, with_rowsum=True)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(xq), xq_ref)
    assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))


# Many rows longer than 4096 (one 256-lane group per row, up to 16 float4 per lane), with and without the code
# sums; a zero row and a tie row placed late.
@pytest.mark.parametrize("M,K,rowsum", [(2048, 14336, True), (1500, 8192, False), (3000, 12288, True),
                                        (700, 16384, False)])
def test_quantize_act_long_rows(M, K, rowsum):
    _announce("quantize long rows", M, K, rowsum)
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(9, 6000 + M + K))
    x[M - 3] = 0.0
    x[M - 2, :6] = torch.tensor([127.0, 63.5, -0.5, 1.5, 2.5, -127.0])
    x[M - 2, 6:] = 0.25
    out = H.quantize(x, with_rowsum=rowsum)
    xq, s = out[0], out[1]
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(xq), xq_ref)
    if rowsum:
        assert np.array_equal(H.to_np(out[2]), xq_ref.astype(np.int64).sum(1))


def test_quantize_act_constructed_ties_and_zero_rows():
    _announce("quantize constructed")
    x = torch.zeros((3, 64), dtype=torch.float32)
    x[0, :6] = torch.tensor([127.0, 63.5, -0.5, 1.5, 2.5, -127.0])
    x[1, :3] = torch.tensor([1.0, 0.5, -0.25])
    xq, s = H.quantize(x)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(xq), xq_ref)


# ------------------------------------------------------------------------------------------------
# a1 + a2: ternarisation and I2_S packing
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("N,K", [(16, 64), (32, 320), (48, 832), (64, 1536), (208, 3200), (1024, 4096)])
def test_pack_i2s_bit_exact(N, K):
    _announce("pack i2s", N, K)
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(8, N + K))
    packed, w_scale = H.pack(W, "i2s")
    t_ref, beta_ref = O.ternarize(W.numpy())
    assert H.to_np(w_scale).view(np.uint32)[0] == np.float32(beta_ref).view(np.uint32)
    assert np.array_equal(H.to_np(packed), O.pack_i2s(t_ref))


def test_pack_beta_constructed():
    _announce("pack constructed beta")
    one = np.float32(1.0)
    e = np.float32(2.0 ** -23)
    W = np.zeros((16, 64), np.float32)
    W[0, :4] = [0.5, -0.5, 1.5, -1.5]
    W[1, 0] = 60.0     # mean now (0.5+0.5+1.5+1.5+60)/1024
    packed, w_scale = H.pack(torch.from_numpy(W), "i2s")
    t_ref, beta_ref = O.ternarize(W)
    assert H.to_np(w_scale)[0] == beta_ref
    assert np.array_equal(H.to_np(packed), O.pack_i2s(t_ref))
    # ties of the exact mean itself (values chosen so the mean is a float32 midpoint)
    for vals, want in (([one, one + e], one), ([one + e, one + 2 * e], one + 2 * e)):
        W = np.tile(np.array(vals, np.float32), (16, 32))
        _, w_scale = H.pack(torch.from_numpy(W), "i2s")
        assert H.to_np(w_scale)[0] == want
    # all-zero weight: beta = 0 and every code is "0"
    packed, w_scale = H.pack(torch.zeros((16, 64)), "i2s")
    assert H.to_np(w_scale)[0] == 0.0
    assert np.all(H.to_np(packed) == 0b01010101)


# ------------------------------------------------------------------------------------------------
# a5 + a7: decode accumulation and epilogue
# ------------------------------------------------------------------------------------------------
def _path_vs_oracle(M, N, K, seed, layout="i2s", repeat=True, rowsum=True):
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 500)
    packed, w_scale = H.pack(W, layout)
    xq, s, rs = H.quantize(x, with_rowsum=True)
    ws = H.workspace(layout, M, N, K)
    y, acc = H.mpgemm(layout, packed, w_scale, N, K, xq, s, ws, x_rowsum=rs if rowsum else None)
    y_ref, acc_ref, xq_ref, s_ref, t_ref, beta_ref = O.mpgemm_reference(x.numpy(), W.numpy())
    acc_np = H.to_np(acc)
    assert np.array_equal(acc_np, acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)
    if repeat:   # the other way to remove the code offset, same workspace: identical results
        y2, acc2 = H.mpgemm(layout, packed, w_scale, N, K, xq, s, ws, x_rowsum=None if rowsum else rs)
        assert np.array_equal(H.to_np(acc2), acc_np)
        assert np.array_equal(H.to_np(y2), H.to_np(y))


@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (1, 32, 320), (2, 48, 832), (5, 64, 1536), (8, 208, 3200),
                                   (16, 96, 1024), (1, 1024, 4096), (3, 16, 8640), (1, 4096, 1536),
                                   (17, 64, 576), (33, 48, 448), (1, 16, 132096), (4, 32, 65600),
                                   (16, 16, 20480)])
@pytest.mark.parametrize("rowsum", [True, False])
def test_i2s_mpgemm_parity(M, N, K, rowsum):
    _announce("i2s mpgemm", M, N, K, rowsum)
    _path_vs_oracle(M, N, K, seed=inputs.seed_for(7, M * 131 + N * 7 + K), rowsum=rowsum)


def test_i2s_mpgemm_extreme_values():
    _announce("i2s extremes")
    N, K = 32, 512
    W = torch.full((N, K), 0.02)            # all +1 after ternarisation
    W[1::2] *= -1                           # odd rows all -1
    x = torch.full((2, K), 5.0)             # every code = 127 ...
    x[1] = -5.0                             # ... or -127
    packed, w_scale = H.pack(W, "i2s")
    xq, s = H.quantize(x)
    y, acc = H.mpgemm("i2s", packed, w_scale, N, K, xq, s)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.abs(acc_ref).max() == 127 * K
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)


def test_i2s_mpgemm_without_acc_output():
    _announce("i2s y only")
    N, K, M = 64, 1024, 2
    W = inputs.weight_f32(N, K, seed=11)
    x = inputs.activation_f32(M, K, seed=12)
    packed, w_scale = H.pack(W)
    xq, s = H.quantize(x)
    y, _ = H.mpgemm("i2s", packed, w_scale, N, K, xq, s, want_acc=False)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    H.check_y(H.to_np(y), y_ref, acc_ref)


# ------------------------------------------------------------------------------------------------
# Full workload shapes, in the launch configuration the benchmark uses
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("workload", [0, 1, 2])
def test_i2s_workload_shapes(workload):
    spec = inputs.WORKLOADS[workload]
    for i, (name, K, N, _) in enumerate(spec["linears"]):
        for M in spec["tokens"]:
            _announce("workload", workload, name, M, N, K)
            _path_vs_oracle(M, N, K, seed=inputs.seed_for(workload, i), repeat=False)
