"""GPU parity of the TL1 layout (Table 1 "TL1_1", Algorithm TL1, Table 5): packing, the decode GEMV (pair codes
expanded to int8 in registers for MFMA), one-token fused launches, and more than 16 tokens (weights rewritten in
the I2_S layout for the prefill GEMM), against the oracle, and bit-identical to I2_S on the same weights."""
import numpy as np
import pytest
import torch

import paper_2502_11880_amd as B
from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _announce(*what):
    print("case:", *what, flush=True)


@pytest.mark.parametrize("N,K", [(16, 64), (32, 320), (48, 832), (64, 1600), (208, 3200), (16, 4096)])
def test_pack_tl1_bit_exact(N, K):
    _announce("pack tl1", N, K)
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(11, N + K))
    packed, w_scale = H.pack(W, "tl1")
    t_ref, beta_ref = O.ternarize(W.numpy())
    assert np.array_equal(H.to_np(w_scale).view(np.uint32), np.array([beta_ref], np.float32).view(np.uint32))
    assert np.array_equal(H.to_np(packed), O.pack_tl1(t_ref))


def _vs_oracle(M, N, K, seed, rowsum=True):
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 1)
    packed, w_scale = H.pack(W, "tl1")
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y, acc = H.mpgemm("tl1", packed, w_scale, N, K, xq, s, x_rowsum=rs if rowsum else None)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)
    # the same weights in I2_S give the same integers and the same fp32 outputs
    p2, b2 = H.pack(W, "i2s")
    y2, acc2 = H.mpgemm("i2s", p2, b2, N, K, xq, s, x_rowsum=rs if rowsum else None)
    assert np.array_equal(H.to_np(acc2), H.to_np(acc))
    assert np.array_equal(H.to_np(y2), H.to_np(y))


# Decode GEMV, 1..16 tokens: short last blocks (K = 320, 832, 1600), the 3B / 8B shapes, every launch shape of the
# multi-token kernels (4- and 16-wave streaming groups, the one-group-per-row-group kernel at K = 16448 > 16384).
@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (1, 32, 320), (2, 48, 832), (3, 64, 1600), (5, 208, 3200),
                                   (8, 4096, 4096), (16, 64, 4096), (1, 3200, 8640), (4, 4096, 14336),
                                   (8, 32, 16448), (16, 9600, 4096), (1, 16000, 1088)])
@pytest.mark.parametrize("rowsum", [True, False])
def test_tl1_decode_parity(M, N, K, rowsum):
    _announce("tl1 decode", M, N, K, rowsum)
    _vs_oracle(M, N, K, seed=inputs.seed_for(11, 100 + 7 * M + N + K), rowsum=rowsum)


# More than 16 tokens: the TL1 words rewritten as I2_S words in the workspace, then the prefill GEMM (split-K too).
@pytest.mark.parametrize("M,N,K", [(17, 16, 64), (33, 48, 320), (129, 208, 3200), (300, 512, 4096),
                                   (2048, 4096, 4096)])
@pytest.mark.parametrize("rowsum", [True, False])
def test_tl1_prefill_parity(M, N, K, rowsum):
    _announce("tl1 prefill", M, N, K, rowsum)
    _vs_oracle(M, N, K, seed=inputs.seed_for(11, 300 + M + N + K), rowsum=rowsum)


def test_tl1_extreme_values():
    _announce("tl1 extremes")
    for M in (1, 40):
        N, K = 64, 768
        W = torch.full((N, K), 0.02)
        W[1::2] *= -1
        x = torch.full((M, K), 5.0)
        x[1::2] = -5.0
        packed, w_scale = H.pack(W, "tl1")
        xq, s = H.quantize(x)
        y, acc = H.mpgemm("tl1", packed, w_scale, N, K, xq, s)
        y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
        assert np.abs(acc_ref).max() == 127 * K
        assert np.array_equal(H.to_np(acc), acc_ref)
        H.check_y(H.to_np(y), y_ref, acc_ref)


# Fused calls: several tokens (quantiser + one decode launch), more than 16 (one transcoding launch for all the
# weights + one prefill launch).  One token is covered with the other layouts in test_gpu_fused.py.
@pytest.mark.parametrize("M,K,Ns,split_ws", [(8, 4096, [4096, 1024, 1024], False), (5, 3200, [8640, 8640], False),
                                             (16, 14336, [4096], False), (40, 832, [48, 16, 64], True),
                                             (600, 1536, [512, 1024, 2048], True), (2048, 4096, [14336], True)])
def test_tl1_fused(M, K, Ns, split_ws):
    _announce("tl1 fused", M, K, Ns, split_ws)
    from tests.test_gpu_fused import _fused_case
    _fused_case("tl1", M, K, Ns, seed=inputs.seed_for(11, 700 + M + K), split_ws=split_ws)
