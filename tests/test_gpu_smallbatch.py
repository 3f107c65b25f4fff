"""GPU parity of the small-batch regime (17 to 112 tokens): the decode GEMV in token slices of up to 16 (8 or 12 where
a slice's codes must fit in LDS), one launch for all slices, for I2_S and TL1 weights, against the oracle, through
bitnet_mpgemm and bitnet_mpgemm_fused; and the boundaries of the regime (113 tokens, no token sums: the prefill
GEMM)."""
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


def _vs_oracle(layout, M, N, K, seed, rowsum=True):
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 1)
    packed, w_scale = H.pack(W, layout)
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y, acc = H.mpgemm(layout, packed, w_scale, N, K, xq, s, x_rowsum=rs if rowsum else None)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)


# Slices of 16 (K <= 8176), 12 (K = 8640) and 8 (K = 14336); last slices of 1..15 tokens; 4-wave groups (K <= 4096,
# many row groups) and 16-wave groups; a short last block (K = 320).
@pytest.mark.parametrize("layout", ["i2s", "tl1"])
@pytest.mark.parametrize("M,N,K", [(17, 64, 320), (24, 9600, 4096), (32, 4096, 4096), (48, 208, 3200),
                                   (64, 1024, 8640), (100, 512, 14336), (112, 4096, 4096), (33, 16, 64)])
def test_small_batch_parity(layout, M, N, K):
    _announce("small batch", layout, M, N, K)
    _vs_oracle(layout, M, N, K, seed=inputs.seed_for(14, M * 7 + N + K))


@pytest.mark.parametrize("layout", ["i2s", "tl1"])
@pytest.mark.parametrize("M,rowsum", [(113, True), (40, False)])
def test_small_batch_boundaries(layout, M, rowsum):
    _announce("small batch boundary", layout, M, rowsum)
    _vs_oracle(layout, M, 256, 1536, seed=inputs.seed_for(14, 900 + M), rowsum=rowsum)


# The 8B-class groups at 32 and 112 tokens through the fused call (quantiser + one sliced launch per group).
@pytest.mark.parametrize("layout", ["i2s", "tl1"])
@pytest.mark.parametrize("M,K,Ns", [(32, 4096, [4096, 1024, 1024]), (112, 4096, [14336, 14336]),
                                    (64, 14336, [4096])])
def test_small_batch_fused(layout, M, K, Ns):
    _announce("small batch fused", layout, M, K, Ns)
    from tests.test_gpu_fused import _fused_case
    _fused_case(layout, M, K, Ns, seed=inputs.seed_for(14, 2000 + M + K + len(Ns)))
