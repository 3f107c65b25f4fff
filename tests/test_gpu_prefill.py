"""GPU parity of the prefill path (M > 16 tokens, int8-MFMA GEMM) against the oracle.

Every test compares every output with the oracle, including the 8B-class prefill shapes (M = 512 and 2048).
"""
import numpy as np
import pytest

from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _announce(*what):
    print("case:", *what, flush=True)


def _prefill_vs_oracle(M, N, K, seed, sample_rows=None, layout="i2s", rowsum=True):
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 500)
    packed, w_scale = H.pack(W, layout)
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y, acc = H.mpgemm(layout, packed, w_scale, N, K, xq, s, x_rowsum=rs if rowsum else None)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    t_ref, beta_ref = O.ternarize(W.numpy())
    assert np.array_equal(H.to_np(xq), xq_ref)
    rows = np.arange(M) if sample_rows is None else np.unique(
        np.concatenate([[0, M - 1], np.random.default_rng(seed).choice(M, size=sample_rows, replace=False)]))
    acc_ref = O.mad_gemm(xq_ref[rows], t_ref)
    y_ref = O.epilogue(acc_ref, beta_ref, s_ref[rows])
    acc_np = H.to_np(acc)[rows]
    assert np.array_equal(acc_np, acc_ref)
    H.check_y(H.to_np(y)[rows], y_ref, acc_ref)


@pytest.mark.parametrize("M,N,K", [(17, 16, 64), (33, 48, 320), (64, 128, 256), (100, 208, 832), (128, 256, 1536),
                                   (129, 1040, 448), (200, 64, 3200), (256, 384, 8640), (300, 512, 4096)])
@pytest.mark.parametrize("rowsum", [True, False])
def test_i2s_prefill_parity(M, N, K, rowsum):
    _announce("i2s prefill", M, N, K, rowsum)
    _prefill_vs_oracle(M, N, K, seed=inputs.seed_for(4, M * 131 + N * 7 + K), rowsum=rowsum)


@pytest.mark.parametrize("M,N,K", [(2048, 8192, 512), (2000, 8208, 320)])
@pytest.mark.parametrize("rowsum", [True, False])
def test_i2s_prefill_wide_tiles(M, N, K, rowsum):
    # grids of at least one 128 x 512 tile per CU take the widest tile; K = 320 ends in a short block
    _announce("i2s prefill wide tiles", M, N, K, rowsum)
    _prefill_vs_oracle(M, N, K, seed=inputs.seed_for(4, 7 * M + N + K), rowsum=rowsum)


def test_i2s_prefill_extreme_values():
    _announce("i2s prefill extremes")
    import torch
    M, N, K = 40, 64, 768
    W = torch.full((N, K), 0.02)
    W[1::2] *= -1
    x = torch.full((M, K), 5.0)
    x[1::2] = -5.0
    packed, w_scale = H.pack(W, "i2s")
    xq, s = H.quantize(x)
    y, acc = H.mpgemm("i2s", packed, w_scale, N, K, xq, s)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.abs(acc_ref).max() == 127 * K
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)


@pytest.mark.parametrize("M", [512, 2048])
def test_i2s_prefill_workload_shapes(M):
    spec = inputs.WORKLOADS[3]
    for i, (name, K, N, _) in enumerate(spec["linears"]):
        if name in ("k", "v", "up"):        # same shapes as q / gate; keep the suite short
            continue
        _announce("prefill workload", name, M, N, K)
        _prefill_vs_oracle(M, N, K, seed=inputs.seed_for(3, i))
