"""GPU parity of bitnet_mpgemm_fused (quantise once, several products in one launch) against the oracle and
against the separate quantise + mpGEMM calls."""
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


def _fused_case(layout, M, K, Ns, seed, split_ws=False, sample_rows=None):
    Ws = [inputs.weight_f32(N, K, seed=seed + i) for i, N in enumerate(Ns)]
    x = inputs.activation_f32(M, K, seed=seed + 100)
    packs = [H.pack(W, layout) for W in Ws]
    xd = x.to(H.DEV)
    xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.empty(M, dtype=torch.float32, device=H.DEV)
    rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
    ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    need = max(B.bitnet_mpgemm_workspace_bytes(layout, M, N, K) for N in Ns)
    if split_ws:
        need = max(need, B.bitnet_mpgemm_fused_workspace_bytes(layout, Ns, K, M))
    ws = torch.zeros(max(16, need), dtype=torch.uint8, device=H.DEV)
    B.bitnet_mpgemm_fused(layout, [p for p, _ in packs], [b for _, b in packs], xd, xq, s, rs, ys, ws)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(xq), xq_ref)
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))
    rows = np.arange(M) if sample_rows is None else np.unique(
        np.concatenate([[0, M - 1], np.random.default_rng(seed).choice(M, size=sample_rows, replace=False)]))
    for i, (W, (p, b), y) in enumerate(zip(Ws, packs, ys)):
        t_ref, beta_ref = O.ternarize(W.numpy())
        acc_ref = O.mad_gemm(xq_ref[rows], t_ref)
        H.check_y(H.to_np(y)[rows], O.epilogue(acc_ref, beta_ref, s_ref[rows]), acc_ref)
        y_sep, _ = H.mpgemm(layout, p, b, Ns[i], K, xq, s, x_rowsum=rs)
        assert np.array_equal(H.to_np(y), H.to_np(y_sep))      # identical to the separate calls
    # the products alone, on the activation quantised above (x = NULL)
    ys2 = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    B.bitnet_mpgemm_fused(layout, [p for p, _ in packs], [b for _, b in packs], None, xq, s, rs, ys2, ws)
    for y, y2 in zip(ys, ys2):
        assert np.array_equal(H.to_np(y), H.to_np(y2))


@pytest.mark.parametrize("M,K,Ns", [(1, 64, [16]), (1, 320, [16, 48, 32]), (2, 832, [64, 16]),
                                    (1, 3200, [3200, 3200, 3200]), (1, 3200, [8640, 8640]), (1, 8640, [3200]),
                                    (8, 4096, [4096, 1024, 1024]), (5, 1536, [208, 96, 16, 64, 32, 48, 128, 16]),
                                    (16, 3840, [48]), (8, 14336, [64, 32]), (16, 4096, [32])])
def test_fused_i2s(M, K, Ns):
    _announce("fused i2s", M, K, Ns)
    _fused_case("i2s", M, K, Ns, seed=inputs.seed_for(2, M * 7 + K + len(Ns)))


# One token at sizes that reach every launch configuration of the streaming single-token kernel on a 256-CU
# MI355X: 2900 row groups (several row groups per work group, both ping-pong tails, a 64-k last block);
# K = 16448 (two weight batches per row group, two row groups per work group); K = 33024 (three batches,
# the widest activation register set).
@pytest.mark.parametrize("K,Ns", [(1088, [16000, 16000, 14400]), (16448, [4800]), (33024, [2400])])
def test_fused_i2s_streaming(K, Ns):
    _announce("fused i2s streaming", 1, K, Ns)
    _fused_case("i2s", 1, K, Ns, seed=inputs.seed_for(2, 500 + K))


# Several tokens at sizes where the multi-token streaming kernel walks several row groups per work group
# (2900, 600 and 1080 row groups), with a 64-k last block in the first case.
@pytest.mark.parametrize("M,K,Ns", [(8, 1088, [16000, 16000, 14400]), (16, 4096, [9600]), (5, 3200, [8640, 8640])])
def test_fused_i2s_streaming_tokens(M, K, Ns):
    _announce("fused i2s streaming tokens", M, K, Ns)
    _fused_case("i2s", M, K, Ns, seed=inputs.seed_for(2, 700 + M + K))


# More than 16 tokens: one prefill launch over the weights' concatenated row tiles; with a workspace from
# bitnet_mpgemm_fused_workspace_bytes small grids also split K over all the weights.
@pytest.mark.parametrize("M,K,Ns", [(40, 832, [48, 16, 64]), (300, 3200, [3200, 3200, 3200]),
                                    (129, 8640, [3200, 16]), (600, 1536, [512, 1024, 2048])])
@pytest.mark.parametrize("split_ws", [False, True])
def test_fused_i2s_prefill(M, K, Ns, split_ws):
    _announce("fused i2s prefill", M, K, Ns, split_ws)
    _fused_case("i2s", M, K, Ns, seed=inputs.seed_for(2, 900 + M + K + len(Ns)), split_ws=split_ws)


# The 8B-class q/k/v and gate/up groups at 2048 tokens (sampled rows against the oracle; every output against the
# separate calls).
@pytest.mark.parametrize("Ns", [[4096, 1024, 1024], [14336, 14336]])
def test_fused_i2s_prefill_workload(Ns):
    _announce("fused i2s prefill workload", 2048, 4096, Ns)
    _fused_case("i2s", 2048, 4096, Ns, seed=inputs.seed_for(3, 50 + len(Ns)), split_ws=True, sample_rows=6)


@pytest.mark.parametrize("M,K,Ns", [(1, 448, [16, 32]), (3, 4096, [64, 48])])
def test_fused_tl2(M, K, Ns):
    _announce("fused tl2", M, K, Ns)
    _fused_case("tl2", M, K, Ns, seed=inputs.seed_for(2, 99 + M + K))
