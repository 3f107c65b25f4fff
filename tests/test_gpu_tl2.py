"""GPU parity of the TL2 path (packing, the ELUT tables and the table-lookup accumulation) against the oracle."""
import numpy as np
import pytest
import torch

from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
import paper_2502_11880_amd as B
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _announce(*what):
    print("case:", *what, flush=True)


@pytest.mark.parametrize("N,K", [(16, 64), (16, 384), (32, 448), (48, 832), (64, 1600), (208, 3200), (64, 4096),
                                 (32, 8640), (16, 14336)])
def test_pack_tl2_bit_exact(N, K):
    _announce("pack tl2", N, K)
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(8, 3 * N + K))
    packed, w_scale = H.pack(W, "tl2")
    t_ref, beta_ref = O.ternarize(W.numpy())
    assert H.to_np(w_scale)[0] == beta_ref
    got = H.to_np(packed)
    ref = O.pack_tl2(t_ref)
    assert got.size == ref.size
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("M,K", [(1, 384), (2, 448), (3, 4096), (1, 8640), (5, 14336)])
def test_elut_tables_bit_exact(M, K):
    _announce("elut tables", M, K)
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(6, M + K))
    xq, _ = H.quantize(x)
    three, two = O.tl2_split(K)
    lut = torch.empty((M, three // 3, 16), dtype=torch.int16, device=H.DEV)
    lut1 = torch.empty((M, max(two // 2, 1), 16), dtype=torch.int16, device=H.DEV)
    B.bitnet_elut_tables(xq, lut, lut1 if two else None)
    ref, ref1 = O.elut_tables(H.to_np(xq))
    got = H.to_np(lut).astype(np.int64)
    assert np.array_equal(got[..., :14], ref)
    assert not got[..., 14:].any()
    if two:
        got1 = H.to_np(lut1).astype(np.int64)
        assert np.array_equal(got1[..., :9], ref1)
        assert not got1[..., 9:].any()


def _tl2_vs_oracle(M, N, K, seed, repeat=True):
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 500)
    packed, w_scale = H.pack(W, "tl2")
    xq, s = H.quantize(x)
    y, acc = H.mpgemm("tl2", packed, w_scale, N, K, xq, s)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    acc_np = H.to_np(acc)
    assert np.array_equal(acc_np, acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)
    if repeat:
        y2, acc2 = H.mpgemm("tl2", packed, w_scale, N, K, xq, s)
        assert np.array_equal(H.to_np(acc2), acc_np)


@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (1, 16, 384), (1, 32, 448), (2, 48, 832), (3, 64, 1600),
                                   (4, 208, 3200), (5, 16, 4096), (8, 96, 1536), (9, 32, 8640), (16, 16, 768),
                                   (17, 48, 448), (1, 1024, 4096)])
def test_tl2_mpgemm_parity(M, N, K):
    _announce("tl2 mpgemm", M, N, K)
    _tl2_vs_oracle(M, N, K, seed=inputs.seed_for(5, M * 131 + N * 7 + K))


def test_tl2_elut_matches_i2s_on_same_weights():
    _announce("tl2 == i2s")
    M, N, K = 3, 64, 3200
    W = inputs.weight_f32(N, K, seed=44)
    x = inputs.activation_f32(M, K, seed=45)
    xq, s = H.quantize(x)
    p1, b1 = H.pack(W, "i2s")
    p2, b2 = H.pack(W, "tl2")
    y1, a1 = H.mpgemm("i2s", p1, b1, N, K, xq, s)
    y2, a2 = H.mpgemm("tl2", p2, b2, N, K, xq, s)
    assert np.array_equal(H.to_np(a1), H.to_np(a2))
    assert np.array_equal(H.to_np(y1), H.to_np(y2))


def test_tl2_extreme_values():
    _announce("tl2 extremes")
    N, K = 32, 832
    W = torch.full((N, K), 0.02)
    W[1::2] *= -1
    W[:, 5::7] = 0.0
    x = torch.full((2, K), 5.0)
    x[1] = -5.0
    packed, w_scale = H.pack(W, "tl2")
    xq, s = H.quantize(x)
    y, acc = H.mpgemm("tl2", packed, w_scale, N, K, xq, s)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)


@pytest.mark.parametrize("workload", [0, 1, 2])
def test_tl2_workload_shapes(workload):
    spec = inputs.WORKLOADS[workload]
    for i, (name, K, N, _) in enumerate(spec["linears"]):
        for M in spec["tokens"]:
            _announce("tl2 workload", workload, name, M, N, K)
            _tl2_vs_oracle(M, N, K, seed=inputs.seed_for(workload, i), repeat=False)


# One token through the streaming kernel (tables of the whole row built once per work group): every wave /
# blocks-per-wave configuration (4x1, 8x1, 8x2, 16x2, 16x3), with and without a TL1 tail, the largest K whose
# tables fit in LDS, and enough row groups that work groups walk several of them (both ping-pong tails).
@pytest.mark.parametrize("N,K", [(16, 1536), (48, 1600), (32, 3200), (2400, 4096), (64, 8640), (4112, 12288),
                                 (32, 14336), (9616, 448)])
def test_tl2_stream_one_token(N, K):
    _announce("tl2 stream one token", N, K)
    _tl2_vs_oracle(1, N, K, seed=inputs.seed_for(8, 77 + N + K))


# One token as one launch for several weights that share the activation, quantised inside the launch (the MFMA
# kernel with the row converted in each work group): every wave configuration, 1 to 8 float4 of the row per
# thread (K = 16512: five, rounded up to eight), with and without a TL1 tail; past 48 blocks, row groups in two or
# three batches with 8 float4 per thread (K = 19264 with a 1-unit tail; K = 32768) or 9 (K = 33024, the 100B-class
# down projection; K = 36864, the longest such row), and past 9 float4 per thread the quantiser followed by the
# multi-batch kernel (K = 36928; K = 65472 with a 3-unit tail).
@pytest.mark.parametrize("K,Ns", [(3200, [3200, 3200, 3200]), (4096, [4096, 1024, 1024]), (8640, [3200, 16]),
                                  (14336, [4096]), (1536, [64, 48]), (16512, [32]), (448, [2400]),
                                  (2304, [48]), (4480, [64, 32]), (19264, [48]), (32768, [64, 16]),
                                  (33024, [64, 16]), (36864, [32]), (36928, [16]), (65472, [32])])
def test_tl2_one_token_fused(K, Ns):
    _announce("tl2 one token fused", K, Ns)
    from tests.test_gpu_fused import _fused_case
    _fused_case("tl2", 1, K, Ns, seed=inputs.seed_for(8, 300 + K + len(Ns)))


# Several tokens through the MFMA kernel (triples expanded to int8 through the LDS tables): every wave / blocks-per-
# wave configuration (4x1, 8x1, 8x2, 16x2, 16x3), TL1 tails of 1 to 5 units, 1 to 16 tokens per launch (both
# staging widths), token slices (16 tokens at K = 14336 take two launches of 8; 40 tokens take 16 + 16 + 8), one
# token where the single-token streaming kernel's tables do not fit (K = 16384); past 48 blocks, row groups in
# several batches with token slices sized to LDS (K = 19200 and 19264: 50 blocks, the second with a 1-unit tail;
# K = 33024: three tokens per slice; K = 20480: five per slice and a 2-unit tail; K = 65600: one per slice; K = 121536:
# the longest row whose codes fit), and past that the table-lookup kernel (K = 132096, the largest K).
@pytest.mark.parametrize("M,N,K", [(2, 48, 832), (3, 64, 1600), (8, 96, 1536), (4, 208, 3200), (16, 64, 4096),
                                   (9, 32, 8640), (12, 48, 6080), (5, 16, 14336), (16, 32, 14336), (40, 48, 4096),
                                   (1, 64, 16384), (2, 16, 19200), (7, 16, 384), (1, 64, 19264), (3, 48, 33024),
                                   (8, 32, 33024), (16, 16, 20480), (2, 16, 65600), (1, 16, 121536),
                                   (1, 16, 132096)])
def test_tl2_mfma_decode(M, N, K):
    _announce("tl2 mfma decode", M, N, K)
    _tl2_vs_oracle(M, N, K, seed=inputs.seed_for(8, 900 + M * 17 + N + K))


# Enough row groups that work groups walk 2, 3 or more of them (both ends of the two-register-set pipeline).
@pytest.mark.parametrize("M,N", [(8, 16 * 2000), (3, 16 * 3000), (8, 16 * 5000)])
def test_tl2_mfma_decode_streaming(M, N):
    _announce("tl2 mfma decode streaming", M, N, 448)
    _tl2_vs_oracle(M, N, 448, seed=inputs.seed_for(8, 1300 + M + N), repeat=False)


# The 8B-class groups at 8 tokens as one launch per group (quantised once).
@pytest.mark.parametrize("K,Ns", [(4096, [4096, 1024, 1024]), (4096, [14336]), (14336, [4096])])
def test_tl2_mfma_fused(K, Ns):
    _announce("tl2 mfma fused", 8, K, Ns)
    from tests.test_gpu_fused import _fused_case
    _fused_case("tl2", 8, K, Ns, seed=inputs.seed_for(8, 1500 + K + len(Ns)))


# More than 16 tokens: the TL2 weights rewritten in the I2_S layout (in the workspace), then the I2_S prefill GEMM
# on them; TL1 tails of 0 to 5 units (K = 320 has no 384-k block at all), ragged token tiles, with and without
# the token sums given (split-K needs them).
@pytest.mark.parametrize("M,N,K", [(17, 48, 448), (40, 48, 832), (33, 16, 320), (64, 96, 1536), (129, 208, 3200),
                                   (300, 512, 4096), (200, 64, 6080)])
@pytest.mark.parametrize("rowsum", [False, True])
def test_tl2_prefill(M, N, K, rowsum):
    _announce("tl2 prefill", M, N, K, rowsum)
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(8, 1700 + M + N + K))
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(8, 1800 + M + K))
    packed, w_scale = H.pack(W, "tl2")
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y, acc = H.mpgemm("tl2", packed, w_scale, N, K, xq, s, x_rowsum=rs if rowsum else None)
    y_ref, acc_ref, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), y_ref, acc_ref)


# The 8B-class shapes at 2048 tokens (every output) and a fused group (one prefill launch for all weights).
def test_tl2_prefill_workload():
    _announce("tl2 prefill workload", 2048, 14336, 4096)
    M, N, K = 2048, 14336, 4096
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(8, 1900))
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(8, 1901))
    packed, w_scale = H.pack(W, "tl2")
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y, acc = H.mpgemm("tl2", packed, w_scale, N, K, xq, s, x_rowsum=rs)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    t_ref, beta = O.ternarize(W.numpy())
    acc_ref = O.mad_gemm(xq_ref, t_ref)
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), O.epilogue(acc_ref, beta, s_ref), acc_ref)


@pytest.mark.parametrize("M,K,Ns,split_ws", [(600, 1536, [512, 1024, 2048], True), (40, 832, [48, 16, 64], False),
                                             (2048, 4096, [4096, 1024, 1024], True)])
def test_tl2_prefill_fused(M, K, Ns, split_ws):
    _announce("tl2 prefill fused", M, K, Ns, split_ws)
    from tests.test_gpu_fused import _fused_case
    _fused_case("tl2", M, K, Ns, seed=inputs.seed_for(8, 2000 + M + K), split_ws=split_ws)
