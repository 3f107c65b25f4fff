"""GPU parity of the lossy TL2_0 and TL1_0 kernels (Table 1; Sec. 3.2.1): table lookups on tables quantised to int8
with a power-of-two scale per token and table block.  The accumulators are the oracle's lossy integers exactly and
the outputs within 1e-5 of their float64 epilogue; with codes small enough for every table entry to fit int8 they
are the exact MAD sums."""
import numpy as np
import pytest
import torch

from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _announce(*what):
    print("case:", *what, flush=True)


def _route(layout):
    if layout == "tl2_0":
        return O.pack_tl2, O.elut_gemm_lossy
    return O.pack_tl1, O.elut_gemm_tl1_lossy


@pytest.mark.parametrize("layout", ["tl2_0", "tl1_0"])
@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (1, 32, 448), (2, 48, 832), (3, 64, 1600), (8, 208, 3200),
                                   (5, 64, 4096), (1, 3200, 8640), (11, 32, 14336), (17, 16, 384), (1, 48, 384),
                                   (1, 1024, 4096), (1, 64, 14336), (1, 16, 12352)])
def test_lossy_parity(layout, M, N, K):
    _announce("lossy", layout, M, N, K)
    pack_ref, gemm_ref = _route(layout)
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(15, M + N + K))
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(15, 7 + M + N + K))
    packed, w_scale = H.pack(W, layout)
    xq, s = H.quantize(x)
    y, acc = H.mpgemm(layout, packed, w_scale, N, K, xq, s)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    t_ref, beta = O.ternarize(W.numpy())
    assert np.array_equal(H.to_np(packed), pack_ref(t_ref))
    acc_ref = gemm_ref(xq_ref, pack_ref(t_ref), N, K)
    assert np.array_equal(H.to_np(acc), acc_ref)
    H.check_y(H.to_np(y), O.epilogue(acc_ref, beta, s_ref), acc_ref)


@pytest.mark.parametrize("layout", ["tl2_0", "tl1_0"])
@pytest.mark.parametrize("M", [1, 3])
def test_lossy_is_exact_when_tables_fit_int8(layout, M):
    _announce("lossy exact", layout, M)
    N, K = 64, 832
    W = inputs.weight_f32(N, K, seed=inputs.seed_for(15, 900))
    packed, w_scale = H.pack(W, layout)
    rng = np.random.default_rng(4)
    xq_np = rng.integers(-42, 43, size=(M, K)).astype(np.int8)          # every TL2 entry within 126
    xq = torch.from_numpy(xq_np).to(H.DEV)
    s = torch.ones(M, dtype=torch.float32, device=H.DEV)
    y, acc = H.mpgemm(layout, packed, w_scale, N, K, xq, s)
    t_ref, _ = O.ternarize(W.numpy())
    assert np.array_equal(H.to_np(acc), O.mad_gemm(xq_np, t_ref))


@pytest.mark.parametrize("layout", ["tl2_0", "tl1_0"])
@pytest.mark.parametrize("M,K,Ns", [(3, 1600, (64, 208)), (1, 1600, (64, 208)), (1, 4096, (4096, 1024, 1024)),
                                    (1, 8640, (3200,)), (1, 14336, (16, 32)), (1, 448, (16,)), (11, 832, (48, 16)),
                                    (8, 3200, (208, 16, 32))])
def test_lossy_fused(layout, M, K, Ns):
    _announce("lossy fused", layout, M, K, Ns)
    from tests.test_gpu_fused import _fused_case_lossy
    _fused_case_lossy(layout, M, K, Ns)


# The 100B-class groups at one token, as the stack benchmark runs them on the lossy layouts: q/k/v (2304 row groups)
# and o (768) on the persistent kernels (the whole row's tables in LDS), down (K = 33024) on the lookup kernels with
# the row quantised inside.  The oracle's lossy route runs on sampled row groups.
@pytest.mark.parametrize("layout", ["tl2_0", "tl1_0"])
@pytest.mark.parametrize("K,Ns", [(12288, (12288, 12288, 12288)), (12288, (12288,)), (33024, (12288,))])
def test_lossy_fused_100b_groups(layout, K, Ns):
    _announce("lossy fused 100B-class", layout, K, Ns)
    from tests.test_gpu_fused import _fused_case_lossy
    _fused_case_lossy(layout, 1, K, Ns, sample_groups=6)


# The 8B-class layer groups at one and eight tokens, as the benchmark runs them on the lossy layouts (one token: the
# persistent kernels; eight: the quantiser, then the lookup kernels); the oracle's lossy route on sampled row groups.
@pytest.mark.parametrize("layout", ["tl2_0", "tl1_0"])
@pytest.mark.parametrize("M", [1, 8])
@pytest.mark.parametrize("K,Ns", [(4096, (4096, 1024, 1024)), (4096, (4096,)), (4096, (14336, 14336)),
                                  (14336, (4096,))])
def test_lossy_fused_8b_groups(layout, M, K, Ns):
    _announce("lossy fused 8B-class", layout, M, K, Ns)
    from tests.test_gpu_fused import _fused_case_lossy
    _fused_case_lossy(layout, M, K, Ns, sample_groups=6)
