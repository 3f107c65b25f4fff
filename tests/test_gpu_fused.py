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
    """One fused call per layout in `layout` (a name or a tuple of names) on the same seeded weights and
    activation, every output (or every output of a seeded sample of token rows) against the oracle, and
    bit-identical to the separate quantise + bitnet_mpgemm calls and to the fused call on the quantised input."""
    layouts = (layout,) if isinstance(layout, str) else tuple(layout)
    Ws = [inputs.weight_f32(N, K, seed=seed + i) for i, N in enumerate(Ns)]
    x = inputs.activation_f32(M, K, seed=seed + 100)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    refs = [O.ternarize(W.numpy()) for W in Ws]
    rows = np.arange(M) if sample_rows is None else np.unique(
        np.concatenate([[0, M - 1], np.random.default_rng(seed).choice(M, size=sample_rows, replace=False)]))
    acc_refs = [O.mad_gemm(xq_ref[rows], t_ref) for t_ref, _ in refs]
    xd = x.to(H.DEV)
    for lay in layouts:
        _announce("  layout", lay)
        packs = [H.pack(W, lay) for W in Ws]
        xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
        s = torch.empty(M, dtype=torch.float32, device=H.DEV)
        rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
        ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
        need = max(B.bitnet_mpgemm_workspace_bytes(lay, M, N, K) for N in Ns)
        if split_ws:
            need = max(need, B.bitnet_mpgemm_fused_workspace_bytes(lay, Ns, K, M))
        ws = torch.zeros(max(16, need), dtype=torch.uint8, device=H.DEV)
        B.bitnet_mpgemm_fused(lay, [p for p, _ in packs], [b for _, b in packs], xd, xq, s, rs, ys, ws)
        assert np.array_equal(H.to_np(xq), xq_ref)
        assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
        assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))
        for i, ((p, b), y, (_, beta_ref), acc_ref) in enumerate(zip(packs, ys, refs, acc_refs)):
            H.check_y(H.to_np(y)[rows], O.epilogue(acc_ref, beta_ref, s_ref[rows]), acc_ref)
            y_sep, _ = H.mpgemm(lay, p, b, Ns[i], K, xq, s, x_rowsum=rs)
            assert np.array_equal(H.to_np(y), H.to_np(y_sep))      # identical to the separate calls
            del y_sep
        # the products alone, on the activation quantised above (x = NULL)
        ys2 = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
        B.bitnet_mpgemm_fused(lay, [p for p, _ in packs], [b for _, b in packs], None, xq, s, rs, ys2, ws)
        for y, y2 in zip(ys, ys2):
            assert np.array_equal(H.to_np(y), H.to_np(y2))
        del packs, ys, ys2, ws
        torch.cuda.empty_cache()


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


# The 8B-class layer groups at the token counts the benchmark times, every output against the oracle: 8 and 16 tokens
# (the multi-token stream for I2_S and TL1, the TL2 MFMA expansion on codes given) and the small-batch regime
# (32, 64 and 112 tokens: token slices of the stream for I2_S and TL1).
GROUPS_8B = [(4096, [4096, 1024, 1024]), (4096, [4096]), (4096, [14336, 14336]), (14336, [4096])]


@pytest.mark.parametrize("M", [8, 16])
@pytest.mark.parametrize("K,Ns", GROUPS_8B)
def test_fused_few_tokens_8b_groups(M, K, Ns):
    _announce("fused 8B-class group", M, K, Ns)
    _fused_case(("i2s", "tl2", "tl1"), M, K, Ns, seed=inputs.seed_for(18, M * 31 + K + len(Ns)))


@pytest.mark.parametrize("M", [32, 64, 112])
@pytest.mark.parametrize("K,Ns", GROUPS_8B)
def test_fused_small_batch_8b_groups(M, K, Ns):
    _announce("fused 8B-class group, small batch", M, K, Ns)
    _fused_case(("i2s", "tl1"), M, K, Ns, seed=inputs.seed_for(19, M * 31 + K + len(Ns)))


# The same groups at 512 tokens (the prefill GEMM; split-K over the workspace where a launch has fewer tiles than
# CUs), every output against the oracle, for the three layouts.
@pytest.mark.parametrize("K,Ns", GROUPS_8B)
def test_fused_prefill_512_8b_groups(K, Ns):
    _announce("fused 8B-class group, 512 tokens", K, Ns)
    _fused_case(("i2s", "tl2", "tl1"), 512, K, Ns, seed=inputs.seed_for(20, K + len(Ns)), split_ws=True)


# 2..12 tokens through the fused call, both word formats: 1, 2 and 3 token groups of the multi-token stream,
# K = 4160 (a 64-k last block), K = 4032 (a 192-k last block), K = 8192, several row groups per work group
# (2900 row groups) and a single row group.
@pytest.mark.parametrize("M,K,Ns", [(4, 4096, [1024, 2048]), (12, 4096, [4096, 1024]), (7, 4032, [640, 16]),
                                    (3, 4160, [512]), (4, 8192, [2048, 2048]), (2, 8192, [16]),
                                    (9, 1088, [16000, 16000, 14400])])
def test_fused_few_tokens(M, K, Ns):
    _announce("fused few tokens", M, K, Ns)
    _fused_case(("i2s", "tl1"), M, K, Ns, seed=inputs.seed_for(17, M * 13 + K + len(Ns)))


# More than 16 tokens: one prefill launch over the weights' concatenated row tiles; with a workspace from
# bitnet_mpgemm_fused_workspace_bytes small grids also split K over all the weights.
@pytest.mark.parametrize("M,K,Ns", [(40, 832, [48, 16, 64]), (300, 3200, [3200, 3200, 3200]),
                                    (129, 8640, [3200, 16]), (600, 1536, [512, 1024, 2048])])
@pytest.mark.parametrize("split_ws", [False, True])
def test_fused_i2s_prefill(M, K, Ns, split_ws):
    _announce("fused i2s prefill", M, K, Ns, split_ws)
    _fused_case("i2s", M, K, Ns, seed=inputs.seed_for(2, 900 + M + K + len(Ns)), split_ws=split_ws)


# The 8B-class q/k/v and gate/up groups at 2048 tokens: every output against the oracle (these groups take the
# 128 x 512 tile, four 32 x 32 tiles per wave column) and against the separate calls.
@pytest.mark.parametrize("Ns", [[4096, 1024, 1024], [14336, 14336]])
def test_fused_i2s_prefill_workload(Ns):
    _announce("fused i2s prefill workload", 2048, 4096, Ns)
    _fused_case("i2s", 2048, 4096, Ns, seed=inputs.seed_for(3, 50 + len(Ns)), split_ws=True)


@pytest.mark.parametrize("M,K,Ns", [(1, 448, [16, 32]), (3, 4096, [64, 48])])
def test_fused_tl2(M, K, Ns):
    _announce("fused tl2", M, K, Ns)
    _fused_case("tl2", M, K, Ns, seed=inputs.seed_for(2, 99 + M + K))


# One token through the fused call (one launch that also quantises) on the exact linear groups the benchmark times,
# and one shape for each remaining instance of the single-token streaming kernel, in the three layouts (TL1 runs the
# same instances as I2_S).  Instance (waves, 256-k blocks per wave per batch, float4 of the row per thread) that
# each shape selects on a 256-CU MI355X, I2_S and TL1:
ONE_TOKEN_GROUPS = [
    (1536, [4096]),                  # the 1536 x 4096 linear: <4, 2, 2>
    (3200, [3200]),                  # 3B-class o: <4, 4, 4>
    (4096, [4096, 1024, 1024]),      # 8B-class q/k/v: <4, 4, 4>
    (4096, [4096]),                  # 8B-class o: <4, 4, 4>
    (4096, [14336, 14336]),          # 8B-class gate/up: <4, 4, 4>
    (14336, [4096]),                 # 8B-class down: <8, 4, 8>, two batches per row group
    (8640, [3200]),                  # 3B-class down: <8, 3, 8>, two batches per row group
    (1024, [4096]),                  # <4, 1, 1>
    (2560, [4096]),                  # <4, 3, 4>
    (6144, [1024]),                  # <16, 2, 2>
    (28672, [1024]),                 # <8, 4, 16>, four batches per row group
    (32768, [48]),                   # <8, 4, 16>, the longest row on 8-wave groups
    (33024, [16]),                   # one block longer: <16, 3, 9>, three batches per row group
    (40960, [512]),                  # <16, 4, 12>, three batches per row group
    (61440, [32]),                   # the longest row one launch quantises itself (<16, 4, 16>, 4 batches)
    (61504, [16]),                   # one 64-k unit longer: the quantiser, then the GEMV reading the codes
    (132096, [16]),                  # the largest K
]


@pytest.mark.parametrize("K,Ns", ONE_TOKEN_GROUPS)
def test_fused_one_token_workload_groups(K, Ns):
    _announce("fused one token", K, Ns)
    _fused_case(("i2s", "tl2", "tl1"), 1, K, Ns, seed=inputs.seed_for(2, 3000 + K + len(Ns)))


# The 100B-class layer's groups at one token (the launches of the stack benchmark), every layout.  I2_S and TL1: q/k/v
# (2304 row groups: 256 work groups of <16, 3, 4> walking nine row groups each), o and down (768 row groups:
# three per work group; down <16, 3, 9> with three batches per row group), gate/up (4128 row groups).  TL2: every
# group on the MFMA expansion with the row quantised inside; down (K = 33024, 86 blocks: 9 float4 of the row per
# thread) in two batches per row group.
@pytest.mark.parametrize("K,Ns", [(12288, [12288, 12288, 12288]), (12288, [12288]), (12288, [33024, 33024]),
                                  (33024, [12288])])
def test_fused_one_token_100b_groups(K, Ns):
    _announce("fused one token 100B-class", K, Ns)
    _fused_case(("i2s", "tl2", "tl1"), 1, K, Ns, seed=inputs.seed_for(4, 10 * len(Ns) + K % 7))


def _fused_case_lossy(layout, M=3, K=1600, Ns=(64, 208), sample_groups=None):
    """bitnet_mpgemm_fused on a lossy layout: one table-lookup launch per slice of up to 8 tokens over every weight
    (one token quantised inside it, else the quantiser first); the codes, scales and sums bit-exact, the outputs
    equal to the separate calls and to the oracle's lossy route.  sample_groups: the oracle route runs on the first,
    the last and that many seeded random 16-row groups of each weight (rows are independent in the packing and in
    the route, so packing only those rows gives their exact values); the separate calls are compared everywhere."""
    Ws = [inputs.weight_f32(N, K, seed=inputs.seed_for(15, 500 + i)) for i, N in enumerate(Ns)]
    x = inputs.activation_f32(M, K, seed=inputs.seed_for(15, 599))
    packs = [H.pack(W, layout) for W in Ws]
    xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.empty(M, dtype=torch.float32, device=H.DEV)
    rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
    ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    B.bitnet_mpgemm_fused(layout, [p for p, _ in packs], [b for _, b in packs], x.to(H.DEV), xq, s, rs, ys)
    xq_ref, s_ref = O.quantize_act(x.numpy())
    assert np.array_equal(H.to_np(xq), xq_ref)
    assert np.array_equal(H.to_np(s).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(H.to_np(rs), xq_ref.astype(np.int64).sum(1))
    route = O.elut_gemm_lossy if layout == "tl2_0" else O.elut_gemm_tl1_lossy
    pack = O.pack_tl2 if layout == "tl2_0" else O.pack_tl1
    for i, (W, (p, b), y, N) in enumerate(zip(Ws, packs, ys, Ns)):
        t_ref, beta = O.ternarize(W.numpy())
        if sample_groups is None:
            rows = np.arange(N)
        else:
            groups = N // 16
            pick = np.random.default_rng(inputs.seed_for(15, 700 + i)).choice(groups, size=sample_groups,
                                                                                 replace=False)
            groups_sel = np.unique(np.concatenate([[0, groups - 1], pick]))
            rows = (groups_sel[:, None] * 16 + np.arange(16)[None, :]).ravel()
        acc_ref = route(xq_ref, pack(np.ascontiguousarray(t_ref[rows])), len(rows), K)
        H.check_y(H.to_np(y)[:, rows], O.epilogue(acc_ref, beta, s_ref), acc_ref)
        y_sep, _ = H.mpgemm(layout, p, b, N, K, xq, s)
        assert np.array_equal(H.to_np(y), H.to_np(y_sep))
