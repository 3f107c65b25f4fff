"""HIP-graph capture and replay of the calls the benchmark times (bitnet_mpgemm_fused, one launch group per
activation) and of the no-allocation entry point: each case runs once eagerly, is captured in a graph on the same
stream, and is replayed three times with eager work in between (the outputs overwritten by fill kernels on that
stream) and a host synchronisation after each replay.  Every replay must reproduce the eager outputs bit for bit:
the same kernels on the same inputs, with fixed reduction orders.  The library records no memset or copy nodes, so
nothing in a replay depends on state the first run left behind other than what the calls themselves rewrite."""
import pytest
import torch

import paper_2502_11880_amd as B
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu

INT_LAYOUTS = {"c4g2": 4, "c5g2": 5, "c3g5": 3}


def _announce(*what):
    print("case:", *what, flush=True)


def _weights(layout, Ns, K, seed):
    packs, scales = [], []
    for i, N in enumerate(Ns):
        if layout in INT_LAYOUTS:
            w = inputs.int_weights(N, K, INT_LAYOUTS[layout], seed=seed + i)
            p = torch.empty(B.bitnet_packed_bytes(layout, N, K), dtype=torch.uint8, device=H.DEV)
            B.bitnet_pack_int_weights(layout, w.to(H.DEV).contiguous(), p)
            sc = torch.full((1,), 0.02, dtype=torch.float32, device=H.DEV)
        else:
            p, sc = H.pack(inputs.weight_f32(N, K, seed=seed + i), layout)
        packs.append(p)
        scales.append(sc)
    return packs, scales


def _bits(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else t


def _replays_match(call, outs, stream, poison):
    """Eager run, capture, three replays; every replay equals the eager outputs bit for bit."""
    with torch.cuda.stream(stream):
        call()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(stream):
            poison()
            g.replay()
        torch.cuda.synchronize()
        for i, (o, r) in enumerate(zip(outs, ref)):
            assert torch.equal(_bits(o), _bits(r)), f"replay {rep}: output {i} differs from the eager run"
    del g


# (layout, tokens, K, output rows of the group): the single-token fused launches (I2_S 4- and 8-wave shapes, the TL2
# expansion with and without its multi-batch form, the TL1 words, the persistent lossy table kernels, the ELUT
# lookups), the quantiser + multi-token stream, token slices, and the prefill GEMM with its split-K finish pass.
CASES = [("i2s", 1, 4096, [4096, 1024, 1024]), ("i2s", 1, 14336, [4096]), ("i2s", 1, 12288, [768]),
         ("i2s", 8, 4096, [2048, 1024]), ("i2s", 40, 4096, [1024]), ("i2s", 512, 4096, [1024, 512]),
         ("tl2", 1, 4096, [1024]), ("tl2", 1, 33024, [16]), ("tl2", 8, 4096, [512]), ("tl1", 1, 4096, [2048]),
         ("tl2_0", 1, 4096, [1024, 32]), ("tl1_0", 1, 4096, [1024, 32]), ("tl2_0", 3, 1600, [64]),
         ("c4g2", 1, 3200, [3200]), ("c3g5", 2, 640, [208])]


@pytest.mark.parametrize("layout,M,K,Ns", CASES)
def test_fused_call_graph_replays(layout, M, K, Ns):
    _announce("graph fused", layout, M, K, Ns)
    seed = inputs.seed_for(21, M + K + len(Ns))
    packs, scales = _weights(layout, Ns, K, seed)
    x = inputs.activation_f32(M, K, seed=seed + 50).to(H.DEV)
    xq = torch.empty((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.empty(M, dtype=torch.float32, device=H.DEV)
    rs = torch.empty(M, dtype=torch.int32, device=H.DEV)
    ys = [torch.empty((M, N), dtype=torch.float32, device=H.DEV) for N in Ns]
    ws = torch.zeros(max(16, B.bitnet_mpgemm_fused_workspace_bytes(layout, Ns, K, M)), dtype=torch.uint8,
                     device=H.DEV)
    args = B.FusedArgs(packs, scales, ys)
    stream = torch.cuda.Stream()
    sptr = stream.cuda_stream
    torch.cuda.synchronize()

    def call():
        B.bitnet_mpgemm_fused(layout, None, None, x, xq, s, rs, None, ws, sptr, args=args)

    def poison():
        for y in ys:
            y.fill_(float("nan"))
        xq.fill_(-7)
        s.fill_(-1.0)
        rs.fill_(123)

    _replays_match(call, ys + [xq, s, rs], stream, poison)


# The no-allocation entry point is for callers that capture graphs: its split-K slices live in the library's
# static scratch, which each replay rewrites before reading.
@pytest.mark.parametrize("layout,M,N,K", [("i2s", 512, 1024, 4096), ("i2s", 1, 2048, 4096), ("tl2", 200, 512, 1536),
                                          ("tl1", 300, 256, 2048)])
def test_noalloc_graph_replays(layout, M, N, K):
    _announce("graph noalloc", layout, M, N, K)
    seed = inputs.seed_for(22, M + N + K)
    (packed,), (w_scale,) = _weights(layout, [N], K, seed)
    x = inputs.activation_f32(M, K, seed=seed + 50)
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y = torch.empty((M, N), dtype=torch.float32, device=H.DEV)
    acc = torch.empty((M, N), dtype=torch.int32, device=H.DEV)
    stream = torch.cuda.Stream()
    sptr = stream.cuda_stream
    torch.cuda.synchronize()

    def call():
        B.bitnet_mpgemm_noalloc(layout, packed, w_scale, N, K, xq, s, y, acc, stream=sptr, x_rowsum=rs)

    def poison():
        y.fill_(float("nan"))
        acc.fill_(-5)

    _replays_match(call, [y, acc], stream, poison)
