"""GPU check of bitnet_mpgemm_noalloc (the workspace from the library's static scratch) against bitnet_mpgemm with
a caller workspace: two calls in a row on shapes that use the scratch, the second with a smaller input, each
bit-identical to bitnet_mpgemm (acc and y) and to the oracle."""
import numpy as np
import pytest
import torch

import paper_2502_11880_amd as B
from oracle import bitnet_oracle as O
from paper_2502_11880_amd import inputs
from tests import hip_runner as H

pytestmark = pytest.mark.gpu


def _call_pair(layout, M, N, K, seed):
    print("case: no-alloc", layout, M, N, K, flush=True)
    need = B.bitnet_mpgemm_workspace_bytes(layout, M, N, K)
    assert 0 < need <= B.NOALLOC_SCRATCH_BYTES          # the shape really uses the scratch
    W = inputs.weight_f32(N, K, seed=seed)
    x = inputs.activation_f32(M, K, seed=seed + 1)
    packed, w_scale = H.pack(W, layout)
    xq, s, rs = H.quantize(x, with_rowsum=True)
    y_ref_gpu, acc_ref_gpu = H.mpgemm(layout, packed, w_scale, N, K, xq, s, x_rowsum=rs)
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device=H.DEV)
    acc = torch.full((M, N), -7, dtype=torch.int32, device=H.DEV)
    B.bitnet_mpgemm_noalloc(layout, packed, w_scale, N, K, xq, s, y, acc, x_rowsum=rs)
    assert np.array_equal(H.to_np(acc), H.to_np(acc_ref_gpu))
    assert np.array_equal(H.to_np(y), H.to_np(y_ref_gpu))
    y_o, acc_o, *_ = O.mpgemm_reference(x.numpy(), W.numpy())
    assert np.array_equal(H.to_np(acc), acc_o)
    H.check_y(H.to_np(y), y_o, acc_o)


# I2_S prefill with K split across work groups (the int32 slices in the scratch), then a smaller one; TL2 prefill
# (weights rewritten in the I2_S layout in the scratch), then a smaller one.
@pytest.mark.parametrize("layout,shapes", [("i2s", [(64, 1024, 4096), (40, 256, 1536)]),
                                           ("tl2", [(300, 2048, 4096), (33, 256, 832)]),
                                           ("tl1", [(300, 2048, 4096), (33, 256, 832)])])
def test_noalloc_matches_mpgemm_twice(layout, shapes):
    for i, (M, N, K) in enumerate(shapes):
        _call_pair(layout, M, N, K, seed=inputs.seed_for(9, 40 * i + M + N + K))


def test_noalloc_rejects_shapes_beyond_scratch():
    # TL2 prefill rewrites N*K/4 bytes: past the scratch the call fails on the host, before any launch
    M, N, K = 64, 16384, 16384
    assert B.bitnet_mpgemm_workspace_bytes("tl2", M, N, K) > B.NOALLOC_SCRATCH_BYTES
    xq = torch.zeros((M, K), dtype=torch.int8, device=H.DEV)
    s = torch.ones(M, dtype=torch.float32, device=H.DEV)
    packed = torch.zeros(B.bitnet_packed_bytes("tl2", N, K), dtype=torch.uint8, device=H.DEV)
    w_scale = torch.ones(1, dtype=torch.float32, device=H.DEV)
    y = torch.empty((M, N), dtype=torch.float32, device=H.DEV)
    with pytest.raises(B.BitnetError) as e:
        B.bitnet_mpgemm_noalloc("tl2", packed, w_scale, N, K, xq, s, y)
    assert e.value.status == 5 and "scratch" in str(e.value)
