"""Host-side checks of the C ABI: every declared symbol is exported, size queries agree with the layout
definitions, and argument validation returns the documented status before anything touches a GPU."""
import os
import re

import pytest

import paper_2502_11880_amd as B
from oracle import bitnet_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = []
    for fn in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"\b(bitnet_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = _declared_functions()
    assert len(names) >= 8
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(n for n, _, _ in B._SIGNATURES) == names


@pytest.mark.parametrize("N,K", [(16, 64), (32, 448), (4096, 4096), (3200, 8640), (12288, 33024)])
def test_packed_bytes_match_layout_definitions(N, K):
    assert B.bitnet_packed_bytes("i2s", N, K) == O.i2s_packed_bytes(N, K)
    assert B.bitnet_packed_bytes("tl2", N, K) == O.tl2_packed_bytes(N, K)
    assert B.bitnet_packed_bytes("tl1", N, K) == O.tl1_packed_bytes(N, K)
    assert B.bitnet_packed_bytes("tl2_0", N, K) == O.tl2_packed_bytes(N, K)      # the lossy kernels' formats
    assert B.bitnet_packed_bytes("tl1_0", N, K) == O.tl1_packed_bytes(N, K)
    for fmt in O.ELUT_FORMATS:
        ok = K % (320 if fmt == "c3g5" else 64) == 0
        assert B.bitnet_packed_bytes(fmt, N, K) == (O.elut_packed_bytes(fmt, N, K) if ok else 0)


def test_packed_bytes_rejects_bad_shapes():
    for layout in ("i2s", "tl2", "tl1", "c4g2", "c5g2", "c3g5"):
        assert B.bitnet_packed_bytes(layout, 15, 64) == 0
        assert B.bitnet_packed_bytes(layout, 16, 65) == 0
        assert B.bitnet_packed_bytes(layout, 0, 64) == 0
    assert B.bitnet_packed_bytes(8, 16, 64) == 0
    assert B.bitnet_packed_bytes("c3g5", 16, 640) == 16 * 640 // 5 and B.bitnet_packed_bytes("c3g5", 16, 384) == 0


FAKE = 1 << 20          # aligned, never dereferenced: validation fails before any launch


def _gpu_visible():
    import torch
    return torch.cuda.device_count() > 0


# The placeholder pointers are only safe where nothing can launch: a validation regression on a machine with a
# GPU would send them to a kernel.  These tests run in the CPU suite.
cpu_only = pytest.mark.skipif(_gpu_visible(), reason="placeholder device pointers: validation checks run without a GPU")


def _mpgemm(**kw):
    a = dict(layout=0, packed=FAKE, packed_bytes=1 << 30, w_scale=FAKE, N=64, K=256, xq=FAKE, x_scale=FAKE,
             x_rowsum=None, M=1, y=FAKE, acc=None, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return B.lib().bitnet_mpgemm(a["layout"], a["packed"], a["packed_bytes"], a["w_scale"], a["N"], a["K"], a["xq"],
                                 a["x_scale"], a["x_rowsum"], a["M"], a["y"], a["acc"], a["ws"], a["ws_bytes"],
                                 a["stream"])


@cpu_only
def test_mpgemm_validation_statuses():
    assert _mpgemm(layout=9) == 4 and _mpgemm(layout=8) == 4
    assert _mpgemm(packed=None) == 1
    assert _mpgemm(y=None) == 1
    assert _mpgemm(N=40) == 2
    assert _mpgemm(K=100) == 2
    assert _mpgemm(K=132096 + 64) == 2
    assert _mpgemm(M=0) == 2
    assert _mpgemm(xq=FAKE + 4) == 3
    assert _mpgemm(acc=FAKE + 8) == 3
    assert _mpgemm(x_rowsum=FAKE + 2) == 3
    assert _mpgemm(packed_bytes=10) == 1
    for layout, M, N, K in ((0, 1, 64, 256 * 64), (1, 1, 64, 4096), (0, 512, 4096, 4096), (1, 512, 4096, 4096)):
        need = B.bitnet_mpgemm_workspace_bytes(layout, M, N, K)
        if need:
            assert _mpgemm(layout=layout, M=M, N=N, K=K, ws=None, ws_bytes=0) == 5
            assert _mpgemm(layout=layout, M=M, N=N, K=K, ws_bytes=need - 1) == 5
            assert "workspace" in B.bitnet_last_error()


@cpu_only
def test_mpgemm_noalloc_validation_statuses():
    lib = B.lib()

    def call(**kw):
        a = dict(layout=1, packed=FAKE, packed_bytes=1 << 30, w_scale=FAKE, N=16384, K=16384, xq=FAKE, x_scale=FAKE,
                 x_rowsum=None, M=64, y=FAKE, acc=None, stream=None)
        a.update(kw)
        return lib.bitnet_mpgemm_noalloc(a["layout"], a["packed"], a["packed_bytes"], a["w_scale"], a["N"], a["K"],
                                         a["xq"], a["x_scale"], a["x_rowsum"], a["M"], a["y"], a["acc"], a["stream"])

    assert call(packed=None) == 1
    assert call(layout=9) == 4
    assert call(K=100) == 2
    assert call(xq=FAKE + 4) == 3
    # TL2 prefill at 16384 x 16384 rewrites 64 MiB of weights: more than the static scratch holds
    assert B.bitnet_mpgemm_workspace_bytes("tl2", 64, 16384, 16384) > B.NOALLOC_SCRATCH_BYTES
    assert call() == 5 and "scratch" in B.bitnet_last_error()


@cpu_only
def test_quantize_and_pack_validation_statuses():
    lib = B.lib()
    assert lib.bitnet_quantize_act(None, 1, 64, FAKE, FAKE, None, None) == 1
    assert lib.bitnet_quantize_act(FAKE, 0, 64, FAKE, FAKE, None, None) == 2
    assert lib.bitnet_quantize_act(FAKE, 1, 0, FAKE, FAKE, None, None) == 2
    assert lib.bitnet_quantize_act(FAKE + 4, 1, 64, FAKE, FAKE, None, None) == 3
    assert lib.bitnet_quantize_act(FAKE, 1, 64, FAKE, FAKE, FAKE + 1, None) == 3
    ws = B.bitnet_pack_workspace_bytes(64, 64)
    assert lib.bitnet_pack_weights(3, FAKE, 64, 64, FAKE, 1 << 20, FAKE, FAKE, ws, None) == 4
    assert lib.bitnet_pack_weights(0, FAKE, 60, 64, FAKE, 1 << 20, FAKE, FAKE, ws, None) == 2
    assert lib.bitnet_pack_weights(0, FAKE, 64, 64, FAKE, 100, FAKE, FAKE, ws, None) == 1
    assert lib.bitnet_pack_weights(0, FAKE, 64, 64, FAKE, 1 << 20, FAKE, FAKE, ws - 8, None) == 5
    assert lib.bitnet_pack_weights(0, FAKE, 64, 64, FAKE + 2, 1 << 20, FAKE, FAKE, ws, None) == 3


@cpu_only
def test_pack_int_weights_validation_statuses():
    lib = B.lib()
    assert lib.bitnet_pack_int_weights(0, FAKE, 64, 640, FAKE, 1 << 20, None) == 4          # ternary layouts: no
    assert lib.bitnet_pack_int_weights(5, FAKE, 64, 448, FAKE, 1 << 20, None) == 2          # c3g5 needs K % 320
    assert lib.bitnet_pack_int_weights(3, None, 64, 640, FAKE, 1 << 20, None) == 1
    assert lib.bitnet_pack_int_weights(4, FAKE, 64, 640, FAKE, 100, None) == 1
    assert lib.bitnet_pack_int_weights(3, FAKE + 4, 64, 640, FAKE, 1 << 20, None) == 3
    ws = B.bitnet_pack_workspace_bytes(64, 640)
    assert lib.bitnet_pack_weights(3, FAKE, 64, 640, FAKE, 1 << 20, FAKE, FAKE, ws, None) == 4   # integer layouts
    assert _mpgemm(layout=5, K=448) == 2


@cpu_only
def test_elut_tables_validation_statuses():
    lib = B.lib()
    assert lib.bitnet_elut_tables(None, 1, 384, FAKE, FAKE, None) == 1
    assert lib.bitnet_elut_tables(FAKE, 1, 320, FAKE, FAKE, None) == 2      # no TL2 block
    assert lib.bitnet_elut_tables(FAKE, 1, 400, FAKE, FAKE, None) == 2      # K % 64
    assert lib.bitnet_elut_tables(FAKE, 1, 448, FAKE, None, None) == 1      # tail needs lut1
    assert lib.bitnet_elut_tables(FAKE + 2, 1, 384, FAKE, None, None) == 3


def test_status_strings():
    for st in range(7):
        assert B.bitnet_status_string(st)
    assert B.bitnet_status_string(99) == "unknown status"


def test_fused_workspace_query():
    # decode needs no workspace; a fused prefill split holds whole M x sum(N) int32 slices; bad input gives 0
    assert B.bitnet_mpgemm_fused_workspace_bytes("i2s", [4096, 1024, 1024], 4096, 8) == 0
    for M, Ns, K in [(512, [4096, 1024, 1024], 4096), (40, [48, 16, 64], 832), (300, [3200] * 3, 3200)]:
        w = B.bitnet_mpgemm_fused_workspace_bytes("i2s", Ns, K, M)
        single = max(B.bitnet_mpgemm_workspace_bytes("i2s", M, N, K) for N in Ns)
        assert w >= single
        assert w == single or w % (M * sum(Ns) * 4) == 0
    assert B.bitnet_mpgemm_fused_workspace_bytes("i2s", [4096, 1000], 4096, 512) == 0
    assert B.bitnet_mpgemm_fused_workspace_bytes("i2s", [], 4096, 512) == 0
    assert B.bitnet_mpgemm_fused_workspace_bytes("i2s", [64] * 9, 256, 512) == 0
