"""Host-side checks of the MLP mapper's C ABI (no GPU needed).

Calls pass placeholder addresses 16 MiB apart (every tensor of these sizes
fits in its slot).  Each rejected call also carries a second defect, a
workspace that is too small, so that a missed check still cannot reach a
launch."""

import ctypes

import numpy as np
import pytest

from paper_2608_03893_amd import kvx
from tests.test_abi_host import L, _gpu_visible  # noqa: F401  (the library fixture)

B = 1 << 24


def _rope(style=0):
    return kvx.Rope(theta=1e6, style=style, original_max_pos=8192, factor=1.0,
                    low_freq_factor=1.0, high_freq_factor=4.0)


class MlpCall:
    def __init__(self, **kw):
        self.dims = kvx.Dims(L_s=4, L_t=3, H=2, T=300, d=128, k=2)
        self.dtype = 0
        self.F = 256
        self.idx = np.array([[0, 1], [2, 3], [1, 0]], dtype=np.int32)
        self.src = B
        self.nk = kvx.Mlp(2 * B, 3 * B, 4 * B, 5 * B, 6 * B, 7 * B)
        self.nv = kvx.Mlp(8 * B, 9 * B, 10 * B, 11 * B, 12 * B, None)
        self.rs, self.rt = _rope(), _rope()
        self.pos, self.tgt, self.ws = 13 * B, 14 * B, 16 * B
        self.wsb = 1 << 40
        self.flags = 0
        self.layer = None
        for k, v in kw.items():
            setattr(self, k, v)

    def run(self, L):
        idx = None if self.idx is None else self.idx.ctypes.data_as(ctypes.c_void_p)
        dims = None if self.dims is None else ctypes.byref(self.dims)
        nk = None if self.nk is None else ctypes.byref(self.nk)
        nv = None if self.nv is None else ctypes.byref(self.nv)
        rs = None if self.rs is None else ctypes.byref(self.rs)
        rt = None if self.rt is None else ctypes.byref(self.rt)
        if self.layer is None:
            return L.kvx_mlp_map_cache(dims, self.dtype, self.F, self.src, idx, nk, nv, rs, rt,
                                       self.pos, self.tgt, self.ws, self.wsb, self.flags, None)
        return L.kvx_mlp_map_layer(dims, self.dtype, self.F, self.layer, self.src, idx, nk, nv,
                                   rs, rt, self.pos, self.tgt, self.ws, self.wsb, self.flags, None)


def _expect(L, status, **kw):
    st = MlpCall(**{"wsb": 1, **kw}).run(L)
    assert st == status, (kvx.STATUS.get(st), L.kvx_last_error())
    assert L.kvx_last_error() != b""


def test_mlp_workspace_bytes(L):
    d = kvx.Dims(L_s=40, L_t=64, H=8, T=32768, d=128, k=4)
    tables = 12 * 32768 * 128
    xs = 40 * 8 * 32768 * 128 * 2
    act = 2 * 8 * 32768 * 1024 * 2
    assert kvx.mlp_workspace_bytes(d, 1024) == tables + xs + 2 * act
    assert kvx.mlp_workspace_bytes(kvx.Dims(L_s=40, L_t=64, H=8, T=0, d=128, k=4), 1024) == 0
    assert kvx.mlp_workspace_bytes(d, 1000) == 0        # F not a multiple of 256
    assert kvx.mlp_workspace_bytes(d, 0) == 0
    assert kvx.mlp_workspace_bytes(kvx.Dims(L_s=4, L_t=3, H=2, T=8, d=64, k=2), 256) == 0
    assert L.kvx_mlp_workspace_bytes(None, 256) == 0


def test_mlp_rejections(L):
    _expect(L, 1, dims=None)
    _expect(L, 1, idx=None)
    _expect(L, 1, nk=None)
    _expect(L, 1, nv=kvx.Mlp(8 * B, 9 * B, None, 11 * B, 12 * B, None))   # W2_V missing
    _expect(L, 1, src=None)
    _expect(L, 1, pos=None)
    _expect(L, 1, tgt=None)
    _expect(L, 1, rs=None)
    _expect(L, 2, dims=kvx.Dims(L_s=4, L_t=3, H=0, T=300, d=128, k=2))
    _expect(L, 2, F=0)
    _expect(L, 5, F=300)                                  # not a multiple of 256
    _expect(L, 5, dims=kvx.Dims(L_s=4, L_t=3, H=2, T=300, d=64, k=2))
    _expect(L, 5, dims=kvx.Dims(L_s=10, L_t=1, H=2, T=300, d=128, k=9),
            idx=np.zeros((1, 9), np.int32))              # k above 8
    _expect(L, 5, dims=kvx.Dims(L_s=4, L_t=3, H=2, T=1 << 21, d=128, k=2), F=1024)
    _expect(L, 5, dtype=1)                                # fp32 not built
    _expect(L, 4, dtype=7)
    _expect(L, 3, idx=np.array([[0, 1], [2, 4], [1, 0]], np.int32))
    _expect(L, 5, nk=kvx.Mlp(2 * B + 8, 3 * B, 4 * B, 5 * B, 6 * B, 7 * B))  # misaligned
    _expect(L, 5, rt=_rope(style=1))                      # mixed RoPE styles
    _expect(L, 9, rs=kvx.Rope(theta=0.5, style=0, original_max_pos=8192, factor=1.0,
                              low_freq_factor=1.0, high_freq_factor=4.0))
    _expect(L, 3, layer=3)
    _expect(L, 3, layer=-1)


def test_mlp_workspace_checks(L):
    # second defect: the target sits on the source
    assert MlpCall(wsb=100, tgt=B).run(L) == 7
    assert MlpCall(ws=None, tgt=B).run(L) == 7
    assert MlpCall(ws=16 * B + 16, tgt=B).run(L) == 7


def test_mlp_empty_call_is_ok(L):
    c = MlpCall(dims=kvx.Dims(L_s=4, L_t=3, H=2, T=0, d=128, k=2), src=None, pos=None,
                tgt=None, ws=None, wsb=0)
    assert c.run(L) == 0, L.kvx_last_error()


@pytest.mark.skipif(_gpu_visible(), reason="alias checks are the last line; run where no GPU is visible")
def test_mlp_alias_checks(L):
    assert MlpCall(tgt=B).run(L) == 6                    # target == source
    assert MlpCall(tgt=4 * B + 64).run(L) == 6           # target inside W2_K
    assert MlpCall(ws=3 * B).run(L) == 6                 # workspace on b1_K
    assert MlpCall(ws=12 * B + 256).run(L) == 6          # workspace inside W3_V
    assert MlpCall(ws=14 * B + 4096).run(L) == 6         # workspace inside the target
