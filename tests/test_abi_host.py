"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function that include/kvx.h declares,
and reject malformed calls with the documented status before touching the
GPU.  Calls here pass placeholder addresses; each one also carries a second
defect that the validator checks later, so that a missed check still cannot
reach a kernel launch.  Tests that need a call with no other defect run only
where no GPU is visible.
"""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_03893_amd import kvx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvx.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(kvx.lib_path()):
        from paper_2608_03893_amd import build
        build.build()
    return kvx.load()


def _gpu_visible():
    import torch
    return torch.cuda.is_available()


def test_exports_every_declared_function(L):
    text = open(HEADER).read()
    names = set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(kvx_\w+)\s*\(", text, flags=re.M))
    assert {"kvx_map_cache", "kvx_map_layer", "kvx_map_cache_slots", "kvx_workspace_bytes",
            "kvx_rope_prepare", "kvx_last_error", "kvx_version", "kvx_map_kernel_name",
            "kvx_map_cache_xhead", "kvx_xhead_workspace_bytes", "kvx_map_layer_xhead",
            "kvx_map_cache_slots_xhead"} <= names
    for n in sorted(names):
        assert hasattr(L, n), f"libkvx.so does not export {n}"


def test_map_kernel_name_follows_the_selection_rule(L):
    """Host-only: which kernel a call would launch (no GPU needed)."""
    from paper_2608_03893_amd import kvx
    q = kvx.Dims(L_s=40, L_t=64, H=8, T=32768, d=128, k=4)
    assert kvx.map_kernel_name(q, "bf16") == "map_ks2_kernel"
    assert kvx.map_kernel_name(q, "bf16", n_layers=1) == "map_w_kernel"
    assert kvx.map_kernel_name(q, "f32") == "map_kernel"
    small = kvx.Dims(L_s=28, L_t=36, H=8, T=4096, d=128, k=3)
    assert kvx.map_kernel_name(small, "bf16") == "map_ks_kernel"
    assert kvx.map_kernel_name(small, "bf16", n_layers=15) == "map_w_kernel"
    odd_heads = kvx.Dims(L_s=28, L_t=36, H=3, T=4096, d=128, k=3)
    assert kvx.map_kernel_name(odd_heads, "bf16") == "map_w_kernel"
    wide = kvx.Dims(L_s=40, L_t=64, H=8, T=4096, d=128, k=5)
    assert kvx.map_kernel_name(wide, "bf16") == "map_kernel"
    d64 = kvx.Dims(L_s=4, L_t=64, H=2, T=256, d=64, k=2)
    assert kvx.map_kernel_name(d64, "bf16") == "map_kernel"
    with pytest.raises(ValueError):
        kvx.map_kernel_name(q, "bf16", n_layers=0)


def test_version_and_empty_error(L):
    assert L.kvx_version() == 100
    assert isinstance(L.kvx_last_error(), bytes)


def test_workspace_bytes(L):
    d = kvx.Dims(L_s=40, L_t=64, H=8, T=32768, d=128, k=4)
    tables = 12 * 32768 * 128
    assert kvx.workspace_bytes(d) == tables + 2 * 64 * 8 * 4 * 128 * 128 * 2
    assert kvx.workspace_bytes(d, "bf16") == kvx.workspace_bytes(d)
    # fp32 calls never use packed maps: the tables only
    assert kvx.workspace_bytes(d, "f32") == tables
    # bf16 calls that the general tile kernel serves (k > 4, d = 64): the tables only
    assert kvx.workspace_bytes(kvx.Dims(L_s=40, L_t=64, H=8, T=32768, d=128, k=5)) == tables
    assert kvx.workspace_bytes(kvx.Dims(L_s=4, L_t=6, H=2, T=256, d=64, k=2)) == 12 * 256 * 64
    # an empty call needs no workspace at all
    assert kvx.workspace_bytes(kvx.Dims(L_s=40, L_t=64, H=8, T=0, d=128, k=4)) == 0
    assert L.kvx_workspace_bytes(None, 0) == 0
    assert L.kvx_workspace_bytes(ctypes.byref(d), 7) == 0          # unknown dtype
    bad = kvx.Dims(L_s=1, L_t=1, H=1, T=5, d=7, k=1)
    assert kvx.workspace_bytes(bad) == 0


# ---------------------------------------------------------------- fake calls
A = 1 << 20  # placeholder "device" addresses, 256-byte aligned, never dereferenced


class Call:
    def __init__(self, **kw):
        self.dims = kvx.Dims(L_s=4, L_t=3, H=2, T=8, d=64, k=2)
        self.dtype = 0
        self.idx = np.array([[0, 1], [2, 3], [1, 0]], dtype=np.int32)
        self.src, self.wk, self.wv = A, 2 * A, 3 * A
        self.bk, self.bv = None, None
        self.rs = kvx.Rope(theta=1e4, style=0, original_max_pos=8192, factor=1.0,
                           low_freq_factor=1.0, high_freq_factor=4.0)
        self.rt = kvx.Rope(theta=1e4, style=0, original_max_pos=8192, factor=1.0,
                           low_freq_factor=1.0, high_freq_factor=4.0)
        self.pos, self.tgt, self.ws = 4 * A, 5 * A, 6 * A
        self.wsb = 10 ** 6
        self.flags = 0
        for k, v in kw.items():
            setattr(self, k, v)

    def run(self, L):
        idx = None if self.idx is None else np.ascontiguousarray(self.idx, dtype=np.int32)
        return L.kvx_map_cache(
            None if self.dims is None else ctypes.byref(self.dims), self.dtype,
            self.src, None if idx is None else idx.ctypes.data_as(ctypes.c_void_p),
            self.wk, self.wv, self.bk, self.bv,
            None if self.rs is None else ctypes.byref(self.rs),
            None if self.rt is None else ctypes.byref(self.rt),
            self.pos, self.tgt, self.ws, self.wsb, self.flags, None)


SAFETY = dict(wsb=1)  # workspace too small: checked after everything except aliasing


def _expect(L, status, **kw):
    st = Call(**{**SAFETY, **kw}).run(L)
    assert st == status, (kvx.STATUS.get(st), L.kvx_last_error())
    assert L.kvx_last_error() != b""


@pytest.mark.parametrize("d", [64, 128])
def test_empty_call_is_ok_and_launches_nothing(L, d):
    # at d = 128 a non-empty bf16 call needs packed-map space; an empty one needs none
    c = Call(dims=kvx.Dims(L_s=4, L_t=3, H=2, T=0, d=d, k=2), src=None, pos=None,
             tgt=None, ws=None, wsb=0)
    assert c.run(L) == 0, L.kvx_last_error()
    c.dtype = 1
    assert c.run(L) == 0, L.kvx_last_error()


def test_null_arguments(L):
    _expect(L, 1, dims=None)
    _expect(L, 1, idx=None)
    _expect(L, 1, wk=None)
    _expect(L, 1, wv=None)
    _expect(L, 1, src=None)
    _expect(L, 1, pos=None)
    _expect(L, 1, tgt=None)
    _expect(L, 1, rs=None)
    _expect(L, 1, rt=None)


def test_bad_shapes(L):
    for dims in [dict(L_s=0), dict(L_t=0), dict(H=0), dict(T=-1), dict(k=0), dict(d=65)]:
        base = dict(L_s=4, L_t=3, H=2, T=8, d=64, k=2)
        base.update(dims)
        _expect(L, 2, dims=kvx.Dims(**base))


def test_unsupported(L):
    _expect(L, 5, dims=kvx.Dims(L_s=4, L_t=3, H=2, T=8, d=96, k=2))
    _expect(L, 5, dims=kvx.Dims(L_s=300, L_t=3, H=2, T=8, d=64, k=2))
    _expect(L, 5, src=A + 8)                                # misaligned
    big = kvx.Dims(L_s=4, L_t=1100, H=2, T=8, d=64, k=2)    # 2200 index entries
    _expect(L, 5, dims=big, idx=np.zeros((1100, 2), np.int32))
    rt = kvx.Rope(theta=1e4, style=1, original_max_pos=8192, factor=1.0,
                  low_freq_factor=1.0, high_freq_factor=4.0)
    _expect(L, 5, rt=rt)                                    # mixed RoPE styles


def test_bad_dtype(L):
    _expect(L, 4, dtype=7)


def test_index_out_of_range(L):
    _expect(L, 3, idx=np.array([[0, 1], [2, 4], [1, 0]], np.int32))
    _expect(L, 3, idx=np.array([[0, -1], [2, 3], [1, 0]], np.int32))


def test_bad_rope(L):
    def r(**kw):
        base = dict(theta=1e4, style=0, original_max_pos=8192, factor=1.0,
                    low_freq_factor=1.0, high_freq_factor=4.0)
        base.update(kw)
        return kvx.Rope(**base)
    _expect(L, 9, rs=r(theta=0.5))
    _expect(L, 9, rs=r(theta=float("nan")))
    _expect(L, 9, rt=r(style=2))
    _expect(L, 9, rt=r(factor=0.5))
    _expect(L, 9, rt=r(factor=8.0, low_freq_factor=4.0, high_freq_factor=1.0))
    _expect(L, 9, rt=r(factor=8.0, original_max_pos=0))


def test_workspace_checks(L):
    # safety defect for these: target aliases the source
    st = Call(wsb=100, tgt=A).run(L)
    assert st == 7
    st = Call(ws=None, tgt=A).run(L)
    assert st == 7
    st = Call(ws=6 * A + 16, tgt=A).run(L)
    assert st == 7


@pytest.mark.skipif(_gpu_visible(), reason="alias checks are the last line; run where no GPU is visible")
def test_alias_checks(L):
    assert Call(tgt=A).run(L) == 6                 # target == source
    assert Call(tgt=2 * A + 64).run(L) == 6        # inside W_K
    assert Call(ws=5 * A + 256).run(L) == 6        # workspace inside target
    # the workspace is written (tables, packed maps) while the inputs are read
    assert Call(ws=2 * A).run(L) == 6              # workspace on W_K
    assert Call(ws=A + 256).run(L) == 6            # workspace inside the source
    assert Call(ws=3 * A + 1024).run(L) == 6       # workspace inside W_V
    assert Call(bv=7 * A, ws=7 * A).run(L) == 6    # workspace on b_V
    assert Call(bk=7 * A, ws=7 * A - 256).run(L) == 6   # workspace running into b_K
    assert Call(ws=4 * A - 256).run(L) == 6        # workspace running into positions
    d128 = kvx.Dims(L_s=4, L_t=3, H=2, T=8, d=128, k=2)
    assert Call(dims=d128, ws=2 * A).run(L) == 6   # also with packed maps in the workspace


def test_noalloc_rejects_oversized_workspace(L):
    """The no-allocation entry point refuses, before any HIP call, a call
    whose workspace would not fit the library's static scratch."""
    c = Call(dims=kvx.Dims(L_s=40, L_t=2, H=8, T=200000, d=128, k=4))
    assert kvx.workspace_bytes(c.dims) > kvx.SCRATCH_MAX_BYTES
    st = L.kvx_map_cache_noalloc(ctypes.byref(c.dims), 0, c.src,
                                 c.idx.ctypes.data_as(ctypes.c_void_p), c.wk, c.wv, None, None,
                                 ctypes.byref(c.rs), ctypes.byref(c.rt), c.pos, c.tgt, 0, None)
    assert st == 7, L.kvx_last_error()
    assert b"static scratch" in L.kvx_last_error()
    # invalid calls report through the regular checks, also without a GPU
    st = L.kvx_map_cache_noalloc(None, 0, c.src, None, c.wk, c.wv, None, None,
                                 ctypes.byref(c.rs), ctypes.byref(c.rt), c.pos, c.tgt, 0, None)
    assert st == 1
    empty = kvx.Dims(L_s=4, L_t=3, H=2, T=0, d=128, k=2)
    st = L.kvx_map_cache_noalloc(ctypes.byref(empty), 0, None,
                                 c.idx.ctypes.data_as(ctypes.c_void_p), c.wk, c.wv, None, None,
                                 ctypes.byref(c.rs), ctypes.byref(c.rt), None, None, 0, None)
    assert st == 0, L.kvx_last_error()


def test_map_layer_rejects_bad_layer(L):
    c = Call(wsb=1)
    for lt in (-1, 3):
        st = L.kvx_map_layer(ctypes.byref(c.dims), 0, lt, c.src,
                             c.idx.ctypes.data_as(ctypes.c_void_p), c.wk, c.wv, None, None,
                             ctypes.byref(c.rs), ctypes.byref(c.rt), c.pos, c.tgt, c.ws, 1, 0,
                             None)
        assert st == 3


def test_slots_checks(L):
    c = Call()
    def run(slots, num_slots, wsb=1):
        return L.kvx_map_cache_slots(ctypes.byref(c.dims), 0, c.src,
                                     c.idx.ctypes.data_as(ctypes.c_void_p), c.wk, c.wv,
                                     None, None, ctypes.byref(c.rs), ctypes.byref(c.rt),
                                     c.pos, slots, num_slots, c.tgt, c.ws, wsb, 0, None)
    assert run(7 * A, 0) == 2
    assert run(7 * A, 1 << 31) == 2
    assert run(None, 16) == 1


def test_python_binding_rejects_bad_tensors():
    import torch
    src = torch.zeros((2, 2, 1, 4, 64))
    with pytest.raises(ValueError):
        kvx._ptr(src)  # CPU tensor


# ------------------------------------------------------- cross-head form calls
def test_xhead_workspace_bytes(L):
    m = kvx.XDims(L_s=40, L_t=64, H_s=8, H_t=8, T=32768, d=128, k=4)
    assert kvx.xhead_workspace_bytes(m) == (12 * 32768 * 128 + 40 * 8 * 32768 * 128 * 2
                                            + 2 * 64 * 8 * 128 * 4 * 8 * 128 * 2)
    assert L.kvx_xhead_workspace_bytes(None) == 0
    assert kvx.xhead_workspace_bytes(kvx.XDims(L_s=2, L_t=2, H_s=1, H_t=1, T=4, d=96, k=1)) == 0
    assert kvx.xhead_workspace_bytes(kvx.XDims(L_s=2, L_t=2, H_s=0, H_t=1, T=4, d=64, k=1)) == 0


class XCall(Call):
    def __init__(self, **kw):
        super().__init__()
        self.dims = kvx.XDims(L_s=4, L_t=3, H_s=2, H_t=3, T=8, d=64, k=2)
        for k, v in kw.items():
            setattr(self, k, v)

    def run(self, L):
        idx = None if self.idx is None else np.ascontiguousarray(self.idx, dtype=np.int32)
        return L.kvx_map_cache_xhead(
            None if self.dims is None else ctypes.byref(self.dims), self.dtype,
            self.src, None if idx is None else idx.ctypes.data_as(ctypes.c_void_p),
            self.wk, self.wv, self.bk, self.bv,
            None if self.rs is None else ctypes.byref(self.rs),
            None if self.rt is None else ctypes.byref(self.rt),
            self.pos, self.tgt, self.ws, self.wsb, self.flags, None)


def _xexpect(L, status, **kw):
    st = XCall(**{**SAFETY, **kw}).run(L)
    assert st == status, (kvx.STATUS.get(st), L.kvx_last_error())
    assert L.kvx_last_error() != b""


def test_xhead_rejections(L):
    _xexpect(L, 1, dims=None)
    _xexpect(L, 1, idx=None)
    _xexpect(L, 1, wk=None)
    _xexpect(L, 1, src=None)
    _xexpect(L, 2, dims=kvx.XDims(L_s=4, L_t=3, H_s=0, H_t=3, T=8, d=64, k=2))
    _xexpect(L, 2, dims=kvx.XDims(L_s=4, L_t=3, H_s=2, H_t=3, T=8, d=63, k=2))
    _xexpect(L, 5, dims=kvx.XDims(L_s=4, L_t=3, H_s=2, H_t=3, T=8, d=96, k=2))
    _xexpect(L, 5, dims=kvx.XDims(L_s=4, L_t=3, H_s=2, H_t=3, T=2 ** 24, d=128, k=2))
    _xexpect(L, 5, dtype=1)                         # fp32 not built for this form
    _xexpect(L, 4, dtype=7)
    _xexpect(L, 3, idx=np.array([[0, 1], [2, 4], [1, 0]], dtype=np.int32))
    _xexpect(L, 5, wk=2 * A + 8)                    # not 16-byte aligned
    _xexpect(L, 5, rt=kvx.Rope(theta=1e4, style=1, original_max_pos=8192, factor=1.0,
                               low_freq_factor=1.0, high_freq_factor=4.0))
    # workspace: too small, missing, misaligned (each with the target aliasing
    # the source as a second defect)
    assert XCall(wsb=100, tgt=A).run(L) == 7
    assert XCall(ws=None, tgt=A).run(L) == 7
    assert XCall(ws=6 * A + 16, tgt=A).run(L) == 7


def test_xhead_empty_call_is_ok(L):
    c = XCall(dims=kvx.XDims(L_s=4, L_t=3, H_s=2, H_t=3, T=0, d=64, k=2), src=None, pos=None,
              tgt=None, ws=None, wsb=0)
    assert c.run(L) == 0


@pytest.mark.skipif(_gpu_visible(), reason="alias checks are the last line; run where no GPU is visible")
def test_xhead_alias_checks(L):
    assert XCall(tgt=A).run(L) == 6                 # target == source
    assert XCall(ws=2 * A + 256).run(L) == 6        # workspace inside W_K
    assert XCall(ws=5 * A + 256).run(L) == 6        # workspace inside the target


def test_xhead_layer_and_slots_checks(L):
    c = XCall(wsb=1)
    idx = c.idx.ctypes.data_as(ctypes.c_void_p)
    for lt in (-1, 3):
        st = L.kvx_map_layer_xhead(ctypes.byref(c.dims), 0, lt, c.src, idx, c.wk, c.wv, None, None,
                                   ctypes.byref(c.rs), ctypes.byref(c.rt), c.pos, c.tgt, c.ws,
                                   1, 0, None)
        assert st == 3, (lt, L.kvx_last_error())

    def run(slots, num_slots, wsb=1):
        return L.kvx_map_cache_slots_xhead(ctypes.byref(c.dims), 0, c.src, idx, c.wk, c.wv, None,
                                           None, ctypes.byref(c.rs), ctypes.byref(c.rt), c.pos,
                                           slots, num_slots, c.tgt, c.ws, wsb, 0, None)
    assert run(7 * A, 0) == 2                     # num_slots < 1
    assert run(7 * A, 1 << 31) == 2
    assert run(None, 100) == 1                    # slot_mapping NULL
    assert run(7 * A + 2, 100) == 5               # misaligned
    assert run(7 * A, 100) == 7                   # the safety defect: workspace too small
