"""ctypes binding of libkvx.so (argument marshalling only).

Every step of the mapping runs in the library's HIP kernels.  This module
checks tensor placement, dtype and contiguity, derives the problem sizes from
the shapes, passes raw pointers and the current HIP stream, and turns a
non-OK status into ``KvxError``.  There is no fallback: if the library is not
built, ``load()`` raises.

Entry points mirror include/kvx.h: ``workspace_bytes``, ``rope_prepare``,
``map_cache``, ``map_layer``, ``map_cache_slots``.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

__all__ = ["KvxError", "KvxNotBuilt", "load", "lib_path", "Dims", "Rope",
           "workspace_bytes", "rope_prepare", "map_cache", "map_layer",
           "map_cache_slots", "make_rope", "STATUS", "FLAG_TABLES_READY",
           "FLAG_WEIGHTS_PACKED", "FLAG_KEYS_STRIPPED", "FLAG_PLANES_READY", "map_kernel_name", "XDims",
           "xhead_workspace_bytes", "map_cache_xhead", "map_layer_xhead",
           "map_cache_slots_xhead", "map_cache_noalloc", "SCRATCH_MAX_BYTES",
           "fit_workspace_bytes", "fit_cache", "probe_workspace_bytes", "probe_r2",
           "select_topk", "Mlp", "mlp_workspace_bytes", "mlp_map_cache", "mlp_map_layer"]

_PKG = os.path.dirname(os.path.abspath(__file__))
FLAG_TABLES_READY = 1
FLAG_WEIGHTS_PACKED = 2
FLAG_KEYS_STRIPPED = 4
FLAG_PLANES_READY = 8
SCRATCH_MAX_BYTES = 256 << 20   # KVX_SCRATCH_MAX_BYTES of include/kvx.h

STATUS = {
    0: "KVX_OK", 1: "KVX_ERR_NULL", 2: "KVX_ERR_SHAPE", 3: "KVX_ERR_INDEX",
    4: "KVX_ERR_DTYPE", 5: "KVX_ERR_UNSUPPORTED", 6: "KVX_ERR_ALIAS",
    7: "KVX_ERR_WORKSPACE", 8: "KVX_ERR_HIP", 9: "KVX_ERR_ROPE",
}


class KvxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class KvxNotBuilt(RuntimeError):
    pass


class Dims(ctypes.Structure):
    _fields_ = [("L_s", ctypes.c_int32), ("L_t", ctypes.c_int32),
                ("H", ctypes.c_int32), ("T", ctypes.c_int32),
                ("d", ctypes.c_int32), ("k", ctypes.c_int32)]


class XDims(ctypes.Structure):
    """kvx_xdims: sizes of the cross-head form."""
    _fields_ = [("L_s", ctypes.c_int32), ("L_t", ctypes.c_int32), ("H_s", ctypes.c_int32),
                ("H_t", ctypes.c_int32), ("T", ctypes.c_int32), ("d", ctypes.c_int32),
                ("k", ctypes.c_int32)]


class Mlp(ctypes.Structure):
    """Device pointers of one set of MLP mapper weights (kvx_mlp)."""
    _fields_ = [("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("W2", ctypes.c_void_p),
                ("b2", ctypes.c_void_p), ("W3", ctypes.c_void_p), ("b3", ctypes.c_void_p)]


class Rope(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("style", ctypes.c_int32),
                ("original_max_pos", ctypes.c_int32), ("factor", ctypes.c_double),
                ("low_freq_factor", ctypes.c_double),
                ("high_freq_factor", ctypes.c_double)]


def make_rope(p) -> Rope:
    """Rope struct from a dict with keys theta, style, factor, low_freq_factor,
    high_freq_factor, original_max_pos (missing keys take the defaults)."""
    if isinstance(p, Rope):
        return p
    return Rope(theta=float(p["theta"]), style=int(p.get("style", 0)),
                original_max_pos=int(p.get("original_max_pos", 8192)),
                factor=float(p.get("factor", 1.0)),
                low_freq_factor=float(p.get("low_freq_factor", 1.0)),
                high_freq_factor=float(p.get("high_freq_factor", 4.0)))


_LIB = None


def lib_path() -> str:
    return os.path.join(_PKG, "libkvx.so")


def load():
    """Load libkvx.so once and declare every exported signature."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise KvxNotBuilt(f"{path} is missing; run python -m paper_2608_03893_amd.build")
    L = ctypes.CDLL(path)
    P, I32, U32, SZ, I64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32,
                            ctypes.c_size_t, ctypes.c_int64)
    DP, RP = ctypes.POINTER(Dims), ctypes.POINTER(Rope)
    L.kvx_workspace_bytes.argtypes = [DP, I32]
    L.kvx_workspace_bytes.restype = SZ
    L.kvx_rope_prepare.argtypes = [DP, RP, RP, P, P, SZ, P]
    L.kvx_rope_prepare.restype = I32
    common = [P, P, P, P, P, P, RP, RP, P]
    L.kvx_map_cache.argtypes = [DP, I32, *common, P, P, SZ, U32, P]
    L.kvx_map_cache.restype = I32
    L.kvx_map_layer.argtypes = [DP, I32, I32, *common, P, P, SZ, U32, P]
    L.kvx_map_layer.restype = I32
    L.kvx_map_cache_slots.argtypes = [DP, I32, *common, P, I64, P, P, SZ, U32, P]
    L.kvx_map_cache_slots.restype = I32
    XP = ctypes.POINTER(XDims)
    L.kvx_xhead_workspace_bytes.argtypes = [XP]
    L.kvx_xhead_workspace_bytes.restype = SZ
    L.kvx_map_cache_xhead.argtypes = [XP, I32, *common, P, P, SZ, U32, P]
    L.kvx_map_cache_xhead.restype = I32
    L.kvx_map_layer_xhead.argtypes = [XP, I32, I32, *common, P, P, SZ, U32, P]
    L.kvx_map_layer_xhead.restype = I32
    L.kvx_map_cache_slots_xhead.argtypes = [XP, I32, *common, P, I64, P, P, SZ, U32, P]
    L.kvx_map_cache_slots_xhead.restype = I32
    D64 = ctypes.c_double
    L.kvx_fit_workspace_bytes.argtypes = [DP]
    L.kvx_fit_workspace_bytes.restype = SZ
    L.kvx_fit_cache.argtypes = [DP, I32, P, P, P, RP, RP, P, D64, P, P, P, P, P, SZ, U32, P]
    L.kvx_fit_cache.restype = I32
    L.kvx_probe_workspace_bytes.argtypes = [DP]
    L.kvx_probe_workspace_bytes.restype = SZ
    L.kvx_probe_r2.argtypes = [DP, I32, P, P, RP, RP, P, P, P, SZ, U32, P]
    L.kvx_probe_r2.restype = I32
    L.kvx_select_topk.argtypes = [I32, I32, I32, I32, P, P, P]
    L.kvx_select_topk.restype = I32
    L.kvx_map_cache_noalloc.argtypes = [DP, I32, *common, P, U32, P]
    L.kvx_map_cache_noalloc.restype = I32
    MP = ctypes.POINTER(Mlp)
    L.kvx_mlp_workspace_bytes.argtypes = [DP, I32]
    L.kvx_mlp_workspace_bytes.restype = SZ
    L.kvx_mlp_map_cache.argtypes = [DP, I32, I32, P, P, MP, MP, RP, RP, P, P, P, SZ, U32, P]
    L.kvx_mlp_map_cache.restype = I32
    L.kvx_mlp_map_layer.argtypes = [DP, I32, I32, I32, P, P, MP, MP, RP, RP, P, P, P, SZ, U32, P]
    L.kvx_mlp_map_layer.restype = I32
    L.kvx_last_error.argtypes = []
    L.kvx_last_error.restype = ctypes.c_char_p
    L.kvx_version.argtypes = []
    L.kvx_version.restype = I32
    L.kvx_map_kernel_name.argtypes = [DP, I32, I32]
    L.kvx_map_kernel_name.restype = ctypes.c_char_p
    _LIB = L
    return L


def _check(status: int):
    if status != 0:
        msg = load().kvx_last_error().decode(errors="replace")
        raise KvxError(status, msg)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return 0
    if t.dtype == torch.float32:
        return 1
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor arguments must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _idx_host(idx) -> np.ndarray:
    if isinstance(idx, torch.Tensor):
        idx = idx.detach().cpu().numpy()
    a = np.ascontiguousarray(np.asarray(idx, dtype=np.int32))
    if a.ndim != 2:
        raise ValueError("src_idx must be 2-D [L_t, k]")
    return a


def _torch_stream(stream, device):
    return torch.cuda.current_stream(device) if stream is None else stream


def _stream(stream, device):
    return ctypes.c_void_p(_torch_stream(stream, device).cuda_stream)


def _dims(src, idx, T=None) -> Dims:
    L_s, two, H, Ts, d = src.shape
    if two != 2:
        raise ValueError("src_kv must be [L_s, 2, H, T, d]")
    return Dims(L_s=L_s, L_t=idx.shape[0], H=H, T=Ts if T is None else T, d=d,
                k=idx.shape[1])


def map_kernel_name(dims: Dims, dtype: str = "bf16", n_layers: int | None = None) -> str:
    """Kernel the library would launch for these sizes ("map_sweep_kernel",
    "map_w_kernel" or "map_kernel")."""
    r = load().kvx_map_kernel_name(ctypes.byref(dims), 0 if dtype == "bf16" else 1,
                                   dims.L_t if n_layers is None else n_layers)
    if r is None:
        raise ValueError("invalid sizes or dtype")
    return r.decode()


def workspace_bytes(dims: Dims, dtype: str = "bf16") -> int:
    """Workspace bytes of a call with these sizes and element type ("bf16" or
    "f32")."""
    if dtype not in ("bf16", "f32"):
        raise ValueError("dtype must be 'bf16' or 'f32'")
    return int(load().kvx_workspace_bytes(ctypes.byref(dims), 0 if dtype == "bf16" else 1))


def _scratch(nbytes, device, stream):
    """A temporary workspace allocated on the launch stream: the caching
    allocator reuses its bytes only for later allocations on that stream, whose
    work runs after the kernels enqueued here."""
    with torch.cuda.stream(_torch_stream(stream, device)):
        return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def _workspace(dims: Dims, src, workspace, stream):
    need = workspace_bytes(dims, "bf16" if src.dtype == torch.bfloat16 else "f32")
    if workspace is None:
        workspace = _scratch(need, src.device, stream)
    return workspace, need


def _check_shapes(src, W_K, W_V, b_K, b_V, positions, idx):
    L_s, _, H, T, d = src.shape
    L_t, k = idx.shape
    for name, W in (("W_K", W_K), ("W_V", W_V)):
        if tuple(W.shape) != (L_t, H, k * d, d):
            raise ValueError(f"{name} must be [L_t, H, k*d, d] = {(L_t, H, k * d, d)}, got {tuple(W.shape)}")
        if W.dtype != src.dtype:
            raise TypeError(f"{name} dtype {W.dtype} differs from src_kv {src.dtype}")
    for name, b in (("b_K", b_K), ("b_V", b_V)):
        if b is not None:
            if tuple(b.shape) != (L_t, H, d):
                raise ValueError(f"{name} must be [L_t, H, d]")
            if b.dtype != src.dtype:
                raise TypeError(f"{name} dtype {b.dtype} differs from src_kv {src.dtype}")
    if positions.dtype != torch.int32 or positions.shape != (T,):
        raise ValueError("positions must be int32 [T]")


def rope_prepare(positions, rope_src, rope_tgt, d, workspace, L_s=1, L_t=1, H=1, k=1,
                 stream=None):
    """Build the cos/sin tables for ``positions`` into ``workspace``."""
    dims = Dims(L_s=L_s, L_t=L_t, H=H, T=positions.shape[0], d=d, k=k)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_rope_prepare(ctypes.byref(dims), ctypes.byref(rs), ctypes.byref(rt),
                                   _ptr(positions), _ptr(workspace), workspace.numel(),
                                   _stream(stream, positions.device)))


def map_cache(src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions, out,
              workspace=None, flags=0, stream=None):
    """Map the whole cache into ``out`` [L_t, 2, H, T, d] (enqueued on the stream)."""
    idx = _idx_host(idx)
    _check_shapes(src, W_K, W_V, b_K, b_V, positions, idx)
    dims = _dims(src, idx)
    if tuple(out.shape) != (dims.L_t, 2, dims.H, dims.T, dims.d) or out.dtype != src.dtype:
        raise ValueError("out must be [L_t, 2, H, T, d] with the source dtype")
    ws, need = _workspace(dims, src, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_cache(
        ctypes.byref(dims), _dtype_code(src), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(ws),
        ws.numel(), flags, _stream(stream, src.device)))
    return out


def map_cache_noalloc(src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions, out,
                      flags=0, stream=None):
    """map_cache through the entry point that allocates nothing: the library's
    static device scratch serves as the workspace (calls on one device must
    not overlap)."""
    idx = _idx_host(idx)
    _check_shapes(src, W_K, W_V, b_K, b_V, positions, idx)
    dims = _dims(src, idx)
    if tuple(out.shape) != (dims.L_t, 2, dims.H, dims.T, dims.d) or out.dtype != src.dtype:
        raise ValueError("out must be [L_t, 2, H, T, d] with the source dtype")
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_cache_noalloc(
        ctypes.byref(dims), _dtype_code(src), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), flags,
        _stream(stream, src.device)))
    return out


def map_layer(l_t, src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions, out,
              workspace=None, flags=0, stream=None):
    """Map target layer ``l_t`` only; writes ``out[l_t]``."""
    idx = _idx_host(idx)
    _check_shapes(src, W_K, W_V, b_K, b_V, positions, idx)
    dims = _dims(src, idx)
    if tuple(out.shape) != (dims.L_t, 2, dims.H, dims.T, dims.d) or out.dtype != src.dtype:
        raise ValueError("out must be [L_t, 2, H, T, d] with the source dtype")
    ws, need = _workspace(dims, src, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_layer(
        ctypes.byref(dims), _dtype_code(src), int(l_t), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(ws),
        ws.numel(), flags, _stream(stream, src.device)))
    return out


def map_cache_slots(src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions,
                    slot_mapping, pool, workspace=None, flags=0, stream=None):
    """Map packed rows into the slot-addressed pool [L_t, 2, H, num_slots, d]."""
    idx = _idx_host(idx)
    _check_shapes(src, W_K, W_V, b_K, b_V, positions, idx)
    dims = _dims(src, idx)
    if (pool.dim() != 5 or tuple(pool.shape[:3]) != (dims.L_t, 2, dims.H)
            or pool.shape[4] != dims.d or pool.dtype != src.dtype):
        raise ValueError("pool must be [L_t, 2, H, num_slots, d] with the source dtype")
    if slot_mapping.dtype != torch.int32 or slot_mapping.shape != (dims.T,):
        raise ValueError("slot_mapping must be int32 [T]")
    ws, need = _workspace(dims, src, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_cache_slots(
        ctypes.byref(dims), _dtype_code(src), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(slot_mapping),
        int(pool.shape[3]), _ptr(pool), _ptr(ws), ws.numel(), flags,
        _stream(stream, src.device)))
    return pool


def xhead_workspace_bytes(dims: XDims) -> int:
    return int(load().kvx_xhead_workspace_bytes(ctypes.byref(dims)))


def _xhead_args(src, idx, W_K, W_V, b_K, b_V, positions):
    idx = _idx_host(idx)
    L_s, two, H_s, T, d = src.shape
    if two != 2:
        raise ValueError("src_kv must be [L_s, 2, H_s, T, d]")
    L_t, k = idx.shape
    if W_K.dim() != 4:
        raise ValueError("W_K must be [L_t, H_t, k*H_s*d, d]")
    H_t = W_K.shape[1]
    for name, W in (("W_K", W_K), ("W_V", W_V)):
        if tuple(W.shape) != (L_t, H_t, k * H_s * d, d) or W.dtype != src.dtype:
            raise ValueError(f"{name} must be [L_t, H_t, k*H_s*d, d] = {(L_t, H_t, k * H_s * d, d)}"
                             f" with the source dtype, got {tuple(W.shape)} {W.dtype}")
    for name, b in (("b_K", b_K), ("b_V", b_V)):
        if b is not None and (tuple(b.shape) != (L_t, H_t, d) or b.dtype != src.dtype):
            raise ValueError(f"{name} must be [L_t, H_t, d] with the source dtype")
    if positions.dtype != torch.int32 or positions.shape != (T,):
        raise ValueError("positions must be int32 [T]")
    return idx, XDims(L_s=L_s, L_t=L_t, H_s=H_s, H_t=H_t, T=T, d=d, k=k)


def _xhead_workspace(dims, device, workspace, stream):
    if workspace is None:
        workspace = _scratch(xhead_workspace_bytes(dims), device, stream)
    return workspace


def map_cache_xhead(src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions, out,
                    workspace=None, flags=0, stream=None):
    """Cross-head map of the whole cache into ``out`` [L_t, 2, H_t, T, d].

    src [L_s, 2, H_s, T, d]; W_K, W_V [L_t, H_t, k*H_s*d, d]; b_K, b_V
    [L_t, H_t, d] or None (enqueued on the stream)."""
    idx, dims = _xhead_args(src, idx, W_K, W_V, b_K, b_V, positions)
    if (tuple(out.shape) != (dims.L_t, 2, dims.H_t, dims.T, dims.d)
            or out.dtype != src.dtype):
        raise ValueError("out must be [L_t, 2, H_t, T, d] with the source dtype")
    ws = _xhead_workspace(dims, src.device, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_cache_xhead(
        ctypes.byref(dims), _dtype_code(src), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(ws),
        ws.numel(), flags, _stream(stream, src.device)))
    return out


def map_layer_xhead(l_t, src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions, out,
                    workspace=None, flags=0, stream=None):
    """Cross-head map of target layer ``l_t`` only; writes ``out[l_t]``."""
    idx, dims = _xhead_args(src, idx, W_K, W_V, b_K, b_V, positions)
    if (tuple(out.shape) != (dims.L_t, 2, dims.H_t, dims.T, dims.d)
            or out.dtype != src.dtype):
        raise ValueError("out must be [L_t, 2, H_t, T, d] with the source dtype")
    ws = _xhead_workspace(dims, src.device, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_layer_xhead(
        ctypes.byref(dims), _dtype_code(src), int(l_t), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(ws),
        ws.numel(), flags, _stream(stream, src.device)))
    return out


def map_cache_slots_xhead(src, idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt, positions,
                          slot_mapping, pool, workspace=None, flags=0, stream=None):
    """Cross-head map of packed rows into the pool [L_t, 2, H_t, num_slots, d]."""
    idx, dims = _xhead_args(src, idx, W_K, W_V, b_K, b_V, positions)
    if (pool.dim() != 5 or tuple(pool.shape[:3]) != (dims.L_t, 2, dims.H_t)
            or pool.shape[4] != dims.d or pool.dtype != src.dtype):
        raise ValueError("pool must be [L_t, 2, H_t, num_slots, d] with the source dtype")
    if slot_mapping.dtype != torch.int32 or slot_mapping.shape != (dims.T,):
        raise ValueError("slot_mapping must be int32 [T]")
    ws = _xhead_workspace(dims, src.device, workspace, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_map_cache_slots_xhead(
        ctypes.byref(dims), _dtype_code(src), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), _ptr(W_K), _ptr(W_V), _ptr(b_K), _ptr(b_V),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(slot_mapping),
        int(pool.shape[3]), _ptr(pool), _ptr(ws), ws.numel(), flags,
        _stream(stream, src.device)))
    return pool


# ---------------------------------------------------------------- fitting

def _calib_dims(src, tgt, k=1):
    L_s, two, H, N, d = src.shape
    if two != 2 or tgt.dim() != 5 or tgt.shape[1] != 2 or tuple(tgt.shape[2:]) != (H, N, d):
        raise ValueError("caches must be [L_s, 2, H, N, d] and [L_t, 2, H, N, d]")
    if src.dtype != tgt.dtype:
        raise TypeError("source and target caches must share the dtype")
    return Dims(L_s=L_s, L_t=tgt.shape[0], H=H, T=N, d=d, k=k)


def fit_workspace_bytes(dims: Dims) -> int:
    return int(load().kvx_fit_workspace_bytes(ctypes.byref(dims)))


def probe_workspace_bytes(dims: Dims) -> int:
    return int(load().kvx_probe_workspace_bytes(ctypes.byref(dims)))


def fit_cache(src, idx, tgt, rope_src, rope_tgt, positions, lam=0.01, out=None,
              workspace=None, flags=0, stream=None):
    """Fit the per-head mapper from calibration caches; returns fp32 tensors
    (W_K, W_V [L_t, H, k*d, d], b_K, b_V [L_t, H, d]) (enqueued on the stream)."""
    idx = _idx_host(idx)
    dims = _calib_dims(src, tgt, k=idx.shape[1])
    if idx.shape[0] != dims.L_t:
        raise ValueError("src_idx must have one row per target layer")
    if positions.dtype != torch.int32 or positions.shape != (dims.T,):
        raise ValueError("positions must be int32 [N]")
    if out is None:
        with torch.cuda.stream(_torch_stream(stream, src.device)):
            kd = dims.k * dims.d
            out = (torch.empty((dims.L_t, dims.H, kd, dims.d), dtype=torch.float32, device=src.device),
                   torch.empty((dims.L_t, dims.H, kd, dims.d), dtype=torch.float32, device=src.device),
                   torch.empty((dims.L_t, dims.H, dims.d), dtype=torch.float32, device=src.device),
                   torch.empty((dims.L_t, dims.H, dims.d), dtype=torch.float32, device=src.device))
    if workspace is None:
        workspace = _scratch(fit_workspace_bytes(dims), src.device, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_fit_cache(
        ctypes.byref(dims), _dtype_code(src), _ptr(src), idx.ctypes.data_as(ctypes.c_void_p),
        _ptr(tgt), ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), float(lam),
        *[_ptr(t) for t in out], _ptr(workspace), workspace.numel(), flags,
        _stream(stream, src.device)))
    return out


def probe_r2(src, tgt, rope_src, rope_tgt, positions, out=None, workspace=None, flags=0,
             stream=None):
    """Single-source OLS R2 of every (source layer, target layer, head) for
    stripped keys and values: fp32 [L_s, L_t, H, 2] (enqueued on the stream)."""
    dims = _calib_dims(src, tgt)
    if positions.dtype != torch.int32 or positions.shape != (dims.T,):
        raise ValueError("positions must be int32 [N]")
    if out is None:
        with torch.cuda.stream(_torch_stream(stream, src.device)):
            out = torch.empty((dims.L_s, dims.L_t, dims.H, 2), dtype=torch.float32,
                              device=src.device)
    if workspace is None:
        workspace = _scratch(probe_workspace_bytes(dims), src.device, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_probe_r2(
        ctypes.byref(dims), _dtype_code(src), _ptr(src), _ptr(tgt), ctypes.byref(rs),
        ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(workspace), workspace.numel(), flags,
        _stream(stream, src.device)))
    return out


def select_topk(r2, k, out=None, stream=None):
    """Top-k source layers per target layer from an R2 table [L_s, L_t, H, 2]:
    device int32 [L_t, k], each row ascending."""
    if r2.dtype != torch.float32 or r2.dim() != 4 or r2.shape[3] != 2:
        raise ValueError("r2 must be float32 [L_s, L_t, H, 2]")
    L_s, L_t, H, _ = r2.shape
    if out is None:
        with torch.cuda.stream(_torch_stream(stream, r2.device)):
            out = torch.empty((L_t, k), dtype=torch.int32, device=r2.device)
    _check(load().kvx_select_topk(L_s, L_t, H, int(k), _ptr(r2), _ptr(out),
                                  _stream(stream, r2.device)))
    return out


# ---------------------------------------------------------------- MLP mapper

def mlp_workspace_bytes(dims: Dims, F: int) -> int:
    return int(load().kvx_mlp_workspace_bytes(ctypes.byref(dims), int(F)))


def _mlp_args(src, idx, mlp_K, mlp_V, positions, out):
    idx = _idx_host(idx)
    dims = _dims(src, idx)
    L_t, H, d, kd = dims.L_t, dims.H, dims.d, dims.k * dims.d
    if len(mlp_K) != 6 or len(mlp_V) != 6:
        raise ValueError("mlp_K / mlp_V must be (W1, b1, W2, b2, W3, b3)")
    F = int(mlp_K[0].shape[2]) if mlp_K[0].dim() == 4 else -1
    shapes = ((L_t, H, F, kd), (L_t, H, F), (L_t, H, F, F), (L_t, H, F), (L_t, H, d, F),
              (L_t, H, d))
    for which, net in (("mlp_K", mlp_K), ("mlp_V", mlp_V)):
        for i, (t, shp) in enumerate(zip(net, shapes)):
            if t is None and i % 2 == 1:
                continue
            if t is None or tuple(t.shape) != shp or t.dtype != src.dtype:
                raise ValueError(f"{which}[{i}] must be {shp} with the source dtype")
    if positions.dtype != torch.int32 or positions.shape != (dims.T,):
        raise ValueError("positions must be int32 [T]")
    if tuple(out.shape) != (L_t, 2, H, dims.T, d) or out.dtype != src.dtype:
        raise ValueError("out must be [L_t, 2, H, T, d] with the source dtype")
    return idx, dims, F, Mlp(*[_ptr(t) for t in mlp_K]), Mlp(*[_ptr(t) for t in mlp_V])


def mlp_map_cache(src, idx, mlp_K, mlp_V, rope_src, rope_tgt, positions, out, workspace=None,
                  flags=0, stream=None):
    """MLP mapper of the whole cache into ``out`` [L_t, 2, H, T, d].

    mlp_K, mlp_V: (W1 [L_t, H, F, k*d], b1 [L_t, H, F] or None, W2 [L_t, H, F, F],
    b2, W3 [L_t, H, d, F], b3 [L_t, H, d] or None), weights in nn.Linear's
    [out, in] layout (enqueued on the stream)."""
    idx, dims, F, nk, nv = _mlp_args(src, idx, mlp_K, mlp_V, positions, out)
    if workspace is None:
        workspace = _scratch(mlp_workspace_bytes(dims, F), src.device, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_mlp_map_cache(
        ctypes.byref(dims), _dtype_code(src), F, _ptr(src), idx.ctypes.data_as(ctypes.c_void_p),
        ctypes.byref(nk), ctypes.byref(nv), ctypes.byref(rs), ctypes.byref(rt), _ptr(positions),
        _ptr(out), _ptr(workspace), workspace.numel(), flags, _stream(stream, src.device)))
    return out


def mlp_map_layer(l_t, src, idx, mlp_K, mlp_V, rope_src, rope_tgt, positions, out,
                  workspace=None, flags=0, stream=None):
    """MLP mapper of target layer ``l_t`` only; writes ``out[l_t]``."""
    idx, dims, F, nk, nv = _mlp_args(src, idx, mlp_K, mlp_V, positions, out)
    if workspace is None:
        workspace = _scratch(mlp_workspace_bytes(dims, F), src.device, stream)
    rs, rt = make_rope(rope_src), make_rope(rope_tgt)
    _check(load().kvx_mlp_map_layer(
        ctypes.byref(dims), _dtype_code(src), F, int(l_t), _ptr(src),
        idx.ctypes.data_as(ctypes.c_void_p), ctypes.byref(nk), ctypes.byref(nv),
        ctypes.byref(rs), ctypes.byref(rt), _ptr(positions), _ptr(out), _ptr(workspace),
        workspace.numel(), flags, _stream(stream, src.device)))
    return out
