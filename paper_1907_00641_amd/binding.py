"""Thin Python binding of the C ABI in include/pam_lattice.h (and the benchmark's
row-copy probe in include/pam_probe.h).

Argument marshalling only: every step of the filter runs in the HIP
library ``libpam_lattice.so``.  PyTorch provides device memory and the
current stream; tensors are passed to the library as raw pointers.  There is
no fallback: if the library is not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libpam_lattice.so")

PAM_OK = 0
PAM_ERR_INVALID_ARGUMENT = 1
PAM_ERR_OUT_OF_MEMORY = 2
PAM_ERR_CAPACITY = 3
PAM_ERR_KEY_RANGE = 4
PAM_ERR_STATE = 5
PAM_ERR_DEVICE = 6
PAM_NORMALIZE = 1
PAM_EGRAD_AUGMENTED = 2
PAM_MAX_D = 16
PAM_MAX_C = 1024
PAM_MAX_GROUPS = 65536

# every symbol the header declares
EXPORTS = (
    "pam_lattice_build", "pam_filter_fwd", "pam_filter_bwd", "pam_lattice_stats",
    "pam_lattice_export", "pam_lattice_set_capacity", "pam_timing_enable", "pam_kernel_count",
    "pam_kernel_name", "pam_timing_read", "pam_lattice_destroy", "pam_status_string",
    "pam_last_error", "pam_lattice_build_groups", "pam_lattice_export_groups", "pam_filter_fwd_asym",
    "pam_filter_bwd_asym", "pam_block_fwd", "pam_block_bwd_workspace", "pam_block_bwd", "pam_block_bwd_noalloc",
    "pam_probe_copy_rows",
)


class BlockDesc(ctypes.Structure):
    """pam_block_desc_t of the C header."""
    _fields_ = [("c_in", ctypes.c_int32), ("d_tot", ctypes.c_int32), ("c_tot", ctypes.c_int32),
                ("groups", ctypes.c_int32), ("dims", ctypes.c_int32 * 3), ("mesh_scale", ctypes.c_float),
                ("slope", ctypes.c_float)]

_lib = None
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_u32 = ctypes.c_uint32


class PamError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {status_string(status)} ({detail})")
        self.status = status


def lib():
    """Load libpam_lattice.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_1907_00641_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.pam_lattice_build.restype = ctypes.c_int
    L.pam_lattice_build.argtypes = [_vp, _i64, _i32, _vp, ctypes.POINTER(_vp)]
    L.pam_lattice_build_groups.restype = ctypes.c_int
    L.pam_lattice_build_groups.argtypes = [_vp, _i64, _i32, _vp, _i32, _vp, ctypes.POINTER(_vp)]
    L.pam_lattice_export_groups.restype = ctypes.c_int
    L.pam_lattice_export_groups.argtypes = [_vp, _vp]
    L.pam_filter_fwd.restype = ctypes.c_int
    L.pam_filter_fwd.argtypes = [_vp, _vp, _i32, _u32, _vp, _vp]
    L.pam_filter_fwd_asym.restype = ctypes.c_int
    L.pam_filter_fwd_asym.argtypes = [_vp, _i64, _vp, _i32, _u32, _vp, _vp]
    L.pam_filter_bwd_asym.restype = ctypes.c_int
    L.pam_filter_bwd_asym.argtypes = [_vp, _i64, _vp, _vp, _i32, _u32, _vp, _vp, _vp]
    L.pam_block_fwd.restype = ctypes.c_int
    L.pam_block_fwd.argtypes = [ctypes.POINTER(BlockDesc)] + [_vp] * 8
    L.pam_block_bwd_workspace.restype = ctypes.c_size_t
    L.pam_block_bwd_workspace.argtypes = [ctypes.POINTER(BlockDesc)]
    L.pam_block_bwd.restype = ctypes.c_int
    L.pam_block_bwd.argtypes = [ctypes.POINTER(BlockDesc)] + [_vp] * 13
    L.pam_block_bwd_noalloc.restype = ctypes.c_int
    L.pam_block_bwd_noalloc.argtypes = [ctypes.POINTER(BlockDesc)] + [_vp] * 12
    L.pam_filter_bwd.restype = ctypes.c_int
    L.pam_filter_bwd.argtypes = [_vp, _vp, _vp, _i32, _u32, _vp, _vp, _vp]
    L.pam_lattice_stats.restype = ctypes.c_int
    L.pam_lattice_stats.argtypes = [_vp, ctypes.POINTER(_i64), ctypes.POINTER(_i64)]
    L.pam_lattice_export.restype = ctypes.c_int
    L.pam_lattice_export.argtypes = [_vp, _vp, _vp, _vp, _vp]
    L.pam_lattice_set_capacity.restype = ctypes.c_int
    L.pam_lattice_set_capacity.argtypes = [_vp, _i64, _i32]
    L.pam_timing_enable.restype = ctypes.c_int
    L.pam_timing_enable.argtypes = [_vp, _i32]
    L.pam_kernel_count.restype = _i32
    L.pam_kernel_count.argtypes = []
    L.pam_kernel_name.restype = ctypes.c_char_p
    L.pam_kernel_name.argtypes = [_i32]
    L.pam_timing_read.restype = ctypes.c_int
    L.pam_timing_read.argtypes = [_vp, _i32, ctypes.POINTER(_i64), ctypes.POINTER(ctypes.c_double)]
    L.pam_probe_copy_rows.restype = ctypes.c_int
    L.pam_probe_copy_rows.argtypes = [_vp, _vp, _vp, _i64, _i32, _i32, _vp]
    L.pam_lattice_destroy.restype = None
    L.pam_lattice_destroy.argtypes = [_vp]
    L.pam_status_string.restype = ctypes.c_char_p
    L.pam_status_string.argtypes = [ctypes.c_int]
    L.pam_last_error.restype = ctypes.c_char_p
    L.pam_last_error.argtypes = []
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().pam_status_string(status).decode()


def last_error() -> str:
    return lib().pam_last_error().decode()


def _check(status: int, where: str):
    if status != PAM_OK:
        raise PamError(status, where, last_error())


def _stream_ptr(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _dev_ptr(t: torch.Tensor | None, dtype, name: str) -> int | None:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


class Lattice:
    """A built lattice handle plus the borrowed feature tensor it reads."""

    def __init__(self, handle: int, feat: torch.Tensor, d: int):
        self.handle = ctypes.c_void_p(handle)
        self.feat = feat  # kept alive: the augmented-channel backward re-reads it
        self.n = feat.shape[0]
        self.d = d

    def __del__(self):
        if getattr(self, "handle", None) is not None and self.handle.value and _lib is not None:
            _lib.pam_lattice_destroy(self.handle)
            self.handle = None

    def destroy(self):
        if self.handle is not None and self.handle.value:
            lib().pam_lattice_destroy(self.handle)
        self.handle = None


def pam_lattice_build(feat: torch.Tensor, stream=None, lat: Lattice | None = None, group_start=None) -> Lattice:
    """Build (or rebuild in place) the lattice of ``feat`` (n x d fp32, device).
    ``group_start`` (G + 1 offsets, host) makes a batched build of G
    independent point groups (pam_lattice_build_groups)."""
    if feat.dim() != 2:
        raise ValueError("feat must be n x d")
    n, d = feat.shape
    ptr = _dev_ptr(feat, torch.float32, "feat")
    h = ctypes.c_void_p(lat.handle.value if lat is not None else None)
    if group_start is None:
        _check(lib().pam_lattice_build(ptr, n, d, _stream_ptr(stream), ctypes.byref(h)), "pam_lattice_build")
    else:
        import numpy as np

        gs = np.ascontiguousarray(np.asarray(group_start, dtype=np.int64))
        _check(lib().pam_lattice_build_groups(ptr, n, d, gs.ctypes.data, len(gs) - 1, _stream_ptr(stream),
                                              ctypes.byref(h)), "pam_lattice_build_groups")
    if lat is not None:
        lat.feat, lat.n, lat.d = feat, n, d
        return lat
    return Lattice(h.value, feat, d)


def pam_filter_fwd(lat: Lattice, val: torch.Tensor, flags: int = 0, out: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Forward filter; returns ``out`` (n x C fp32, allocated if not given)."""
    if val.dim() != 2 or val.shape[0] != lat.n:
        raise ValueError("val must be n x C")
    if out is None:
        out = torch.empty_like(val)
    _check(lib().pam_filter_fwd(lat.handle, _dev_ptr(val, torch.float32, "val"), val.shape[1], flags,
                                _dev_ptr(out, torch.float32, "out"), _stream_ptr(stream)),
           "pam_filter_fwd")
    return out


def pam_filter_bwd(lat: Lattice, val: torch.Tensor, grad_out: torch.Tensor, flags: int = 0,
                   grad_val: torch.Tensor | bool | None = True, grad_feat: torch.Tensor | bool | None = True,
                   stream=None):
    """Backward filter; returns (grad_val, grad_feat), each None if skipped.
    Pass True to allocate an output, a tensor to fill it, None/False to skip."""
    if grad_val is True:
        grad_val = torch.empty_like(val)
    elif grad_val is False:
        grad_val = None
    if grad_feat is True:
        grad_feat = torch.empty_like(lat.feat)
    elif grad_feat is False:
        grad_feat = None
    _check(lib().pam_filter_bwd(lat.handle, _dev_ptr(val, torch.float32, "val"),
                                _dev_ptr(grad_out, torch.float32, "grad_out"), val.shape[1], flags,
                                _dev_ptr(grad_val, torch.float32, "grad_val"),
                                _dev_ptr(grad_feat, torch.float32, "grad_feat"), _stream_ptr(stream)),
           "pam_filter_bwd")
    return grad_val, grad_feat


def pam_filter_fwd_asym(lat: Lattice, n_keys: int, val: torch.Tensor, flags: int = 0,
                        out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Asymmetric forward filter over a lattice built on [keys; queries]:
    ``val`` holds the n_keys key values (n_keys x C); returns ``out`` for the
    n - n_keys queries."""
    if val.dim() != 2 or val.shape[0] != n_keys:
        raise ValueError("val must be n_keys x C")
    if out is None:
        out = torch.empty((lat.n - n_keys, val.shape[1]), dtype=val.dtype, device=val.device)
    _check(lib().pam_filter_fwd_asym(lat.handle, n_keys, _dev_ptr(val, torch.float32, "val"), val.shape[1], flags,
                                     _dev_ptr(out, torch.float32, "out"), _stream_ptr(stream)),
           "pam_filter_fwd_asym")
    return out


def pam_filter_bwd_asym(lat: Lattice, n_keys: int, val: torch.Tensor, grad_out: torch.Tensor, flags: int = 0,
                        grad_val: torch.Tensor | bool | None = True, grad_feat: torch.Tensor | bool | None = True,
                        stream=None):
    """Backward pass of the asymmetric filter; returns (grad_val (n_keys x C),
    grad_feat (n x d)), each None if skipped."""
    if grad_val is True:
        grad_val = torch.empty_like(val)
    elif grad_val is False:
        grad_val = None
    if grad_feat is True:
        grad_feat = torch.empty_like(lat.feat)
    elif grad_feat is False:
        grad_feat = None
    _check(lib().pam_filter_bwd_asym(lat.handle, n_keys, _dev_ptr(val, torch.float32, "val"),
                                     _dev_ptr(grad_out, torch.float32, "grad_out"), val.shape[1], flags,
                                     _dev_ptr(grad_val, torch.float32, "grad_val"),
                                     _dev_ptr(grad_feat, torch.float32, "grad_feat"), _stream_ptr(stream)),
           "pam_filter_bwd_asym")
    return grad_val, grad_feat


def block_desc(c_in: int, d_tot: int, c_tot: int, groups: int, dims, mesh_scale: float, slope: float) -> BlockDesc:
    return BlockDesc(c_in, d_tot, c_tot, groups, (ctypes.c_int32 * 3)(*dims), mesh_scale, slope)


def pam_block_fwd(desc: BlockDesc, x: torch.Tensor, wf: torch.Tensor, bf: torch.Tensor, wv: torch.Tensor,
                  bv: torch.Tensor, stream=None):
    """Permutohedral block prologue; returns (feat, val) in the grouped layout
    ((groups N) x d_tot/groups and (groups N) x c_tot/groups)."""
    n = desc.dims[0] * desc.dims[1] * desc.dims[2]
    G = desc.groups
    feat = torch.empty((G * n, desc.d_tot // G), dtype=torch.float32, device=x.device)
    val = torch.empty((G * n, desc.c_tot // G), dtype=torch.float32, device=x.device)
    f32 = torch.float32
    _check(lib().pam_block_fwd(ctypes.byref(desc), _dev_ptr(x, f32, "x"), _dev_ptr(wf, f32, "wf"),
                               _dev_ptr(bf, f32, "bf"), _dev_ptr(wv, f32, "wv"), _dev_ptr(bv, f32, "bv"),
                               feat.data_ptr(), val.data_ptr(), _stream_ptr(stream)), "pam_block_fwd")
    return feat, val


def pam_block_bwd(desc: BlockDesc, x: torch.Tensor, wf: torch.Tensor, bf: torch.Tensor, wv: torch.Tensor,
                  grad_feat: torch.Tensor, grad_val: torch.Tensor, stream=None):
    """Backward of the prologue; returns (grad_x, grad_wf, grad_bf, grad_wv, grad_bv)."""
    f32 = torch.float32
    outs = [torch.empty_like(x), torch.empty_like(wf), torch.empty_like(bf), torch.empty_like(wv),
            torch.empty((desc.c_tot,), dtype=f32, device=x.device)]
    ws_bytes = lib().pam_block_bwd_workspace(ctypes.byref(desc))
    ws = torch.empty((max(ws_bytes, 4) + 3) // 4, dtype=f32, device=x.device)
    _check(lib().pam_block_bwd(ctypes.byref(desc), _dev_ptr(x, f32, "x"), _dev_ptr(wf, f32, "wf"),
                               _dev_ptr(bf, f32, "bf"), _dev_ptr(wv, f32, "wv"),
                               _dev_ptr(grad_feat, f32, "grad_feat"), _dev_ptr(grad_val, f32, "grad_val"),
                               *[o.data_ptr() for o in outs], ws.data_ptr(), _stream_ptr(stream)), "pam_block_bwd")
    return tuple(outs)


def pam_block_bwd_noalloc(desc: BlockDesc, x: torch.Tensor, wf: torch.Tensor, bf: torch.Tensor, wv: torch.Tensor,
                          grad_feat: torch.Tensor, grad_val: torch.Tensor, out, stream=None):
    """pam_block_bwd through the allocation-free entry point: ``out`` is the
    caller's (grad_x, grad_wf, grad_bf, grad_wv, grad_bv), written in full."""
    f32 = torch.float32
    shapes = (tuple(x.shape), tuple(wf.shape), tuple(bf.shape), tuple(wv.shape), (desc.c_tot,))
    ptrs = [_dev_ptr(o, f32, name) for o, name in zip(out, ("grad_x", "grad_wf", "grad_bf", "grad_wv", "grad_bv"))]
    for o, shp in zip(out, shapes):
        if tuple(o.shape) != shp:
            raise ValueError(f"output of shape {tuple(o.shape)}, expected {shp}")
    _check(lib().pam_block_bwd_noalloc(ctypes.byref(desc), _dev_ptr(x, f32, "x"), _dev_ptr(wf, f32, "wf"),
                                       _dev_ptr(bf, f32, "bf"), _dev_ptr(wv, f32, "wv"),
                                       _dev_ptr(grad_feat, f32, "grad_feat"), _dev_ptr(grad_val, f32, "grad_val"),
                                       *ptrs, _stream_ptr(stream)), "pam_block_bwd_noalloc")
    return tuple(out)


def pam_lattice_stats(lat: Lattice):
    """Returns (num_vertices, table_capacity)."""
    m, cap = _i64(0), _i64(0)
    _check(lib().pam_lattice_stats(lat.handle, ctypes.byref(m), ctypes.byref(cap)), "pam_lattice_stats")
    return m.value, cap.value


def pam_lattice_export(lat: Lattice):
    """Host copies: keys (M x d), vert (n x (d+1)), bary (n x (d+1)), nbr (M x (d+1) x 2)."""
    import numpy as np

    M, _ = pam_lattice_stats(lat)
    d, n = lat.d, lat.n
    keys = np.zeros((M, d), dtype=np.int32)
    vert = np.zeros((n, d + 1), dtype=np.int32)
    bary = np.zeros((n, d + 1), dtype=np.float32)
    nbr = np.zeros((M, d + 1, 2), dtype=np.int32)
    _check(lib().pam_lattice_export(lat.handle, keys.ctypes.data, vert.ctypes.data, bary.ctypes.data,
                                    nbr.ctypes.data), "pam_lattice_export")
    return keys, vert, bary, nbr


def pam_lattice_export_groups(lat: Lattice):
    """Host copy of the group id of every vertex (M int32)."""
    import numpy as np

    M, _ = pam_lattice_stats(lat)
    vg = np.zeros(M, dtype=np.int32)
    if M:
        _check(lib().pam_lattice_export_groups(lat.handle, vg.ctypes.data), "pam_lattice_export_groups")
    return vg


def pam_lattice_set_capacity(lat: Lattice, table_capacity: int, allow_regrow: bool = True):
    _check(lib().pam_lattice_set_capacity(lat.handle, table_capacity, int(allow_regrow)),
           "pam_lattice_set_capacity")


def pam_timing_enable(lat: Lattice, enable: bool):
    _check(lib().pam_timing_enable(lat.handle, int(enable)), "pam_timing_enable")


def pam_kernel_names():
    L = lib()
    return [L.pam_kernel_name(k).decode() for k in range(L.pam_kernel_count())]


def pam_timing_read(lat: Lattice):
    """Synchronise; returns {kernel name: (launches, total_ms)}."""
    L = lib()
    res = {}
    for k, name in enumerate(pam_kernel_names()):
        cnt, ms = _i64(0), ctypes.c_double(0.0)
        _check(L.pam_timing_read(lat.handle, k, ctypes.byref(cnt), ctypes.byref(ms)), "pam_timing_read")
        if cnt.value:
            res[name] = (cnt.value, ms.value)
    return res


def pam_probe_copy_rows(src: torch.Tensor, dst: torch.Tensor, perm: torch.Tensor | None, mode: int,
                        stream=None):
    """Measurement utility: dst row (perm[i] if mode & 2 else i) = src row
    (perm[i] if mode & 1 else i) for the n rows of the n x c fp32 tensors."""
    if src.dim() != 2 or src.shape != dst.shape:
        raise ValueError("src and dst must be n x c tensors of one shape")
    n, c = src.shape
    ps = _dev_ptr(src, torch.float32, "src")
    pd = _dev_ptr(dst, torch.float32, "dst")
    pp = _dev_ptr(perm, torch.int32, "perm") if mode else None
    if mode and perm.numel() != n:
        raise ValueError("perm must hold n entries")
    _check(lib().pam_probe_copy_rows(ps, pd, pp, n, c, mode, _stream_ptr(stream)), "pam_probe_copy_rows")


def pam_lattice_destroy(lat: Lattice):
    lat.destroy()
