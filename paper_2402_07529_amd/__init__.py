"""Python binding of libhc (include/hc.h): lossless homomorphic gradient
compression on MI355X.

Argument marshalling only.  Every stage runs in the library's gfx950 kernels;
PyTorch supplies device memory and the current stream.  The names mirror the
C ABI:

    hc_geometry   sketch sizing, |Y| >= gamma * n (section 3.2, gamma = 1.23)
    hc_geometry_blocked  the same for a blocked sketch (section 3.2 blocking)
    hc_geometry_bloom    the same with a Bloom-filter index (section 3.3)
    hc_sizes      byte sizes of Y, B and the decode workspace
    hc_plan_bytes, hc_plan_build   inverse row map of a geometry (c >= 256)
    hc_encode     Algorithm 1 phase I on a dense gradient (sections 3.1-3.4)
    hc_encode_gather, hc_encode_staged  the same through a plan (dense or
                  sparse gradients), without global atomics
    hc_encode_coo the same from COO input
    hc_aggregate  sum of sketches and OR of bitmaps over W workers (section 3)
    hc_decode     Algorithm 1 phase II: parallel peeling + median estimate

The library must be built (``python -m paper_2402_07529_amd.build``); there is
no fallback: importing this package without libhc.so raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhc.so")

HC_OK, HC_EINVAL, HC_EWORKSPACE, HC_EHIP, HC_EUNSUPPORTED = range(5)
HC_I32, HC_F32 = 0, 1
GAMMA = 1.23
INFO_BYTES = 32

EXPORTS = ("hc_geometry", "hc_geometry_blocked", "hc_geometry_bloom", "hc_sizes", "hc_plan_bytes",
           "hc_plan_build", "hc_encode", "hc_encode_gather", "hc_encode_staged_bytes",
           "hc_encode_staged", "hc_encode_coo", "hc_aggregate",
           "hc_decode", "hc_decode_noalloc", "hc_status_string", "hc_last_error")
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024


class HCError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: status {status}: {msg}")
        self.status = status


class hc_params(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("k", ctypes.c_uint32), ("c", ctypes.c_uint32),
                ("rows", ctypes.c_uint64), ("seed", ctypes.c_uint64),
                ("vtype", ctypes.c_uint32), ("block", ctypes.c_uint32),
                ("bloom_k", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("bloom_rows", ctypes.c_uint64)]

    @property
    def cells(self) -> int:
        return int(self.rows) * int(self.c)

    @property
    def words(self) -> int:
        """Words of an n-bit bitmap (the bitmap index, the recovered mask)."""
        return (int(self.n) + 31) // 32

    @property
    def index_words(self) -> int:
        """Words of the index B: the bitmap, or the Bloom filter."""
        if int(self.bloom_k) == 0:
            return self.words
        return (int(self.bloom_rows) * int(self.c) + 31) // 32

    @property
    def is_f32(self) -> bool:
        return int(self.vtype) == HC_F32

    @property
    def nblocks(self) -> int:
        if int(self.block) == 0:
            return 1
        return ((int(self.n) + int(self.c) - 1) // int(self.c) + int(self.block) - 1) // int(self.block)

    @property
    def block_rows(self) -> int:
        return int(self.rows) // self.nblocks


if not os.path.exists(LIB_PATH):
    raise ImportError(f"libhc.so not built at {LIB_PATH}; run python -m paper_2402_07529_amd.build")

_lib = ctypes.CDLL(LIB_PATH)
_P = ctypes.c_void_p
_PP = ctypes.POINTER(hc_params)
_lib.hc_geometry.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double, ctypes.c_uint32,
                             ctypes.c_uint64, ctypes.c_int, _PP]
_lib.hc_geometry_blocked.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                     ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64,
                                     ctypes.c_int, _PP]
_lib.hc_geometry_bloom.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                   ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int, _PP,
                                   ctypes.POINTER(ctypes.c_double)]
_lib.hc_sizes.argtypes = [_PP, ctypes.c_uint64, ctypes.POINTER(ctypes.c_size_t),
                          ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]
_lib.hc_encode.argtypes = [_PP, _P, _P, _P, _P]
_lib.hc_encode_gather.argtypes = [_PP, _P, ctypes.c_size_t, _P, _P, _P, _P]
_lib.hc_encode_staged_bytes.argtypes = [_PP, ctypes.POINTER(ctypes.c_size_t)]
_lib.hc_encode_staged.argtypes = [_PP, _P, ctypes.c_size_t, _P, ctypes.c_size_t, _P, _P, _P, _P]
_lib.hc_encode_coo.argtypes = [_PP, _P, _P, ctypes.c_uint64, _P, _P, _P]
_lib.hc_aggregate.argtypes = [_PP, _P, _P, ctypes.c_uint32, _P, _P, _P]
_lib.hc_decode.argtypes = [_PP, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, ctypes.c_uint64,
                           _P, ctypes.c_size_t, _P]
_lib.hc_decode_noalloc.argtypes = [_PP, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P,
                                   ctypes.c_uint64, _P]
_lib.hc_plan_bytes.argtypes = [_PP, ctypes.POINTER(ctypes.c_size_t)]
_lib.hc_plan_build.argtypes = [_PP, _P, ctypes.c_size_t, _P]
for _f in ("hc_geometry", "hc_geometry_blocked", "hc_geometry_bloom", "hc_sizes", "hc_plan_bytes",
           "hc_plan_build", "hc_encode", "hc_encode_gather", "hc_encode_staged_bytes",
           "hc_encode_staged", "hc_encode_coo", "hc_aggregate",
           "hc_decode", "hc_decode_noalloc"):
    getattr(_lib, _f).restype = ctypes.c_int
_lib.hc_status_string.argtypes = [ctypes.c_int]
_lib.hc_status_string.restype = ctypes.c_char_p
_lib.hc_last_error.argtypes = []
_lib.hc_last_error.restype = ctypes.c_char_p


def lib():
    return _lib


def _check(status: int, where: str):
    if status != HC_OK:
        raise HCError(status, where, (_lib.hc_last_error() or b"").decode())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, name, dtype=None, numel=None):
    """Device pointer of a contiguous CUDA tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _vdtypes(p: hc_params):
    import torch
    return (torch.float32,) if p.is_f32 else (torch.int32,)


def _u32():
    import torch
    return (torch.int32, torch.uint32) if hasattr(torch, "uint32") else (torch.int32,)


def hc_geometry(n: int, n_nonzero: int, gamma: float = GAMMA, c: int = 1024, seed: int = 0,
                vtype: str = "i32") -> hc_params:
    p = hc_params()
    vt = HC_F32 if vtype in ("f32", HC_F32) else HC_I32
    _check(_lib.hc_geometry(n, n_nonzero, gamma, c, seed & (2**64 - 1), vt, ctypes.byref(p)),
           "hc_geometry")
    return p


def hc_geometry_blocked(n: int, n_nonzero: int, gamma: float = 1.3, c: int = 1024,
                        block_rows: int = 0, seed: int = 0, vtype: str = "i32") -> hc_params:
    """block_rows = 0: the library's choice for the current device."""
    p = hc_params()
    vt = HC_F32 if vtype in ("f32", HC_F32) else HC_I32
    _check(_lib.hc_geometry_blocked(n, n_nonzero, gamma, c, block_rows, seed & (2**64 - 1), vt,
                                    ctypes.byref(p)), "hc_geometry_blocked")
    return p


def hc_geometry_bloom(n: int, n_nonzero: int, gamma: float = GAMMA, c: int = 1024, seed: int = 0,
                      vtype: str = "i32"):
    """(params with a Bloom-filter index, the paper's eps)."""
    p = hc_params()
    eps = ctypes.c_double()
    vt = HC_F32 if vtype in ("f32", HC_F32) else HC_I32
    _check(_lib.hc_geometry_bloom(n, n_nonzero, gamma, c, seed & (2**64 - 1), vt, ctypes.byref(p),
                                  ctypes.byref(eps)), "hc_geometry_bloom")
    return p, eps.value


def make_params(n: int, rows: int, seed: int, c: int = 1024, vtype: str = "i32",
                block: int = 0, bloom_k: int = 0, bloom_rows: int = 0) -> hc_params:
    return hc_params(n, 3, c, rows, seed & (2**64 - 1), HC_F32 if vtype == "f32" else HC_I32,
                     block, bloom_k, 0, bloom_rows)


def hc_sizes(p: hc_params, max_support: int = 0):
    y = ctypes.c_size_t()
    b = ctypes.c_size_t()
    w = ctypes.c_size_t()
    _check(_lib.hc_sizes(ctypes.byref(p), max_support, ctypes.byref(y), ctypes.byref(b),
                         ctypes.byref(w)), "hc_sizes")
    return y.value, b.value, w.value


def hc_encode(p: hc_params, x, y, b, stream=None):
    _check(_lib.hc_encode(ctypes.byref(p), _ptr(x, "x", _vdtypes(p), p.n),
                          _ptr(y, "y", _vdtypes(p), p.cells),
                          _ptr(b, "b", _u32(), p.index_words), _stream(stream)), "hc_encode")


def hc_encode_gather(p: hc_params, plan, x, y, b, stream=None):
    import torch
    _check(_lib.hc_encode_gather(ctypes.byref(p), _ptr(plan, "plan", (torch.uint8,)), plan.numel(),
                                 _ptr(x, "x", _vdtypes(p), p.n),
                                 _ptr(y, "y", _vdtypes(p), p.cells),
                                 _ptr(b, "b", _u32(), p.index_words), _stream(stream)),
           "hc_encode_gather")


def hc_encode_staged_bytes(p: hc_params) -> int:
    b = ctypes.c_size_t()
    _check(_lib.hc_encode_staged_bytes(ctypes.byref(p), ctypes.byref(b)), "hc_encode_staged_bytes")
    return b.value


def hc_encode_staged(p: hc_params, plan, ws, x, y, b, stream=None):
    import torch
    _check(_lib.hc_encode_staged(ctypes.byref(p), _ptr(plan, "plan", (torch.uint8,)), plan.numel(),
                                 _ptr(ws, "ws", (torch.uint8,)), ws.numel(),
                                 _ptr(x, "x", _vdtypes(p), p.n),
                                 _ptr(y, "y", _vdtypes(p), p.cells),
                                 _ptr(b, "b", _u32(), p.index_words), _stream(stream)),
           "hc_encode_staged")


def alloc_stage_workspace(p: hc_params, device="cuda"):
    import torch
    return torch.empty(hc_encode_staged_bytes(p), dtype=torch.uint8, device=device)


def hc_encode_coo(p: hc_params, idx, val, y, b, stream=None):
    nnz = idx.numel()
    if val.numel() != nnz:
        raise ValueError("idx and val differ in length")
    _check(_lib.hc_encode_coo(ctypes.byref(p), _ptr(idx, "idx", _u32()),
                              _ptr(val, "val", _vdtypes(p)), nnz,
                              _ptr(y, "y", _vdtypes(p), p.cells),
                              _ptr(b, "b", _u32(), p.index_words), _stream(stream)),
           "hc_encode_coo")


def hc_aggregate(p: hc_params, y_in, b_in, W: int, y_out, b_out, stream=None):
    _check(_lib.hc_aggregate(ctypes.byref(p), _ptr(y_in, "y_in", _vdtypes(p), W * p.cells),
                             _ptr(b_in, "b_in", _u32(), W * p.index_words), W,
                             _ptr(y_out, "y_out", _vdtypes(p), p.cells),
                             _ptr(b_out, "b_out", _u32(), p.index_words), _stream(stream)),
           "hc_aggregate")


def hc_plan_bytes(p: hc_params) -> int:
    b = ctypes.c_size_t()
    _check(_lib.hc_plan_bytes(ctypes.byref(p), ctypes.byref(b)), "hc_plan_bytes")
    return b.value


def hc_plan_build(p: hc_params, plan, stream=None):
    import torch
    _check(_lib.hc_plan_build(ctypes.byref(p), _ptr(plan, "plan", (torch.uint8,)), plan.numel(),
                              _stream(stream)), "hc_plan_build")


def make_plan(p: hc_params, device="cuda", stream=None):
    """Allocate and build the inverse row map of a geometry (c >= 256)."""
    import torch
    plan = torch.empty(hc_plan_bytes(p), dtype=torch.uint8, device=device)
    hc_plan_build(p, plan, stream)
    return plan


def _coo_cap(coo_idx, coo_val) -> int:
    """COO capacity: the decode writes up to coo_idx.numel() entries of both."""
    if (coo_idx is None) != (coo_val is None):
        raise ValueError("coo_idx and coo_val must both be given or both be None")
    if coo_idx is None:
        return 0
    if coo_val.numel() < coo_idx.numel():
        raise ValueError(f"coo_val has {coo_val.numel()} elements, fewer than coo_idx's "
                         f"{coo_idx.numel()} (the decode writes that many of each)")
    return coo_idx.numel()


def hc_decode(p: hc_params, y_agg, b_agg, info, ws, x_out=None, coo_idx=None, coo_val=None,
              mask=None, max_support: int = 0, stream=None, plan=None):
    import torch
    coo_cap = _coo_cap(coo_idx, coo_val)
    _check(_lib.hc_decode(ctypes.byref(p), _ptr(plan, "plan", (torch.uint8,)),
                          _ptr(y_agg, "y_agg", _vdtypes(p), p.cells),
                          _ptr(b_agg, "b_agg", _u32(), p.index_words),
                          _ptr(x_out, "x_out", _vdtypes(p), p.n),
                          _ptr(coo_idx, "coo_idx", _u32()),
                          _ptr(coo_val, "coo_val", _vdtypes(p), coo_cap), coo_cap,
                          _ptr(mask, "mask", _u32(), p.words),
                          _ptr(info, "info", (torch.uint8,), INFO_BYTES),
                          max_support, _ptr(ws, "ws", (torch.uint8,)),
                          ws.numel() if ws is not None else 0, _stream(stream)), "hc_decode")


def hc_decode_noalloc(p: hc_params, y_agg, b_agg, info, x_out=None, coo_idx=None, coo_val=None,
                      mask=None, max_support: int = 0, stream=None, plan=None):
    """hc_decode with the library's static scratch array as its workspace."""
    import torch
    coo_cap = _coo_cap(coo_idx, coo_val)
    _check(_lib.hc_decode_noalloc(ctypes.byref(p), _ptr(plan, "plan", (torch.uint8,)),
                                  _ptr(y_agg, "y_agg", _vdtypes(p), p.cells),
                                  _ptr(b_agg, "b_agg", _u32(), p.index_words),
                                  _ptr(x_out, "x_out", _vdtypes(p), p.n),
                                  _ptr(coo_idx, "coo_idx", _u32()),
                                  _ptr(coo_val, "coo_val", _vdtypes(p), coo_cap), coo_cap,
                                  _ptr(mask, "mask", _u32(), p.words),
                                  _ptr(info, "info", (torch.uint8,), INFO_BYTES),
                                  max_support, _stream(stream)), "hc_decode_noalloc")


@dataclass(frozen=True)
class DecodeInfo:
    n_support: int
    n_recovered: int
    rounds: int
    success: int
    status: int


def read_info(info) -> DecodeInfo:
    """Copy a device hc_decode_info to the host (synchronises its stream)."""
    import numpy as np
    raw = info[:INFO_BYTES].cpu().numpy().tobytes()
    u64 = np.frombuffer(raw[:24], dtype=np.uint64)
    u32 = np.frombuffer(raw[24:32], dtype=np.uint32)
    return DecodeInfo(int(u64[0]), int(u64[1]), int(u64[2]), int(u32[0]), int(u32[1]))


def alloc_info(device="cuda"):
    import torch
    return torch.zeros(64, dtype=torch.uint8, device=device)


def alloc_workspace(p: hc_params, max_support: int = 0, device="cuda"):
    import torch
    _, _, w = hc_sizes(p, max_support)
    return torch.empty(w, dtype=torch.uint8, device=device)
