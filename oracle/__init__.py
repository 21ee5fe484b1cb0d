"""CPU oracle for lossless homomorphic gradient compression.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU library and its Python
binding never do.  It wraps the plain C implementation in ``hco.c`` (built by
``oracle/build.py`` with gcc) with numpy marshalling and nothing else.

Paper passages each entry point follows:
  encode     Algorithm 1 phase I; Count Sketch update (section 3.1), bitmap
             index (section 3.2), batching with a random rotation (section 3.4)
  aggregate  the aggregation API between the phases: sum of sketches, OR of
             bitmaps (section 3, Algorithm 1)
  decode     Algorithm 1 phase II: synchronous peeling (section 3.2) and the
             Count Sketch median estimate for what cannot be peeled (3.1)
  rows_for   sketch size at least gamma * n with gamma = 1.23 (section 3.2)
  bloom_geometry  Bloom-filter index sizing: false positive rate
             eps = (ln^2 2 gamma C lambda)^-1, log(1/eps) hashes, (n / ln 2)
             log(1/eps) bits, sketch for the support plus the false positives
             (section 3.3); bloom_bits: a parameter's filter bits
  decode_bound  how far floating-point rounding of the sketch can move each
             decoded value (the imprecision section 4.1 concedes), carried
             through the decode's schedule; used to set fp32 tolerances
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# HCO_LIB selects another build of hco.c (the sanitizer build in the tests)
_LIB_PATH = os.environ.get("HCO_LIB") or os.path.join(_HERE, "libhco.so")
_lib = None

GAMMA = 1.23  # section 3.2


class _Geom(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("k", ctypes.c_uint32), ("c", ctypes.c_uint32),
                ("rows", ctypes.c_uint64), ("seed", ctypes.c_uint64),
                ("block", ctypes.c_uint32), ("bloom_k", ctypes.c_uint32),
                ("bloom_rows", ctypes.c_uint64)]


class _Info(ctypes.Structure):
    _fields_ = [("n_support", ctypes.c_uint64), ("n_recovered", ctypes.c_uint64),
                ("rounds", ctypes.c_uint64), ("success", ctypes.c_uint32),
                ("pad", ctypes.c_uint32)]


@dataclass(frozen=True)
class Geom:
    n: int
    rows: int
    seed: int
    c: int = 1024
    k: int = 3
    block: int = 0  # batches per parameter block of a blocked sketch; 0 = one sketch
    bloom_k: int = 0     # Bloom filter hashes (section 3.3); 0 = bitmap index
    bloom_rows: int = 0  # rows of c bits in the Bloom filter

    @property
    def cells(self) -> int:
        return self.rows * self.c

    @property
    def nblocks(self) -> int:
        if self.block == 0:
            return 1
        return ((self.n + self.c - 1) // self.c + self.block - 1) // self.block

    @property
    def block_rows(self) -> int:
        return self.rows // self.nblocks

    @property
    def words(self) -> int:
        """Words of an n-bit bitmap (the bitmap index, the recovered mask)."""
        return (self.n + 31) // 32

    @property
    def index_words(self) -> int:
        """Words of the index B: the bitmap, or the Bloom filter."""
        if self.bloom_k == 0:
            return self.words
        return (self.bloom_rows * self.c + 31) // 32

    def _c(self) -> _Geom:
        return _Geom(self.n, self.k, self.c, self.rows, self.seed & (2**64 - 1), self.block,
                     self.bloom_k, self.bloom_rows)


@dataclass(frozen=True)
class Info:
    n_support: int
    n_recovered: int
    rounds: int
    success: int


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build
            _build.build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        G = ctypes.POINTER(_Geom)
        L.hco_check_geom.argtypes = [G]
        L.hco_check_geom.restype = ctypes.c_int
        L.hco_rows_for.argtypes = [ctypes.c_uint64, ctypes.c_double, ctypes.c_uint32]
        L.hco_rows_for.restype = ctypes.c_uint64
        L.hco_blocked_geometry.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                           ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                           ctypes.POINTER(ctypes.c_uint32),
                                           ctypes.POINTER(ctypes.c_uint64)]
        L.hco_blocked_geometry.restype = ctypes.c_int
        L.hco_bloom_geometry.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                         ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.POINTER(ctypes.c_uint32),
                                         ctypes.POINTER(ctypes.c_uint64),
                                         ctypes.POINTER(ctypes.c_uint64),
                                         ctypes.POINTER(ctypes.c_double)]
        L.hco_bloom_geometry.restype = ctypes.c_int
        L.hco_index_words.argtypes = [G]
        L.hco_index_words.restype = ctypes.c_uint64
        L.hco_bloom_bits.argtypes = [G, ctypes.c_uint64, P]
        L.hco_bloom_bits.restype = None
        L.hco_bloom_query.argtypes = [G, P, P, ctypes.c_uint64, P]
        L.hco_bloom_query.restype = None
        L.hco_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64, P]
        L.hco_splitmix64.restype = None
        L.hco_batch_hash.argtypes = [G, ctypes.c_uint64, P, P, P]
        L.hco_batch_hash.restype = None
        L.hco_cells.argtypes = [G, P, ctypes.c_uint64, P, P]
        L.hco_cells.restype = None
        for name in ("hco_encode_i32", "hco_encode_f64"):
            getattr(L, name).argtypes = [G, P, P, P]
            getattr(L, name).restype = ctypes.c_int
        for name in ("hco_encode_coo_i32", "hco_encode_coo_f64"):
            getattr(L, name).argtypes = [G, P, P, ctypes.c_uint64, P, P]
            getattr(L, name).restype = ctypes.c_int
        for name in ("hco_aggregate_i32", "hco_aggregate_f64"):
            getattr(L, name).argtypes = [ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                         P, P, P, P]
            getattr(L, name).restype = None
        for name in ("hco_decode_i32", "hco_decode_f64"):
            getattr(L, name).argtypes = [G, P, P, P, P, ctypes.POINTER(_Info), P]
            getattr(L, name).restype = ctypes.c_int
        L.hco_decode_bound_f64.argtypes = [G, P, P, P]
        L.hco_decode_bound_f64.restype = ctypes.c_int
        L.hco_decode_queue_i32.argtypes = [G, P, P, P, P, ctypes.POINTER(_Info)]
        L.hco_decode_queue_i32.restype = ctypes.c_int
        L.hco_query_i32.argtypes = [G, P, ctypes.c_uint64]
        L.hco_query_i32.restype = ctypes.c_int32
        L.hco_query_f64.argtypes = [G, P, ctypes.c_uint64]
        L.hco_query_f64.restype = ctypes.c_double
        L.hco_median3_i32.argtypes = [ctypes.c_int32] * 3
        L.hco_median3_i32.restype = ctypes.c_int32
        L.hco_median3_f64.argtypes = [ctypes.c_double] * 3
        L.hco_median3_f64.restype = ctypes.c_double
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _is_int(dtype) -> bool:
    return np.dtype(dtype) == np.int32


def rows_for(n_nonzero: int, gamma: float = GAMMA, c: int = 1024) -> int:
    return int(lib().hco_rows_for(n_nonzero, gamma, c))


def geometry(n: int, n_nonzero: int, seed: int, c: int = 1024, gamma: float = GAMMA) -> Geom:
    return Geom(n=n, rows=rows_for(n_nonzero, gamma, c), seed=seed, c=c)


def blocked_geometry(n: int, n_nonzero: int, seed: int, c: int = 1024, gamma: float = GAMMA,
                     block_rows: int = 16, max_block: int = 1024) -> Geom:
    """Blocked sketch sized for an expected n_nonzero (hco_blocked_geometry)."""
    blk = ctypes.c_uint32()
    rows = ctypes.c_uint64()
    if lib().hco_blocked_geometry(n, n_nonzero, gamma, c, block_rows, max_block,
                                  ctypes.byref(blk), ctypes.byref(rows)):
        raise ValueError("invalid blocked geometry arguments")
    return Geom(n=n, rows=int(rows.value), seed=seed, c=c, block=int(blk.value))


def bloom_geometry(n: int, n_nonzero: int, seed: int, c: int = 1024, gamma: float = GAMMA,
                   bits: int = 32):
    """(Geom with a Bloom-filter index sized by section 3.3, the paper's eps)."""
    k = ctypes.c_uint32()
    brows = ctypes.c_uint64()
    rows = ctypes.c_uint64()
    eps = ctypes.c_double()
    if lib().hco_bloom_geometry(n, n_nonzero, gamma, c, bits, ctypes.byref(k), ctypes.byref(brows),
                                ctypes.byref(rows), ctypes.byref(eps)):
        raise ValueError("invalid Bloom geometry arguments (or too dense for a filter)")
    return Geom(n=n, rows=int(rows.value), seed=seed, c=c, bloom_k=int(k.value),
                bloom_rows=int(brows.value)), float(eps.value)


def bloom_bits(g: Geom, p: int) -> np.ndarray:
    out = np.zeros(max(g.bloom_k, 1), np.uint64)
    lib().hco_bloom_bits(ctypes.byref(g._c()), p, _ptr(out))
    return out[:g.bloom_k]


def bloom_query(g: Geom, B: np.ndarray, idx) -> np.ndarray:
    """Section 3.3 query: True where all of a parameter's filter bits are set."""
    idx = np.ascontiguousarray(idx, np.uint64)
    B = np.ascontiguousarray(B, np.uint32)
    out = np.zeros(idx.size, np.uint8)
    lib().hco_bloom_query(ctypes.byref(g._c()), _ptr(B), _ptr(idx), idx.size, _ptr(out))
    return out.astype(bool)


def check(g: Geom) -> bool:
    return lib().hco_check_geom(ctypes.byref(g._c())) == 0


def splitmix64(seed: int, count: int) -> np.ndarray:
    out = np.zeros(count, np.uint64)
    lib().hco_splitmix64(seed & (2**64 - 1), count, _ptr(out))
    return out


def batch_hash(g: Geom, b: int):
    row = np.zeros(3, np.uint64)
    bias = np.zeros(3, np.uint32)
    sign = np.zeros(3, np.int32)
    lib().hco_batch_hash(ctypes.byref(g._c()), b, _ptr(row), _ptr(bias), _ptr(sign))
    return row, bias, sign


def cells(g: Geom, idx) -> tuple[np.ndarray, np.ndarray]:
    """(cells[m,3], signs[m,3]) of the parameters idx."""
    idx = np.ascontiguousarray(idx, np.uint64)
    m = idx.size
    cl = np.zeros((m, 3), np.uint64)
    sg = np.zeros((m, 3), np.int32)
    lib().hco_cells(ctypes.byref(g._c()), _ptr(idx), m, _ptr(cl), _ptr(sg))
    return cl, sg


def encode(g: Geom, x: np.ndarray):
    """Dense encode.  int32 input -> int32 sketch; float input -> fp64 sketch."""
    B = np.zeros(g.index_words, np.uint32)
    if _is_int(x.dtype):
        x = np.ascontiguousarray(x, np.int32)
        Y = np.zeros(g.cells, np.int32)
        rc = lib().hco_encode_i32(ctypes.byref(g._c()), _ptr(x), _ptr(Y), _ptr(B))
    else:
        x = np.ascontiguousarray(x, np.float64)
        Y = np.zeros(g.cells, np.float64)
        rc = lib().hco_encode_f64(ctypes.byref(g._c()), _ptr(x), _ptr(Y), _ptr(B))
    if rc != 0:
        raise ValueError("oracle encode: invalid geometry")
    assert x.size == g.n
    return Y, B


def encode_coo(g: Geom, idx: np.ndarray, val: np.ndarray):
    idx = np.ascontiguousarray(idx, np.uint32)
    B = np.zeros(g.index_words, np.uint32)
    if _is_int(val.dtype):
        val = np.ascontiguousarray(val, np.int32)
        Y = np.zeros(g.cells, np.int32)
        rc = lib().hco_encode_coo_i32(ctypes.byref(g._c()), _ptr(idx), _ptr(val), idx.size,
                                      _ptr(Y), _ptr(B))
    else:
        val = np.ascontiguousarray(val, np.float64)
        Y = np.zeros(g.cells, np.float64)
        rc = lib().hco_encode_coo_f64(ctypes.byref(g._c()), _ptr(idx), _ptr(val), idx.size,
                                      _ptr(Y), _ptr(B))
    if rc != 0:
        raise ValueError("oracle encode_coo: invalid geometry or index out of range")
    return Y, B


def aggregate(Ys: np.ndarray, Bs: np.ndarray):
    """Ys[W, cells], Bs[W, words] -> (sum of Ys, OR of Bs)."""
    Ys = np.ascontiguousarray(Ys)
    Bs = np.ascontiguousarray(Bs, np.uint32)
    W, C = Ys.shape
    words = Bs.shape[1]
    Bout = np.zeros(words, np.uint32)
    if _is_int(Ys.dtype):
        Yout = np.zeros(C, np.int32)
        lib().hco_aggregate_i32(W, C, words, _ptr(Ys), _ptr(Bs), _ptr(Yout), _ptr(Bout))
    else:
        Ys = np.ascontiguousarray(Ys, np.float64)
        Yout = np.zeros(C, np.float64)
        lib().hco_aggregate_f64(W, C, words, _ptr(Ys), _ptr(Bs), _ptr(Yout), _ptr(Bout))
    return Yout, Bout


def decode(g: Geom, Y: np.ndarray, B: np.ndarray, want_rounds: bool = False):
    """Synchronous-round peeling decode -> (x[n], mask[words], Info[, round_of[n]])."""
    B = np.ascontiguousarray(B, np.uint32)
    mask = np.zeros(g.words, np.uint32)
    info = _Info()
    rof = np.zeros(g.n, np.uint32) if want_rounds else None
    rptr = _ptr(rof) if want_rounds else None
    if _is_int(Y.dtype):
        Y = np.ascontiguousarray(Y, np.int32)
        x = np.zeros(g.n, np.int32)
        rc = lib().hco_decode_i32(ctypes.byref(g._c()), _ptr(Y), _ptr(B), _ptr(x), _ptr(mask),
                                  ctypes.byref(info), rptr)
    else:
        Y = np.ascontiguousarray(Y, np.float64)
        x = np.zeros(g.n, np.float64)
        rc = lib().hco_decode_f64(ctypes.byref(g._c()), _ptr(Y), _ptr(B), _ptr(x), _ptr(mask),
                                  ctypes.byref(info), rptr)
    if rc != 0:
        raise ValueError("oracle decode: invalid geometry or out of memory")
    inf = Info(info.n_support, info.n_recovered, info.rounds, info.success)
    return (x, mask, inf, rof) if want_rounds else (x, mask, inf)


def decode_bound(g: Geom, dY: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Per-parameter bound on the decoded value's error given per-cell bounds
    dY on the sketch's error, carried through the decode's own schedule."""
    dY = np.ascontiguousarray(dY, np.float64)
    B = np.ascontiguousarray(B, np.uint32)
    out = np.zeros(g.n, np.float64)
    if lib().hco_decode_bound_f64(ctypes.byref(g._c()), _ptr(dY), _ptr(B), _ptr(out)) != 0:
        raise ValueError("oracle decode_bound: invalid geometry or out of memory")
    return out


def decode_queue(g: Geom, Y: np.ndarray, B: np.ndarray):
    B = np.ascontiguousarray(B, np.uint32)
    Y = np.ascontiguousarray(Y, np.int32)
    mask = np.zeros(g.words, np.uint32)
    x = np.zeros(g.n, np.int32)
    info = _Info()
    rc = lib().hco_decode_queue_i32(ctypes.byref(g._c()), _ptr(Y), _ptr(B), _ptr(x), _ptr(mask),
                                    ctypes.byref(info))
    if rc != 0:
        raise ValueError("oracle decode_queue: invalid geometry or out of memory")
    return x, mask, Info(info.n_support, info.n_recovered, info.rounds, info.success)


def query(g: Geom, Y: np.ndarray, p: int):
    if _is_int(Y.dtype):
        Y = np.ascontiguousarray(Y, np.int32)
        return int(lib().hco_query_i32(ctypes.byref(g._c()), _ptr(Y), p))
    Y = np.ascontiguousarray(Y, np.float64)
    return float(lib().hco_query_f64(ctypes.byref(g._c()), _ptr(Y), p))


def median3(a, b, c):
    if all(isinstance(v, (int, np.integer)) for v in (a, b, c)):
        return int(lib().hco_median3_i32(a, b, c))
    return float(lib().hco_median3_f64(a, b, c))
