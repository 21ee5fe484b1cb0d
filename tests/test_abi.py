"""The C-ABI library loads on the host and exports every entry point that
include/hc.h declares; host-side validation (no GPU work) behaves as the
header documents."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_entry_points():
    with open(os.path.join(ROOT, "include", "hc.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hc_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    import paper_2402_07529_amd as hc
    names = declared_entry_points()
    assert set(names) == set(hc.EXPORTS)
    lib = ctypes.CDLL(hc.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_geometry_and_sizes_host_only():
    import oracle
    import paper_2402_07529_amd as hc
    for n, nnz, c in ((65536, 1636, 1024), (109_482_240, 9_305_915, 1024), (1000, 10, 1),
                      (2**32 - 1, 10**6, 64)):
        p = hc.hc_geometry(n, nnz, 1.23, c, 7, "i32")
        assert p.rows == oracle.rows_for(nnz, 1.23, c)
        y, b, ws = hc.hc_sizes(p)
        assert y == p.rows * c * 4 and b == (n + 31) // 32 * 4
        assert ws > 8 * p.cells
        _, _, ws_small = hc.hc_sizes(p, max_support=1000)
        assert ws_small < ws or n <= 1000


@pytest.mark.parametrize("kw", [dict(c=3), dict(c=2048), dict(n=0), dict(n=2**32)])
def test_geometry_rejects_invalid(kw):
    import paper_2402_07529_amd as hc
    args = dict(n=1000, nnz=100, c=1024)
    args.update(kw)
    with pytest.raises(hc.HCError) as ei:
        hc.hc_geometry(args["n"], args["nnz"], 1.23, args["c"], 1)
    assert ei.value.status == hc.HC_EINVAL


def test_sizes_reject_bad_params():
    import paper_2402_07529_amd as hc
    for p, st in ((hc.make_params(1000, 2, 1), hc.HC_EINVAL),
                  (hc.hc_params(1000, 2, 1024, 5, 1, 0, 0), hc.HC_EUNSUPPORTED),
                  (hc.hc_params(1000, 3, 1024, 5, 1, 7, 0), hc.HC_EINVAL),
                  (hc.hc_params(1000, 3, 1024, 2**23, 1, 0, 0), hc.HC_EINVAL)):
        with pytest.raises(hc.HCError) as ei:
            hc.hc_sizes(p)
        assert ei.value.status == st
        assert hc.lib().hc_last_error()


def test_null_and_misaligned_pointers_rejected_before_launch():
    import paper_2402_07529_amd as hc
    L = hc.lib()
    p = hc.make_params(1000, 3, 1)
    assert L.hc_encode(ctypes.byref(p), None, None, None, None) == hc.HC_EINVAL
    assert L.hc_aggregate(ctypes.byref(p), ctypes.c_void_p(16), ctypes.c_void_p(16), 0,
                          ctypes.c_void_p(16), ctypes.c_void_p(16), None) == hc.HC_EINVAL
    assert L.hc_encode(ctypes.byref(p), ctypes.c_void_p(18), ctypes.c_void_p(32),
                       ctypes.c_void_p(48), None) == hc.HC_EINVAL
    assert b"aligned" in L.hc_last_error()
    V = ctypes.c_void_p
    assert L.hc_decode(ctypes.byref(p), None, V(16), V(16), None, None, None, 0, None, V(16), 0,
                       V(64), 10**9, None) == hc.HC_EINVAL
    assert b"aligned" in L.hc_last_error()
    assert L.hc_decode(ctypes.byref(p), None, V(16), V(16), None, None, None, 0, None, V(16), 0,
                       V(256), 10, None) == hc.HC_EWORKSPACE
    # a plan is rejected for c < 256
    p1 = hc.make_params(1000, 3, 1, c=1)
    assert L.hc_decode(ctypes.byref(p1), V(256), V(16), V(16), None, None, None, 0, None, V(16), 0,
                       V(256), 10**9, None) == hc.HC_EINVAL


def test_plan_sizes():
    import paper_2402_07529_amd as hc
    p = hc.hc_geometry(109_482_240, 9_305_915, 1.23, 1024, 3)
    nb = (109_482_240 + 1023) // 1024
    bytes_ = hc.hc_plan_bytes(p)
    assert bytes_ >= 3 * nb * 8 + (p.rows + 1) * 4
    with pytest.raises(hc.HCError) as ei:
        hc.hc_plan_bytes(hc.hc_geometry(100000, 1000, 1.23, 64, 3))
    assert ei.value.status == hc.HC_EUNSUPPORTED
    L = hc.lib()
    assert L.hc_plan_build(ctypes.byref(p), ctypes.c_void_p(256), 10, None) == hc.HC_EWORKSPACE
    assert L.hc_plan_build(ctypes.byref(p), ctypes.c_void_p(100), 10**9, None) == hc.HC_EINVAL


def test_blocked_geometry_matches_oracle():
    import oracle
    import paper_2402_07529_amd as hc
    for n, nnz, gamma, c, br in ((109_482_240, 9_305_915, 1.3, 1024, 14),
                                 (109_482_240, 273_579, 1.3, 1024, 14),
                                 (143_667_240, 8_476_348, 1.3, 1024, 12),
                                 (10_000, 500, 1.3, 8, 4), (65_536, 1636, 1.6, 64, 16),
                                 (1_000_000, 999_999, 1.25, 256, 12)):
        p = hc.hc_geometry_blocked(n, nnz, gamma, c, br, 5, "i32")
        g = oracle.blocked_geometry(n, nnz, 5, c, gamma, br)
        assert (int(p.block), int(p.rows)) == (g.block, g.rows)
        assert p.nblocks == g.nblocks and p.block_rows == g.block_rows
        _, _, ws = hc.hc_sizes(p)
        assert ws < 4096 + (n // 32 // 1024 + 1) * 4 + 512  # control blocks and chunk offsets only


def test_blocked_params_rejected():
    import paper_2402_07529_amd as hc
    L = hc.lib()
    V = ctypes.c_void_p
    bad = ((hc.make_params(10_000, 84, 1, c=8, block=61), hc.HC_EINVAL),    # 61 * 8 % 32
           (hc.make_params(10_000, 85, 1, c=8, block=60), hc.HC_EINVAL),    # 85 % 21 blocks
           (hc.make_params(10_000, 42, 1, c=8, block=60), hc.HC_EINVAL))    # 2 rows per block
    for p, st in bad:
        with pytest.raises(hc.HCError) as ei:
            hc.hc_sizes(p)
        assert ei.value.status == st
    # valid format, beyond the LDS kernels: 30 rows of 1024 cells per block
    with pytest.raises(hc.HCError) as ei:
        hc.hc_geometry_blocked(109_482_240, 9_305_915, 1.3, 1024, 18, 3)
    assert ei.value.status == hc.HC_EUNSUPPORTED
    p = hc.make_params(2_000_000, 30 * 62, 1, c=1024, block=32)
    hc.hc_sizes(p)
    assert L.hc_encode(ctypes.byref(p), V(256), V(256), V(256), None) == hc.HC_EUNSUPPORTED
    assert L.hc_decode(ctypes.byref(p), None, V(256), V(256), None, None, None, 0, None, V(256), 0,
                       V(256), 10**9, None) == hc.HC_EUNSUPPORTED
    assert b"LDS" in L.hc_last_error()
    # more than 1024 batches per block
    p = hc.make_params(2 * 1050 * 1024, 3 * 2, 1, c=1024, block=1050)
    assert L.hc_encode(ctypes.byref(p), V(256), V(256), V(256), None) == hc.HC_EUNSUPPORTED
    # a blocked sketch takes no plan
    p = hc.hc_geometry_blocked(109_482_240, 9_305_915, 1.3, 1024, 14, 3)
    with pytest.raises(hc.HCError) as ei:
        hc.hc_plan_bytes(p)
    assert ei.value.status == hc.HC_EUNSUPPORTED
    assert L.hc_decode(ctypes.byref(p), V(256), V(256), V(256), None, None, None, 0, None, V(256), 0,
                       V(256), 10**9, None) == hc.HC_EINVAL
    # workspace too small
    assert L.hc_decode(ctypes.byref(p), None, V(256), V(256), None, None, None, 0, None, V(256), 0,
                       V(256), 64, None) == hc.HC_EWORKSPACE



def test_bloom_geometry_matches_oracle():
    # section 3.3 sizing, computed by the library and by the oracle separately
    import oracle
    import paper_2402_07529_amd as hc
    for n, nnz, c in ((1 << 30, 1_551_680, 1024), (109_482_240, 9_305_915, 1024),
                      (109_482_240, 273_579, 256), (2_000_000, 8_000, 64), (50_000, 900, 1),
                      (1000, 900, 8)):
        p, eps = hc.hc_geometry_bloom(n, nnz, 1.23, c, 11, "i32")
        g, eps_o = oracle.bloom_geometry(n, nnz, 11, c)
        assert (int(p.bloom_k), int(p.bloom_rows), int(p.rows)) == (g.bloom_k, g.bloom_rows, g.rows)
        assert eps == pytest.approx(eps_o, rel=1e-12)
        _, b_bytes, _ = hc.hc_sizes(p)
        assert b_bytes == 4 * g.index_words == 4 * p.index_words
    with pytest.raises(hc.HCError) as ei:
        hc.hc_geometry_bloom(1000, 950, 1.23, 1024, 1)   # log2(1/eps) rounds to 0
    assert ei.value.status == hc.HC_EINVAL


def test_bloom_params_rejected():
    import paper_2402_07529_amd as hc
    bad = ((hc.make_params(10_000, 9, 1, c=64, bloom_k=65, bloom_rows=10), hc.HC_EINVAL),
           (hc.make_params(10_000, 9, 1, c=64, bloom_k=3, bloom_rows=0), hc.HC_EINVAL),
           (hc.make_params(10_000, 9, 1, c=1024, bloom_k=3, bloom_rows=1 << 22), hc.HC_EINVAL),
           (hc.make_params(10_000, 60, 1, c=64, block=8, bloom_k=3, bloom_rows=10),
            hc.HC_EUNSUPPORTED))
    for p, st in bad:
        with pytest.raises(hc.HCError) as ei:
            hc.hc_sizes(p)
        assert ei.value.status == st
    p = hc.make_params(10_000, 9, 1, c=64, bloom_k=3, bloom_rows=10)
    p.reserved = 1
    with pytest.raises(hc.HCError) as ei:
        hc.hc_sizes(p)
    assert ei.value.status == hc.HC_EINVAL
    # the decode workspace holds the probed candidate bitmap on top
    q = hc.make_params(10_000, 9, 1, c=64, bloom_k=3, bloom_rows=10)
    _, _, ws_bloom = hc.hc_sizes(q, 100)
    _, _, ws_bitmap = hc.hc_sizes(hc.make_params(10_000, 9, 1, c=64), 100)
    assert ws_bloom - ws_bitmap >= 4 * q.words


def test_gather_encode_rejected_before_launch():
    # hc_encode_gather: unblocked sketch, bitmap index, c >= 256, a 256-byte
    # aligned plan of at least hc_plan_bytes
    import paper_2402_07529_amd as hc
    L = hc.lib()
    V = ctypes.c_void_p
    p = hc.hc_geometry(2_000_000, 20_000, 1.23, 1024, 3)
    need = hc.hc_plan_bytes(p)
    ok = (V(256), need, V(256), V(256), V(256), None)
    assert L.hc_encode_gather(ctypes.byref(p), V(100), *ok[1:]) == hc.HC_EINVAL
    assert L.hc_encode_gather(ctypes.byref(p), None, *ok[1:]) == hc.HC_EINVAL
    assert L.hc_encode_gather(ctypes.byref(p), V(256), need - 1, *ok[2:]) == hc.HC_EWORKSPACE
    assert L.hc_encode_gather(ctypes.byref(p), *ok[:2], None, V(256), V(256), None) == hc.HC_EINVAL
    assert L.hc_encode_gather(ctypes.byref(p), *ok[:2], V(18), V(256), V(256), None) == hc.HC_EINVAL
    for q in (hc.hc_geometry(2_000_000, 20_000, 1.23, 64, 3),                  # c < 256
              hc.hc_geometry_blocked(109_482_240, 9_305_915, 1.3, 1024, 14, 3),  # blocked
              hc.hc_geometry_bloom(2_000_000, 20_000, 1.23, 1024, 3)[0]):        # Bloom index
        assert L.hc_encode_gather(ctypes.byref(q), *ok) == hc.HC_EUNSUPPORTED
        assert L.hc_last_error()


def test_decode_binding_checks_coo_lengths_before_launch():
    # the decode writes coo_cap = coo_idx.numel() entries of both COO arrays:
    # a shorter coo_val, or only one of the two, is refused on the host
    import torch

    import paper_2402_07529_amd as hc
    p = hc.hc_geometry(10_000, 100, 1.23, 1024, 3)
    assert hc._coo_cap(None, None) == 0
    assert hc._coo_cap(torch.zeros(8, dtype=torch.int32), torch.zeros(8, dtype=torch.int32)) == 8
    with pytest.raises(ValueError, match="fewer than"):
        hc.hc_decode(p, None, None, None, None, coo_idx=torch.zeros(8, dtype=torch.int32),
                     coo_val=torch.zeros(7, dtype=torch.int32))
    with pytest.raises(ValueError, match="both"):
        hc.hc_decode(p, None, None, None, None, coo_idx=torch.zeros(8, dtype=torch.int32))


def test_staged_encode_rejected_before_launch():
    # hc_encode_staged: unblocked sketch, c >= 256, a 256-byte aligned plan of
    # at least hc_plan_bytes and a 256-byte aligned workspace of at least
    # hc_encode_staged_bytes
    import paper_2402_07529_amd as hc
    L = hc.lib()
    V = ctypes.c_void_p
    p = hc.hc_geometry(2_000_000, 20_000, 1.23, 1024, 3)
    need = hc.hc_plan_bytes(p)
    wsb = hc.hc_encode_staged_bytes(p)
    assert wsb >= ((2_000_000 + 1023) // 1024) * (64 * 8 + 4)
    ok = [V(256), need, V(512), wsb, V(256), V(256), V(256), None]
    bad = [(0, V(100), hc.HC_EINVAL), (0, None, hc.HC_EINVAL), (1, need - 1, hc.HC_EWORKSPACE),
           (2, V(520), hc.HC_EINVAL), (2, None, hc.HC_EINVAL), (3, wsb - 1, hc.HC_EWORKSPACE),
           (4, None, hc.HC_EINVAL), (5, V(18), hc.HC_EINVAL)]
    for k, v, st in bad:
        args = list(ok)
        args[k] = v
        assert L.hc_encode_staged(ctypes.byref(p), *args) == st, (k, v)
    for q in (hc.hc_geometry(2_000_000, 20_000, 1.23, 64, 3),                  # c < 256
              hc.hc_geometry_blocked(109_482_240, 9_305_915, 1.3, 1024, 14, 3)):  # blocked
        assert L.hc_encode_staged(ctypes.byref(q), *ok) == hc.HC_EUNSUPPORTED
        with pytest.raises(hc.HCError):
            hc.hc_encode_staged_bytes(q)
