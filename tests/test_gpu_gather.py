"""hc_encode_gather: the dense encode assembled row by row through a plan.

Its sketches and bitmaps must equal the oracle's (int32 bit for bit; fp32
within the order-independent bound of a sum of m terms), exactly as
hc_encode's do, on sparse and dense gradients, ragged lengths and every
plan-capable batch width.  A plan built for another geometry must give a
zero sketch and an all-ones bitmap, which the decode reports as a failure."""
import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run, wrap_sum
from test_gpu_parity import U, _hc, check_fp32, check_int, gamma

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("c", [1024, 512, 256])
def test_gather_ragged_sparse_int32(c):
    # several rows and tiles, n not a multiple of c or of the 16-byte vector
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.01, overlap=0.4, data_seed=c + 3)
    g, o = check_int(w, oracle.rows_for(w.n_agg, 1.23, c), c, gather=True, use_plan=True)
    assert g["info"].success
    assert np.array_equal(g["x"], wrap_sum([w.dense(i) for i in range(w.W)]))


@pytest.mark.parametrize("c", [1024, 256])
def test_gather_dense_int32(c):
    # most parameters nonzero (section 4.1's setting), one worker
    _hc()
    # (at this small size, gamma = 1.23 sits too close to the threshold for
    # c = 256 batches of a dense gradient: the oracle fails there too)
    w = wl.make("synthetic", n=300_017, W=1, density=0.696, overlap=0.0, data_seed=c)
    g, o = check_int(w, oracle.rows_for(w.n_agg, 1.3, c), c, gather=True)
    assert g["info"].success


def test_gather_undersized_int32():
    # the encode does not depend on the decode succeeding
    _hc()
    w = wl.make("synthetic", n=200_000, W=2, density=0.5, overlap=0.0, data_seed=9)
    g, o = check_int(w, 3 * (int(0.5 * w.n_agg / 3072) + 1), 1024, gather=True)
    assert not g["info"].success


@pytest.mark.parametrize("n", [1, 31, 255, 1025, 4097])
def test_gather_tiny_lengths(n):
    _hc()
    w = wl.make("synthetic", n=n, W=2, density=0.4, overlap=0.0, data_seed=n)
    check_int(w, 3, 1024 if n > 1000 else 256, gather=True)


def test_gather_fp32():
    _hc()
    w = wl.make("synthetic", n=700_001, W=3, density=0.25, overlap=0.2, vtype="f32", data_seed=21)
    g, o, bnd = check_fp32(w, oracle.rows_for(w.n_agg, 1.23, 1024), 1024, gather=True)
    assert g["info"].success


def test_gather_matches_atomic_encode_bitwise():
    # int32 sums wrap the same in any order: the two encodes agree bit for bit
    import torch
    hc = _hc()
    w = wl.make("synthetic", n=2_000_000, W=1, density=0.2, overlap=0.0, data_seed=4)
    p = hc.hc_geometry(w.n, w.n_agg, 1.23, 1024, w.hash_seed, "i32")
    dev = torch.device("cuda")
    x = torch.from_numpy(w.dense(0)).to(dev)
    plan = hc.make_plan(p, dev)
    Y1 = torch.empty(p.cells, dtype=torch.int32, device=dev)
    B1 = torch.empty(p.words, dtype=torch.int32, device=dev)
    Y2 = torch.full((p.cells,), 7, dtype=torch.int32, device=dev)
    B2 = torch.full((p.words,), 7, dtype=torch.int32, device=dev)
    hc.hc_encode(p, x, Y1, B1)
    hc.hc_encode_gather(p, plan, x, Y2, B2)   # overwrites whatever was there
    assert torch.equal(Y1, Y2) and torch.equal(B1, B2)
    # an unaligned view of the gradient takes the scalar loads
    xs = torch.zeros(w.n + 1, dtype=torch.int32, device=dev)
    xs[1:] = x
    Y3 = torch.empty_like(Y1)
    B3 = torch.empty_like(B1)
    hc.hc_encode_gather(p, plan, xs[1:], Y3, B3)
    assert torch.equal(Y1, Y3) and torch.equal(B1, B3)


def test_gather_plan_for_other_geometry_poisons():
    import torch
    hc = _hc()
    w = wl.make("synthetic", n=500_000, W=1, density=0.05, overlap=0.0, data_seed=8)
    p = hc.hc_geometry(w.n, w.n_agg, 1.23, 1024, w.hash_seed, "i32")
    other = hc.hc_geometry(w.n, w.n_agg, 1.23, 1024, w.hash_seed + 1, "i32")
    dev = torch.device("cuda")
    bad_plan = hc.make_plan(other, dev)
    x = torch.from_numpy(w.dense(0)).to(dev)
    Y = torch.full((p.cells,), 5, dtype=torch.int32, device=dev)
    B = torch.zeros(p.words, dtype=torch.int32, device=dev)
    hc.hc_encode_gather(p, bad_plan, x, Y, B)
    torch.cuda.synchronize()
    assert not Y.any().item()
    assert bool((B == -1).all().item())
    out = torch.empty(w.n, dtype=torch.int32, device=dev)
    info = hc.alloc_info(dev)
    ws = hc.alloc_workspace(p, 0, dev)
    hc.hc_decode(p, Y, B, info, ws, x_out=out)
    torch.cuda.synchronize()
    assert hc.read_info(info).success == 0
