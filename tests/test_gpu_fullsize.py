"""Parity at the full sizes of the named workloads, in the launch
configuration bench.py times: dense hc_encode per worker, hc_aggregate over
the W sketches, hc_decode with the geometry's plan and max_support = the
aggregate's nonzeros.

int32: every stage bit-exact against the CPU oracle (per-worker sketches and
bitmaps, aggregate, decoded gradient, mask, support size, recovered count,
round count, success), and the decoded gradient equals the direct sum of the
workers' sparse gradients.  fp32 (VGG19): structure exact, values within the
per-element bound derived in test_gpu_parity, and the decode stage within 1e-6
relative of the oracle's decode of the GPU's own fp32 aggregate.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run
from test_gpu_parity import (assert_fp32_decode_stage, assert_fp32_values, assert_same_info,
                             fp32_cell_bounds, fp32_normwise_error)

pytestmark = pytest.mark.gpu


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def sparse_direct_sum(w):
    """(indices, int32 wrapped sums) of the workers' COO gradients."""
    idx = np.concatenate(w.idx).astype(np.int64)
    val = np.concatenate(w.val).astype(np.int64)
    order = np.argsort(idx, kind="stable")
    idx, val = idx[order], val[order]
    uniq, start = np.unique(idx, return_index=True)
    sums = np.add.reduceat(val, start)
    return uniq, ((sums + 2**31) % 2**32 - 2**31).astype(np.int32)


@pytest.mark.timeout(900)
def test_fullsize_vgg19_int32_without_plan():
    # no plan: the support kernel builds the counters with atomics and the
    # peel keeps separate residuals; at this sketch size (10.4 M cells) the
    # scan and round 0 run as whole-chip launches before the persistent peel
    _hc()
    w = wl.make("vgg19")
    n_agg = w.n_agg
    rows = oracle.rows_for(n_agg)
    print(f"[fullsize] vgg19 without plan: n={w.n} W={w.W} n_agg={n_agg} rows={rows}", flush=True)
    g = gpu_run(w, rows, 1024, want_coo_out=False, max_support=n_agg, use_plan=False,
                keep_workers=False)
    o = oracle_run(w, rows, 1024)
    assert np.array_equal(g["Ya"], o["Ya"])
    assert_same_info(g["info"], o["info"])
    assert np.array_equal(g["mask"], o["mask"])
    assert np.array_equal(g["x"], o["x"])
    assert g["info"].success


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["tiny", "ncf", "lstm", "vgg19", "bert"])
def test_fullsize_int32(name):
    _hc()
    w = wl.make(name)
    n_agg = w.n_agg
    rows = oracle.rows_for(n_agg)
    print(f"[fullsize] {name}: n={w.n} W={w.W} n_agg={n_agg} rows={rows}", flush=True)
    g = gpu_run(w, rows, 1024, want_coo_out=False, max_support=n_agg, use_plan=True)
    o = oracle_run(w, rows, 1024)
    for i in range(w.W):
        assert np.array_equal(g["Y"][i], o["Y"][i]), f"worker {i} sketch"
        assert np.array_equal(g["B"][i], o["B"][i]), f"worker {i} bitmap"
    assert np.array_equal(g["Ya"], o["Ya"])
    assert np.array_equal(g["Ba"], o["Ba"])
    assert_same_info(g["info"], o["info"])
    assert np.array_equal(g["mask"], o["mask"])
    assert np.array_equal(g["x"], o["x"])
    assert g["info"].success and g["info"].n_support == n_agg
    uniq, sums = sparse_direct_sum(w)
    assert np.array_equal(g["x"][uniq], sums)
    assert np.count_nonzero(g["x"]) == np.count_nonzero(sums)


@pytest.mark.timeout(900)
def test_fullsize_vgg19_fp32():
    _hc()
    w = wl.make("vgg19", vtype="f32")
    rows = oracle.rows_for(w.n_agg)
    g = gpu_run(w, rows, 1024, want_coo_out=False, max_support=w.n_agg, use_plan=True)
    o = oracle_run(w, rows, 1024)
    wb, ab = fp32_cell_bounds(w, o["g"])
    for i in range(w.W):
        assert np.array_equal(g["B"][i], o["B"][i])
        assert np.all(np.abs(g["Y"][i].astype(np.float64) - o["Y"][i]) <= wb[i] * (1 + 1e-6))
    assert np.array_equal(g["Ba"], o["Ba"])
    assert np.all(np.abs(g["Ya"].astype(np.float64) - o["Ya"]) <= ab * (1 + 1e-6))
    assert np.array_equal(g["mask"], o["mask"])
    assert_same_info(g["info"], o["info"])
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    bnd = oracle.decode_bound(o["g"], ab, o["Ba"])
    assert_fp32_values(g["x"], o["x"], bnd, sup)
    assert_fp32_decode_stage(g, o["g"], "vgg19 global")
    fp32_normwise_error(g["x"], o["x"], bnd, "vgg19 global")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("density,overlap", [(0.001, 0.9), (0.05, 0.1)])
def test_fullsize_bert_sweep_corners(density, overlap):
    # the smallest and the largest aggregate of the BERT-base density/overlap
    # sweep, every stage against the oracle (the large corner's 79 M aggregate
    # nonzeros take the oracle's decode about two minutes), and the decode
    # also against the direct sum of the workers' gradients.
    _hc()
    w = wl.make("bert", density=density, overlap=overlap)
    n_agg = w.n_agg
    rows = oracle.rows_for(n_agg)
    print(f"[fullsize] bert d={density} o={overlap}: n_agg={n_agg} rows={rows}", flush=True)
    g = gpu_run(w, rows, 1024, want_coo_out=False, max_support=n_agg, use_plan=True)
    gg = oracle.Geom(n=w.n, rows=rows, seed=w.hash_seed, c=1024)
    Ys, Bs = [], []
    for i in range(w.W):
        Y, B = oracle.encode_coo(gg, w.idx[i], w.val[i])
        assert np.array_equal(g["Y"][i], Y) and np.array_equal(g["B"][i], B), f"worker {i}"
        Ys.append(Y)
        Bs.append(B)
        print(f"[fullsize] bert d={density} o={overlap}: oracle encode of worker {i} equal",
              flush=True)
    Ya, Ba = oracle.aggregate(np.stack(Ys), np.stack(Bs))
    del Ys, Bs
    assert np.array_equal(g["Ya"], Ya) and np.array_equal(g["Ba"], Ba)
    inf = g["info"]
    assert inf.success and inf.n_support == n_agg == inf.n_recovered and inf.status == 0
    assert np.array_equal(g["mask"], Ba)
    uniq, sums = sparse_direct_sum(w)
    assert np.array_equal(g["x"][uniq], sums)
    assert np.count_nonzero(g["x"]) == np.count_nonzero(sums)
    print(f"[fullsize] bert d={density} o={overlap}: oracle decode", flush=True)
    xo, mo, io = oracle.decode(gg, Ya, Ba)
    assert_same_info(inf, io)
    assert np.array_equal(g["mask"], mo)
    assert np.array_equal(g["x"], xo)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,vtype", [("bert", "i32"), ("vgg19", "i32"), ("lstm", "i32"),
                                        ("vgg19", "f32")])
def test_fullsize_blocked(name, vtype):
    # the blocked sketch in bench.py --blocked's configuration: gamma = 1.3 and
    # the library's rows per block for this device
    _hc()
    import paper_2402_07529_amd as hc
    w = wl.make(name, vtype=vtype)
    p = hc.hc_geometry_blocked(w.n, w.n_agg, 1.3, 1024, 0, w.hash_seed, vtype)
    print(f"[fullsize blocked] {name} {vtype}: n={w.n} W={w.W} n_agg={w.n_agg} "
          f"block={int(p.block)} rows={int(p.rows)} nblocks={p.nblocks} seed={int(p.seed)}",
          flush=True)
    g = gpu_run(w, int(p.rows), int(p.c), want_coo_out=False, block=int(p.block),
                seed=int(p.seed))
    o = oracle_run(w, int(p.rows), int(p.c), block=int(p.block), seed=int(p.seed))
    if vtype == "i32":
        for i in range(w.W):
            assert np.array_equal(g["Y"][i], o["Y"][i]), f"worker {i} sketch"
            assert np.array_equal(g["B"][i], o["B"][i]), f"worker {i} bitmap"
        assert np.array_equal(g["Ya"], o["Ya"])
        assert np.array_equal(g["x"], o["x"])
    else:
        wb, ab = fp32_cell_bounds(w, o["g"])
        for i in range(w.W):
            assert np.array_equal(g["B"][i], o["B"][i])
            assert np.all(np.abs(g["Y"][i].astype(np.float64) - o["Y"][i]) <= wb[i] * (1 + 1e-6))
        assert np.all(np.abs(g["Ya"].astype(np.float64) - o["Ya"]) <= ab * (1 + 1e-6))
        sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
        bnd = oracle.decode_bound(o["g"], ab, o["Ba"])
        assert_fp32_values(g["x"], o["x"], bnd, sup)
        assert_fp32_decode_stage(g, o["g"], f"{name} blocked")
        fp32_normwise_error(g["x"], o["x"], bnd, f"{name} blocked")
    assert np.array_equal(g["Ba"], o["Ba"])
    assert np.array_equal(g["mask"], o["mask"])
    assert_same_info(g["info"], o["info"])
    assert g["info"].success and g["info"].n_support == w.n_agg
    if vtype == "i32":
        uniq, sums = sparse_direct_sum(w)
        assert np.array_equal(g["x"][uniq], sums)
        assert np.count_nonzero(g["x"]) == np.count_nonzero(sums)


def _hot_cell_workload(n, rows, density, seed):
    """A synthetic gradient plus one nonzero in every batch that hashes into
    the busiest row, at the offset that lands on that row's cell 0: a cell of
    far more elements than any random one, whose deg * 2^k + (sum of
    positions) does not fit 32 bits."""
    w = wl.make("synthetic", n=n, W=1, density=density, data_seed=seed)
    g = oracle.Geom(n=n, rows=rows, seed=w.hash_seed, c=1024)
    nb = n // 1024
    cl, _ = oracle.cells(g, np.arange(nb, dtype=np.uint64) * 1024)
    r = (cl // 1024).astype(np.int64)
    bias = (cl % 1024).astype(np.int64)
    busiest = int(np.argmax(np.bincount(r.reshape(-1), minlength=rows)))
    bb, jj = np.nonzero(r == busiest)
    hot = (bb.astype(np.int64) * 1024 + ((0 - bias[bb, jj]) & 1023)).astype(np.uint32)
    idx = np.union1d(w.idx[0], hot).astype(np.uint32)
    vals = np.ones(idx.size, np.int32)
    pos = np.searchsorted(w.idx[0], idx)
    old = (pos < w.idx[0].size) & (w.idx[0][np.minimum(pos, w.idx[0].size - 1)] == idx)
    vals[old] = w.val[0][pos[old]]
    w.idx, w.val = [idx], [vals]
    kp = int(np.ceil(np.log2(idx.size)))
    hot_pos = np.searchsorted(idx, hot)
    assert hot.size * 2**kp + int(hot_pos.sum()) >= 2**32  # the busy cell cannot pack
    return w, idx, hot


def _check_unpackable(w, idx, rows, label):
    print(f"[{label}] n={w.n} nonzeros={idx.size} rows={rows} cells={rows * 1024}", flush=True)
    gr = gpu_run(w, rows, 1024, want_coo_out=False, use_plan=True, max_support=idx.size)
    o = oracle_run(w, rows, 1024)
    assert np.array_equal(gr["Ya"], o["Ya"])
    assert np.array_equal(gr["x"], o["x"])
    assert np.array_equal(gr["mask"], o["mask"])
    assert_same_info(gr["info"], o["info"])
    assert 0 < gr["info"].n_recovered < idx.size


@pytest.mark.timeout(900)
def test_unpackable_counters_sketch_half_the_support():
    # 16 M cells (16,384 rows) over 33.6 M elements (positions take 26 bits)
    # with one cell of at least 77 elements that cannot pack: the int32 peel
    # keeps counters and residuals apart.  With fewer cells than support
    # elements the decode takes the counter gather and the entry-by-entry
    # round 0 (round 0 by rows needs a cell per element).  Round 0 recovers
    # the elements with a pure cell, a few rounds follow, the rest get median
    # estimates.  Exact against the oracle.
    _hc()
    n, rows = 1 << 28, 16384
    w, idx, hot = _hot_cell_workload(n, rows, 0.13, 515)
    assert rows * 1024 < idx.size
    _check_unpackable(w, idx, rows, "unpackable, half the support")


@pytest.mark.timeout(900)
def test_round0_by_rows_with_unpackable_counters():
    # 25.2 M cells (24,576 rows, wide enough for round 0 by rows) over 21.5 M
    # elements of a 2^30-parameter gradient (positions take 25 bits) with one
    # cell of 177 elements: its deg * 2^25 + (sum of positions) does not fit
    # 32 bits, so round 0 by rows takes its unpacked path (counters and
    # residuals apart, two passes over the row).  The sketch is 1.17 cells per
    # element, under the peeling threshold: the decode ends with median
    # estimates for what the 2-core keeps.  Exact against the oracle.
    _hc()
    n, rows = 1 << 30, 24576
    w, idx, hot = _hot_cell_workload(n, rows, 0.02, 515)
    assert rows * 1024 >= idx.size  # round 0 by rows: a cell per support element
    assert rows >= 8 * 256  # rows to spare (8 per CU of a 256-CU GPU)
    _check_unpackable(w, idx, rows, "round0 rows unpacked")
