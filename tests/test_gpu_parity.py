"""GPU (gfx950) parity of encode -> aggregate -> decode against the CPU oracle.

Bar: int32 fixed-point results are bit-exact (sketches, bitmaps, decoded
gradient, recovered mask, COO, and the support size / recovered count / round
count / success flag).

fp32: the structural outputs (bitmaps, mask, counts, rounds, success) are
exact.  Values are compared with the oracle's fp64 computation under a
tolerance derived from the arithmetic, element by element:
  * a worker's fp32 sketch cell is a sum of m terms added in an unspecified
    order (atomics): |error| <= gamma_(m-1) * S, S the sum of the terms'
    magnitudes, gamma_k = k u / (1 - k u), u = 2^-24;
  * the aggregate adds W such cells in worker order: per cell
    |error| <= gamma_K * S with K = (largest per-worker term count - 1) + (W - 1);
  * decoding peels in fp64, so each decoded value's error is at most these
    cell bounds carried through the peeling schedule (oracle.decode_bound),
    plus one rounding to fp32 (u |x|) and fp64 noise (1e-12 of the largest
    value).
A flat 1e-6 normwise tolerance against the exact sum is not attainable by any
decoder of an fp32 sketch: rounding the exact aggregate sketch to fp32 once
already moves the exactly peeled result by about 1.3e-6 of its largest value
on these inputs (pinned on the CPU in test_oracle).  The decode stage alone
meets the 1e-6 bar: the oracle decodes the GPU's own fp32 aggregate (widened
to fp64, the same synchronous rounds, each element read from the pure cell of
smallest j, as the GPU's fp32 peel does), and every decoded value agrees
within 1e-6 of its own magnitude (plus 1e-12 of the largest value).
"""
import math

import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run, wrap_sum

pytestmark = pytest.mark.gpu

U = 2.0 ** -24  # fp32 unit roundoff


def gamma(k):
    k = np.asarray(k, np.float64)
    return k * U / (1 - k * U)


def fp32_cell_bounds(w, g):
    """Per-cell error bounds of each worker's fp32 sketch and of the fp32
    aggregate (see the module docstring)."""
    S = np.zeros(g.cells)
    mmax = np.zeros(g.cells)
    per_worker = []
    for i in range(w.W):
        cl, _ = oracle.cells(g, w.idx[i].astype(np.uint64))
        a = np.abs(w.val[i].astype(np.float64))
        Si = np.zeros(g.cells)
        mi = np.zeros(g.cells)
        for j in range(3):
            Si += np.bincount(cl[:, j].astype(np.int64), weights=a, minlength=g.cells)
            mi += np.bincount(cl[:, j].astype(np.int64), minlength=g.cells)
        per_worker.append(gamma(np.maximum(mi - 1, 0)) * Si)
        S += Si
        mmax = np.maximum(mmax, mi)
    agg = gamma(np.maximum(mmax - 1, 0) + (w.W - 1)) * S
    return per_worker, agg


def assert_fp32_values(x_gpu, x_oracle, bnd, support):
    x64 = x_oracle.astype(np.float64)
    tol = bnd * (1 + 1e-6) + U * np.abs(x64) + 1e-12 * np.max(np.abs(x64))
    err = np.abs(x_gpu.astype(np.float64) - x64)
    bad = np.nonzero(err > tol)[0]
    assert bad.size == 0, (bad[:5], err[bad[:5]], tol[bad[:5]])
    other = np.ones(x_gpu.size, bool)
    other[support] = False
    assert not x_gpu[other].any()


def assert_fp32_decode_stage(g, geom, label=""):
    """The GPU's fp32 decode against the oracle's decode of the same fp32
    aggregate: structure exact, values within 1e-6 relative.  Returns the
    largest element-wise relative difference."""
    xo, mo, io = oracle.decode(geom, g["Ya"].astype(np.float64), g["Ba"])
    assert np.array_equal(g["mask"], mo), label
    assert_same_info(g["info"], io)
    err = np.abs(g["x"].astype(np.float64) - xo)
    tol = 1e-6 * np.abs(xo) + 1e-12 * max(float(np.max(np.abs(xo))), 1e-300)
    bad = np.nonzero(err > tol)[0]
    assert bad.size == 0, (label, bad[:5], g["x"][bad[:5]], xo[bad[:5]])
    rel = float(np.max(err / np.maximum(np.abs(xo), 1e-300), initial=0.0))
    print(f"[fp32 decode stage] {label} max |gpu - oracle(gpu aggregate)| / |x| = {rel:.3e}",
          flush=True)
    return rel


def fp32_normwise_error(x_gpu, truth, bnd=None, label=""):
    """max |x - truth| / max |truth| (printed, with max error / bound)."""
    t = truth.astype(np.float64)
    err = np.abs(x_gpu.astype(np.float64) - t)
    nw = float(np.max(err) / max(float(np.max(np.abs(t))), 1e-300))
    msg = f"[fp32 vs exact sum] {label} normwise error {nw:.3e}"
    if bnd is not None:
        tol = bnd + U * np.abs(t) + 1e-12 * np.max(np.abs(t))
        msg += f", max error / bound {float(np.max(err / np.maximum(tol, 1e-300))):.3f}"
    print(msg, flush=True)
    return nw


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2402_07529_amd as hc
    return hc


def assert_same_info(gi, oi):
    assert (gi.n_support, gi.n_recovered, gi.rounds, gi.success) == \
        (oi.n_support, oi.n_recovered, oi.rounds, oi.success), (gi, oi)
    assert gi.status == 0


def check_int(w, rows, c, coo_input=False, use_plan=False, gather=False, staged=False):
    g = gpu_run(w, rows, c, coo_input=coo_input, use_plan=use_plan, gather=gather, staged=staged)
    o = oracle_run(w, rows, c)
    for i in range(w.W):
        assert np.array_equal(g["Y"][i], o["Y"][i]), f"worker {i} sketch"
        assert np.array_equal(g["B"][i], o["B"][i]), f"worker {i} bitmap"
    assert np.array_equal(g["Ya"], o["Ya"])
    assert np.array_equal(g["Ba"], o["Ba"])
    assert np.array_equal(g["x"], o["x"])
    assert np.array_equal(g["mask"], o["mask"])
    assert_same_info(g["info"], o["info"])
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    assert np.array_equal(g["coo_idx"], sup.astype(np.uint32))
    assert np.array_equal(g["coo_val"], o["x"][sup])
    return g, o


def test_tiny_int32_all_stages():
    _hc()
    w = wl.make("tiny")
    rows = oracle.rows_for(w.n_agg)
    g, o = check_int(w, rows, 1024)
    assert g["info"].success
    assert np.array_equal(g["x"], wrap_sum([w.dense(i) for i in range(w.W)]))


@pytest.mark.parametrize("c", [1024, 512, 256, 128, 64, 16, 4, 2, 1])
def test_multi_tile_ragged_int32(c):
    # several rows and tiles, n not a multiple of the tile, the word or c
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.01, overlap=0.4, data_seed=c)
    rows = oracle.rows_for(w.n_agg, 1.23, c)
    g, o = check_int(w, rows, c)
    assert g["info"].success
    assert np.array_equal(g["x"], wrap_sum([w.dense(i) for i in range(w.W)]))


@pytest.mark.parametrize("c", [1024, 512, 256])
def test_multi_tile_ragged_int32_planned(c):
    # the decode's per-cell counters gathered row by row through the plan
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.01, overlap=0.4, data_seed=c + 7)
    rows = oracle.rows_for(w.n_agg, 1.23, c)
    g, o = check_int(w, rows, c, use_plan=True)
    assert g["info"].success


@pytest.mark.parametrize("c,frac", [(1024, 0.5), (512, 2.0), (256, 0.4)])
def test_wide_sketch_planned(c, frac):
    # a sketch of frac * n cells: at most 8 plan entries per row, so the
    # counters are built one wave per row and the round-0 frontier comes from
    # the peel kernel's scan; a dense support, so most rows are live
    _hc()
    w = wl.make("synthetic", n=600_011, W=2, density=0.3, overlap=0.2, data_seed=c + 11)
    rows = max(3, int(frac * w.n / c))
    assert 3 * ((w.n + c - 1) // c) <= 8 * rows
    g, o = check_int(w, rows, c, use_plan=True)
    assert g["info"].success == o["info"].success


def test_wide_sketch_planned_fp32():
    _hc()
    w = wl.make("synthetic", n=400_009, W=2, density=0.3, overlap=0.2, vtype="f32", data_seed=31)
    rows = int(0.8 * w.n / 1024)
    g, o, bnd = check_fp32(w, rows, 1024, use_plan=True)
    assert g["info"].success


@pytest.mark.parametrize("ratio", [1.10, 0.8])
def test_undersized_sketch_failure_parity_planned(ratio):
    _hc()
    w = wl.make("synthetic", n=2_000_000, W=4, density=0.01, overlap=0.3,
                data_seed=int(ratio * 100) + 1)
    rows = max(3, int(math.ceil(ratio * w.n_agg / 1024)))
    g, o = check_int(w, rows, 1024, use_plan=True)
    assert not g["info"].success


def test_plan_for_other_geometry_is_reported():
    # a plan built for another seed: detected on the device, nothing peeled,
    # every member of the support gets the estimate from the aggregate
    hc = _hc()
    import torch
    w = wl.make("synthetic", n=300_000, W=2, density=0.01, overlap=0.5, data_seed=19)
    rows = oracle.rows_for(w.n_agg, 1.23, 1024)
    other = hc.make_params(w.n, rows, w.hash_seed + 1, 1024)
    plan = hc.make_plan(other, torch.device("cuda"))
    g = gpu_run(w, rows, 1024, plan=plan)
    o = oracle_run(w, rows, 1024)
    inf = g["info"]
    assert (inf.status, inf.success, inf.n_recovered) == (3, 0, 0)
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    est = np.array([oracle.query(o["g"], o["Ya"], int(p)) for p in sup], np.int32)
    assert np.array_equal(g["x"][sup], est)


@pytest.mark.parametrize("c", [1024, 64, 1])
def test_coo_encode_matches_dense(c):
    _hc()
    w = wl.make("synthetic", n=777_777, W=3, density=0.02, overlap=0.5, data_seed=40 + c)
    rows = oracle.rows_for(w.n_agg, 1.23, c)
    check_int(w, rows, c, coo_input=True)


@pytest.mark.parametrize("ratio,c", [(1.10, 1024), (1.15, 64), (1.20, 1), (0.8, 1024)])
def test_undersized_sketch_failure_parity(ratio, c):
    # below the peeling threshold: partial recovery, leftover estimates
    _hc()
    w = wl.make("synthetic", n=2_000_000, W=4, density=0.01, overlap=0.3, data_seed=int(ratio * 100))
    rows = max(3, int(math.ceil(ratio * w.n_agg / c)))
    g, o = check_int(w, rows, c)
    assert not g["info"].success and g["info"].n_recovered < g["info"].n_support


def test_forced_failure_three_cells():
    _hc()
    w = wl.make("synthetic", n=5000, W=2, density=0.002, overlap=0.0, data_seed=3)
    g, o = check_int(w, 3, 1)
    assert g["info"].n_recovered == 0 and g["info"].rounds == 0


def check_fp32(w, rows, c, use_plan=False, gather=False, staged=False):
    g = gpu_run(w, rows, c, use_plan=use_plan, gather=gather, staged=staged)
    o = oracle_run(w, rows, c)
    wb, ab = fp32_cell_bounds(w, o["g"])
    for i in range(w.W):
        assert np.array_equal(g["B"][i], o["B"][i])
        err = np.abs(g["Y"][i].astype(np.float64) - o["Y"][i])
        over = np.nonzero(err > wb[i] * (1 + 1e-6))[0]
        assert over.size == 0, (f"worker {i} sketch: {over.size} cells over the bound, e.g. "
                                f"{over[:4]} err {err[over[:4]]} bound {wb[i][over[:4]]} "
                                f"gpu {g['Y'][i][over[:4]]} oracle {o['Y'][i][over[:4]]}")
    assert np.array_equal(g["Ba"], o["Ba"])
    assert np.all(np.abs(g["Ya"].astype(np.float64) - o["Ya"]) <= ab * (1 + 1e-6))
    assert np.array_equal(g["mask"], o["mask"])
    assert_same_info(g["info"], o["info"])
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    bnd = oracle.decode_bound(o["g"], ab, o["Ba"])
    assert_fp32_values(g["x"], o["x"], bnd, sup)
    assert np.array_equal(g["coo_idx"], sup.astype(np.uint32))
    assert np.array_equal(g["coo_val"], g["x"][sup])
    assert_fp32_decode_stage(g, o["g"], f"n={w.n} c={c}")
    return g, o, bnd


@pytest.mark.parametrize("use_plan", [False, True])
def test_fp32_all_stages(use_plan):
    _hc()
    w = wl.make("synthetic", n=1_500_001, W=8, density=0.01, overlap=0.3, vtype="f32",
                data_seed=77)
    rows = oracle.rows_for(w.n_agg, 1.23, 1024)
    g, o, bnd = check_fp32(w, rows, 1024, use_plan=use_plan)
    assert g["info"].success
    truth = sum(w.dense(i).astype(np.float64) for i in range(w.W))
    sup = np.nonzero(truth)[0]
    assert np.all(np.abs(g["x"] - truth) <= bnd * (1 + 1e-6) + U * np.abs(truth) +
                  1e-12 * np.max(np.abs(truth)))
    # against the exact sum the fp32 sketch's own rounding sets the scale:
    # the exact decode of the exact aggregate rounded once to fp32 misses by
    # `floor` (about 1.3e-6 here); the GPU's worker sketches and aggregate
    # round at every addition, so its error may be a few times that
    Yr = o["Ya"].astype(np.float32).astype(np.float64)
    xr, _, ir = oracle.decode(o["g"], Yr, o["Ba"])
    assert ir.success
    floor = float(np.max(np.abs(xr - truth)) / np.max(np.abs(truth)))
    nw = fp32_normwise_error(g["x"], truth, bnd, f"use_plan={use_plan}")
    print(f"[fp32 vs exact sum] single-rounding floor {floor:.3e}, gpu / floor {nw / floor:.2f}",
          flush=True)
    assert floor > 1e-6
    assert nw <= 8 * floor
    # the tolerance is not vacuous: for the typical element it is a few
    # rounding units of the gradient's scale (it grows only along long
    # peeling chains, where worst-case errors add up)
    assert np.median(bnd[sup]) < 1e-6 * np.max(np.abs(truth))


@pytest.mark.parametrize("c", [64, 1])
def test_fp32_small_batches(c):
    _hc()
    w = wl.make("synthetic", n=400_003, W=4, density=0.01, overlap=0.5, vtype="f32",
                data_seed=100 + c)
    check_fp32(w, oracle.rows_for(w.n_agg, 1.23, c), c)


def test_fp32_undersized_structure_exact():
    _hc()
    w = wl.make("synthetic", n=600_000, W=4, density=0.01, overlap=0.3, vtype="f32", data_seed=5)
    rows = int(math.ceil(1.1 * w.n_agg / 1024))
    g, o, bnd = check_fp32(w, rows, 1024)
    assert not g["info"].success


def test_overflow_falls_back_to_estimates():
    # support larger than the workspace capacity: nothing is peeled and every
    # member of the support gets the Count Sketch query of the aggregate
    hc = _hc()
    w = wl.make("synthetic", n=300_000, W=2, density=0.01, overlap=0.5, data_seed=9)
    rows = oracle.rows_for(w.n_agg, 1.23, 1024)
    g = gpu_run(w, rows, 1024, max_support=100)
    o = oracle_run(w, rows, 1024)
    inf = g["info"]
    assert (inf.status, inf.success, inf.n_recovered, inf.rounds) == (1, 0, 0, 0)
    assert inf.n_support == w.n_agg
    assert not g["mask"].any()
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    est = np.array([oracle.query(o["g"], o["Ya"], int(p)) for p in sup], np.int32)
    assert np.array_equal(g["x"][sup], est)
    other = np.ones(w.n, bool)
    other[sup] = False
    assert not g["x"][other].any()


@pytest.mark.parametrize("n", [1, 31, 32, 33, 1023, 1025, 4097])
def test_tiny_and_ragged_lengths(n):
    _hc()
    rng = np.random.default_rng(n)
    k = max(1, n // 10)
    idx = np.sort(rng.choice(n, k, replace=False)).astype(np.uint32)
    vals = rng.integers(1, 1000, k).astype(np.int32)
    w = wl.Workload("edge", n, 1, "i32", [idx], [vals], 0, 99)
    for c in (1, 32, 1024):
        check_int(w, 3 + n // 16, c)


def test_empty_support():
    _hc()
    w = wl.Workload("empty", 100_000, 2, "i32", [np.zeros(0, np.uint32)] * 2,
                    [np.zeros(0, np.int32)] * 2, 0, 5)
    g, o = check_int(w, 5, 1024)
    assert g["info"].success and g["info"].n_support == 0 and not g["x"].any()


def test_int32_wraparound_sums():
    _hc()
    n = 200_000
    rng = np.random.default_rng(1)
    idx = np.sort(rng.choice(n, 2000, replace=False)).astype(np.uint32)
    big = [rng.integers(2**30, 2**31 - 1, idx.size).astype(np.int32) for _ in range(3)]
    w = wl.Workload("wrap", n, 3, "i32", [idx] * 3, big, 0, 17)
    g, o = check_int(w, oracle.rows_for(idx.size), 1024)
    assert np.array_equal(g["x"], wrap_sum([w.dense(i) for i in range(3)]))


@pytest.mark.parametrize("use_plan", [False, True])
def test_deterministic_int32_repeat(use_plan):
    _hc()
    w = wl.make("synthetic", n=3_000_000, W=4, density=0.01, overlap=0.5, data_seed=123)
    rows = oracle.rows_for(w.n_agg)
    a = gpu_run(w, rows, 1024, keep_workers=False, use_plan=use_plan)
    b = gpu_run(w, rows, 1024, keep_workers=False, use_plan=use_plan)
    for k in ("Ya", "Ba", "x", "mask", "coo_idx", "coo_val"):
        assert np.array_equal(a[k], b[k]), k
    assert a["info"] == b["info"]


def test_coo_capacity_truncates():
    _hc()
    w = wl.make("tiny")
    rows = oracle.rows_for(w.n_agg)
    g = gpu_run(w, rows, 1024, coo_cap=100)
    o = oracle_run(w, rows, 1024)
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    assert np.array_equal(g["coo_idx"], sup[:100].astype(np.uint32))
    assert np.array_equal(g["coo_val"], o["x"][sup[:100]])


@pytest.mark.parametrize("use_plan,density", [(False, 0.01), (True, 0.01), (True, 0.12)])
def test_decode_unaligned_views(use_plan, density):
    # the decode reads the aggregate and writes its outputs through views 4
    # bytes past a 16-byte boundary (the ABI asks for 4-byte alignment): the
    # index is then read word by word, and the result must not change.  At
    # 0.12 per worker the aggregate is about 0.4 dense, so the support pass
    # takes its dense-segment path.
    import torch
    hc = _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=density, overlap=0.1,
                data_seed=int(density * 1000) + use_plan)
    rows = oracle.rows_for(w.n_agg)
    a = gpu_run(w, rows, 1024, keep_workers=False, want_coo_out=False, use_plan=use_plan)
    assert a["info"].success
    p = a["p"]
    dev = torch.device("cuda")
    vt = torch.int32
    Ya = torch.zeros(p.cells + 1, dtype=vt, device=dev)
    Ba = torch.zeros(p.index_words + 1, dtype=torch.int32, device=dev)
    Ya[1:] = torch.from_numpy(a["Ya"]).to(dev)
    Ba[1:] = torch.from_numpy(a["Ba"].view(np.int32)).to(dev)
    out = torch.empty(w.n + 1, dtype=vt, device=dev)
    mask = torch.empty(p.words + 1, dtype=torch.int32, device=dev)
    info = hc.alloc_info(dev)
    ws = hc.alloc_workspace(p, 0, dev)
    plan = hc.make_plan(p, dev) if use_plan else None
    hc.hc_decode(p, Ya[1:], Ba[1:], info, ws, x_out=out[1:], mask=mask[1:], plan=plan)
    torch.cuda.synchronize()
    assert hc.read_info(info) == a["info"]
    assert np.array_equal(out[1:].cpu().numpy(), a["x"])
    assert np.array_equal(mask[1:].cpu().numpy().view(np.uint32), a["mask"])
    assert np.array_equal(a["x"], wrap_sum([w.dense(i) for i in range(w.W)]))


def test_unpackable_counters_fall_back():
    # 4.2 M elements on three rows: every cell holds about 1,400 of them, so
    # deg * 2^k + (sum of positions) overflows 32 bits and the int32 peel keeps
    # its residuals apart from the counters; nothing peels and every element
    # gets the median estimate.  Exact against the oracle all the same.
    _hc()
    w = wl.make("synthetic", n=6_000_011, W=1, density=0.7, data_seed=4242)
    rows = 3
    print(f"[unpackable] n={w.n} nonzeros={w.n_agg} rows={rows}", flush=True)
    g = gpu_run(w, rows, 1024, want_coo_out=False, use_plan=True, max_support=w.n_agg)
    o = oracle_run(w, rows, 1024)
    assert np.array_equal(g["Ya"], o["Ya"])
    assert np.array_equal(g["x"], o["x"])
    assert np.array_equal(g["mask"], o["mask"])
    assert_same_info(g["info"], o["info"])
    assert g["info"].n_recovered == 0


@pytest.mark.parametrize("density", [0.1, 0.12])
def test_round0_paths_either_side_of_the_support_bound(density):
    # 2,048 rows (8 per CU of a 256-CU GPU: enough for round 0 by rows) over a
    # 2^24-parameter gradient.  max_support = cells takes round 0 by rows,
    # max_support = cells + 1 the entry-by-entry round; both decodes are exact
    # against the oracle.  Density 0.1 gives 1.68 M elements (1.25 cells per
    # element: the sketch peels), 0.12 gives 2.0 M (1.04: peeling stops at the
    # 2-core and the rest get median estimates).
    _hc()
    n, rows = 1 << 24, 2048
    cells = rows * 1024
    w = wl.make("synthetic", n=n, W=1, density=density, data_seed=77)
    assert w.n_agg <= cells
    o = oracle_run(w, rows, 1024)
    for ms in (cells, cells + 1):
        print(f"[round0 paths] density={density} nonzeros={w.n_agg} max_support={ms}", flush=True)
        g = gpu_run(w, rows, 1024, want_coo_out=False, use_plan=True, max_support=ms)
        assert np.array_equal(g["x"], o["x"])
        assert np.array_equal(g["mask"], o["mask"])
        assert_same_info(g["info"], o["info"])
    assert (o["info"].success == 1) == (density == 0.1)


@pytest.mark.parametrize("n", [4096 * 32, 4098 * 32, 4094 * 32 + 5, 4097 * 32 + 1])
@pytest.mark.parametrize("offset", [0, 1, 2])
def test_aggregate_every_vector_width(n, offset):
    # bitmap word counts that are multiples of 4, of 2 only, and odd, on
    # buffers offset by 0, 1 or 2 words (16-, 8- and 4-byte aligned): the
    # aggregate takes vectors of 4, 2 or 1 words accordingly, always exact
    import torch
    hc = _hc()
    dev = torch.device("cuda")
    p = hc.make_params(n, 3, 17, c=1)  # 3 cells: the sketch is odd-sized too
    W = 3
    rng = np.random.default_rng(n + offset)
    Yh = rng.integers(-2**31, 2**31, (W, p.cells), dtype=np.int64).astype(np.int32)
    Bh = rng.integers(0, 2**32, (W, p.words), dtype=np.uint64).astype(np.uint32)
    Yb = torch.zeros(W * p.cells + offset, dtype=torch.int32, device=dev)
    Bb = torch.zeros(W * p.words + offset, dtype=torch.int32, device=dev)
    Yb[offset:] = torch.from_numpy(Yh.reshape(-1)).to(dev)
    Bb[offset:] = torch.from_numpy(Bh.reshape(-1).view(np.int32)).to(dev)
    Yo = torch.empty(p.cells + offset, dtype=torch.int32, device=dev)
    Bo = torch.empty(p.words + offset, dtype=torch.int32, device=dev)
    hc.hc_aggregate(p, Yb[offset:], Bb[offset:], W, Yo[offset:], Bo[offset:])
    torch.cuda.synchronize()
    assert np.array_equal(Yo[offset:].cpu().numpy(), wrap_sum(list(Yh)))
    assert np.array_equal(Bo[offset:].cpu().numpy().view(np.uint32),
                          np.bitwise_or.reduce(Bh, axis=0))


@pytest.mark.parametrize("W", [1, 3, 5, 8, 16])
@pytest.mark.parametrize("vtype", ["i32", "f32"])
def test_aggregate_worker_counts_and_strides(W, vtype):
    # per-worker counts of every residue mod 4 (so worker w starts (w * count)
    # mod 4 words off the 16-byte grid), worker counts that leave a partial
    # group of four, and a bitmap long enough for several passes of the
    # whole grid: sums (fp32 in worker order) and ORs stay exact
    import torch
    hc = _hc()
    dev = torch.device("cuda")
    cases = [(4097 * 32 + 7, 4097), (4098 * 32, 4098), (4099 * 32 + 31, 4099), (4100 * 32, 4100)]
    if W == 8 and vtype == "i32":
        cases.append(((5 * 2**20 + 3) * 32, 5))  # 5 M + 3 bitmap words per worker
    for n, rows in cases:
        p = hc.make_params(n, rows, 23, c=1, vtype=vtype)
        rng = np.random.default_rng(n * 31 + W)
        if vtype == "i32":
            Yh = rng.integers(-2**31, 2**31, (W, p.cells), dtype=np.int64).astype(np.int32)
            want_y = wrap_sum(list(Yh))
            tdt = torch.int32
        else:
            Yh = rng.standard_normal((W, p.cells)).astype(np.float32)
            want_y = Yh[0].copy()
            for w in range(1, W):
                want_y = (want_y + Yh[w]).astype(np.float32)
            tdt = torch.float32
        Bh = rng.integers(0, 2**32, (W, p.words), dtype=np.uint64).astype(np.uint32)
        Y = torch.from_numpy(Yh).to(dev)
        B = torch.from_numpy(Bh.view(np.int32)).to(dev)
        Yo = torch.empty(p.cells, dtype=tdt, device=dev)
        Bo = torch.empty(p.words, dtype=torch.int32, device=dev)
        print(f"[aggregate] W={W} {vtype} n={n} cells={p.cells} words={p.words}", flush=True)
        hc.hc_aggregate(p, Y, B, W, Yo, Bo)
        torch.cuda.synchronize()
        got_y = Yo.cpu().numpy()
        if vtype == "i32":
            assert np.array_equal(got_y, want_y)
        else:
            assert np.array_equal(got_y.view(np.uint32), want_y.view(np.uint32))
        assert np.array_equal(Bo.cpu().numpy().view(np.uint32), np.bitwise_or.reduce(Bh, axis=0))
