"""GPU parity of the Bloom-filter index (section 3.3) against the CPU oracle.

The filter replaces the bitmap: each worker's encode ORs its nonzeros' bits
into the filter, the aggregation ORs the filters, and the decode treats every
parameter whose filter bits are all set as the support (the nonzeros plus the
filter's false positives, which peel to 0).  Bar: int32 sketches, filters,
decoded gradient, recovered mask and support size / recovered count / round
count / success flag bit-exact; fp32 values within the per-element bounds of
test_gpu_parity.  At the NCF size the decode is also checked against the
direct sum and the candidate count against the filter's false-positive
rate.
"""
import math

import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run, wrap_sum
from test_gpu_parity import (assert_fp32_decode_stage, assert_fp32_values, assert_same_info,
                             fp32_cell_bounds)

pytestmark = pytest.mark.gpu


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2402_07529_amd as hc
    return hc


def check_bloom_int(w, g, coo_input=False, use_plan=False):
    print(f"[bloom] {w.name} n={w.n} c={g.c} rows={g.rows} k={g.bloom_k} brows={g.bloom_rows} "
          f"coo_input={coo_input} plan={use_plan}", flush=True)
    r = gpu_run(w, g.rows, g.c, coo_input=coo_input, use_plan=use_plan, seed=g.seed,
                bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    o = oracle_run(w, g.rows, g.c, seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    for i in range(w.W):
        assert np.array_equal(r["Y"][i], o["Y"][i]), f"worker {i} sketch"
        assert np.array_equal(r["B"][i], o["B"][i]), f"worker {i} filter"
    assert np.array_equal(r["Ya"], o["Ya"])
    assert np.array_equal(r["Ba"], o["Ba"])
    assert np.array_equal(r["x"], o["x"])
    assert np.array_equal(r["mask"], o["mask"])
    assert_same_info(r["info"], o["info"])
    return r, o


@pytest.mark.parametrize("c", [1024, 256, 64, 32, 8, 1])
def test_bloom_ragged_int32(c):
    # n not a multiple of c or 32; the filter's last row is partial in words
    # gamma 1.35: a few thousand candidates sit too close to the 2-core
    # threshold at 1.23 to peel every time
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.002, overlap=0.3, data_seed=700 + c)
    _hc()
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, c, gamma=1.35)
    r, o = check_bloom_int(w, g)
    assert r["info"].success and r["info"].n_support > w.n_agg
    assert np.array_equal(r["x"], wrap_sum([w.dense(i) for i in range(w.W)]))
    # COO output: every candidate, false positives with value 0
    cand = np.nonzero(np.unpackbits(r["mask"].view(np.uint8), bitorder="little")[:w.n])[0]
    assert np.array_equal(r["coo_idx"], cand.astype(np.uint32))
    assert np.array_equal(r["coo_val"], r["x"][cand])


@pytest.mark.parametrize("c", [1024, 64])
def test_bloom_coo_encode(c):
    _hc()
    w = wl.make("synthetic", n=600_001, W=3, density=0.003, overlap=0.2, data_seed=710 + c)
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, c)
    check_bloom_int(w, g, coo_input=True)


@pytest.mark.parametrize("c", [1024, 256])
def test_bloom_with_plan(c):
    _hc()
    w = wl.make("synthetic", n=3_000_000, W=4, density=0.001, overlap=0.5, data_seed=720 + c)
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, c)
    check_bloom_int(w, g, use_plan=True)


@pytest.mark.parametrize("ratio", [0.9, 1.1])
def test_bloom_undersized_failure_parity(ratio):
    # sketch below the threshold for the candidates: failures, leftover
    # estimates and masks still bit-exact
    _hc()
    w = wl.make("synthetic", n=2_000_000, W=4, density=0.002, overlap=0.3, data_seed=730)
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, 1024)
    rows = max(3, int(ratio * g.rows / 1.23))
    g = oracle.Geom(n=g.n, rows=rows, seed=g.seed, c=g.c, bloom_k=g.bloom_k,
                    bloom_rows=g.bloom_rows)
    r, o = check_bloom_int(w, g)
    assert not o["info"].success


def test_bloom_tiny_filter_many_false_positives():
    # a filter far too small: most parameters become candidates
    _hc()
    w = wl.make("synthetic", n=200_000, W=2, density=0.01, overlap=0.5, data_seed=740)
    g = oracle.Geom(n=w.n, rows=2000, seed=w.hash_seed, c=64, bloom_k=2, bloom_rows=60)
    r, o = check_bloom_int(w, g)
    assert o["info"].n_support > 10 * w.n_agg


@pytest.mark.parametrize("c", [1024, 64])
def test_bloom_fp32(c):
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.002, overlap=0.4, data_seed=750 + c,
                vtype="f32")
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, c)
    r = gpu_run(w, g.rows, c, seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    o = oracle_run(w, g.rows, c, seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    wb, ab = fp32_cell_bounds(w, o["g"])
    for i in range(w.W):
        assert np.array_equal(r["B"][i], o["B"][i])
        assert np.all(np.abs(r["Y"][i].astype(np.float64) - o["Y"][i]) <= wb[i] * (1 + 1e-6))
    assert np.array_equal(r["Ba"], o["Ba"])
    assert np.array_equal(r["mask"], o["mask"])
    assert_same_info(r["info"], o["info"])
    cand = np.nonzero(np.unpackbits(o["mask"].view(np.uint8), bitorder="little")[:w.n])[0]
    assert_fp32_values(r["x"], o["x"], oracle.decode_bound(o["g"], ab, o["Ba"]), cand)
    assert_fp32_decode_stage(r, o["g"], f"bloom c={c}")


def test_bloom_geometry_call_and_tiny_lengths():
    hc = _hc()
    for n in (1, 31, 33, 1000, 4097):
        W = 2
        rng = np.random.default_rng(n)
        idx = [np.sort(rng.choice(n, max(1, n // 50), replace=False)).astype(np.uint32)
               for _ in range(W)]
        val = [rng.integers(1, 1000, ii.size).astype(np.int32) for ii in idx]
        w = wl.Workload("short", n, W, "i32", idx, val, 1, 5 + n)
        for c in (32, 1024, 8):
            g = oracle.Geom(n=n, rows=3, seed=5 + n, c=c, bloom_k=3, bloom_rows=2)
            check_bloom_int(w, g)
    p, eps = hc.hc_geometry_bloom(10_000_000, 20_000, 1.23, 1024, 3)
    assert int(p.bloom_k) == round(math.log2(1 / eps))


@pytest.mark.timeout(900)
def test_fullsize_ncf_bloom():
    # NCF-shaped (2^30 parameters, 8 workers): the 128 MiB bitmap per worker
    # becomes a filter of a few MiB (section 3.3's case of extreme sparsity)
    hc = _hc()
    w = wl.make("ncf")
    p, _ = hc.hc_geometry_bloom(w.n, w.n_agg, 1.23, 1024, w.hash_seed)
    g = oracle.Geom(n=w.n, rows=int(p.rows), seed=int(p.seed), c=1024, bloom_k=int(p.bloom_k),
                    bloom_rows=int(p.bloom_rows))
    print(f"[bloom fullsize] ncf k={g.bloom_k} filter={4 * g.index_words} B rows={g.rows}",
          flush=True)
    n_cand_max = int(w.n_agg + 4 * 2.0**-g.bloom_k * w.n) + 1000
    r = gpu_run(w, g.rows, 1024, want_coo_out=False, max_support=n_cand_max, use_plan=True,
                seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    Ys, Bs = [], []
    for i in range(w.W):
        Y, B = oracle.encode_coo(g, w.idx[i], w.val[i])
        assert np.array_equal(r["Y"][i], Y) and np.array_equal(r["B"][i], B), f"worker {i}"
        Ys.append(Y)
        Bs.append(B)
    Ya, Ba = oracle.aggregate(np.stack(Ys), np.stack(Bs))
    del Ys, Bs
    assert np.array_equal(r["Ya"], Ya) and np.array_equal(r["Ba"], Ba)
    inf = r["info"]
    assert inf.success and inf.n_recovered == inf.n_support and inf.status == 0
    # decoded gradient: the direct sum, exactly
    from test_gpu_fullsize import sparse_direct_sum
    uniq, sums = sparse_direct_sum(w)
    assert np.array_equal(r["x"][uniq], sums)
    assert np.count_nonzero(r["x"]) == np.count_nonzero(sums)
    # candidates: the support plus about fill^k (N - n) false positives
    fill = np.unpackbits(Ba.view(np.uint8), bitorder="little")[:g.bloom_rows * g.c].mean()
    mu = fill**g.bloom_k * (w.n - w.n_agg)
    fp = inf.n_support - w.n_agg
    assert abs(fp - mu) < 6 * math.sqrt(mu) + 0.05 * mu, (fp, mu)
    # the oracle's whole decode of the same aggregate (about two minutes): the
    # candidate set (every parameter the filter passes, section 3.3), rounds,
    # recovered mask and values, all exact
    print(f"[bloom fullsize] ncf: oracle decode of {inf.n_support} candidates", flush=True)
    xo, mo, io = oracle.decode(g, Ya, Ba)
    assert_same_info(inf, io)
    assert np.array_equal(r["mask"], mo)
    assert np.array_equal(r["x"], xo)
