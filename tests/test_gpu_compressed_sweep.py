"""Section 4.1's microbenchmark at parity-test size: one worker, a gradient at
VGG19's natural density (69.6 % nonzero, Table 1), compressed to sketches of
2 % to 200 % of its size (cells / n) and decompressed at once.

int32: bit-exact against the oracle at every size (decoded gradient, mask,
support, recovered count, rounds, success), including the sizes where
peeling stops early and the median estimate takes over.  fp32: structure
exact, values within the derived bounds.  Against the paper: recovery is
complete from the threshold 1.23 x 69.6 % = 85.6 % on (checked at 100 % and
200 %), and incomplete well below it.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run
from test_gpu_parity import assert_fp32_values, assert_same_info, fp32_cell_bounds

pytestmark = pytest.mark.gpu

SIZES = (0.02, 0.3, 0.7, 0.856, 1.0, 2.0)


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def rows_for_size(n, frac, c=1024):
    return max(3, -(-int(np.ceil(frac * n)) // c))


@pytest.mark.parametrize("frac", SIZES)
def test_compressed_size_int32(frac):
    _hc()
    w = wl.make("synthetic", n=1_500_017, W=1, density=0.696, data_seed=808)
    rows = rows_for_size(w.n, frac)
    print(f"[compressed] int32 size={frac} n={w.n} nonzeros={w.n_agg} rows={rows}", flush=True)
    r = gpu_run(w, rows, 1024, want_coo_out=False, use_plan=True, max_support=w.n_agg)
    o = oracle_run(w, rows, 1024)
    assert np.array_equal(r["Y"][0], o["Y"][0]) and np.array_equal(r["Ya"], o["Ya"])
    assert np.array_equal(r["x"], o["x"])
    assert np.array_equal(r["mask"], o["mask"])
    assert_same_info(r["info"], o["info"])
    rate = r["info"].n_recovered / r["info"].n_support
    if frac >= 1.0:
        assert r["info"].success
        assert np.array_equal(r["x"], w.dense(0))
    if frac <= 0.7:
        assert rate < 0.5


@pytest.mark.parametrize("frac", (0.3, 1.0))
def test_compressed_size_fp32(frac):
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=1, density=0.696, data_seed=809, vtype="f32")
    rows = rows_for_size(w.n, frac)
    r = gpu_run(w, rows, 1024, want_coo_out=False, max_support=w.n_agg)
    o = oracle_run(w, rows, 1024)
    wb, ab = fp32_cell_bounds(w, o["g"])
    assert np.all(np.abs(r["Ya"].astype(np.float64) - o["Ya"]) <= ab * (1 + 1e-6))
    assert np.array_equal(r["mask"], o["mask"])
    assert_same_info(r["info"], o["info"])
    sup = np.nonzero(np.unpackbits(o["Ba"].view(np.uint8), bitorder="little")[:w.n])[0]
    assert_fp32_values(r["x"], o["x"], oracle.decode_bound(o["g"], ab, o["Ba"]), sup)
    if frac >= 1.0:
        x = w.dense(0).astype(np.float64)
        rel = np.abs(r["x"][sup] - x[sup]) / np.abs(x[sup])
        assert rel.mean() < 1e-6
