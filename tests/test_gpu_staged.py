"""hc_encode_staged: a first pass compacts each batch's nonzeros into a list,
a second assembles every sketch row in LDS through the plan.

Its sketches and indexes must equal the oracle's (int32 bit for bit; fp32
within the order-independent bound of a sum of m terms), exactly as
hc_encode's do: on sparse gradients (every batch fits its list), on batches
past the list capacity (read from the gradient by the second pass), at
ragged lengths, every plan-capable batch width and with a Bloom-filter
index.  A plan built for another geometry gives a zero sketch and an
all-ones index, which the decode reports as a failure."""
import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import gpu_run, oracle_run, wrap_sum
from test_gpu_parity import _hc, assert_same_info, check_fp32, check_int

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("c", [1024, 512, 256])
def test_staged_ragged_sparse_int32(c):
    # several rows and tiles, n not a multiple of c, 32 or the 16-byte vector
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.01, overlap=0.4, data_seed=c + 33)
    g, o = check_int(w, oracle.rows_for(w.n_agg, 1.23, c), c, staged=True, use_plan=True)
    assert g["info"].success
    assert np.array_equal(g["x"], wrap_sum([w.dense(i) for i in range(w.W)]))


@pytest.mark.parametrize("c,density,W", [(1024, 0.08, 2), (256, 0.3, 2), (1024, 0.696, 1)])
def test_staged_lists_overflow_int32(c, density, W):
    # more than 64 nonzeros in many (or all) batches: those batches come from
    # the gradient itself in the second pass, the others from their lists
    _hc()
    w = wl.make("synthetic", n=500_009, W=W, density=density, overlap=0.1,
                data_seed=int(density * 1000))
    g, o = check_int(w, oracle.rows_for(w.n_agg, 1.3, c), c, staged=True)


@pytest.mark.parametrize("n", [1, 31, 255, 1025, 4097])
def test_staged_tiny_lengths(n):
    _hc()
    w = wl.make("synthetic", n=n, W=2, density=0.4, overlap=0.0, data_seed=n + 1)
    check_int(w, 3, 1024 if n > 1000 else 256, staged=True)


def test_staged_fp32():
    _hc()
    w = wl.make("synthetic", n=1_500_001, W=8, density=0.01, overlap=0.3, vtype="f32", data_seed=77)
    g, o, bnd = check_fp32(w, oracle.rows_for(w.n_agg, 1.23, 1024), 1024, staged=True,
                           use_plan=True)
    assert g["info"].success


def test_staged_fp32_overflow():
    _hc()
    w = wl.make("synthetic", n=400_009, W=3, density=0.2, overlap=0.2, vtype="f32", data_seed=23)
    g, o, bnd = check_fp32(w, oracle.rows_for(w.n_agg, 1.3, 1024), 1024, staged=True)


@pytest.mark.parametrize("c", [1024, 256])
def test_staged_bloom_int32(c):
    # the first pass writes the filter exactly as hc_encode does
    _hc()
    w = wl.make("synthetic", n=1_000_003, W=4, density=0.002, overlap=0.3, data_seed=800 + c)
    g, _ = oracle.bloom_geometry(w.n, w.n_agg, w.hash_seed, c, gamma=1.35)
    r = gpu_run(w, g.rows, c, seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows,
                staged=True)
    o = oracle_run(w, g.rows, c, seed=g.seed, bloom_k=g.bloom_k, bloom_rows=g.bloom_rows)
    for i in range(w.W):
        assert np.array_equal(r["Y"][i], o["Y"][i]), f"worker {i} sketch"
        assert np.array_equal(r["B"][i], o["B"][i]), f"worker {i} filter"
    assert np.array_equal(r["x"], o["x"])
    assert_same_info(r["info"], o["info"])


def test_staged_matches_atomic_encode_bitwise_and_reuses_workspace():
    # int32 sums wrap the same in any order: the staged and the atomic encode
    # agree bit for bit; a second call on the same workspace (stale lists and
    # counts from another gradient) and an unaligned view of the gradient too
    import torch
    hc = _hc()
    dev = torch.device("cuda")
    w = wl.make("synthetic", n=2_000_000, W=2, density=0.03, overlap=0.0, data_seed=4)
    p = hc.hc_geometry(w.n, w.n_agg, 1.23, 1024, w.hash_seed, "i32")
    plan = hc.make_plan(p, dev)
    ws = hc.alloc_stage_workspace(p, dev)
    for i in range(w.W):
        x = torch.from_numpy(w.dense(i)).to(dev)
        Y1 = torch.empty(p.cells, dtype=torch.int32, device=dev)
        B1 = torch.empty(p.words, dtype=torch.int32, device=dev)
        Y2 = torch.full((p.cells,), 7, dtype=torch.int32, device=dev)
        B2 = torch.full((p.words,), 7, dtype=torch.int32, device=dev)
        hc.hc_encode(p, x, Y1, B1)
        hc.hc_encode_staged(p, plan, ws, x, Y2, B2)
        assert torch.equal(Y1, Y2) and torch.equal(B1, B2), f"worker {i}"
        xs = torch.zeros(w.n + 1, dtype=torch.int32, device=dev)
        xs[1:] = x
        Y3 = torch.empty_like(Y1)
        B3 = torch.empty_like(B1)
        hc.hc_encode_staged(p, plan, ws, xs[1:], Y3, B3)
        assert torch.equal(Y1, Y3) and torch.equal(B1, B3), f"worker {i} unaligned x"
        # and a sketch that is not 16-byte aligned takes the scalar row stores
        Yu = torch.zeros(p.cells + 1, dtype=torch.int32, device=dev)
        hc.hc_encode_staged(p, plan, ws, x, Yu[1:], B3)
        assert torch.equal(Y1, Yu[1:]) and torch.equal(B1, B3), f"worker {i} unaligned y"


def test_staged_plan_for_other_geometry_poisons():
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
    hc.hc_encode_staged(p, bad_plan, hc.alloc_stage_workspace(p, dev), x, Y, B)
    torch.cuda.synchronize()
    assert not Y.any().item()
    assert bool((B == -1).all().item())
    out = torch.empty(w.n, dtype=torch.int32, device=dev)
    info = hc.alloc_info(dev)
    ws = hc.alloc_workspace(p, 0, dev)
    hc.hc_decode(p, Y, B, info, ws, x_out=out)
    torch.cuda.synchronize()
    assert hc.read_info(info).success == 0


@pytest.mark.parametrize("offset", [1, 2, 3])
@pytest.mark.parametrize("path", ["atomic", "staged", "blocked"])
def test_encode_gradient_off_the_16_byte_grid(path, offset):
    # a gradient view 4, 8 or 12 bytes past a 16-byte boundary takes the same
    # 16-byte buffer loads as an aligned one: every worker's sketch and bitmap
    # equal the aligned encode's, bit for bit, also with a ragged tail
    import torch
    hc = _hc()
    dev = torch.device("cuda")
    w = wl.make("synthetic", n=2_000_003, W=2, density=0.02, overlap=0.5, data_seed=500 + offset)
    if path == "blocked":
        g = oracle.blocked_geometry(w.n, w.n_agg, w.hash_seed, 1024, 1.3, 8)
        p = hc.make_params(w.n, g.rows, w.hash_seed, 1024, "i32", block=g.block)
    else:
        p = hc.make_params(w.n, oracle.rows_for(w.n_agg), w.hash_seed, 1024, "i32")
    plan = hc.make_plan(p, dev) if path == "staged" else None
    ws = hc.alloc_stage_workspace(p, dev) if path == "staged" else None
    print(f"[unaligned x] {path} offset={offset} n={w.n} cells={p.cells}", flush=True)
    for i in range(w.W):
        xa = torch.from_numpy(w.dense(i)).to(dev)
        xb = torch.zeros(w.n + offset, dtype=torch.int32, device=dev)
        xb[offset:] = xa
        xu = xb[offset:]
        assert xu.data_ptr() % 16 == 4 * offset
        outs = []
        for x in (xa, xu):
            Y = torch.empty(p.cells, dtype=torch.int32, device=dev)
            B = torch.empty(p.index_words, dtype=torch.int32, device=dev)
            if path == "staged":
                hc.hc_encode_staged(p, plan, ws, x, Y, B)
            else:
                hc.hc_encode(p, x, Y, B)
            torch.cuda.synchronize()
            outs.append((Y.cpu().numpy(), B.cpu().numpy()))
        assert np.array_equal(outs[0][0], outs[1][0]), f"worker {i} sketch"
        assert np.array_equal(outs[0][1], outs[1][1]), f"worker {i} bitmap"
