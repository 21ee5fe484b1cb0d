"""hc_decode_noalloc (the decode whose workspace is the library's static
scratch array) against hc_decode with a caller-allocated workspace, on the
same aggregated sketches: two calls in a row, the second on a smaller input,
so the second runs on scratch that still holds the first call's state.

Bar: int32 outputs (dense gradient, recovered mask, COO, info) bit-exact;
fp32 values within 1e-6 of the largest decoded value, structure exact."""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2402_07529_amd as hc
    return hc


def _aggregate(hc, w, p):
    """Encode every worker of w and aggregate, on the GPU."""
    import torch
    dev = torch.device("cuda")
    vt = torch.int32 if w.vtype == "i32" else torch.float32
    Y = torch.empty((w.W, p.cells), dtype=vt, device=dev)
    B = torch.empty((w.W, p.index_words), dtype=torch.int32, device=dev)
    for i in range(w.W):
        x = torch.from_numpy(w.dense(i)).to(dev)
        hc.hc_encode(p, x, Y[i], B[i])
    Ya = torch.empty(p.cells, dtype=vt, device=dev)
    Ba = torch.empty(p.index_words, dtype=torch.int32, device=dev)
    hc.hc_aggregate(p, Y, B, w.W, Ya, Ba)
    return Ya, Ba


def _decode(hc, p, Ya, Ba, noalloc, max_support, plan):
    import torch
    dev = Ya.device
    vt = Ya.dtype
    out = torch.full((int(p.n),), 7, dtype=vt, device=dev)
    mask = torch.full((p.words,), -1, dtype=torch.int32, device=dev)
    coo_idx = torch.full((int(p.n),), -1, dtype=torch.int32, device=dev)
    coo_val = torch.full((int(p.n),), 7, dtype=vt, device=dev)
    info = hc.alloc_info(dev)
    if noalloc:
        hc.hc_decode_noalloc(p, Ya, Ba, info, x_out=out, coo_idx=coo_idx, coo_val=coo_val,
                             mask=mask, max_support=max_support, plan=plan)
    else:
        ws = hc.alloc_workspace(p, max_support, dev)
        hc.hc_decode(p, Ya, Ba, info, ws, x_out=out, coo_idx=coo_idx, coo_val=coo_val,
                     mask=mask, max_support=max_support, plan=plan)
    torch.cuda.synchronize()
    inf = hc.read_info(info)
    k = int(inf.n_support)
    return dict(x=out.cpu().numpy(), mask=mask.cpu().numpy(), info=inf,
                coo_idx=coo_idx[:k].cpu().numpy(), coo_val=coo_val[:k].cpu().numpy())


def _compare(a, b, f32):
    assert a["info"] == b["info"]
    assert np.array_equal(a["mask"], b["mask"])
    assert np.array_equal(a["coo_idx"], b["coo_idx"])
    if not f32:
        assert np.array_equal(a["x"], b["x"])
        assert np.array_equal(a["coo_val"], b["coo_val"])
        return
    scale = max(float(np.max(np.abs(b["x"]))), 1e-30)
    assert np.max(np.abs(a["x"].astype(np.float64) - b["x"])) <= 1e-6 * scale
    assert np.max(np.abs(a["coo_val"].astype(np.float64) - b["coo_val"])) <= 1e-6 * scale


def _case(hc, w, kind):
    if kind == "blocked":
        p = hc.hc_geometry_blocked(w.n, w.n_agg, 1.3, 1024, 0, w.hash_seed, w.vtype)
    else:
        p = hc.hc_geometry(w.n, w.n_agg, hc.GAMMA, 1024, w.hash_seed, w.vtype)
    max_support = 0 if kind == "blocked" else w.n_agg
    _, _, need = hc.hc_sizes(p, max_support)
    assert need <= hc.NOALLOC_SCRATCH_BYTES, (kind, need)
    plan = hc.make_plan(p) if kind == "plan" else None
    return p, max_support, plan


@pytest.mark.parametrize("vtype", ["i32", "f32"])
@pytest.mark.parametrize("kind", ["global", "plan", "blocked"])
def test_noalloc_decode_matches_decode_twice(vtype, kind):
    hc = _hc()
    # first a larger input (several thousand sketch rows, ragged n), then a
    # smaller one: the second call runs on the first call's leftover scratch
    big = wl.make("synthetic", vtype, n=6_000_011, W=4, density=0.02, overlap=0.5,
                  data_seed=31, hash_seed=32)
    small = wl.make("tiny", vtype)
    for w in (big, small):
        print(f"noalloc {kind} {vtype} n={w.n} n_agg={w.n_agg}", flush=True)
        p, max_support, plan = _case(hc, w, kind)
        Ya, Ba = _aggregate(hc, w, p)
        ref = _decode(hc, p, Ya, Ba, False, max_support, plan)
        got = _decode(hc, p, Ya, Ba, True, max_support, plan)
        assert ref["info"].n_support == w.n_agg
        _compare(got, ref, vtype == "f32")


def test_noalloc_decode_rejects_oversized_workspace():
    hc = _hc()
    import torch
    p = hc.hc_geometry(1 << 28, 10_000_000, hc.GAMMA, 1024, 5, "i32")
    _, _, need = hc.hc_sizes(p, 10_000_000)
    assert need > hc.NOALLOC_SCRATCH_BYTES
    Ya = torch.zeros(p.cells, dtype=torch.int32, device="cuda")
    Ba = torch.zeros(p.words, dtype=torch.int32, device="cuda")
    info = hc.alloc_info()
    with pytest.raises(hc.HCError) as e:
        hc.hc_decode_noalloc(p, Ya, Ba, info, max_support=10_000_000)
    assert e.value.status == hc.HC_EWORKSPACE
