"""Repeated decodes of one aggregated sketch (section 3.2 peeling).

The peel kernel hands each round's frontier, counters and residuals to the
next round through coherent memory operations and a grid barrier whose fences
are workgroup-scope; a value that crossed a round boundary stale would change
the recovered set, the values or the round count.  Every one of many decodes
of the same aggregate must therefore equal the oracle's (int32, bit-exact,
rounds included) or the first decode (fp32: the smallest-j rule makes the
decode independent of the order of the entries, so repeats are bit-identical).
Sizes: a sketch peeled on half the CUs with round 0 in the peel kernel, and a
full-size VGG19-shaped sketch peeled on three quarters of the CUs after round
0 by rows."""
import numpy as np
import pytest

import oracle
import workloads as wl
from hc_pipeline import wrap_sum
from test_gpu_parity import assert_same_info

pytestmark = pytest.mark.gpu


def _hc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2402_07529_amd as hc
    return hc


def _aggregate(hc, w, p):
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


def _decodes(hc, p, Ya, Ba, plan, max_support, reps):
    """reps decodes into the same buffers (poisoned before each one)."""
    import torch
    dev = Ya.device
    out = torch.empty(int(p.n), dtype=Ya.dtype, device=dev)
    mask = torch.empty(p.words, dtype=torch.int32, device=dev)
    info = hc.alloc_info(dev)
    ws = hc.alloc_workspace(p, max_support, dev)
    for k in range(reps):
        out.fill_(7)
        mask.fill_(-1)
        hc.hc_decode(p, Ya, Ba, info, ws, x_out=out, mask=mask, max_support=max_support,
                     plan=plan)
        torch.cuda.synchronize()
        yield k, out.cpu().numpy(), mask.cpu().numpy(), hc.read_info(info)


@pytest.mark.parametrize("kind", ["i32_plan", "i32_noplan", "f32_plan"])
def test_peel_repeat_half_grid(kind):
    import torch
    hc = _hc()
    vt = "f32" if kind.startswith("f32") else "i32"
    w = wl.make("synthetic", n=6_000_011, W=4, density=0.01, overlap=0.5, data_seed=77,
                vtype=vt)
    p = hc.hc_geometry(w.n, w.n_agg, hc.GAMMA, 1024, w.hash_seed, vt)
    plan = hc.make_plan(p, torch.device("cuda")) if kind.endswith("_plan") else None
    Ya, Ba = _aggregate(hc, w, p)
    print(f"[peel repeat] {kind} n={w.n} cells={p.cells} support={w.n_agg}", flush=True)
    if vt == "i32":
        ox, omask, oinfo = oracle.decode(
            oracle.Geom(n=w.n, rows=int(p.rows), seed=w.hash_seed, c=1024),
            Ya.cpu().numpy(), Ba.cpu().numpy().view(np.uint32))
        assert oinfo.success
    first = None
    for k, x, mask, info in _decodes(hc, p, Ya, Ba, plan, w.n_agg, 12):
        if vt == "i32":
            assert np.array_equal(x, ox), f"decode {k}"
            assert np.array_equal(mask.view(np.uint32), omask.view(np.uint32)), f"decode {k}"
            assert_same_info(info, oinfo)
        elif first is None:
            first = (x.copy(), mask.copy(), info)
            assert info.success
        else:
            assert np.array_equal(x.view(np.uint32), first[0].view(np.uint32)), f"decode {k}"
            assert np.array_equal(mask, first[1]), f"decode {k}"
            assert info == first[2], f"decode {k}"


@pytest.mark.timeout(900)
def test_peel_repeat_vgg19_fullsize():
    # full-size VGG19 gradients at 1 % density: 10.4 M cells, peeled on three
    # quarters of the CUs after round 0 by rows (the plan); every decode
    # recovers everything, equals the direct sum and takes the same rounds
    import torch
    hc = _hc()
    w = wl.make("vgg19")
    p = hc.hc_geometry(w.n, w.n_agg, hc.GAMMA, 1024, w.hash_seed, "i32")
    plan = hc.make_plan(p, torch.device("cuda"))
    Ya, Ba = _aggregate(hc, w, p)
    direct = wrap_sum([w.dense(i) for i in range(w.W)])
    print(f"[peel repeat] vgg19 n={w.n} cells={p.cells} support={w.n_agg}", flush=True)
    first = None
    for k, x, mask, info in _decodes(hc, p, Ya, Ba, plan, w.n_agg, 8):
        assert info.success, f"decode {k}"
        assert np.array_equal(x, direct), f"decode {k}"
        if first is None:
            first = (mask.copy(), info)
        else:
            assert np.array_equal(mask, first[0]), f"decode {k}"
            assert info == first[1], f"decode {k}"
