"""Shared drivers for the parity tests: one run of the three stages through
the C ABI (GPU) and the same run through the CPU oracle, on the same seeded
workload.  The two share only the workload generator."""
from __future__ import annotations

import numpy as np

import oracle


def wrap_sum(arrs):
    acc = np.zeros(arrs[0].shape, np.int64)
    for a in arrs:
        acc += a.astype(np.int64)
    return (acc & 0xFFFFFFFF).astype(np.uint32).view(np.int32)


def oracle_run(w, rows: int, c: int, coo: bool = True, block: int = 0, seed=None,
               bloom_k: int = 0, bloom_rows: int = 0):
    """Oracle encode (per worker), aggregate and decode of workload w (hash
    seed: w's unless given; bloom_k > 0: a Bloom-filter index)."""
    seed = w.hash_seed if seed is None else seed
    g = oracle.Geom(n=w.n, rows=rows, seed=seed, c=c, block=block, bloom_k=bloom_k,
                    bloom_rows=bloom_rows)
    Ys, Bs = [], []
    for i in range(w.W):
        if coo:
            val = w.val[i] if w.vtype == "i32" else w.val[i].astype(np.float64)
            Y, B = oracle.encode_coo(g, w.idx[i], val)
        else:
            x = w.dense(i)
            Y, B = oracle.encode(g, x if w.vtype == "i32" else x.astype(np.float64))
        Ys.append(Y)
        Bs.append(B)
    Ya, Ba = oracle.aggregate(np.stack(Ys), np.stack(Bs))
    x, mask, info = oracle.decode(g, Ya, Ba)
    return dict(g=g, Y=Ys, B=Bs, Ya=Ya, Ba=Ba, x=x, mask=mask, info=info)


def gpu_run(w, rows: int, c: int, coo_input: bool = False, want_coo_out: bool = True,
            max_support: int = 0, keep_workers: bool = True, coo_cap=None, use_plan=False,
            plan=None, block: int = 0, seed=None, bloom_k: int = 0, bloom_rows: int = 0,
            gather: bool = False, staged: bool = False):
    """The same pipeline through libhc on the current GPU.  use_plan builds the
    geometry's inverse row map and decodes with it; `plan` passes one in;
    block > 0 selects the blocked sketch; seed overrides w's hash seed;
    bloom_k > 0 selects a Bloom-filter index; gather encodes the dense
    gradients row by row through a plan (hc_encode_gather); staged stages
    each batch's nonzeros and assembles the rows through a plan
    (hc_encode_staged)."""
    import torch

    import paper_2402_07529_amd as hc
    dev = torch.device("cuda")
    p = hc.make_params(w.n, rows, w.hash_seed if seed is None else seed, c, w.vtype, block=block,
                       bloom_k=bloom_k, bloom_rows=bloom_rows)
    vt = torch.int32 if w.vtype == "i32" else torch.float32
    W = w.W
    Y = torch.empty((W, p.cells), dtype=vt, device=dev)
    B = torch.empty((W, p.index_words), dtype=torch.int32, device=dev)
    enc_plan = hc.make_plan(p, dev) if gather or staged else None
    stage_ws = hc.alloc_stage_workspace(p, dev) if staged else None
    for i in range(W):
        if coo_input:
            idx = torch.from_numpy(w.idx[i].view(np.int32)).to(dev)
            val = torch.from_numpy(w.val[i]).to(dev)
            hc.hc_encode_coo(p, idx, val, Y[i], B[i])
        else:
            x = torch.zeros(w.n, dtype=vt, device=dev)
            x[torch.from_numpy(w.idx[i].astype(np.int64)).to(dev)] = torch.from_numpy(w.val[i]).to(dev)
            if gather:
                hc.hc_encode_gather(p, enc_plan, x, Y[i], B[i])
            elif staged:
                hc.hc_encode_staged(p, enc_plan, stage_ws, x, Y[i], B[i])
            else:
                hc.hc_encode(p, x, Y[i], B[i])
            del x
    Ya = torch.empty(p.cells, dtype=vt, device=dev)
    Ba = torch.empty(p.index_words, dtype=torch.int32, device=dev)
    hc.hc_aggregate(p, Y, B, W, Ya, Ba)
    out = torch.empty(w.n, dtype=vt, device=dev)
    mask = torch.empty(p.words, dtype=torch.int32, device=dev)
    info = hc.alloc_info(dev)
    ws = hc.alloc_workspace(p, max_support, dev)
    cap = w.n if coo_cap is None else coo_cap
    coo_idx = torch.empty(cap, dtype=torch.int32, device=dev) if want_coo_out else None
    coo_val = torch.empty(cap, dtype=vt, device=dev) if want_coo_out else None
    if use_plan and plan is None:
        plan = hc.make_plan(p, dev)
    hc.hc_decode(p, Ya, Ba, info, ws, x_out=out, coo_idx=coo_idx, coo_val=coo_val, mask=mask,
                 max_support=max_support, plan=plan)
    torch.cuda.synchronize()
    inf = hc.read_info(info)
    res = dict(p=p, Ya=Ya.cpu().numpy(), Ba=Ba.cpu().numpy().view(np.uint32),
               x=out.cpu().numpy(), mask=mask.cpu().numpy().view(np.uint32), info=inf)
    if keep_workers:
        res["Y"] = Y.cpu().numpy()
        res["B"] = B.cpu().numpy().view(np.uint32)
    if want_coo_out:
        k = min(inf.n_support, cap)
        res["coo_idx"] = coo_idx[:k].cpu().numpy().view(np.uint32)
        res["coo_val"] = coo_val[:k].cpu().numpy()
    return res
