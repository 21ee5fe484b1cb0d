"""Throughput of one simulated aggregation iteration on one MI355X.

One step = W worker encodes of dense gradients (hc_encode), the W-way
aggregation (hc_aggregate) and the peeling decode to a dense gradient
(hc_decode), all through the C ABI, inputs resident in HBM.  The metric is
dense-gradient GB/s: the aggregated gradient's 4N bytes counted once per
iteration (the paper's convention for aggregation throughput, section 4.2),
divided by the iteration time.

Prints ONE JSON line.  Default workload: the NCF-shaped embedding gradient
(2^24 rows x 64 dims, 8 workers, 4096 Zipf rows each, int32 fixed point).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "encode+aggregate+decode dense-gradient GB/s at 1 GPU; % HBM peak; decode success"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MALL_BYTES = 256 * 2**20  # MI355X Infinity Cache (memory-attached last level)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="ncf", choices=["tiny", "ncf", "lstm", "vgg19", "bert"])
    ap.add_argument("--vtype", default="i32", choices=["i32", "f32"])
    ap.add_argument("--density", type=float, default=None)
    ap.add_argument("--overlap", type=float, default=None)
    ap.add_argument("--workers", type=int, default=None,
                    help="simulated workers W (default: the configuration's)")
    ap.add_argument("--ratio", type=float, default=None,
                    help="sketch cells / aggregate nonzeros (default: gamma = 1.23)")
    ap.add_argument("--c", type=int, default=1024)
    ap.add_argument("--index", default="bitmap", choices=["bitmap", "bloom"],
                    help="index of the nonzeros: the bitmap (section 3.2) or a Bloom filter sized "
                         "by section 3.3 (global sketch only)")
    ap.add_argument("--blocked", action="store_true",
                    help="blocked sketch (section 3.2 blocking), one block per workgroup in LDS; "
                         "default ratio 1.3")
    ap.add_argument("--block-rows", type=int, default=None,
                    help="rows per block of the blocked sketch (default: the library's choice "
                         "for this device, hc_geometry_blocked with block_rows = 0)")
    ap.add_argument("--encode", default="auto", choices=["auto", "atomic", "gather", "staged"],
                    help="auto: staged for a global sketch with c >= 256 when a worker has at "
                         "least two nonzeros per batch of c parameters (else the atomic "
                         "encode, whose cost follows the nonzeros while the staged encode's "
                         "second pass visits every batch); atomic: hc_encode (each nonzero adds "
                         "into its cells); gather: "
                         "hc_encode_gather (each sketch row assembled through the plan from "
                         "the gradient; global sketch, bitmap index, c >= 256); staged: "
                         "hc_encode_staged (nonzeros staged per batch, rows assembled through "
                         "the plan; global sketch, c >= 256)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", nargs="?", const="bert", choices=["bert", "compressed"],
                    help="bert: BERT-base density/overlap grid and sketch-width sweep; "
                         "compressed: one worker's compress + decompress over sketch sizes of 2 %% "
                         "to 200 %% of a VGG19-shaped gradient at its natural 69.6 %% density "
                         "(section 4.1's microbenchmark); one JSON object")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 10 times (the known-size kernel "
                         "against which the HBM byte counters are scaled)")
    return ap.parse_args()


def copy_calibration():
    """A plain copy of 1 GiB (2^30 bytes read, 2^30 written) ten times."""
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(2**28, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": 2**30, "copy_calibration_bytes_written": 2**30,
                      "launches": 10}), flush=True)


def make_workload(a):
    import workloads as wl
    kw = {}
    if a.density is not None:
        kw["density"] = a.density
    if a.overlap is not None:
        kw["overlap"] = a.overlap
    if a.workers is not None:
        kw["W"] = a.workers
    return wl.make(a.config, vtype=a.vtype, **kw)


def algorithmic_bytes(n, W, cells, n_sup, index_bytes, blocked=False):
    """Bytes the method must move per stage (reads + writes of HBM).
    index_bytes: the index B (the n-bit bitmap, or a Bloom filter, which the
    decode first probes into an n-bit candidate bitmap)."""
    words_b = (n + 31) // 32 * 4
    enc = 4 * n + index_bytes + 4 * cells                  # read x, write B, clear/write Y
    agg = (W + 1) * (4 * cells + index_bytes)              # W sketches+indexes in, one out
    probe = 0 if index_bytes == words_b else index_bytes + words_b
    if blocked:
        dec = words_b + 4 * cells + 4 * n                  # B, Y, dense out (blocks peel in LDS)
    else:
        dec = probe + words_b + 4 * cells + 8 * n_sup + 4 * n  # B, Y, element list+values, out
    return enc, agg, dec


def measured_traffic(tag, mode, vtype):
    """HBM bytes per encode call (all of its kernels) from the committed
    rocprofv3 counter summary profiles/hbm_counters_<line>_<mode>.md
    (FETCH_SIZE and WRITE_SIZE runs scaled by a plain copy of known size), or
    None if there is none for this line or the encode's sources changed since
    the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"hbm_counters_{tag}_{mode}.md")
    if vtype != "i32" or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "kernel_source_sha256"):
            k, v = line.split(":", 1)
            fields[k] = v.strip()
    if fields.get("kernel_source_sha256") != encode_source_sha256(mode):
        return None
    return int(fields["traffic_bytes_per_launch"])


def line_tag(a, w):
    """The workload's name, plus the density, overlap and worker count when
    they were given on the command line (names the counter summaries)."""
    tag = w.name
    for flag, v in (("d", a.density), ("o", a.overlap), ("w", a.workers)):
        if v is not None:
            tag += f"_{flag}{v}"
    return tag


def encode_source_sha256(mode):
    """sha256 of the sources an encode mode's kernels are built from (a
    blocked sketch with fewer blocks than CUs is encoded by the dense kernels)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2402_07529_amd", "csrc")
    files = ["hc_blocked.hip", "hc_encode.hip"] if mode == "blocked" else ["hc_encode.hip"]
    src = b"".join(open(os.path.join(csrc, f), "rb").read() for f in files + ["hc_device.h"])
    return hashlib.sha256(src).hexdigest()


def host_cpu():
    """(CPU model, logical CPUs of the host, CPUs this process may run on)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return model, os.cpu_count(), usable


def cpu_baseline(w, rows, c, block, seed, min_s=10.0, max_reps=4):
    """The CPU oracle, as it stands, on whole iterations of the same workload:
    every worker's dense encode, the W-way aggregate and the decode, each
    timed (building a worker's dense input is not).  Iterations repeat until
    `min_s` seconds of oracle work have been timed, at most `max_reps` of
    them, and the median iteration is reported."""
    import oracle
    g = oracle.Geom(n=w.n, rows=rows, seed=seed, c=c, block=block)
    dt = np.int32 if w.vtype == "i32" else np.float64
    its, info = [], None
    while not its or (sum(t[0] for t in its) < min_s and len(its) < max_reps):
        Ys, Bs, t_enc = None, None, 0.0
        for i in range(w.W):
            x = w.dense(i).astype(dt, copy=False)
            t0 = time.perf_counter()
            Y, B = oracle.encode(g, x)
            t_enc += time.perf_counter() - t0
            del x
            if Ys is None:
                Ys = np.empty((w.W,) + Y.shape, Y.dtype)
                Bs = np.empty((w.W,) + B.shape, B.dtype)
            Ys[i], Bs[i] = Y, B
        t0 = time.perf_counter()
        Ya, Ba = oracle.aggregate(Ys, Bs)
        t_agg = time.perf_counter() - t0
        del Ys, Bs
        t0 = time.perf_counter()
        _, _, info = oracle.decode(g, Ya, Ba)
        t_dec = time.perf_counter() - t0
        its.append((t_enc + t_agg + t_dec, t_enc, t_agg, t_dec))
    t_iter, t_enc, t_agg, t_dec = sorted(its)[len(its) // 2]
    model, nproc, usable = host_cpu()
    return dict(value=round(4 * w.n / t_iter / 1e9, 4), unit="GB/s", cores=1, kind="oracle",
                cpu_model=model, nproc=nproc, cpus_usable=usable,
                sample=(f"{w.name}: {len(its)} whole iterations, {sum(t[0] for t in its):.1f} s "
                        f"timed; the median: {w.W} dense encodes {t_enc:.2f} s, aggregate "
                        f"{t_agg:.2f} s, decode {t_dec:.2f} s; single-threaded C"),
                success=int(info.success), rounds=int(info.rounds))


def auto_encode(w, c, blocked):
    """The encode 'auto' picks: staged for a global sketch with c >= 256 when a
    worker has at least two nonzeros per batch of c parameters (its second
    pass visits every batch), else the atomic encode.  Measured on MI355X at
    c = 1024 (per worker, BERT-base / VGG19 shapes): 2 per batch 0.098 / 0.126
    ms atomic against 0.095 / 0.125 staged; 4 per batch 0.114 / 0.146 against
    0.098 / 0.127; 1 per batch (BERT-base, Bloom index) 0.124 against 0.156."""
    nnz_w = float(np.mean([w.nnz(i) for i in range(w.W)]))
    batches = (w.n + c - 1) // c
    return "staged" if not blocked and c >= 256 and nnz_w >= 2 * batches else "atomic"


def core_fraction(lam):
    """Edges left in the 2-core of a random 3-uniform hypergraph with lam edges
    per vertex (x^3 for the largest root of x = 1 - exp(-3 lam x^2)); the
    textbook prediction of the unpeeled fraction."""
    xs = np.linspace(1e-9, 1.0, 200001)
    f = xs - (1 - np.exp(-3 * lam * xs**2))
    idx = np.nonzero(np.sign(f[:-1]) != np.sign(f[1:]))[0]
    if idx.size == 0:
        return 0.0
    lo, hi = xs[idx[-1]], xs[idx[-1] + 1]
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        if (mid - (1 - np.exp(-3 * lam * mid * mid))) * (lo - (1 - np.exp(-3 * lam * lo * lo))) > 0:
            lo = mid
        else:
            hi = mid
    return float(lo) ** 3


class Runner:
    """Device buffers of one workload and the timed W-encode + aggregate +
    decode iteration through the C ABI."""

    def __init__(self, w, c, dev):
        import torch
        self.torch = torch
        self.w, self.c, self.dev = w, c, dev
        self.vt = torch.int32 if w.vtype == "i32" else torch.float32
        # each worker's gradient starts on a 256-byte boundary, as separate
        # per-worker buffers would (the rows of one (W, n) tensor start off
        # the 16-byte grid when n mod 4 != 0, as LSTM's n does)
        n_pad = (w.n + 63) // 64 * 64
        self.x_rows = torch.zeros((w.W, n_pad), dtype=self.vt, device=dev)
        self.x = self.x_rows[:, :w.n]
        for i in range(w.W):
            self.x[i][torch.from_numpy(w.idx[i].astype(np.int64)).to(dev)] = \
                torch.from_numpy(w.val[i]).to(dev)
        self.n_agg = w.n_agg
        self.out = torch.empty(w.n, dtype=self.vt, device=dev)
        self.mask = torch.empty((w.n + 31) // 32, dtype=torch.int32, device=dev)

    def run(self, ratio, steps, warmup, check=True, block_rows=None, bloom=False, gather=False,
            staged=False):
        """block_rows: None for the global sketch, else the rows per block of
        a blocked sketch; bloom: a Bloom-filter index instead of the bitmap;
        gather: encode row by row through the plan (hc_encode_gather);
        staged: stage each batch's nonzeros, then assemble the rows through
        the plan (hc_encode_staged)."""
        import paper_2402_07529_amd as hc
        torch, w, dev, W = self.torch, self.w, self.dev, self.w.W
        max_support = self.n_agg
        if bloom:
            p, _ = hc.hc_geometry_bloom(w.n, self.n_agg, ratio, self.c, w.hash_seed, w.vtype)
            # room for four times the filter's expected false positives
            max_support = int(self.n_agg + 4 * 2.0**-int(p.bloom_k) * (w.n - self.n_agg)) + 1024
        elif block_rows is None:
            p = hc.hc_geometry(w.n, self.n_agg, ratio, self.c, w.hash_seed, w.vtype)
        else:
            p = hc.hc_geometry_blocked(w.n, self.n_agg, ratio, self.c, block_rows, w.hash_seed,
                                       w.vtype)
        cells, words = p.cells, p.index_words
        Y = torch.empty((W, cells), dtype=self.vt, device=dev)
        B = torch.empty((W, words), dtype=torch.int32, device=dev)
        Ya = torch.empty(cells, dtype=self.vt, device=dev)
        Ba = torch.empty(words, dtype=torch.int32, device=dev)
        info = hc.alloc_info(dev)
        ws = hc.alloc_workspace(p, max_support, dev)
        stream = torch.cuda.current_stream()
        # the inverse row map depends only on the geometry: built once, like
        # the sketch geometry itself, before any iteration
        torch.cuda.synchronize()
        t_plan = time.perf_counter()
        plan = hc.make_plan(p, dev) if self.c >= 256 and block_rows is None else None
        torch.cuda.synchronize()
        plan_ms = (time.perf_counter() - t_plan) * 1e3
        stage_ws = hc.alloc_stage_workspace(p, dev) if staged else None
        x, out, mask = self.x, self.out, self.mask

        def step(ev=None):
            if ev is not None:
                ev[0].record(stream)
            for i in range(W):
                if gather:
                    hc.hc_encode_gather(p, plan, x[i], Y[i], B[i], stream)
                elif staged:
                    hc.hc_encode_staged(p, plan, stage_ws, x[i], Y[i], B[i], stream)
                else:
                    hc.hc_encode(p, x[i], Y[i], B[i], stream)
            if ev is not None:
                ev[1].record(stream)
            hc.hc_aggregate(p, Y, B, W, Ya, Ba, stream)
            if ev is not None:
                ev[2].record(stream)
            hc.hc_decode(p, Ya, Ba, info, ws, x_out=out, mask=mask, max_support=max_support,
                         stream=stream, plan=plan)
            if ev is not None:
                ev[3].record(stream)

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for k in range(steps):
            step(evs[k])
        stop.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / steps
        step_ms = [e[0].elapsed_time(e[3]) for e in evs]
        enc_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) / W
        agg_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
        dec_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
        inf = hc.read_info(info)
        # the decode alone without the plan (per-cell counters by atomics), for
        # a geometry that changes every iteration and so cannot reuse a plan
        dec_noplan_ms = None
        if plan is not None:
            info2 = hc.alloc_info(dev)
            dev_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            times = []
            for k in range(max(steps // 2, 2) + 1):
                dev_ev[0].record(stream)
                hc.hc_decode(p, Ya, Ba, info2, ws, x_out=out, mask=mask,
                             max_support=max_support, stream=stream)
                dev_ev[1].record(stream)
                torch.cuda.synchronize()
                if k > 0:
                    times.append(dev_ev[0].elapsed_time(dev_ev[1]))
            dec_noplan_ms = float(np.median(times))
            assert hc.read_info(info2) == inf, "decode without a plan differs"
            # the timed iterations' outputs again (the check below reads them)
            hc.hc_decode(p, Ya, Ba, info, ws, x_out=out, mask=mask, max_support=max_support,
                         stream=stream, plan=plan)
            torch.cuda.synchronize()
        exact = None
        if check:
            # correctness of the timed result against the direct sum of the inputs
            direct = x.sum(dim=0, dtype=torch.int64 if self.vt == torch.int32 else torch.float64)
            if self.vt == torch.int32:
                direct = ((direct + 2**31) % 2**32 - 2**31).to(torch.int32)
                exact = bool(torch.equal(out, direct)) if inf.success else False
            else:
                exact = bool((out.double() - direct).abs().max().item() <=
                             1e-5 * direct.abs().max().item()) if inf.success else False
            del direct
        return dict(p=p, ms=ms, enc_ms=enc_ms, agg_ms=agg_ms, dec_ms=dec_ms, info=inf,
                    exact=exact, plan_ms=plan_ms, step_ms=step_ms, dec_noplan_ms=dec_noplan_ms,
                    ws_bytes=int(ws.numel()))


# sketch sizes (cells / n) of section 4.1's microbenchmark, 2 % to 200 %, with
# the threshold 1.23 x 0.696 = 85.6 % among them
COMPRESSED_SIZES = (0.02, 0.05, 0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.856, 0.9, 1.0, 1.2,
                    1.5, 2.0)


def sweep_compressed(a, dev):
    """Section 4.1's microbenchmark on one worker: a VGG19-shaped gradient at
    its natural density (69.6 % nonzero, Table 1) compressed to sketches of 2 %
    to 200 % of its size and decompressed at once.  Per size: the average
    relative error |x_hat - x| / |x| over the nonzeros, the recovery rate
    (fraction recovered by peeling), the recovery iterations (rounds), and the
    compress + decompress throughput of the single worker (the paper's
    single-worker, single-GPU aggregation throughput)."""
    import workloads as wl
    w = wl.make("vgg19", vtype=a.vtype, W=1, density=0.696)
    r = Runner(w, 1024, dev)
    x = r.x[0].double()
    nz = x != 0
    absx = x[nz].abs()
    points = []
    for frac in COMPRESSED_SIZES:
        # the atomic encode first, for its time alone; then the timed run with
        # the encode gathered through the plan, which suits a dense gradient
        atomic_ms = r.run(frac * w.n / r.n_agg, 3, 1, check=False)["enc_ms"]
        m = r.run(frac * w.n / r.n_agg, 3, 1, check=False, gather=True)
        inf = m["info"]
        err = ((r.out.double()[nz] - x[nz]).abs() / absx).mean().item()
        t = m["enc_ms"] + m["dec_ms"]  # W = 1: the aggregate of one sketch is a copy
        pt = dict(compressed_size=frac, cells=m["p"].cells,
                  index_bytes_frac=round(4 * m["p"].index_words / (4 * w.n), 4),
                  avg_relative_error=err,
                  recovery_rate=round(inf.n_recovered / max(inf.n_support, 1), 6),
                  recovery_iterations=inf.rounds, success=inf.success,
                  encode_ms=round(m["enc_ms"], 4), encode_atomic_ms=round(atomic_ms, 4),
                  decode_ms=round(m["dec_ms"], 4),
                  compress_decompress_gbs=round(4 * w.n / (t * 1e-3) / 1e9, 2))
        log(f"[sweep] {pt}")
        points.append(pt)
    print(json.dumps({"sweep": "compressed-size", "workload": "vgg19 natural density",
                      "n": w.n, "nonzeros": r.n_agg, "dtype": "int32" if w.vtype == "i32" else "fp32",
                      "points": points}), flush=True)


def sweep(a, dev):
    """BERT-base: density x overlap grid at gamma = 1.23, then sketch widths
    around gamma at 1 % / 50 % overlap, to chart the decode-failure boundary
    against the 2-core closed form."""
    import workloads as wl
    points = []
    for density in (0.001, 0.01, 0.05):
        for overlap in (0.1, 0.3, 0.5, 0.7, 0.9):
            w = wl.make("bert", density=density, overlap=overlap)
            r = Runner(w, 1024, dev)
            enc = auto_encode(w, 1024, False)
            m = r.run(1.23, 3, 1, staged=enc == "staged")
            inf = m["info"]
            pt = dict(kind="density_overlap", density=density, overlap=overlap, n_agg=r.n_agg,
                      encode=enc,
                      ratio=round(m["p"].cells / r.n_agg, 4), value=round(4 * w.n / m["ms"] / 1e6, 2),
                      ms_per_step=round(m["ms"], 4), encode_ms=round(m["enc_ms"], 4),
                      aggregate_ms=round(m["agg_ms"], 4), decode_ms=round(m["dec_ms"], 4),
                      success=inf.success, rounds=inf.rounds,
                      recovered_frac=round(inf.n_recovered / max(inf.n_support, 1), 6),
                      equals_direct_sum=m["exact"])
            log(f"[sweep] {pt}")
            points.append(pt)
            del r
    w = wl.make("bert", density=0.01, overlap=0.5)
    r = Runner(w, 1024, dev)
    enc = auto_encode(w, 1024, False)
    for ratio in (1.10, 1.15, 1.20, 1.22, 1.23, 1.25, 1.30, 1.50, 2.00):
        m = r.run(ratio, 2, 1, check=False, staged=enc == "staged")
        inf = m["info"]
        lam = r.n_agg / m["p"].cells
        pt = dict(kind="width", density=0.01, overlap=0.5, ratio=round(m["p"].cells / r.n_agg, 4),
                  success=inf.success, rounds=inf.rounds,
                  unpeeled_frac=round(1 - inf.n_recovered / max(inf.n_support, 1), 6),
                  predicted_unpeeled=round(core_fraction(lam), 6),
                  decode_ms=round(m["dec_ms"], 4), ms_per_step=round(m["ms"], 4))
        log(f"[sweep] {pt}")
        points.append(pt)
    print(json.dumps({"sweep": "bert-base", "points": points}), flush=True)


def main():
    a = parse()
    if a.copy_calibration:
        copy_calibration()
        return
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (the W workers are simulated on it); "
              f"--gpus {a.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if a.sweep == "compressed":
        sweep_compressed(a, dev)
        return
    if a.sweep:
        sweep(a, dev)
        return

    import paper_2402_07529_amd as hc
    t0 = time.perf_counter()
    w = make_workload(a)
    block_rows = None
    ratio = a.ratio if a.ratio is not None else (1.3 if a.blocked else hc.GAMMA)
    if a.blocked:
        block_rows = a.block_rows or 0  # 0: the library's choice for this device
    log(f"[bench] workload {w.name} n={w.n} W={w.W} gen {time.perf_counter() - t0:.1f}s")
    r = Runner(w, a.c, dev)
    if a.index == "bloom" and a.blocked:
        print("bench.py: the Bloom-filter index needs the global sketch", file=sys.stderr)
        sys.exit(2)
    encode = a.encode
    if encode == "auto":
        encode = auto_encode(w, a.c, a.blocked)
    gather = encode == "gather"
    staged = encode == "staged"
    if gather and (a.blocked or a.index == "bloom" or a.c < 256):
        print("bench.py: --encode gather needs the global sketch, the bitmap index and c >= 256",
              file=sys.stderr)
        sys.exit(2)
    if staged and (a.blocked or a.c < 256):
        print("bench.py: --encode staged needs the global sketch and c >= 256", file=sys.stderr)
        sys.exit(2)
    m = r.run(ratio, a.steps, a.warmup, block_rows=block_rows, bloom=a.index == "bloom",
              gather=gather, staged=staged)
    p, inf, W, n_agg = m["p"], m["info"], w.W, r.n_agg
    ms, enc_ms, agg_ms, dec_ms = m["ms"], m["enc_ms"], m["agg_ms"], m["dec_ms"]
    cells = p.cells

    enc_b, agg_b, dec_b = algorithmic_bytes(w.n, W, cells, inf.n_support, 4 * p.index_words,
                                            a.blocked)
    iter_b = W * enc_b + agg_b + dec_b
    value = 4 * w.n / (ms * 1e-3) / 1e9
    nnz_w = float(np.mean([w.nnz(i) for i in range(W)]))  # nonzeros one worker encodes
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    enc_gbs = enc_b / (enc_ms * 1e-3) / 1e9
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "GB/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32" if w.vtype == "i32" else "fp32", "data": "synthetic",
        "config": {"workload": w.name, "n": w.n, "workers": W, "n_agg": n_agg,
                   "rows": int(p.rows), "c": int(p.c), "cells": cells, "ratio": round(cells / max(n_agg, 1), 4),
                   "sketch": (f"blocked: {int(p.block)} batches and {p.block_rows} rows per block, "
                              f"{p.nblocks} blocks") if a.blocked else "global",
                   "index": (f"bloom: {int(p.bloom_k)} hashes, {4 * p.index_words} bytes"
                             if a.index == "bloom" else "bitmap"),
                   "encode": encode,
                   **{k: v for k, v in w.params.items() if k in ("density", "overlap", "rows_per_worker")}},
        "roofline": {"bound": "hbm",
                     "kernel": (("hc_encode (blocked LDS encode)" if p.nblocks >= cus else
                                 "hc_encode (blocked sketch, fewer blocks than CUs: Y clear + "
                                 "dense encode over the whole GPU)") if a.blocked
                                else "hc_encode_gather (rows through the plan)" if gather
                                else "hc_encode_staged (staging pass + rows through the plan)"
                                if staged else "hc_encode (Y clear + dense encode)"),
                     "achieved": round(enc_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(enc_gbs / HBM_PEAK_GBS, 4),
                     "traffic": (None if a.index == "bloom" else
                                 measured_traffic(line_tag(a, w), "blocked" if a.blocked
                                                  else encode, w.vtype)),
                     "bytes_per_launch": enc_b, "avg_launch_ms": round(enc_ms, 4)},
        "ms_per_step_median": round(float(np.median(m["step_ms"])), 4),
        "hbm_frac_iteration": round(iter_b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "stages_ms": {"encode_per_worker": round(enc_ms, 4), "aggregate": round(agg_ms, 4),
                      "decode": round(dec_ms, 4)},
        "stages_gbs_dense": {"encode": round(4 * w.n / (enc_ms * 1e-3) / 1e9, 1),
                             "aggregate": round(4 * w.n / (agg_ms * 1e-3) / 1e9, 1),
                             "decode": round(4 * w.n / (dec_ms * 1e-3) / 1e9, 1)},
        # nonzeros handled per second: one worker's nonzeros per encode, the
        # aggregate's nonzeros for the aggregate and the decode
        "stages_nonzeros_per_s": {"encode": round(nnz_w / (enc_ms * 1e-3), 1),
                                  "aggregate": round(n_agg / (agg_ms * 1e-3), 1),
                                  "decode": round(n_agg / (dec_ms * 1e-3), 1)},
        "plan_build_ms_once": round(m["plan_ms"], 3),
        "decode_ms_without_plan": (round(m["dec_noplan_ms"], 4) if m["dec_noplan_ms"] is not None
                                   else None),
        # whether the sketch (and the decode's working set) fit the 256 MiB
        # Infinity Cache that backs HBM; the W dense inputs never do
        "mall": {"capacity_bytes": MALL_BYTES, "sketch_bytes": 4 * cells,
                 "sketch_resident": 4 * cells <= MALL_BYTES,
                 "all_worker_sketches_resident": W * (4 * cells + 4 * p.index_words) <= MALL_BYTES,
                 "decode_workspace_bytes": m["ws_bytes"],
                 "decode_workspace_resident": m["ws_bytes"] + 4 * cells <= MALL_BYTES},
        "decode": {"success": inf.success, "n_support": inf.n_support,
                   "n_recovered": inf.n_recovered, "rounds": inf.rounds, "status": inf.status,
                   "equals_direct_sum": m["exact"]},
    }
    del r
    torch.cuda.empty_cache()
    if not a.no_cpu_baseline and a.index == "bloom":
        # the oracle's filter query visits every parameter with every hash: far
        # beyond the bounded sample the baseline is meant to take
        log("[bench] no CPU baseline for the Bloom-filter index")
    elif not a.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        res["cpu_baseline"] = cpu_baseline(w, int(p.rows), int(p.c), int(p.block), int(p.seed))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
