"""Seeded synthetic gradients shaped like the paper's workloads.

This module only draws inputs: supports (which parameters are nonzero on each
worker) and their values.  It holds none of the compression method's
arithmetic, so both the CPU oracle and the GPU path can take their inputs from
it.  The paper trains NCF, LSTM, VGG19 and BERT-base (section 4, Table 1); none
of those datasets or trained weights are used here.  Instead each workload is a
per-tensor gradient layout of that model's shape with seeded random supports:

* shared-pool overlap (all but NCF): per tensor of m parameters and density d,
  each worker has n_w = round(d*m) nonzeros; s = round(o*n_w) of them are drawn
  once and shared by every worker, the other n_w - s are private to the worker
  (disjoint across workers), so the aggregate has s + W*(n_w - s) nonzeros;
* NCF: each worker touches 4096 distinct rows of a 2^24 x 64 embedding table,
  rows drawn by Zipf(s=1.1) rank through a seeded bijection of row ids, every
  element of a touched row nonzero;
* values: N(0, sigma) per worker and index; the int32 path quantizes them to
  fixed point at scale 2^20 (round half to even, saturating to +-(2^31-1)) and
  redraws any value that would be 0, so the dense and COO supports agree.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

FIXED_POINT_SCALE = 2.0 ** 20
INT32_MAX = 2**31 - 1

# ------------------------------------------------------------ model layouts

def lstm_tensors():
    """2-layer LSTM, hidden 1500, tied 33,278-word embedding (85,974,278)."""
    t = [("embedding", 33278 * 1500)]
    for layer in range(2):
        t += [(f"l{layer}.w_ih", 6000 * 1500), (f"l{layer}.w_hh", 6000 * 1500),
              (f"l{layer}.b_ih", 6000), (f"l{layer}.b_hh", 6000)]
    t += [("decoder.bias", 33278)]
    return t


def vgg19_tensors():
    """VGG19: 16 conv 3x3 layers and 3 FC layers with biases (143,667,240)."""
    chans = [(3, 64), (64, 64), (64, 128), (128, 128), (128, 256), (256, 256), (256, 256),
             (256, 256), (256, 512), (512, 512), (512, 512), (512, 512), (512, 512),
             (512, 512), (512, 512), (512, 512)]
    t = []
    for i, (ci, co) in enumerate(chans):
        t += [(f"conv{i}.w", ci * co * 9), (f"conv{i}.b", co)]
    for i, (fi, fo) in enumerate([(25088, 4096), (4096, 4096), (4096, 1000)]):
        t += [(f"fc{i}.w", fi * fo), (f"fc{i}.b", fo)]
    return t


def bert_base_tensors():
    """BERT-base encoder with embeddings and pooler, no task head (109,482,240)."""
    h, f = 768, 3072
    t = [("emb.word", 30522 * h), ("emb.pos", 512 * h), ("emb.type", 2 * h), ("emb.ln", 2 * h)]
    for layer in range(12):
        p = f"l{layer}."
        for name in ("q", "k", "v", "o"):
            t += [(p + name + ".w", h * h), (p + name + ".b", h)]
        t += [(p + "attn_ln", 2 * h), (p + "ffn1.w", h * f), (p + "ffn1.b", f),
              (p + "ffn2.w", f * h), (p + "ffn2.b", h), (p + "out_ln", 2 * h)]
    t += [("pooler.w", h * h), ("pooler.b", h)]
    return t


# ---------------------------------------------------------------- workloads

@dataclass
class Workload:
    name: str
    n: int                      # gradient length N
    W: int                      # simulated workers
    vtype: str                  # "i32" or "f32"
    idx: list                   # per worker: sorted uint32 indices
    val: list                   # per worker: int32 or float32 values (nonzero)
    data_seed: int
    hash_seed: int
    params: dict = field(default_factory=dict)

    @property
    def n_agg(self) -> int:
        """Nonzeros of the aggregate's support (union over workers)."""
        return int(np.unique(np.concatenate(self.idx)).size) if self.idx else 0

    @property
    def dtype(self):
        return np.int32 if self.vtype == "i32" else np.float32

    def dense(self, w: int) -> np.ndarray:
        x = np.zeros(self.n, self.dtype)
        x[self.idx[w]] = self.val[w]
        return x

    def nnz(self, w: int) -> int:
        return int(self.idx[w].size)


def _values(rng: np.random.Generator, size: int, sigma: float, vtype: str) -> np.ndarray:
    if vtype == "i32":
        out = np.empty(size, np.int32)
        todo = np.arange(size)
        while todo.size:
            v = rng.normal(0.0, sigma, todo.size)
            q = np.clip(np.rint(v * FIXED_POINT_SCALE), -INT32_MAX, INT32_MAX).astype(np.int64)
            out[todo] = q.astype(np.int32)
            todo = todo[q == 0]
        return out
    if vtype == "f32":
        out = np.empty(size, np.float32)
        todo = np.arange(size)
        while todo.size:
            v = rng.normal(0.0, sigma, todo.size).astype(np.float32)
            out[todo] = v
            todo = todo[v == 0]
        return out
    raise ValueError(f"unknown vtype {vtype!r}")


def overlap_supports(rng: np.random.Generator, tensors, W: int, density: float,
                     overlap: float):
    """Per-worker supports under the shared-pool overlap model (module doc)."""
    parts = [[] for _ in range(W)]
    base = 0
    for _, m in tensors:
        n_w = int(round(density * m))
        s = int(round(overlap * n_w))
        total = s + W * (n_w - s)
        if total > m:
            raise ValueError(f"tensor of {m} cannot hold {total} distinct nonzeros")
        if n_w > 0:
            pick = rng.choice(m, total, replace=False).astype(np.int64) + base
            shared = pick[:s]
            for w in range(W):
                lo = s + w * (n_w - s)
                parts[w].append(shared)
                parts[w].append(pick[lo:lo + n_w - s])
        base += m
    return [np.sort(np.concatenate(p)).astype(np.uint32) if p else np.zeros(0, np.uint32)
            for p in parts], base


def overlap_workload(name: str, tensors, W: int, density: float, overlap: float,
                     sigma: float, vtype: str, data_seed: int, hash_seed: int,
                     **params) -> Workload:
    rng = np.random.default_rng([data_seed, 0])
    idx, n = overlap_supports(rng, tensors, W, density, overlap)
    val = [_values(np.random.default_rng([data_seed, 1, w]), idx[w].size, sigma, vtype)
           for w in range(W)]
    p = dict(density=density, overlap=overlap, sigma=sigma, tensors=len(tensors))
    p.update(params)
    return Workload(name, n, W, vtype, idx, val, data_seed, hash_seed, p)


def ncf_workload(vtype: str = "i32", W: int = 8, rows: int = 2**24, dim: int = 64,
                 rows_per_worker: int = 4096, zipf_s: float = 1.1, sigma: float = 1e-2,
                 data_seed: int = 1001, hash_seed: int = 2001) -> Workload:
    """Row-sparse embedding gradient: Zipf-chosen rows, full rows nonzero."""
    mix = np.random.default_rng([data_seed, 2])
    mult = int(mix.integers(0, rows // 2)) * 2 + 1  # odd => bijection mod 2^24
    add = int(mix.integers(0, rows))
    idx = []
    for w in range(W):
        rng = np.random.default_rng([data_seed, 0, w])
        chosen: set = set()
        while len(chosen) < rows_per_worker:
            r = rng.zipf(zipf_s, 4 * rows_per_worker)
            for v in r[r <= rows]:
                chosen.add(int(v))
                if len(chosen) == rows_per_worker:
                    break
        ranks = np.fromiter(chosen, np.int64)
        row_ids = ((ranks - 1) * mult + add) % rows
        p = (np.sort(row_ids)[:, None] * dim + np.arange(dim)[None, :]).reshape(-1)
        idx.append(p.astype(np.uint32))
    val = [_values(np.random.default_rng([data_seed, 1, w]), idx[w].size, sigma, vtype)
           for w in range(W)]
    return Workload("ncf", rows * dim, W, vtype, idx, val, data_seed, hash_seed,
                    dict(rows=rows, dim=dim, rows_per_worker=rows_per_worker, zipf_s=zipf_s,
                         sigma=sigma))


def make(name: str, vtype: str = "i32", **kw) -> Workload:
    """The named workloads with their default parameters (overridable)."""
    if name == "tiny":
        return overlap_workload("tiny", [("x", 65536)], kw.get("W", 4),
                                kw.get("density", 655 / 65536), kw.get("overlap", 0.5),
                                kw.get("sigma", 1e-3), vtype, kw.get("data_seed", 1000),
                                kw.get("hash_seed", 2000))
    if name == "ncf":
        return ncf_workload(vtype=vtype, **kw)
    if name == "lstm":
        return overlap_workload("lstm", lstm_tensors(), kw.get("W", 8), kw.get("density", 0.01),
                                kw.get("overlap", 0.3), kw.get("sigma", 1e-3), vtype,
                                kw.get("data_seed", 1002), kw.get("hash_seed", 2002))
    if name == "vgg19":
        return overlap_workload("vgg19", vgg19_tensors(), kw.get("W", 8),
                                kw.get("density", 0.01), kw.get("overlap", 0.3),
                                kw.get("sigma", 1e-3), vtype, kw.get("data_seed", 1003),
                                kw.get("hash_seed", 2003))
    if name == "bert":
        return overlap_workload("bert", bert_base_tensors(), kw.get("W", 16),
                                kw.get("density", 0.01), kw.get("overlap", 0.5),
                                kw.get("sigma", 1e-3), vtype, kw.get("data_seed", 1004),
                                kw.get("hash_seed", 2004))
    if name == "synthetic":
        n = kw["n"]
        return overlap_workload("synthetic", [("x", n)], kw.get("W", 4), kw.get("density", 0.02),
                                kw.get("overlap", 0.5), kw.get("sigma", 1e-3), vtype,
                                kw.get("data_seed", 7), kw.get("hash_seed", 8))
    raise ValueError(f"unknown workload {name!r}")


NAMES = ("tiny", "ncf", "lstm", "vgg19", "bert")
