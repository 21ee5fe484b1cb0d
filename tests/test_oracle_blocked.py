"""Pins of the oracle's blocked sketch (section 3.2: the Count Sketch split
into blocks of a fixed size so that peeling ends in O(1) rounds).

The blocked layout changes only where an element's three cells lie: block q of
K batches owns R_b consecutive rows.  The checks below fix that map from the
outside -- one block is exactly the global sketch, every cell stays in its
block, local rows are uniform -- and then pin what blocking must mean for the
decode: blocks are disconnected parts of the hypergraph, so decoding the whole
sketch equals decoding each block alone (values, mask, recovered counts), the
round count is the largest of the blocks', brute-force 2-cores hold per block,
and a successful decode returns the direct sum of the workers.
"""
import numpy as np
import pytest

import oracle as o
import workloads as wl
from test_oracle import check_against_brute, mask_set, wrap_sum


def blocked(n, block, brows, seed, c):
    nb = ((n + c - 1) // c + block - 1) // block
    return o.Geom(n=n, rows=nb * brows, seed=seed, c=c, block=block)


def test_blocked_geometry_closed_form():
    # BERT-base, 1 % per worker and 50 % overlap (aggregate 9,305,915):
    # K = floor(18 * 109482240 / (1.3 * 9305915)) = 162 batches; the expected
    # share of 162 * 1024 parameters is 14100.5 -> 14101; 1.3 * 14101 = 18331.3
    # -> 18332 cells -> 18 rows; ceil(106917 / 162) = 660 blocks
    g = o.blocked_geometry(109_482_240, 9_305_915, 7, 1024, 1.3, 18)
    assert (g.block, g.rows, g.nblocks, g.block_rows) == (162, 11880, 660, 18)
    # sparse: K = 5540 clamps to 1024; share ceil(2620.2) = 2621; 1.3 * 2621 =
    # 3407.3 -> 3408 cells -> 4 rows; ceil(106917 / 1024) = 105 blocks
    g = o.blocked_geometry(109_482_240, 273_579, 7, 1024, 1.3, 18)
    assert (g.block, g.rows, g.block_rows) == (1024, 420, 4)
    # c = 8: K = floor(4 * 10000 / 650) = 61, rounded down to a multiple of
    # 32 / 8 = 4 -> 60; share 500 * 480 / 10000 = 24; 1.3 * 24 = 31.2 -> 32
    # cells -> 4 rows; ceil(1250 / 60) = 21 blocks
    g = o.blocked_geometry(10_000, 500, 7, 8, 1.3, 4)
    assert (g.block, g.rows, g.block_rows) == (60, 84, 4)
    assert o.check(g)


def test_blocked_geometry_invalid():
    assert not o.check(o.Geom(n=10_000, rows=84, seed=1, c=8, block=61))  # 61 * 8 % 32 != 0
    assert not o.check(o.Geom(n=10_000, rows=85, seed=1, c=8, block=60))  # 85 % 21 != 0
    assert not o.check(o.Geom(n=10_000, rows=42, seed=1, c=8, block=60))  # 2 rows per block
    assert o.check(o.Geom(n=10_000, rows=63, seed=1, c=8, block=60))


@pytest.mark.parametrize("c", [1024, 64, 1])
def test_one_block_has_the_global_rows(c):
    # a single block draws the same three rows per batch as the global sketch
    # (taken in ascending order), the same signs and the same first rotation
    n = 300_000
    batches = (n + c - 1) // c
    g0 = o.Geom(n=n, rows=57, seed=5, c=c)
    g1 = o.Geom(n=n, rows=57, seed=5, c=c, block=batches + (32 - batches % 32) % 32 if c == 1 else batches)
    assert g1.nblocks == 1
    for b in np.random.default_rng(3).choice(batches, min(500, batches), replace=False):
        r0, b0, s0 = o.batch_hash(g0, int(b))
        r1, b1, s1 = o.batch_hash(g1, int(b))
        assert np.array_equal(np.sort(r0), r1)
        assert np.array_equal(s0, s1) and b0[0] == b1[0]


def relative_rotation_keys(g):
    """(block, rows in ascending order, rotations of the 2nd and 3rd row
    relative to the 1st) of every batch, from the cells of its column 0."""
    nb = (g.n + g.c - 1) // g.c
    cl, _ = o.cells(g, np.arange(nb, dtype=np.uint64) * g.c)
    rows, rot = cl // g.c, cl % g.c
    order = np.argsort(rows, axis=1)
    rows = np.take_along_axis(rows, order, 1)
    rot = np.take_along_axis(rot, order, 1)
    return np.stack([np.arange(nb) // max(g.block, 1), rows[:, 0], rows[:, 1], rows[:, 2],
                     (rot[:, 1] - rot[:, 0]) % g.c, (rot[:, 2] - rot[:, 0]) % g.c], 1)


@pytest.mark.parametrize("n,nnz,gamma,c,brows", [(109_482_240, 273_579, 1.3, 1024, 18),
                                                 (143_667_240, 8_476_348, 1.3, 1024, 11),
                                                 (20_000_000, 100_000, 1.3, 64, 200)])
def test_no_whole_batch_collisions_in_a_block(n, nnz, gamma, c, brows):
    # Section 3.4 rotates a batch onto consecutive columns of one row per hash,
    # so two batches on the same three rows with the same relative rotations
    # would pair all their corresponding elements on the same three cells
    # (stopping sets of two).  With 4 rows per block (the sparse BERT-base
    # sketch), independent rotations would give about 13 such pairs per
    # sketch; the blocked hash admits none.
    g = o.blocked_geometry(n, nnz, 2003, c, gamma, brows)
    key = relative_rotation_keys(g)
    assert len(np.unique(key, axis=0)) == len(key)


def test_blocked_rotations_uniform():
    # each hash's rotation stays uniform over the columns: chi-square of the
    # second and third rotations over 64 column bins
    g = blocked(20_000 * 256, 40, 6, 33, 256)
    nb = 20_000
    cl, _ = o.cells(g, np.arange(nb, dtype=np.uint64) * 256)
    for j in range(3):
        counts = np.bincount((cl[:, j] % 256) // 4, minlength=64).astype(float)
        exp = nb / 64
        assert float(((counts - exp) ** 2 / exp).sum()) < 130  # 63 dof: P(> 130) < 1e-6


@pytest.mark.parametrize("c,block,brows", [(1024, 7, 5), (64, 16, 3), (8, 12, 9), (1, 64, 4)])
def test_cells_stay_in_their_block(c, block, brows):
    n = 5_000_000 if c >= 64 else 200_000
    g = blocked(n, block, brows, 9, c)
    assert o.check(g)
    idx = np.random.default_rng(c + block).choice(n, 20_000, replace=False).astype(np.uint64)
    cl, sg = o.cells(g, idx)
    q = (idx // c) // block
    rows = cl // c
    assert np.all(rows // brows == q[:, None])
    assert np.all((rows[:, 0] != rows[:, 1]) & (rows[:, 0] != rows[:, 2]) & (rows[:, 1] != rows[:, 2]))
    assert set(np.unique(sg).tolist()) <= {-1, 1}
    # within a batch (section 3.4) each hash keeps one row, one rotation of the
    # column and one sign
    for b in (0, 5, (n // c) - 1):
        ps = np.arange(b * c, min((b + 1) * c, n), dtype=np.uint64)
        cb, sb = o.cells(g, ps)
        for j in range(3):
            assert len(set((cb[:, j] // c).tolist())) == 1
            assert len(set(((cb[:, j] % c - ps % c) % c).tolist())) == 1
            assert len(set(sb[:, j].tolist())) == 1


def test_local_rows_uniform():
    # rows of a blocked sketch are uniform within the block: chi-square over
    # R_b = 9 local rows, 30,000 batches x 3 hashes
    g = blocked(30_000 * 1024, 50, 9, 21, 1024)
    counts = np.zeros(9)
    for b in range(0, 30_000):
        r, _, _ = o.batch_hash(g, b)
        for v in r:
            counts[int(v) % 9] += 1
    exp = counts.sum() / 9
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 40.0  # 8 degrees of freedom: P(chi2 > 40) < 1e-5


@pytest.mark.parametrize("c,block,brows", [(8, 4, 3), (8, 4, 5), (4, 8, 4), (1, 32, 6)])
def test_blocked_supports_vs_stopping_sets(c, block, brows):
    # brute-force 2-cores and round numbers over the blocked cell map; blocks of
    # 32 parameters, 64 parameters in all (two blocks)
    rng = np.random.default_rng(c * 1000 + block * 10 + brows)
    g = blocked(64, block, brows, c + brows, c)
    assert g.nblocks == 2
    for trial in range(25):
        m = int(rng.integers(1, 15))
        S = sorted(rng.choice(64, m, replace=False).tolist())
        vals = rng.integers(1, 2**20, m) * rng.choice([-1, 1], m)
        check_against_brute(g, S, vals)


def test_blocks_peel_independently():
    # six blocks, one of them overloaded so that it cannot be peeled: decoding
    # the whole sketch equals decoding each block's part alone
    c, block, brows = 64, 8, 5          # 512 parameters and 320 cells per block
    n = 6 * block * c
    g = blocked(n, block, brows, 17, c)
    rng = np.random.default_rng(4)
    x = np.zeros(n, np.int32)
    for q in range(6):
        m = 330 if q == 2 else int(rng.integers(60, 230))
        S = rng.choice(block * c, m, replace=False) + q * block * c
        x[S] = rng.integers(1, 2**20, m) * rng.choice([-1, 1], m)
    Y, B = o.encode(g, x)
    xo, mask, info = o.decode(g, Y, B)
    assert not info.success
    xs = np.zeros(n, np.int32)
    masks = np.zeros_like(mask)
    rec = rounds = sup = 0
    for q in range(6):
        xq = np.zeros(n, np.int32)
        sl = slice(q * block * c, (q + 1) * block * c)
        xq[sl] = x[sl]
        Yq, Bq = o.encode(g, xq)
        # block q's sketch is zero outside its rows, and the parts add up
        rows_q = np.zeros(g.cells, bool)
        rows_q[q * brows * c:(q + 1) * brows * c] = True
        assert not np.any(Yq[~rows_q])
        oq, mq, iq = o.decode(g, Yq, Bq)
        xs[sl] = oq[sl]
        masks |= mq
        rec += iq.n_recovered
        sup += iq.n_support
        rounds = max(rounds, iq.rounds)
        assert (iq.success == 0) == (q == 2)
    assert np.array_equal(xo, xs)
    assert np.array_equal(mask, masks)
    assert (info.n_recovered, info.n_support, info.rounds) == (rec, sup, rounds)
    # everything outside the overloaded block is exact
    outside = np.ones(n, bool)
    outside[2 * block * c:3 * block * c] = False
    assert np.array_equal(xo[outside], x[outside])


@pytest.mark.parametrize("c,block_rows,gamma", [(1024, 3, 1.3), (256, 4, 1.5), (64, 16, 1.6)])
def test_blocked_decode_equals_direct_sum(c, block_rows, gamma):
    # blocks of a few hundred elements need more room than gamma = 1.23
    w = wl.make("tiny")
    g = o.blocked_geometry(w.n, w.n_agg, w.hash_seed, c, gamma, block_rows)
    assert g.nblocks > 1 or c == 1024
    Ys, Bs = [], []
    for i in range(w.W):
        Y, B = o.encode(g, w.dense(i))
        Yc, Bc = o.encode_coo(g, w.idx[i], w.val[i])
        assert np.array_equal(Y, Yc) and np.array_equal(B, Bc)
        Ys.append(Y)
        Bs.append(B)
    Ya, Ba = o.aggregate(np.stack(Ys), np.stack(Bs))
    assert np.array_equal(Ya, wrap_sum(Ys))
    x, mask, info = o.decode(g, Ya, Ba)
    direct = wrap_sum([w.dense(i) for i in range(w.W)])
    assert info.success and info.n_support == w.n_agg
    assert np.array_equal(x, direct)
    assert mask_set(mask, w.n) == set(np.nonzero(direct)[0].tolist())


def test_blocked_linearity():
    g = blocked(40_000, 10, 4, 77, 256)
    rng = np.random.default_rng(8)
    a = np.zeros(g.n, np.int32)
    b = np.zeros(g.n, np.int32)
    a[rng.choice(g.n, 900, replace=False)] = rng.integers(-2**31, 2**31 - 1, 900, dtype=np.int64).astype(np.int32)
    b[rng.choice(g.n, 900, replace=False)] = rng.integers(-2**31, 2**31 - 1, 900, dtype=np.int64).astype(np.int32)
    Ya, _ = o.encode(g, a)
    Yb, _ = o.encode(g, b)
    s = wrap_sum([a, b])
    Ys, _ = o.encode(g, s)
    # linear wherever no nonzero cancels (a cancelled entry drops out of the
    # bitmap but contributes 0 to Y either way, so Y stays linear)
    assert np.array_equal(Ys, wrap_sum([Ya, Yb]))


def test_small_blocks_peel_at_low_load():
    # 3 rows per block, so every batch of a block has the same three rows:
    # only the rotations separate them.  At about 0.26 members per cell the
    # blocks must all peel; offsets with arithmetic structure (an affine map
    # of the batch index) leave small stopping sets here
    c, block, brows, nbk = 1024, 4, 3, 150
    n = nbk * block * c
    rng = np.random.default_rng(44)
    parts = [rng.choice(block * c, 800, replace=False) + q * block * c for q in range(nbk)]
    idx = np.sort(np.concatenate(parts)).astype(np.uint32)
    val = (rng.integers(1, 2**20, idx.size) * rng.choice([-1, 1], idx.size)).astype(np.int32)
    g = o.Geom(n=n, rows=nbk * brows, seed=91, c=c, block=block)
    Y, B = o.encode_coo(g, idx, val)
    x, mask, info = o.decode(g, Y, B)
    assert info.success and info.n_support == idx.size
    assert np.array_equal(x[idx], val)
