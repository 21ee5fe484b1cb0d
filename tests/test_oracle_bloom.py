"""Pins of the oracle's Bloom-filter index (section 3.3) against what the paper
and the mathematics fix, independently of the oracle's own code path:

  * the space claim of section 3.3: with eps = (ln^2 2 gamma C lambda)^-1 the
    sketch plus the filter stay below 1.6 S_min, S_min from the entropy bound
    the section derives (computed here from its own definition);
  * a Bloom filter never reports a nonzero as zero (section 3.3);
  * the filter is homomorphic under bitwise OR (section 3.3);
  * the textbook fill and false-positive rate of a Bloom filter with k
    hashes and m bits after n insertions, 1 - exp(-k n / m) and its k-th power
    (Bloom 1970), checked statistically with and without batching;
  * decoding peels the candidates (the support plus the false positives):
    exactly the candidates outside the largest stopping set, by enumeration
    of every subset, with the false positives recovered as 0, and the result
    equal to the direct sum of the workers' gradients on success.
"""
import math

import numpy as np
import pytest

import oracle as o
import workloads as wl
from test_oracle import brute_two_core, mask_set, support_bits, wrap_sum

LN2 = math.log(2.0)


def entropy(x):
    return -x * math.log2(x) - (1 - x) * math.log2(1 - x)


def s_min_per_nonzero(lam, C):
    """Section 3.3's lower bound per nonzero: f(0, lambda) + log2(2^C - 1),
    with f(0, x) = (x + 1) H(1 / (x + 1))."""
    return (lam + 1) * entropy(1 / (lam + 1)) + math.log2(2.0**C - 1)


def candidates(g, B):
    """Parameters whose filter bits are all set, by direct probing."""
    bits = np.unpackbits(B.view(np.uint8), bitorder="little")
    return [p for p in range(g.n) if all(bits[int(q)] for q in o.bloom_bits(g, p))]


@pytest.mark.parametrize("n,nnz,c", [(1 << 30, 1_551_680, 1024), (109_482_240, 9_305_915, 1024),
                                     (109_482_240, 273_579, 1024), (143_667_240, 8_476_348, 1024),
                                     (1_000_000, 300_000, 1024), (65_536, 1_636, 1)])
def test_space_below_paper_bound(n, nnz, c):
    # S = S_1 + S_2 (filter bits + C bits per sketch cell) < 1.6 S_min; the
    # bound ignores rounding to whole rows, so the tiny case uses rows of 1
    C = 32
    g, eps = o.bloom_geometry(n, nnz, seed=1, c=c)
    lam = (n - nnz) / nnz
    assert abs(eps * LN2 * LN2 * o.GAMMA * C * lam - 1.0) < 1e-12
    S = g.bloom_rows * g.c + C * g.cells
    assert S / (nnz * s_min_per_nonzero(lam, C)) < 1.6
    # and the filter replaces an n-bit bitmap by far fewer bits once the
    # gradient is sparse (at lambda ~ 10 the two are about the same size)
    if lam > 100:
        assert g.bloom_rows * g.c < n / 4


def test_hash_count_and_size_follow_eps():
    # log(1/eps) hashes (rounded), n / ln 2 bits per hash: about half the bits
    # set, and a sketch sized for the support plus the expected false positives
    for n, nnz in ((1 << 30, 1_551_680), (109_482_240, 9_305_915), (10_000_000, 2_000_000)):
        g, eps = o.bloom_geometry(n, nnz, seed=3, c=1024)
        assert g.bloom_k == round(math.log2(1 / eps))
        m = g.bloom_rows * g.c
        assert m - g.c < g.bloom_k * nnz / LN2 <= m
        cand = nnz + (n - nnz) * 2.0**-g.bloom_k
        assert g.cells >= o.GAMMA * cand > g.cells - g.c


def test_too_dense_for_a_filter():
    # lambda below about 0.075: eps above 2^-1/2, log(1/eps) rounds to no hash
    with pytest.raises(ValueError):
        o.bloom_geometry(1000, 950, seed=1)
    g, eps = o.bloom_geometry(1000, 900, seed=1)
    assert g.bloom_k == 1 and 0.4 < eps < 0.5
    with pytest.raises(ValueError):
        o.bloom_geometry(1000, 1000, seed=1)


@pytest.mark.parametrize("c", [1, 8, 64, 1024])
def test_no_false_negatives(c):
    rng = np.random.default_rng(c)
    n = 50_000
    for trial in range(3):
        m = int(rng.integers(50, 2000))
        S = np.sort(rng.choice(n, m, replace=False))
        g, _ = o.bloom_geometry(n, m, seed=17 + trial, c=c)
        x = np.zeros(n, np.int32)
        x[S] = rng.integers(1, 1000, m)
        _, B = o.encode(g, x)
        bits = np.unpackbits(B.view(np.uint8), bitorder="little")
        for p in S[:300]:
            assert all(bits[int(q)] for q in o.bloom_bits(g, int(p)))
        _, _, info = o.decode(g, *o.encode(g, x))
        assert info.n_support >= m


@pytest.mark.parametrize("c", [1, 1024])
def test_fill_and_false_positive_rate(c):
    # m bits, k hashes, n insertions: E[fill] = 1 - (1 - 1/m)^(k n); the false
    # positive rate of a zero is about fill^k.  Batching (section 3.4) places a
    # batch's nonzeros at distinct bits of one row per hash, which leaves both
    # expectations unchanged to first order.
    rng = np.random.default_rng(5 + c)
    n, nnz = 400_000, 4_000
    S = np.sort(rng.choice(n, nnz, replace=False))
    g, _ = o.bloom_geometry(n, nnz, seed=99, c=c)
    x = np.zeros(n, np.int32)
    x[S] = 1
    _, B = o.encode(g, x)
    m = g.bloom_rows * g.c
    k = g.bloom_k
    fill = np.unpackbits(B.view(np.uint8), bitorder="little")[:m].mean()
    e_fill = 1 - (1 - 1 / m) ** (k * nnz)
    sd_fill = math.sqrt(e_fill * (1 - e_fill) / m)
    assert abs(fill - e_fill) < 6 * sd_fill + 2e-3
    _, _, info = o.decode(g, *o.encode(g, x))
    fp = info.n_support - nnz
    p_fp = e_fill**k
    mu = p_fp * (n - nnz)
    assert abs(fp - mu) < 6 * math.sqrt(mu) + 0.1 * mu, (fp, mu)


def test_filter_is_homomorphic_under_or():
    # B(sum X) = OR of B(X_w) when no sum cancels (section 3.3)
    w = wl.make("synthetic", n=300_000, W=4, density=0.01, overlap=0.3, data_seed=8)
    g, _ = o.bloom_geometry(w.n, w.n_agg, seed=w.hash_seed, c=1024)
    enc = [o.encode(g, w.dense(i)) for i in range(w.W)]
    Ya, Ba = o.aggregate(np.stack([e[0] for e in enc]), np.stack([e[1] for e in enc]))
    total = wrap_sum([w.dense(i) for i in range(w.W)])
    assert np.count_nonzero(total) == w.n_agg  # nothing cancelled
    Yd, Bd = o.encode(g, total)
    assert np.array_equal(Bd, Ba)
    assert np.array_equal(Yd, Ya)
    assert Ba.size == g.index_words < g.words


def test_decode_over_candidates_vs_stopping_sets():
    # every support of a 12-parameter gradient with a deliberately small
    # filter (many false positives): the recovered set is the candidate set
    # minus its largest stopping set, the false positives come back as 0, and
    # a candidate that stays in the core gets the median estimate
    rng = np.random.default_rng(21)
    fps = fails = 0
    for c, rows, brows, seed in ((1, 9, 12, 4), (2, 6, 5, 7)):
        g = o.Geom(n=12, rows=rows, seed=seed, c=c, bloom_k=2, bloom_rows=brows)
        for code in range(1, 1 << g.n):
            S = [p for p in range(g.n) if code >> p & 1]
            x = np.zeros(g.n, np.int32)
            x[S] = rng.integers(1, 1000, len(S)) * rng.choice([-1, 1], len(S))
            Y, B = o.encode(g, x)
            cand = candidates(g, B)
            assert set(S) <= set(cand)
            out, mask, info = o.decode(g, Y, B)
            cl, _ = o.cells(g, np.array(cand, np.uint64))
            core = brute_two_core([tuple(int(v) for v in r) for r in cl])
            peeled = {cand[i] for i in range(len(cand)) if i not in core}
            assert mask_set(mask, g.n) == peeled
            assert (info.n_support, info.n_recovered) == (len(cand), len(peeled))
            for p in peeled:
                assert out[p] == x[p]
            assert not out[[p for p in range(g.n) if p not in cand]].any()
            fps += len(cand) - len(S)
            fails += not info.success
    assert fps > 0 and fails > 0


@pytest.mark.parametrize("c", [1, 64, 1024])
def test_decode_equals_direct_sum(c):
    w = wl.make("synthetic", n=2_000_000, W=4, density=0.002, overlap=0.4, data_seed=40 + c)
    g, _ = o.bloom_geometry(w.n, w.n_agg, seed=w.hash_seed, c=c)
    enc = [o.encode_coo(g, w.idx[i], w.val[i]) for i in range(w.W)]
    Ya, Ba = o.aggregate(np.stack([e[0] for e in enc]), np.stack([e[1] for e in enc]))
    x, mask, info = o.decode(g, Ya, Ba)
    direct = wrap_sum([w.dense(i) for i in range(w.W)])
    assert info.success
    assert np.array_equal(x, direct)
    assert info.n_support > w.n_agg  # false positives exist and decode to 0
    rec = support_bits(mask, g.n)
    assert rec.size == info.n_support
    assert set(np.nonzero(direct)[0].tolist()) <= set(rec.tolist())
