"""Pins of the oracle's sampler against the paper and the mathematics
(eq. 3-6, Sec. 3.3, Alg. 2-3, App. C.1), not against itself."""
import itertools
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import philox, sampler


def _kat_rows(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split("->")
            v = [int(x, 16) for x in lhs.split()[1:]]
            rows.append((v[:4], v[4:6], [int(x, 16) for x in rhs.split()]))
    return rows


def test_philox_known_answers(golden_dir):
    rows = _kat_rows(golden_dir)
    assert len(rows) == 3
    for ctr, key, want in rows:
        assert philox.philox4x32_10(ctr, key) == want
        got = philox.philox4x32_10_np(*ctr, *key)
        assert [int(g) for g in got] == want


def test_unrank_matches_itertools_order():
    for n in range(1, 9):
        for c in range(1, n + 1):
            combos = list(itertools.combinations(range(n), c))
            for q, comb in enumerate(combos):
                assert tuple(sampler.unrank(n, c, q)) == comb


@pytest.mark.parametrize("n,c", [(5, 2), (6, 3), (7, 2), (8, 4)])
def test_floyd_uniform_over_subsets(n, c):
    rows = np.arange(30000)
    sel = sampler.floyd_rows(n, c, rows, seed=12345, stream=7)
    assert (sel.sum(axis=1) == c).all()
    codes = (sel * (1 << np.arange(n))).sum(axis=1)
    subsets = [sum(1 << i for i in s) for s in itertools.combinations(range(n), c)]
    counts = np.array([(codes == s).sum() for s in subsets])
    assert counts.sum() == rows.size           # every draw is a valid c-subset
    _, pval = stats.chisquare(counts)
    assert pval > 1e-4


def test_floyd_exact_size_large():
    for M, c in [(60, 11), (400, 150), (1000, 499), (64, 64), (65, 1)]:
        sel = sampler.floyd_rows(M, c, np.arange(200), seed=99, stream=3)
        assert (sel.sum(axis=1) == c).all()


def _pi(M, s):
    """Kernel SHAP weight of a single coalition of size s (eq. 3)."""
    return (M - 1) / (math.comb(M, s) * s * (M - s))


@pytest.mark.parametrize("M", list(range(2, 11)))
def test_enumeration_regime_is_every_coalition_with_kernel_weight(M):
    p = 2 ** M - 2
    pl = sampler.plan(M, p)
    assert pl["k"] == p
    masks, w = sampler.sample(pl, seed=1, stream=2)
    codes = (masks * (1 << np.arange(M))).sum(axis=1)
    assert sorted(codes.tolist()) == list(range(1, 2 ** M - 1))
    rho_sum = sum((M - 1) / (s * (M - s)) for s in range(1, M))
    sizes = masks.sum(axis=1)
    want = np.array([_pi(M, s) / rho_sum for s in sizes])
    np.testing.assert_allclose(w, want, rtol=1e-13, atol=0)


@pytest.mark.parametrize("M,p", [(20, 10000), (60, 2000), (400, 10000), (33, 5000),
                                 (4000, 25000), (13, 8190), (12, 50), (2, 2), (3, 100)])
def test_plan_invariants(M, p):
    pl = sampler.plan(M, p)
    k, half = pl["k"], pl["half"]
    assert k <= p and k % 2 == 0 and k == 2 * half
    masks, w = sampler.sample(pl, seed=0xABCDEF, stream=42)
    # complement pairing (App. C.1)
    np.testing.assert_array_equal(masks[half:], ~masks[:half])
    np.testing.assert_array_equal(w[half:], w[:half])
    # "50% sparse" (Sec. 3.5): with complements exactly half the bits are set
    assert masks.sum() == half * M
    assert abs(w.sum() - 1.0) < 1e-12
    # every representative row has the size of its class
    for cl in pl["classes"]:
        rows = masks[cl["row_begin"]:cl["row_begin"] + cl["row_count"]]
        assert (rows.sum(axis=1) == cl["c"]).all()
        if cl["full"] and 2 * cl["c"] == M:     # enumerated middle class: contains player 0
            assert rows[:, 0].all()
    # no coalition is empty or full
    sizes = masks.sum(axis=1)
    assert sizes.min() >= 1 and sizes.max() <= M - 1


def test_random_class_counts_follow_eq5():
    """Random rows are spread over sizes in proportion to rho (eq. 4-5)."""
    for M, p in [(30, 25000), (400, 10000), (4000, 25000)]:
        pl = sampler.plan(M, p)
        rnd = [cl for cl in pl["classes"] if not cl["full"]]
        full_c = {cl["c"] for cl in pl["classes"] if cl["full"]}
        total = pl["random_pairs"]
        rest = [c for c in range(1, M // 2 + 1) if c not in full_c]
        omega = {c: (2.0 if 2 * c < M else 1.0) * (M - 1) / (c * (M - c)) for c in rest}
        wsum = sum(omega.values())
        got = {cl["c"]: cl["row_count"] for cl in rnd}
        assert sum(got.values()) == total
        for c in rest:
            assert abs(got.get(c, 0) - total * omega[c] / wsum) < 1.0


def test_surplus_goes_to_enumeration_of_small_sizes():
    """Sizes whose quota exceeds the number of coalitions are enumerated
    (Sec. 3.3.1); M = 20, p = 10,000 enumerates sizes 1, 2 and 18, 19."""
    pl = sampler.plan(20, 10000)
    full = [cl["c"] for cl in pl["classes"] if cl["full"]]
    assert full == [1, 2]
    assert pl["classes"][0]["row_count"] == 20 and pl["classes"][1]["row_count"] == 190
    masks, _ = sampler.sample(pl, seed=5, stream=6)
    size1 = masks[:20]
    np.testing.assert_array_equal(size1, np.eye(20, dtype=bool))


def test_pack_layout():
    rng = np.random.default_rng(3)
    for M in [1, 63, 64, 65, 130]:
        m = rng.random((7, M)) < 0.5
        words = sampler.pack(m)
        assert words.shape == (7, (M + 63) // 64)
        for b in range(7):
            for j in range(M):
                assert ((int(words[b, j // 64]) >> (j % 64)) & 1) == int(m[b, j])
            if M % 64:
                assert int(words[b, -1]) >> (M % 64) == 0
        np.testing.assert_array_equal(sampler.unpack(words, M), m)


def test_plan_rejects_bad_arguments():
    with pytest.raises(ValueError):
        sampler.plan(1, 10)
    with pytest.raises(ValueError):
        sampler.plan(10, 11)
    with pytest.raises(ValueError):
        sampler.plan(10, 0)


@pytest.mark.parametrize("M,p", [(10, 1022), (11, 600), (12, 600), (20, 10000), (63, 2000), (64, 2000),
                                 (65, 2000), (128, 1000), (129, 1000), (200, 4000)])
def test_sample_rows_equals_rows_of_sample(M, p):
    """sample_rows builds each requested row on its own (unranked subset,
    Floyd subset or complement of its representative); the parity tests of
    large targets use it as the reference for masks and weights.  Every row
    it builds must equal the same row of the whole matrix from sample(),
    which the tests above pin against eq. 3-6 and Alg. 2-3: enumerated
    classes (the middle class of even M included), random classes, the
    boundary between them, complement rows and rows whose players cross
    uint64 word boundaries."""
    seed, stream = 0x5EED0007 + M, 1000 + M
    pl = sampler.plan(M, p)
    masks, w = sampler.sample(pl, seed, stream)
    k, half, rb = pl["k"], pl["half"], pl["random_begin"]
    rng = np.random.Generator(np.random.PCG64(M * 7919 + p))
    edges = {0, max(rb - 1, 0), rb, half - 1, half, min(half + rb, k - 1), k - 1}
    rows = np.unique(np.concatenate([np.fromiter((r for r in edges if 0 <= r < k), dtype=np.int64),
                                     rng.integers(0, k, size=min(k, 64))]))
    got, gw = sampler.sample_rows(pl, rows, seed, stream)
    np.testing.assert_array_equal(got, masks[rows])
    np.testing.assert_array_equal(gw, w[rows])
    # the packed form of the selected rows is the packed form of the matrix rows
    np.testing.assert_array_equal(sampler.pack(got), sampler.pack(masks)[rows])
    kinds = {bool(cl["full"]) for cl in pl["classes"]}
    if M in (10, 12, 20):
        assert True in kinds              # enumerated classes are covered
    if M >= 11:
        assert False in kinds             # random classes are covered
