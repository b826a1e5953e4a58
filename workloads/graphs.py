"""Seeded random graph generators (numpy PCG64)."""
import numpy as np


def _unique_pairs(a, b, n):
    """Undirected pairs (min, max) without self loops, deduplicated, as uint64 keys."""
    lo = np.minimum(a, b).astype(np.uint64)
    hi = np.maximum(a, b).astype(np.uint64)
    keep = lo != hi
    return np.unique(lo[keep] * np.uint64(n) + hi[keep])


def _draw_exact(n, n_pairs, draw, rng):
    """Draws candidate pairs with `draw(count)` until exactly n_pairs distinct
    undirected pairs exist; keeps a seeded random subset of the last batch."""
    keys = np.zeros(0, dtype=np.uint64)
    while keys.size < n_pairs:
        need = n_pairs - keys.size
        a, b = draw(int(need * 1.3) + 1024)
        new = _unique_pairs(a, b, n)
        new = np.setdiff1d(new, keys, assume_unique=True)
        if new.size > need:
            new = rng.choice(new, size=need, replace=False)
        keys = np.union1d(keys, new)
    lo = (keys // np.uint64(n)).astype(np.int64)
    hi = (keys % np.uint64(n)).astype(np.int64)
    return lo, hi


def chung_lu_pairs(n, n_pairs, exponent, seed):
    """Chung-Lu graph with power-law expected degrees.

    Expected-degree weights w_i = (i + 1)^(-1/(exponent-1)); endpoints are drawn
    i.i.d. with probability proportional to w until exactly `n_pairs` distinct
    undirected pairs exist.  Returns (lo, hi) int64 arrays of relabelled ids.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    w = (np.arange(n, dtype=np.float64) + 1.0) ** (-1.0 / (exponent - 1.0))
    cdf = np.cumsum(w)
    cdf /= cdf[-1]

    def draw(count):
        a = np.searchsorted(cdf, rng.random(count), side="right")
        b = np.searchsorted(cdf, rng.random(count), side="right")
        return np.minimum(a, n - 1), np.minimum(b, n - 1)

    lo, hi = _draw_exact(n, n_pairs, draw, rng)
    perm = rng.permutation(n)
    return perm[lo], perm[hi]


def dcsbm_pairs(n, n_pairs, n_blocks, p_in, degree_weights, seed):
    """Degree-corrected stochastic block model.

    Nodes are split into `n_blocks` communities of near-equal size; an edge
    endpoint is drawn with probability proportional to `degree_weights`; with
    probability p_in the second endpoint is drawn from the first endpoint's
    community (again by weight), otherwise from the whole graph.  Exactly
    `n_pairs` distinct undirected pairs.  Returns (lo, hi) int64 arrays.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    w = np.asarray(degree_weights, dtype=np.float64)
    block = np.arange(n) % n_blocks
    order = np.argsort(block, kind="stable")            # nodes grouped by block
    starts = np.searchsorted(block[order], np.arange(n_blocks + 1))
    wcum_all = np.cumsum(w)
    wcum_all /= wcum_all[-1]
    w_sorted = w[order]
    cum_sorted = np.cumsum(w_sorted)

    def draw(count):
        a = np.minimum(np.searchsorted(wcum_all, rng.random(count), side="right"), n - 1)
        b = np.minimum(np.searchsorted(wcum_all, rng.random(count), side="right"), n - 1)
        intra = rng.random(count) < p_in
        ba = block[a[intra]]
        s0, s1 = starts[ba], starts[ba + 1]
        c0 = np.where(s0 > 0, cum_sorted[np.maximum(s0 - 1, 0)], 0.0)
        c1 = cum_sorted[s1 - 1]
        r = c0 + rng.random(ba.size) * (c1 - c0)
        pos = np.minimum(np.searchsorted(cum_sorted, r, side="right"), s1 - 1)
        b[intra] = order[pos]
        return a, b

    lo, hi = _draw_exact(n, n_pairs, draw, rng)
    perm = rng.permutation(n)
    return perm[lo], perm[hi]


def in_csr_from_directed(n, src, dst):
    """In-CSR of the directed edges src -> dst (self loops and duplicates dropped)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    keep = src != dst
    key = np.unique(dst[keep] * np.int64(n) + src[keep])
    d = key // n
    s = key % n
    indptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(d, minlength=n), out=indptr[1:])
    return indptr, s.astype(np.int32)


def in_csr_from_pairs(n, lo, hi):
    """Symmetric in-CSR: both directions of every undirected pair."""
    src = np.concatenate([lo, hi])
    dst = np.concatenate([hi, lo])
    return in_csr_from_directed(n, src, dst)


def random_digraph(n, n_edges, seed, symmetric=False):
    """Small uniform random (di)graph as an in-CSR, for tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    a = rng.integers(0, n, size=n_edges)
    b = rng.integers(0, n, size=n_edges)
    if symmetric:
        return in_csr_from_pairs(n, a, b)
    return in_csr_from_directed(n, a, b)
