"""Seeded random graph generators (numpy PCG64)."""
import numpy as np


def _unique_pairs(a, b, n):
    """Undirected pairs (min, max) without self loops, deduplicated, as uint64 keys."""
    lo = np.minimum(a, b).astype(np.uint64)
    hi = np.maximum(a, b).astype(np.uint64)
    keep = lo != hi
    return np.unique(lo[keep] * np.uint64(n) + hi[keep])


def _draw_exact(n, n_pairs, draw, rng):
    """Draws candidate pairs with `draw(count)` until at least n_pairs distinct
    undirected pairs exist, then keeps a seeded random subset of exactly
    n_pairs.  Returns (lo, hi), sorted by (lo, hi)."""
    keys = np.zeros(0, dtype=np.uint64)
    batch = int(n_pairs * 1.3) + 1024
    while keys.size < n_pairs:
        a, b = draw(batch)
        new = _unique_pairs(a, b, n)
        keys = new if keys.size == 0 else np.union1d(keys, new)
        batch = int((n_pairs - keys.size) * 2) + 1024
    if keys.size > n_pairs:
        pick = rng.permutation(keys.size)[:n_pairs]
        pick.sort()
        keys = keys[pick]
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


def _categorical(rng, prob, count):
    """`count` i.i.d. draws from the categorical distribution `prob`: the
    multinomial counts of every category, repeated and shuffled (the same law
    as independent draws, with sequential memory access)."""
    counts = rng.multinomial(count, prob)
    idx = np.repeat(np.arange(prob.size, dtype=np.int64), counts)
    rng.shuffle(idx)
    return idx


def dcsbm_pairs(n, n_pairs, n_blocks, p_in, degree_weights, seed):
    """Degree-corrected stochastic block model.

    Nodes are split into `n_blocks` communities (node i in community
    i mod n_blocks); an edge endpoint is drawn with probability proportional
    to `degree_weights`; with probability p_in the second endpoint is drawn
    from the first endpoint's community (again by weight), otherwise from the
    whole graph.  Exactly `n_pairs` distinct undirected pairs.  Returns
    (lo, hi) int64 arrays.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    w = np.asarray(degree_weights, dtype=np.float64)
    prob = w / w.sum()
    block = np.arange(n) % n_blocks
    members = [np.flatnonzero(block == c) for c in range(n_blocks)]
    member_prob = [w[m] / w[m].sum() for m in members]

    def draw(count):
        a = _categorical(rng, prob, count)
        b = _categorical(rng, prob, count)
        intra = np.flatnonzero(rng.random(count) < p_in)
        ba = block[a[intra]]
        by_block = np.argsort(ba, kind="stable")
        counts = np.bincount(ba, minlength=n_blocks)
        off = 0
        for c in range(n_blocks):
            sel = intra[by_block[off:off + counts[c]]]
            b[sel] = members[c][_categorical(rng, member_prob[c], int(counts[c]))]
            off += counts[c]
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
    """Symmetric in-CSR: both directions of every undirected pair (self loops
    and repeated pairs dropped)."""
    lo = np.asarray(lo, dtype=np.int64)
    hi = np.asarray(hi, dtype=np.int64)
    if lo.size and (lo == hi).any():
        keep = lo != hi
        lo, hi = lo[keep], hi[keep]
    # sort by (dst, src) with one key sort; dedupe only when a repeat exists
    key = np.concatenate([hi * np.int64(n) + lo, lo * np.int64(n) + hi])
    key.sort()
    if key.size > 1 and (key[1:] == key[:-1]).any():
        key = np.unique(key)
    d = key // n
    s = key % n
    indptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(d, minlength=n), out=indptr[1:])
    return indptr, s.astype(np.int32)


def random_digraph(n, n_edges, seed, symmetric=False):
    """Small uniform random (di)graph as an in-CSR, for tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    a = rng.integers(0, n, size=n_edges)
    b = rng.integers(0, n, size=n_edges)
    if symmetric:
        return in_csr_from_pairs(n, a, b)
    return in_csr_from_directed(n, a, b)
