"""Coalition sampler: plan, unranking, random subsets, complements, packing.

Follows Sec. 3.3 of the paper (eq. 4-6), Alg. 2 (host plan) and Alg. 3 (row
generation), App. C.1 (complement pairing) and App. F (sampling with
replacement).  Readings where the paper is silent or garbled:

* Size classes c = 1..floor(M/2); class c holds coalition sizes c and M-c
  (paired by complementing), except the middle size c = M/2 of even M, which
  is its own complement and is one class of half the c-subsets.
* omega_c = kappa_c * rho_c, rho_s = (M-1)/(s(M-s)) (eq. 4), kappa_c = 2 for a
  paired class and 1 for the middle class; N_c = number of representative
  rows needed to enumerate the class fully.
* Surplus redistribution (Sec. 3.3.1, Alg. 2 "more samples than possible
  coalitions"): classes are tested in ascending c; class c is enumerated when
  its eq. 5 share of the pairs still unassigned is at least N_c (1e-6 slack);
  the test stops at the first class that is not.
* Remaining pairs go to the other classes in proportion to omega_c (eq. 5),
  rounded by largest remainder, ties to the smaller c.
* Enumerated classes carry the Kernel-SHAP weight pi (eq. 3) normalised by
  sum(rho); every random row carries one common weight (Alg. 2, the weight
  spread over the random samples), which equals eq. 6 up to integer rounding.
* Lexicographic order of increasing tuples, rank 0 = {0..c-1} (Sec. 3.3.2).
* rand(c) of Alg. 3 is Floyd's algorithm (Bentley & Floyd, CACM 1987) fed by
  Philox4x32-10 draws; draw s of representative row i uses counter
  (s // 4, i, stream_lo, stream_hi), key (seed_lo, seed_hi), word s % 4, and
  is mapped to [0, j] as floor(u * (j + 1) / 2^32).
* Row i + k/2 is the complement of row i within the M player bits and has
  the same weight.
* Bit j of row b lives in uint64 word b * wpr + j // 64, bit j % 64,
  wpr = ceil(M / 64); padding bits are zero.

All floating point is fp64 with a fixed operation order (plain ascending
sums), so that the plan is reproducible bit for bit.
"""
import math

import numpy as np

from .philox import philox4x32_10_np

SATURATE = 1 << 62


def binom_sat(n, r):
    """C(n, r) saturated at 2^62 (exact integers below that)."""
    if r < 0 or r > n:
        return 0
    r = min(r, n - r)
    v = 1
    for i in range(1, r + 1):
        v = v * (n - r + i) // i          # C(n-r+i, i), exact at every step
        if v >= SATURATE:
            return SATURATE
    return v


def class_tables(M):
    """Per size class c = 1..floor(M/2): (c, kappa, omega, N)."""
    out = []
    for c in range(1, M // 2 + 1):
        paired = 2 * c < M
        kappa = 2.0 if paired else 1.0
        rho = float(M - 1) / (float(c) * float(M - c))      # eq. 4
        omega = kappa * rho
        n_rows = binom_sat(M, c)
        if not paired:
            n_rows = n_rows if n_rows >= SATURATE else n_rows // 2
        out.append((c, kappa, omega, n_rows))
    return out


def ascending_sum(values):
    s = 0.0
    for v in values:
        s = s + v
    return s


def plan(M, p):
    """Host plan of Alg. 2 for M players and a budget of p samples.

    Returns a dict with
      classes: list of dicts (c, full, row_begin, row_count, weight) for every
               class that owns rows, enumerated classes first, both groups in
               ascending c; row ranges index the first half of the mask matrix;
      k:       number of rows actually produced (k_eff <= p);
      half:    k // 2; random_begin: first row of the random part;
      omega_total, full_fraction, random_weight.
    """
    if M < 2:
        raise ValueError("need at least two players")
    if p < 2 or p % 2:
        raise ValueError("sample budget must be even and >= 2")
    tab = class_tables(M)
    omegas = [t[2] for t in tab]
    K = len(tab)
    omega_total = ascending_sum(omegas)

    pairs = p // 2
    n_full = 0
    for idx in range(K):
        c, kappa, omega, n_rows = tab[idx]
        w_rem = ascending_sum(omegas[idx:])
        share = (float(pairs) * omega) / w_rem                 # eq. 5 on what is left
        if n_rows <= pairs and float(n_rows) <= share + 1e-6:
            n_full += 1
            pairs -= n_rows
        else:
            break

    rest = list(range(n_full, K))
    bins = {}
    if rest:
        p_r = pairs
        w_r = ascending_sum([omegas[i] for i in rest])
        q = {}
        for i in rest:
            q[i] = (float(p_r) * omegas[i]) / w_r
            bins[i] = int(math.floor(q[i]))
        extra = p_r - sum(bins.values())
        order = sorted(rest, key=lambda i: (-(q[i] - bins[i]), i))
        for i in order[:extra]:
            bins[i] += 1
    else:
        p_r = 0

    classes = []
    row = 0
    full_fraction = 0.0
    for idx in range(n_full):
        c, kappa, omega, n_rows = tab[idx]
        frac = omega / omega_total
        full_fraction = full_fraction + frac
        classes.append(dict(c=c, full=True, row_begin=row, row_count=n_rows,
                            weight=frac / (2.0 * float(n_rows))))
        row += n_rows
    random_begin = row
    random_weight = (1.0 - full_fraction) / (2.0 * float(p_r)) if p_r > 0 else 0.0
    for i in rest:
        if bins[i] == 0:
            continue
        classes.append(dict(c=tab[i][0], full=False, row_begin=row,
                            row_count=bins[i], weight=random_weight))
        row += bins[i]
    half = row
    return dict(M=M, p=p, classes=classes, k=2 * half, half=half,
                random_begin=random_begin, random_pairs=p_r,
                omega_total=omega_total, full_fraction=full_fraction,
                random_weight=random_weight)


def unrank(M, c, q):
    """q-th c-subset of {0..M-1} in lexicographic order (Sec. 3.3.2, Alg. 3)."""
    out = []
    x = 0
    for j in range(1, c + 1):
        while math.comb(M - x - 1, c - j) <= q:
            q -= math.comb(M - x - 1, c - j)
            x += 1
        out.append(x)
        x += 1
    return out


def floyd_rows(M, c, rows, seed, stream):
    """Floyd's random c-subsets of {0..M-1} for representative rows `rows`.

    `c` is one size or one size per row.  Vectorised over rows; for each row
    the c steps run in order, exactly as Floyd's algorithm prescribes.
    Returns a bool array [len(rows), M].
    """
    rows = np.asarray(rows, dtype=np.uint64)
    nr = rows.shape[0]
    cs = np.broadcast_to(np.asarray(c, dtype=np.int64), (nr,))
    sel = np.zeros((nr, M), dtype=bool)
    seed_lo, seed_hi = seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF
    st_lo, st_hi = stream & 0xFFFFFFFF, (stream >> 32) & 0xFFFFFFFF
    words = None
    for s in range(int(cs.max()) if nr else 0):
        act = np.flatnonzero(cs > s)              # rows that still take a step
        if s % 4 == 0:
            words = philox4x32_10_np(np.uint64(s // 4), rows, st_lo, st_hi, seed_lo, seed_hi)
        u = words[s % 4][act]
        j = M - cs[act] + s
        t = ((u * (j + 1).astype(np.uint64)) >> np.uint64(32)).astype(np.int64)   # uniform in [0, j]
        hit = sel[act, t]
        pick = np.where(hit, j, t)
        sel[act, pick] = True
    return sel


def sample(pl, seed, stream):
    """Mask matrix (bool [k, M]) and weights (fp64 [k]) for a plan (Alg. 2-3)."""
    M, k, half = pl["M"], pl["k"], pl["half"]
    masks = np.zeros((k, M), dtype=bool)
    w = np.zeros(k, dtype=np.float64)
    sizes = np.zeros(half, dtype=np.int64)
    for cl in pl["classes"]:
        r0, n, c = cl["row_begin"], cl["row_count"], cl["c"]
        if cl["full"]:
            for q in range(n):
                masks[r0 + q, unrank(M, c, q)] = True
        sizes[r0:r0 + n] = c
        w[r0:r0 + n] = cl["weight"]
    rb = pl["random_begin"]
    if rb < half:
        masks[rb:half] = floyd_rows(M, sizes[rb:half], np.arange(rb, half), seed, stream)
    masks[half:] = ~masks[:half]                      # complement pairing
    w[half:] = w[:half]
    return masks, w


def pack(masks):
    """Pack bool [k, M] into uint64 [k, ceil(M/64)], LSB first, zero padding."""
    k, M = masks.shape
    wpr = (M + 63) // 64
    padded = np.zeros((k, wpr * 64), dtype=np.uint8)
    padded[:, :M] = masks
    by = np.packbits(padded, axis=1, bitorder="little")        # [k, wpr*8] bytes
    return by.view("<u8").reshape(k, wpr)


def unpack(words, M):
    words = np.ascontiguousarray(words, dtype="<u8")
    k = words.shape[0]
    by = words.view(np.uint8).reshape(k, -1)
    return np.unpackbits(by, axis=1, bitorder="little")[:, :M].astype(bool)


def sample_rows(pl, rows, seed, stream):
    """Masks (bool [len(rows), M]) and weights of selected rows of the plan,
    each built by its own definition: an unranked subset, a Floyd subset, or
    the complement of its representative row."""
    M, half = pl["M"], pl["half"]
    rows = np.asarray(rows, dtype=np.int64)
    rep = np.where(rows >= half, rows - half, rows)
    out = np.zeros((rows.size, M), dtype=bool)
    w = np.zeros(rows.size, dtype=np.float64)
    starts = np.array([cl["row_begin"] for cl in pl["classes"]])
    for t, r in enumerate(rep):
        cl = pl["classes"][int(np.searchsorted(starts, r, side="right")) - 1]
        if cl["full"]:
            out[t, unrank(M, cl["c"], int(r - cl["row_begin"]))] = True
        else:
            out[t] = floyd_rows(M, cl["c"], np.array([r]), seed, stream)[0]
        w[t] = cl["weight"]
    out[rows >= half] = ~out[rows >= half]
    return out, w
