"""Fidelity of an explanation (eq. 7-8, Sec. 4.3; protocol of Sec. 4.6).

Test infrastructure: only tests/, the smoke check and the benchmark's CPU
baseline use this module.

Importance of a player is |phi| (Sec. 2.3: Shapley values can be negative,
so their absolute value ranks the edges).  Order: larger |phi| first, equal
|phi| by lower player index first.  With the importance values given as
float32 (the explainer's output), the order is that of the float32 values.

  G_S        (Fidelity-) all players except the floor(s M) least important
             ones (sparsity s; Sec. 4.6 uses s = 0.3);
  G_{C \\ S}  (Fidelity+) all players except the min(k, M) most important
             ones (Sec. 4.6 uses the top 10).

f(G)_y is the explained output of the model (the logit of the predicted
class, as everywhere in this library), and each target contributes
|f(G_C) - f(G_S)| to Fidelity- and |f(G_C) - f(G_{C\\S})| to Fidelity+;
eq. 7-8 average them over the N targets.
"""
import numpy as np


def importance_order(phi):
    """Player indices from most to least important (|phi| desc, index asc)."""
    a = np.abs(np.asarray(phi, dtype=np.float32)).astype(np.float64)
    idx = np.arange(a.size)
    return np.lexsort((idx, -a))


def fidelity_masks(phi, sparsity, top_k):
    """Boolean rows (G_S, G_{C\\S}) over the M players."""
    M = len(phi)
    order = importance_order(phi)
    n_drop = int(np.floor(sparsity * M))
    keep = np.ones(M, bool)
    if n_drop > 0:
        keep[order[M - n_drop:]] = False
    rest = np.ones(M, bool)
    rest[order[:min(int(top_k), M)]] = False
    return keep, rest


def fidelity_terms(game, phi, sparsity, top_k):
    """(|f(G_C) - f(G_S)|, |f(G_C) - f(G_{C\\S})|, f(G_C)) for one target;
    `game` maps a boolean player mask to the explained output."""
    M = len(phi)
    keep, rest = fidelity_masks(phi, sparsity, top_k)
    full = float(game(np.ones(M, bool)))
    return abs(full - float(game(keep))), abs(full - float(game(rest))), full


def fidelity(terms):
    """eq. 7 and eq. 8: the means over the targets of the first two entries
    of each target's terms."""
    t = np.asarray(terms, dtype=np.float64)[:, :2]
    return float(t[:, 0].mean()), float(t[:, 1].mean())
