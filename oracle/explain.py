"""Alg. 1 end to end for one target node: prune -> sample -> predict -> WLS.

Prediction pruning (Sec. 3.4.1) is not applied here: the oracle evaluates the
game on every sampled coalition, so that the exactness of the shortcut taken
by the product path is checked rather than assumed.
"""
import numpy as np

from . import gcn, sampler, subgraph, wls


def explain(indptr, indices, X, weights, biases, target, hops, p, seed,
            stream=None, cls=None, rows=None):
    """Returns a dict with the subgraph, plan, masks, weights, y, f(empty),
    f(full), the explained class and phi.  `rows` (optional) restricts the
    evaluated coalitions to a subset of row indices (phi is then not computed).
    """
    sub = subgraph.extract(indptr, indices, target, hops)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, weights, biases)
    full_logits = game.logits(np.ones(M, dtype=bool))
    if cls is None:
        cls = gcn.predicted_class(full_logits)
    game.cls = cls
    f_full = float(full_logits[cls])
    f_empty = game(np.zeros(M, dtype=bool))
    out = dict(sub=sub, cls=cls, f_full=f_full, f_empty=f_empty,
               full_logits=full_logits)
    if M < 2:
        out["phi"] = np.array([f_full - f_empty])[:M]
        return out
    pl = sampler.plan(M, p)
    masks, w = sampler.sample(pl, seed, target if stream is None else stream)
    out.update(plan=pl, masks=masks, weights=w)
    if rows is not None:
        out["rows"] = np.asarray(rows)
        out["y"] = game.values(masks[rows])
        return out
    y = game.values(masks)
    out["y"] = y
    out["phi"] = wls.kernel_shap(masks, w, y, f_empty, f_full)
    return out
