"""Pins of the oracle's fidelity (eq. 7-8, Sec. 4.3, protocol of Sec. 4.6):
a hand-worked example (tests/golden/fidelity_worked.json), brute force over
player subsets, and the limits s = 0, s = 1, k = 0, k >= M on a GCN game."""
import itertools
import json
import os

import numpy as np
import pytest

import workloads as W
from oracle import fidelity as F
from oracle import gcn, subgraph

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fidelity_worked.json")


def _additive(a, f0):
    a = np.asarray(a, dtype=np.float64)
    return lambda m: f0 + float(np.asarray(m, dtype=np.float64) @ a)


def test_worked_example():
    g = json.load(open(GOLDEN))
    game = _additive(g["a"], g["f0"])
    keep, rest = F.fidelity_masks(np.float32(g["a"]), g["sparsity"], g["top_k"])
    assert keep.tolist() == g["keep"]
    assert rest.tolist() == g["rest"]
    tm, tp, full = F.fidelity_terms(game, np.float32(g["a"]), g["sparsity"], g["top_k"])
    assert full == pytest.approx(g["f_full"], abs=1e-12)
    assert tm == pytest.approx(g["fidelity_minus_term"], abs=1e-12)
    assert tp == pytest.approx(g["fidelity_plus_term"], abs=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_top_and_bottom_sets(seed):
    """With distinct |a|, the top-k set maximises sum |a| over all k-subsets and
    the dropped floor(sM) set minimises it; the terms are |sum of a| over them."""
    rng = np.random.default_rng(seed)
    M = 8
    a = rng.normal(size=M)
    game = _additive(a, 0.1)
    for k in range(M + 1):
        best = max(itertools.combinations(range(M), k), key=lambda S: sum(abs(a[j]) for j in S))
        _, tp, _ = F.fidelity_terms(game, np.float32(a), 0.0, k)
        assert tp == pytest.approx(abs(sum(a[j] for j in best)), abs=1e-9)
    for s in (0.0, 0.1, 0.3, 0.5, 0.99, 1.0):
        nd = int(np.floor(s * M))
        worst = min(itertools.combinations(range(M), nd), key=lambda S: sum(abs(a[j]) for j in S))
        tm, _, _ = F.fidelity_terms(game, np.float32(a), s, 0)
        assert tm == pytest.approx(abs(sum(a[j] for j in worst)), abs=1e-9)


def test_limits_on_a_gcn_game():
    """s = 0 and k = 0 change nothing; s = 1 and k >= M remove every player,
    leaving f(empty)."""
    cfg = W.make_config("tiny")
    v = cfg["targets"][0]
    sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
    M = sub["num_edges"]
    game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"])
    full_logits = game.logits(np.ones(M, bool))
    game.cls = gcn.predicted_class(full_logits)
    f_empty = game(np.zeros(M, bool))
    phi = np.random.default_rng(1).normal(size=M).astype(np.float32)
    tm, tp, full = F.fidelity_terms(game, phi, 0.0, 0)
    assert tm == 0.0 and tp == 0.0
    tm, tp, _ = F.fidelity_terms(game, phi, 1.0, M + 5)
    assert tm == pytest.approx(abs(full - f_empty), abs=1e-12)
    assert tp == pytest.approx(abs(full - f_empty), abs=1e-12)
    assert F.fidelity([(1.0, 2.0, 9.0), (3.0, 6.0, 9.0)]) == (2.0, 4.0)
