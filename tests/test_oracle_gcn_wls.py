"""Pins of the oracle's game f(S) (Sec. 2.2, 3.4, 4.2) and of its Kernel-SHAP
solve (eq. 1-3, Sec. 3.5) against closed forms, brute force and the Shapley
axioms."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import gcn, sampler, shapley, subgraph, wls


def _small_problem(seed, n=12, edges=22, hops=2, dims=(5, 4, 3), bias="random", m_lo=4, m_hi=10):
    indptr, indices = W.random_digraph(n, edges, seed=seed, symmetric=True)
    X = W.gaussian_features(n, dims[0], seed + 100)
    Ws, bs = W.glorot_gcn(list(dims), seed + 200, bias=bias)
    for v in range(n):
        sub = subgraph.extract(indptr, indices, v, hops)
        if m_lo <= sub["num_edges"] <= m_hi:
            return indptr, indices, X, Ws, bs, v, sub
    pytest.skip("no target of the wanted size")


def test_star_graph_closed_form():
    """One-layer GCN on a star u_1..u_n -> v: under S, deg(v) = 1 + |S| and the
    leaves have degree 1, so y = sum_{i in S} x_i W / sqrt(1+|S|) + x_v W / (1+|S|) + b."""
    n = 5
    src = list(range(1, n + 1))
    indptr, indices = W.in_csr_from_directed(n + 1, src, [0] * n)
    X = W.gaussian_features(n + 1, 3, 7).astype(np.float64)
    Ws, bs = W.glorot_gcn([3, 2], 8, bias="random")
    sub = subgraph.extract(indptr, indices, 0, 1)
    game = gcn.Game(sub, X, Ws, bs)
    rng = np.random.default_rng(0)
    for _ in range(20):
        m = rng.random(n) < 0.5
        S = [1 + i for i in np.flatnonzero(m)]        # leaves in the coalition
        s = len(S)
        Wd, bd = Ws[0].astype(np.float64), bs[0].astype(np.float64)
        want = sum(X[u] @ Wd for u in S) / math.sqrt(1 + s) + (X[0] @ Wd) / (1 + s) + bd
        np.testing.assert_allclose(game.logits(m), want, rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(gcn.forward_dense(sub, X, Ws, bs, m), want, rtol=1e-13, atol=1e-14)


def test_path_graph_two_layers_closed_form():
    """Two-layer GCN on the path a -> b -> v with all edges present:
    deg(v) = deg(b) = 2, deg(a) = 1 (a is outermost)."""
    indptr, indices = W.in_csr_from_directed(3, [2, 1], [1, 0])   # 2->1->0
    X = W.gaussian_features(3, 4, 17).astype(np.float64)
    Ws, bs = W.glorot_gcn([4, 3, 2], 18, bias="random")
    W1, W2 = Ws[0].astype(np.float64), Ws[1].astype(np.float64)
    b1, b2 = bs[0].astype(np.float64), bs[1].astype(np.float64)
    sub = subgraph.extract(indptr, indices, 0, 2)
    game = gcn.Game(sub, X, Ws, bs)
    relu = lambda z: np.maximum(z, 0)
    # full coalition
    h_b = relu(X[2] @ W1 / math.sqrt(2 * 1) + X[1] @ W1 / 2 + b1)
    h_v = relu(X[1] @ W1 / 2 + X[0] @ W1 / 2 + b1)
    y = h_b @ W2 / 2 + h_v @ W2 / 2 + b2
    np.testing.assert_allclose(game.logits(np.ones(2, bool)), y, rtol=1e-13)
    # only 1 -> 0 present: deg(v) = 2, deg(b) = 1
    h_b = relu(X[1] @ W1 + b1)
    h_v = relu(X[1] @ W1 / math.sqrt(2) + X[0] @ W1 / 2 + b1)
    y = h_b @ W2 / math.sqrt(2) + h_v @ W2 / 2 + b2
    players = [(int(sub["node_gid"][s]), int(sub["node_gid"][d])) for s, d in zip(sub["edge_src"], sub["edge_dst"])]
    m = np.array([p == (1, 0) for p in players])
    np.testing.assert_allclose(game.logits(m), y, rtol=1e-13)


@pytest.mark.parametrize("seed", range(4))
def test_dense_and_sparse_forms_agree(seed):
    indptr, indices = W.random_digraph(40, 150, seed=seed, symmetric=True)
    X = W.gaussian_features(40, 6, seed)
    Ws, bs = W.glorot_gcn([6, 5, 4, 3], seed + 1, bias="random")
    sub = subgraph.extract(indptr, indices, 3, 3)
    game = gcn.Game(sub, X, Ws, bs)
    rng = np.random.default_rng(seed)
    for _ in range(10):
        m = rng.random(sub["num_edges"]) < 0.5
        np.testing.assert_allclose(game.logits(m), gcn.forward_dense(sub, X, Ws, bs, m),
                                   rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_empty_coalition_and_prediction_pruning(seed):
    """f(empty) is the MLP on x_v; any coalition without an in-edge of v gives
    exactly f(empty) (Sec. 3.4.1)."""
    indptr, indices = W.random_digraph(40, 150, seed=seed, symmetric=True)
    X = W.gaussian_features(40, 6, seed)
    Ws, bs = W.glorot_gcn([6, 5, 3], seed + 1, bias="random")
    v = int(np.argmax(np.diff(indptr)))
    sub = subgraph.extract(indptr, indices, v, 2)
    game = gcn.Game(sub, X, Ws, bs)
    f0 = game.logits(np.zeros(sub["num_edges"], bool))
    np.testing.assert_allclose(f0, gcn.mlp_at_target(X[v], Ws, bs), rtol=1e-13, atol=1e-14)
    deg_v = sub["dst_ptr"][1]
    rng = np.random.default_rng(seed)
    for _ in range(10):
        m = rng.random(sub["num_edges"]) < 0.6
        m[:deg_v] = False
        np.testing.assert_allclose(game.logits(m), f0, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("seed", range(5))
def test_exhaustive_kernel_shap_equals_exact_shapley(seed):
    """Kernel SHAP over every coalition with the eq. 3 weights and the two
    infinite-weight constraints reproduces eq. 1 exactly."""
    indptr, indices, X, Ws, bs, v, sub = _small_problem(seed)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, Ws, bs)
    game.cls = gcn.predicted_class(game.logits(np.ones(M, bool)))
    vals = shapley.all_values(game, M)
    exact = shapley.exact_shapley(vals, M)
    pl = sampler.plan(M, 2 ** M - 2)
    masks, w = sampler.sample(pl, seed=1, stream=v)
    y = game.values(masks)
    phi = wls.kernel_shap(masks, w, y, vals[0], vals[-1])
    np.testing.assert_allclose(phi, exact, rtol=0, atol=1e-9 * max(1.0, np.abs(exact).max()))
    # efficiency (eq. 1 sums to f(full) - f(empty))
    assert abs(exact.sum() - (vals[-1] - vals[0])) < 1e-12


def test_efficiency_holds_for_any_sample_set():
    indptr, indices, X, Ws, bs, v, sub = _small_problem(11, n=30, edges=60, m_lo=20, m_hi=80)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, Ws, bs, cls=0)
    pl = sampler.plan(M, 600)
    masks, w = sampler.sample(pl, seed=3, stream=v)
    y = game.values(masks)
    f0, f1 = game(np.zeros(M, bool)), game(np.ones(M, bool))
    phi = wls.kernel_shap(masks, w, y, f0, f1)
    assert abs(phi.sum() - (f1 - f0)) < 1e-10


def test_additive_game_is_recovered_exactly():
    rng = np.random.default_rng(5)
    M = 37
    a = rng.normal(size=M)
    f0 = 0.7
    pl = sampler.plan(M, 4000)
    masks, w = sampler.sample(pl, seed=8, stream=1)
    y = f0 + masks @ a
    phi = wls.kernel_shap(masks, w, y, f0, f0 + a.sum())
    np.testing.assert_allclose(phi, a, atol=1e-10)


def test_symmetry_and_dummy_axioms():
    """Two leaves with identical features feeding the same node get equal
    exact values; a player that never changes the game gets zero."""
    # leaves 3, 4 -> node 1 -> v=0, plus 2 -> 0 ; leaves 3 and 4 share features
    indptr, indices = W.in_csr_from_directed(5, [1, 2, 3, 4], [0, 0, 1, 1])
    X = W.gaussian_features(5, 4, 31)
    X[4] = X[3]
    Ws, bs = W.glorot_gcn([4, 3, 2], 32, bias="random")
    sub = subgraph.extract(indptr, indices, 0, 2)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, Ws, bs, cls=1)
    vals = shapley.all_values(game, M)
    exact = shapley.exact_shapley(vals, M)
    g = sub["node_gid"]
    players = [(int(g[s]), int(g[d])) for s, d in zip(sub["edge_src"], sub["edge_dst"])]
    i3, i4 = players.index((3, 1)), players.index((4, 1))
    assert abs(exact[i3] - exact[i4]) < 1e-12
    pl = sampler.plan(M, 2 ** M - 2)
    masks, w = sampler.sample(pl, seed=1, stream=0)
    phi = wls.kernel_shap(masks, w, game.values(masks), vals[0], vals[-1])
    assert abs(phi[i3] - phi[i4]) < 1e-10
    # dummy player: a synthetic game that ignores player 2
    rng = np.random.default_rng(2)
    table = rng.normal(size=1 << M)
    dummy = 2

    def g2(m):
        m = np.array(m, bool).copy()
        m[dummy] = False
        return table[int((m * (1 << np.arange(M))).sum())]

    vals2 = shapley.all_values(g2, M)
    ex2 = shapley.exact_shapley(vals2, M)
    assert abs(ex2[dummy]) < 1e-12
    phi2 = wls.kernel_shap(masks, w, np.array([g2(m) for m in masks]), vals2[0], vals2[-1])
    assert abs(phi2[dummy]) < 1e-10


# -- the batched game and the normal-equation solve, pinned against the forms above -------

@pytest.mark.parametrize("L,hops", [(1, 1), (1, 2), (2, 1), (2, 2), (2, 3), (3, 2), (3, 3), (4, 3)])
def test_values_many_equals_per_coalition_game(L, hops):
    """gcn.values_many (the layer formula over a batch of coalitions, rows
    without entering players computed once) gives Game.values (one sparse
    normalised adjacency per coalition, pinned above against the dense
    textbook form and closed forms) to 1e-12, with tiny batches so that the
    chunking is exercised, on random coalitions including the empty and full
    ones."""
    dims = [5, 7, 6, 4, 3][:L] + [3]
    for seed in range(3):
        indptr, indices = W.random_digraph(45, 140, seed=seed + 10 * L + hops, symmetric=True)
        X = W.gaussian_features(45, dims[0], seed + 1)
        Ws, bs = W.glorot_gcn(dims, seed + 2, bias="random")
        for v in range(0, 45, 4):
            sub = subgraph.extract(indptr, indices, v, hops)
            M = sub["num_edges"]
            if M < 1:
                continue
            game = gcn.Game(sub, X, Ws, bs, cls=v % dims[-1])
            rng = np.random.default_rng(v + seed)
            masks = rng.random((23, M)) < rng.random((23, 1))
            masks[0] = False
            masks[1] = True
            want = game.values(masks)
            got = gcn.values_many(game, masks, chunk_bytes=3000)
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12 * max(1.0, np.abs(want).max()))


def test_values_many_hub_target_many_players():
    """A target whose in-neighbours have hundreds of players each, with edges
    between in-neighbours (sources whose degree varies with the coalition)."""
    rng = np.random.default_rng(4)
    n, src, dst = 3000, [], []
    for x in range(1, 9):
        src.append(x)
        dst.append(0)
        s = rng.choice(np.arange(9, n), size=int(rng.integers(100, 400)), replace=False)
        src += s.tolist()
        dst += [x] * s.size
    src += [1, 2, 3]
    dst += [2, 3, 5]
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, 12, 5)
    Ws, bs = W.glorot_gcn([12, 32, 7], 6, bias="random")
    sub = subgraph.extract(indptr, indices, 0, 2)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, Ws, bs, cls=3)
    pl = sampler.plan(M, 300)
    masks, _ = sampler.sample(pl, seed=9, stream=0)
    np.testing.assert_allclose(gcn.values_many(game, masks), game.values(masks), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("M,p", [(5, 30), (9, 200), (40, 600), (150, 2000), (300, 3000)])
def test_normal_equation_solve_equals_lstsq(M, p):
    """wls.kernel_shap_normal (Cholesky of the normal equations) gives the
    lstsq (SVD) solution of kernel_shap to 1e-9 of max|phi| on sampled rows
    of random games, and keeps efficiency exact."""
    rng = np.random.default_rng(M)
    pl = sampler.plan(M, p)
    masks, w = sampler.sample(pl, seed=4, stream=M)
    inter = rng.normal(size=(M, M)) / M
    y = masks @ rng.normal(size=M) + 0.3 * np.einsum("bi,ij,bj->b", masks, inter, masks) + 0.1
    f0, f1 = 0.1, float(y.max())
    a = wls.kernel_shap(masks, w, y, f0, f1)
    b = wls.kernel_shap_normal(masks, w, y, f0, f1, chunk=97)
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-9 * np.abs(a).max())
    assert abs(b.sum() - (f1 - f0)) < 1e-10


@pytest.mark.parametrize("seed", range(3))
def test_normal_equation_solve_exhaustive_equals_exact_shapley(seed):
    """Over every coalition the normal-equation solve reproduces eq. 1."""
    indptr, indices, X, Ws, bs, v, sub = _small_problem(seed)
    M = sub["num_edges"]
    game = gcn.Game(sub, X, Ws, bs)
    game.cls = gcn.predicted_class(game.logits(np.ones(M, bool)))
    vals = shapley.all_values(game, M)
    exact = shapley.exact_shapley(vals, M)
    pl = sampler.plan(M, 2 ** M - 2)
    masks, w = sampler.sample(pl, seed=1, stream=v)
    phi = wls.kernel_shap_normal(masks, w, gcn.values_many(game, masks), vals[0], vals[-1])
    np.testing.assert_allclose(phi, exact, rtol=0, atol=1e-9 * max(1.0, np.abs(exact).max()))


def test_normal_equation_solve_recovers_additive_game():
    rng = np.random.default_rng(6)
    M = 120
    a = rng.normal(size=M)
    f0 = -0.4
    pl = sampler.plan(M, 4000)
    masks, w = sampler.sample(pl, seed=2, stream=3)
    phi = wls.kernel_shap_normal(masks, w, f0 + masks @ a, f0, f0 + a.sum())
    np.testing.assert_allclose(phi, a, atol=1e-9)
