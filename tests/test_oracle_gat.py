"""Pins of the oracle's GAT game (App. E; one GAT layer as in Velickovic et
al. 2018, with self loops and the softmax renormalised under each
coalition): the dense and edge-list layers agree; zero attention vectors
reduce a layer to the mean over the present in-neighbours and the node;
one present in-edge gives the logistic weight of the two logits; a
coalition without an in-edge of the target gives the closed form of the
target alone (the pruning of Sec. 3.4.1 holds for the GAT)."""
import numpy as np
import pytest

import workloads as W
from oracle import gat as G
from oracle import subgraph


def _case(seed, n=40, e=120, d=6, heads=3, F=4, C=5):
    indptr, indices = W.random_digraph(n, e, seed=seed, symmetric=True)
    X = W.gaussian_features(n, d, seed + 7)
    P = W.glorot_gat(d, heads, F, C, seed + 9, bias="random")
    deg = np.diff(indptr)
    v = int(np.argmax(deg))
    sub = subgraph.extract(indptr, indices, v, 2)
    return sub, X, P


@pytest.mark.parametrize("seed", range(4))
def test_dense_and_edge_layers_agree(seed):
    sub, X, P = _case(seed)
    M = sub["num_edges"]
    rng = np.random.default_rng(seed)
    for _ in range(5):
        mask = rng.random(M) < rng.random()
        a = G.GatGame(sub, X, P, dense=True).logits(mask)
        b = G.GatGame(sub, X, P, dense=False).logits(mask)
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_zero_attention_is_the_mean_over_present_neighbours():
    sub, X, P = _case(11)
    M = sub["num_edges"]
    n = sub["num_nodes"]
    mask = np.random.default_rng(3).random(M) < 0.5
    heads, F = P["att_src1"].shape
    H = np.asarray(X, np.float64)[sub["node_gid"]]
    out = G.layer_edges(H, mask, sub, P["W1"], np.zeros((heads, F)), np.zeros((heads, F)), P["b1"])
    Z = H @ np.asarray(P["W1"], np.float64)
    for w in range(n):
        srcs = [w] + [int(s) for s, t, on in zip(sub["edge_src"], sub["edge_dst"], mask) if on and t == w]
        want = Z[srcs].mean(axis=0) + P["b1"]
        np.testing.assert_allclose(out[w], want, rtol=1e-12, atol=1e-12)


def test_one_present_edge_is_a_logistic_mix():
    sub, X, P = _case(5)
    M = sub["num_edges"]
    heads, F = P["att_src1"].shape
    H = np.asarray(X, np.float64)[sub["node_gid"]]
    Z = (H @ np.asarray(P["W1"], np.float64)).reshape(-1, heads, F)
    for e in range(min(M, 6)):
        mask = np.zeros(M, bool)
        mask[e] = True
        u, w = int(sub["edge_src"][e]), int(sub["edge_dst"][e])
        out = G.layer_edges(H, mask, sub, P["W1"], P["att_src1"], P["att_dst1"], P["b1"]).reshape(-1, heads, F)
        for h in range(heads):
            s = lambda x: float(Z[x, h] @ P["att_src1"][h])
            d = float(Z[w, h] @ P["att_dst1"][h])
            lu = G.leaky(s(u) + d)
            lw = G.leaky(s(w) + d)
            a = 1.0 / (1.0 + np.exp(lw - lu))
            want = a * Z[u, h] + (1 - a) * Z[w, h] + P["b1"].reshape(heads, F)[h]
            np.testing.assert_allclose(out[w, h], want, rtol=1e-12, atol=1e-12)


def test_no_in_edge_of_the_target_gives_the_target_alone():
    sub, X, P = _case(8)
    M = sub["num_edges"]
    indeg_v = int(sub["dst_ptr"][1] - sub["dst_ptr"][0])
    rng = np.random.default_rng(2)
    x_v = np.asarray(X, np.float64)[sub["node_gid"][0]]
    h1 = G.elu(x_v @ np.asarray(P["W1"], np.float64) + P["b1"])
    want = h1 @ np.asarray(P["W2"], np.float64) + P["b2"]
    for _ in range(4):
        mask = rng.random(M) < 0.6
        mask[:indeg_v] = False                 # the target's in-edges come first
        np.testing.assert_allclose(G.GatGame(sub, X, P).logits(mask), want, rtol=1e-12, atol=1e-12)
