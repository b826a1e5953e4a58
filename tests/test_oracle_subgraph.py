"""Pins of the oracle's computational-graph extraction (Sec. 3.2, App. A,
Fig. 2) against brute force and closed forms."""
import numpy as np
import pytest

import workloads as W
from oracle import subgraph


def _reach_within(indptr, indices, v, k):
    """Nodes w with a directed walk w -> ... -> v of length <= k, by boolean
    matrix powers of the dense adjacency (independent of any BFS)."""
    n = indptr.size - 1
    A = np.zeros((n, n), dtype=np.int64)           # A[w, u] = 1 iff u -> w
    for w in range(n):
        A[w, indices[indptr[w]:indptr[w + 1]]] = 1
    reach = np.zeros(n, dtype=bool)
    reach[v] = True
    cur = np.zeros(n, dtype=np.int64)
    cur[v] = 1
    for _ in range(k):
        cur = (cur @ A > 0).astype(np.int64)        # one more step back along in-edges
        reach |= cur > 0
    return reach


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("hops", [1, 2, 3])
def test_players_are_edges_whose_message_reaches_target(seed, hops):
    indptr, indices = W.random_digraph(14, 30, seed=seed)
    for v in range(14):
        sub = subgraph.extract(indptr, indices, v, hops)
        dst_ok = _reach_within(indptr, indices, v, hops - 1)
        want = set()
        for w in range(14):
            if dst_ok[w]:
                for e in range(indptr[w], indptr[w + 1]):
                    want.add(e)
        assert set(sub["edge_gid"].tolist()) == want
        # every player's endpoints map back to the graph's edge
        g = sub["node_gid"]
        for s, d, e in zip(sub["edge_src"], sub["edge_dst"], sub["edge_gid"]):
            assert indices[e] == g[s]
            assert indptr[g[d]] <= e < indptr[g[d] + 1]
        # V_c = nodes within `hops`, sorted by (dist, id); v is local 0
        within = _reach_within(indptr, indices, v, hops)
        assert set(g.tolist()) == set(np.flatnonzero(within).tolist())
        assert g[0] == v
        d = sub["dist"]
        assert all((d[i], g[i]) < (d[i + 1], g[i + 1]) for i in range(len(g) - 1))
        # players sorted by (local dst, source id)
        keys = list(zip(sub["edge_dst"], g[sub["edge_src"]]))
        assert keys == sorted(keys)


def test_two_hop_player_count_closed_form():
    indptr, indices = W.random_digraph(200, 600, seed=9, symmetric=True)
    indeg = np.diff(indptr)
    for v in range(0, 200, 7):
        sub = subgraph.extract(indptr, indices, v, 2)
        nb = indices[indptr[v]:indptr[v + 1]]
        assert sub["num_edges"] == indeg[v] + indeg[nb].sum()


def test_pruned_graph_is_inside_induced_subgraph():
    """Fig. 2: pruning keeps a subset of the l-hop induced subgraph's edges and
    drops the edges between the outermost nodes."""
    indptr, indices = W.random_digraph(60, 240, seed=4, symmetric=True)
    for v in range(0, 60, 5):
        sub = subgraph.extract(indptr, indices, v, 2)
        nodes = set(sub["node_gid"].tolist())
        induced = {e for w in nodes for e in range(indptr[w], indptr[w + 1]) if indices[e] in nodes}
        kept = set(sub["edge_gid"].tolist())
        assert kept <= induced
        outer = {int(u) for u, d in zip(sub["node_gid"], sub["dist"]) if d == 2}
        for e in induced - kept:
            w = next(x for x in nodes if indptr[x] <= e < indptr[x + 1])
            assert w in outer


def test_hand_built_example():
    # edges u->w: 1->0, 2->0, 3->1, 0->1, 4->3, 3->2, 5->4
    indptr, indices = W.in_csr_from_directed(6, [1, 2, 3, 0, 4, 3, 5], [0, 0, 1, 1, 3, 2, 4])
    sub = subgraph.extract(indptr, indices, 0, 2)
    assert sub["node_gid"].tolist() == [0, 1, 2, 3]
    assert sub["hop_ptr"].tolist() == [0, 1, 3, 4]
    # players: in-edges of 0 (from 1, 2), of 1 (from 0, 3), of 2 (from 3)
    g = sub["node_gid"]
    pairs = [(int(g[s]), int(g[d])) for s, d in zip(sub["edge_src"], sub["edge_dst"])]
    assert pairs == [(1, 0), (2, 0), (0, 1), (3, 1), (3, 2)]
    assert sub["dst_ptr"].tolist() == [0, 2, 4, 5]
