"""Pruned computational graph of a target node (Sec. 3.2, App. A, Fig. 2).

The graph is stored as an in-CSR: the sources of the edges u -> w are
indices[indptr[w]:indptr[w+1]], ascending.  For an l-hop explanation:

* dist(u) = length of the shortest directed path u -> ... -> v (BFS over
  in-edges starting at v); H_j = {u : dist(u) <= j}.
* Only edges whose message reaches v within l hops are kept (App. A): the
  players are E_c = {(u -> w) in E : dist(w) <= l - 1}, and V_c = H_l.
* Local node ids sort V_c by (dist, global id), so v is local node 0 and
  H_j is the prefix [0, hop_ptr[j+1]).
* Players are ordered by (local destination, position in the CSR), i.e. by
  (local destination, source global id); the players whose destination is
  local node x are [dst_ptr[x], dst_ptr[x+1]).  Players 0 .. indeg(v)-1 are
  the in-edges of v.
"""
import numpy as np


def bfs_dist(indptr, indices, v, hops):
    dist = {int(v): 0}
    frontier = [int(v)]
    for d in range(1, hops + 1):
        nxt = []
        for w in frontier:
            for e in range(int(indptr[w]), int(indptr[w + 1])):
                u = int(indices[e])
                if u not in dist:
                    dist[u] = d
                    nxt.append(u)
        frontier = nxt
    return dist


def extract(indptr, indices, v, hops):
    if hops < 1:
        raise ValueError("hops must be >= 1")
    dist = bfs_dist(indptr, indices, v, hops)
    nodes = sorted(dist, key=lambda u: (dist[u], u))
    local = {u: i for i, u in enumerate(nodes)}
    hop_ptr = [0]
    for j in range(hops + 1):
        hop_ptr.append(sum(1 for u in nodes if dist[u] <= j))
    n_dst = hop_ptr[hops]                       # |H_{l-1}|
    edge_src, edge_dst, edge_gid, dst_ptr = [], [], [], [0]
    for x in range(n_dst):
        w = nodes[x]
        for e in range(int(indptr[w]), int(indptr[w + 1])):
            edge_src.append(local[int(indices[e])])
            edge_dst.append(x)
            edge_gid.append(e)
        dst_ptr.append(len(edge_src))
    return dict(
        hops=hops,
        node_gid=np.asarray(nodes, dtype=np.int64),
        dist=np.asarray([dist[u] for u in nodes], dtype=np.int64),
        hop_ptr=np.asarray(hop_ptr, dtype=np.int64),
        dst_ptr=np.asarray(dst_ptr, dtype=np.int64),
        edge_src=np.asarray(edge_src, dtype=np.int64),
        edge_dst=np.asarray(edge_dst, dtype=np.int64),
        edge_gid=np.asarray(edge_gid, dtype=np.int64),
        num_nodes=len(nodes),
        num_edges=len(edge_src),
    )
