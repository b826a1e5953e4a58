"""The five synthetic workloads, shaped like the paper's datasets (Sec. 4.1,
Table 1, App. D) and the GCNs of Sec. 4.2.  The real datasets are not used;
these seeded graphs stand in for them.

    tiny    Cora-shaped graph (2,708 nodes, 5,278 undirected pairs), 1,433-dim
            binary features, 2-layer GCN 16 hidden / 7 classes; one target with
            a 2-hop computational graph of 50..70 edges; 2,000 samples.
    cora    same graph and GCN; the first 100 nodes of a seeded permutation
            with 20..400 players; 10,000 samples each.
    pubmed  PubMed-shaped (19,717 nodes, 44,324 pairs), 500-dim TF-IDF-like
            features, 3-layer GCN 64 hidden / 3 classes, 3-hop graphs of
            500..4,000 edges; 200 targets; 25,000 samples.
    arxiv   ogbn-arxiv-shaped (169,343 nodes, 1,166,243 pairs), 128-dim N(0,1)
            features, 3-layer GCN 256 hidden / 40 classes, 2-hop graphs of
            5,000..20,000 edges from nodes of in-degree >= the 95th percentile;
            50 targets; 50,000 samples.
    reddit  Reddit-shaped (232,965 nodes, 57,307,946 pairs, 41 communities),
            602-dim N(0,1) features, 2-layer GCN 128 hidden / 41 classes, 2-hop
            graphs of 10,000..30,000 edges; 20 targets; 100,000 samples.
"""
import functools

import numpy as np

from .graphs import chung_lu_pairs, dcsbm_pairs, in_csr_from_pairs
from .params import binary_features, tfidf_features, gaussian_features, glorot_gcn

CONFIGS = {
    "tiny": dict(graph="cora", features=("binary", 1433, 0.013), dims=[1433, 16, 7],
                 hops=2, p=2000, n_targets=1, m_range=(50, 70), seed=0x5EED0001,
                 target_seed=101, weight_seed=201),
    "cora": dict(graph="cora", features=("binary", 1433, 0.013), dims=[1433, 16, 7],
                 hops=2, p=10000, n_targets=100, m_range=(20, 400), seed=0x5EED0002,
                 target_seed=102, weight_seed=201),
    "pubmed": dict(graph="pubmed", features=("tfidf", 500, 0.10), dims=[500, 64, 64, 3],
                   hops=3, p=25000, n_targets=200, m_range=(500, 4000), seed=0x5EED0003,
                   target_seed=103, weight_seed=203),
    "arxiv": dict(graph="arxiv", features=("gauss", 128), dims=[128, 256, 256, 40],
                  hops=2, p=50000, n_targets=50, m_range=(5000, 20000), seed=0x5EED0004,
                  target_seed=104, weight_seed=204, min_indeg_quantile=0.95),
    "reddit": dict(graph="reddit", features=("gauss", 602), dims=[602, 128, 41],
                   hops=2, p=100000, n_targets=20, m_range=(10000, 30000), seed=0x5EED0005,
                   target_seed=105, weight_seed=205),
}

GRAPHS = {
    "cora": dict(kind="chung_lu", n=2708, pairs=5278, exponent=2.5, seed=11, feat_seed=21),
    "pubmed": dict(kind="chung_lu", n=19717, pairs=44324, exponent=2.5, seed=12, feat_seed=22),
    "arxiv": dict(kind="chung_lu", n=169343, pairs=1166243, exponent=2.2, seed=13, feat_seed=23),
    "reddit": dict(kind="dcsbm", n=232965, pairs=57307946, blocks=41, p_in=0.8,
                   lognormal_sigma=1.18, seed=14, feat_seed=24),
}


@functools.lru_cache(maxsize=4)
def make_graph(name):
    g = GRAPHS[name]
    if g["kind"] == "chung_lu":
        lo, hi = chung_lu_pairs(g["n"], g["pairs"], g["exponent"], g["seed"])
    else:
        rng = np.random.Generator(np.random.PCG64(g["seed"] + 1000))
        w = np.exp(rng.normal(0.0, g["lognormal_sigma"], size=g["n"]))
        lo, hi = dcsbm_pairs(g["n"], g["pairs"], g["blocks"], g["p_in"], w, g["seed"])
    indptr, indices = in_csr_from_pairs(g["n"], lo, hi)
    return indptr, indices


def _features(spec, n, seed):
    if spec[0] == "binary":
        return binary_features(n, spec[1], spec[2], seed)
    if spec[0] == "tfidf":
        return tfidf_features(n, spec[1], spec[2], seed)
    return gaussian_features(n, spec[1], seed)


def _in_neighbours(indptr, indices, nodes):
    parts = [indices[indptr[w]:indptr[w + 1]] for w in nodes]
    if not parts:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(parts).astype(np.int64)


def player_count(indptr, indices, v, hops):
    """Number of edges whose destination lies within hops-1 in-hops of v
    (the size of v's pruned computational graph); a target-selection
    statistic only."""
    seen = {int(v)}
    frontier = np.array([v], dtype=np.int64)
    for _ in range(hops - 1):
        nb = np.unique(_in_neighbours(indptr, indices, frontier))
        new = np.array([u for u in nb if int(u) not in seen], dtype=np.int64)
        seen.update(int(u) for u in new)
        frontier = new
    nodes = np.fromiter(seen, dtype=np.int64)
    return int((indptr[nodes + 1] - indptr[nodes]).sum())


def select_targets(indptr, indices, cfg):
    n = indptr.size - 1
    rng = np.random.Generator(np.random.PCG64(cfg["target_seed"]))
    perm = rng.permutation(n)
    indeg = np.diff(indptr)
    lo_m, hi_m = cfg["m_range"]
    if "min_indeg_quantile" in cfg:
        thr = np.quantile(indeg, cfg["min_indeg_quantile"])
        perm = perm[indeg[perm] >= thr]
    if cfg["hops"] == 2:
        # indeg(v) + sum of the in-degrees of v's in-neighbours (simple graph)
        nb_sum = np.add.reduceat(indeg[indices].astype(np.int64), indptr[:-1].clip(max=max(indices.size - 1, 0)))
        nb_sum = np.where(indeg > 0, nb_sum, 0)
        m_all = indeg + nb_sum
        ok = perm[(m_all[perm] >= lo_m) & (m_all[perm] <= hi_m)]
        return [int(v) for v in ok[:cfg["n_targets"]]]
    out = []
    for v in perm:
        if indeg[v] == 0:
            continue
        m = player_count(indptr, indices, v, cfg["hops"])
        if lo_m <= m <= hi_m:
            out.append(int(v))
            if len(out) == cfg["n_targets"]:
                break
    return out


@functools.lru_cache(maxsize=8)
def make_config(name):
    """All inputs of a named workload (cached per process)."""
    cfg = CONFIGS[name]
    g = GRAPHS[cfg["graph"]]
    indptr, indices = make_graph(cfg["graph"])
    X = _features(cfg["features"], g["n"], g["feat_seed"])
    Ws, bs = glorot_gcn(cfg["dims"], cfg["weight_seed"])
    targets = select_targets(indptr, indices, cfg)
    return dict(name=name, indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs,
                dims=list(cfg["dims"]), hops=cfg["hops"], p=cfg["p"], seed=cfg["seed"],
                targets=targets, m_range=cfg["m_range"])
