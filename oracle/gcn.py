"""The coalition game f(S) (Sec. 2.2-2.3, Sec. 3.4, Sec. 4.2).

A coalition S is a subset of the players (directed edges of the pruned
computational graph).  f(S) is the GCN run on the computational graph with
only the edges of S present; a missing edge is removed from the adjacency,
nodes and features stay (the "background" of eq. 2 for an edge player is its
absence).  The GCN layer is the symmetric-normalised one with self loops:

    A_S[w, u] = 1 iff (u -> w) in S
    deg_S(x)  = 1 + sum_u A_S[x, u]                 (in-degree + self loop)
    Ahat_S    = D_S^-1/2 (A_S + I) D_S^-1/2
    H^0 = X[V_c],  H^l = Ahat_S H^(l-1) W_l + 1 b_l^T,  ReLU after every
    layer except the last.

f(S) is the last layer's output at the target (local node 0) for one class
(a logit, no softmax).  Two implementations: a dense textbook one and a
sparse one; both fp64, pinned against each other.
"""
import numpy as np
import scipy.sparse as sp


def _as64(a):
    return np.asarray(a, dtype=np.float64)


def norm_adj_dense(sub, mask):
    n = sub["num_nodes"]
    A = np.zeros((n, n), dtype=np.float64)
    m = np.asarray(mask, dtype=bool)
    A[sub["edge_dst"][m], sub["edge_src"][m]] = 1.0
    deg = 1.0 + A.sum(axis=1)
    dm = 1.0 / np.sqrt(deg)
    return dm[:, None] * (A + np.eye(n)) * dm[None, :]


def norm_adj_sparse(sub, mask):
    n = sub["num_nodes"]
    m = np.asarray(mask, dtype=bool)
    dst = sub["edge_dst"][m]
    src = sub["edge_src"][m]
    deg = 1.0 + np.bincount(dst, minlength=n).astype(np.float64)
    dm = 1.0 / np.sqrt(deg)
    rows = np.concatenate([dst, np.arange(n)])
    cols = np.concatenate([src, np.arange(n)])
    vals = dm[rows] * dm[cols]
    return sp.csr_matrix((vals, (rows, cols)), shape=(n, n))


def forward_dense(sub, X, weights, biases, mask):
    """Logits of the target under coalition `mask` (dense textbook form)."""
    Ah = norm_adj_dense(sub, mask)
    H = _as64(X)[sub["node_gid"]]
    L = len(weights)
    for l in range(L):
        H = Ah @ H @ _as64(weights[l]) + _as64(biases[l])[None, :]
        if l < L - 1:
            H = np.maximum(H, 0.0)
    return H[0]


class Game:
    """f(S) for one target, sparse form; caches X[V_c] W_1 (a constant of the
    target, identical for every coalition)."""

    def __init__(self, sub, X, weights, biases, cls=None):
        self.sub = sub
        self.W = [_as64(w) for w in weights]
        self.b = [_as64(b) for b in biases]
        self.XW1 = _as64(X)[sub["node_gid"]] @ self.W[0]
        self.cls = cls

    def logits(self, mask):
        Ah = norm_adj_sparse(self.sub, mask)
        H = Ah @ self.XW1 + self.b[0][None, :]
        L = len(self.W)
        for l in range(1, L):
            H = np.maximum(H, 0.0)
            H = Ah @ (H @ self.W[l]) + self.b[l][None, :]
        return H[0]

    def __call__(self, mask):
        return float(self.logits(mask)[self.cls])

    def values(self, masks):
        return np.array([self(m) for m in masks], dtype=np.float64)


def mlp_at_target(x_v, weights, biases):
    """f(empty set): with no edges Ahat = I, so the GCN is an MLP on x_v."""
    h = _as64(x_v)
    L = len(weights)
    for l in range(L):
        h = h @ _as64(weights[l]) + _as64(biases[l])
        if l < L - 1:
            h = np.maximum(h, 0.0)
    return h


def predicted_class(logits):
    """argmax, ties to the lowest index."""
    logits = np.asarray(logits)
    return int(np.flatnonzero(logits == logits.max())[0])
