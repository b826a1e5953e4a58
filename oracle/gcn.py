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


def values_many(game, masks, chunk_bytes=1 << 28):
    """f(S_b) for many coalitions, the same layer formula as Game.logits
    written over a batch of coalitions at once (fp64), for workloads where a
    Python loop over every coalition is too slow.

    A node x into which no player enters has, in every A_S, only its self loop
    with d_S(x) = 1, so its row of every layer's output is the same for all
    coalitions and is computed once ("constant rows").  The nodes with
    players entering them (the destinations D) are computed per coalition:
        deg_b(x)   = 1 + number of the row's players entering x
        H^l_b[x]   = d_b(x)^-1/2 ( sum_{e -> x, e in S_b} d_b(src e)^-1/2 Z^l_b[src e]
                                  + d_b(x)^-1/2 Z^l_b[x] ) + b_l,   Z^l = H^(l-1) W_l,
    with ReLU after every layer but the last, d_b = 1 at constant rows, and the
    sum taken per destination as a product of the coalitions' coefficient
    rows with the sources' Z rows.  Returns the explained class's logit at
    the target for every row of `masks` (bool [k, M])."""
    sub = game.sub
    masks = np.asarray(masks, dtype=bool)
    k, M = masks.shape
    n = sub["num_nodes"]
    src = sub["edge_src"]
    ptr = sub["dst_ptr"]
    nd = ptr.size - 1                                   # destinations are local ids [0, nd)
    L = len(game.W)
    is_var = np.zeros(n, dtype=bool)
    is_var[:nd] = True
    var_pos = np.full(n, -1, dtype=np.int64)
    var_pos[:nd] = np.arange(nd)
    widths = [game.XW1.shape[1]] + [w.shape[1] for w in game.W[1:]]
    # constant rows of every layer's output
    Zc = [game.XW1]                                     # Z^l at every node, constant rows
    for l in range(L - 1):
        H = Zc[l] + game.b[l][None, :]
        Zc.append(np.maximum(H, 0.0) @ game.W[l + 1])
    # per destination: which players come from constant rows, and those rows of Z^l
    parts = []
    for x in range(nd):
        s = src[ptr[x]:ptr[x + 1]]
        cs = ~is_var[s]
        parts.append((s, np.flatnonzero(~cs), [np.where(cs[:, None], Zc[l][s], 0.0) for l in range(L)]))
    per_row = 8 * nd * (3 * max(widths) + 4)
    B = int(max(1, min(k, chunk_bytes // max(per_row, 1))))
    out = np.empty(k, dtype=np.float64)
    for b0 in range(0, k, B):
        m = masks[b0:b0 + B]
        nb = m.shape[0]
        cnt = np.add.reduceat(m, ptr[:-1], axis=1, dtype=np.float64) if M else np.zeros((nb, nd))
        cnt[:, ptr[:-1] == ptr[1:]] = 0.0                # reduceat's value at an empty range
        dm = 1.0 / np.sqrt(1.0 + cnt)                    # d_b^-1/2 at the destinations
        Hv = None                                       # H^(l-1) at the destinations, per row
        for l in range(L):
            Zv = np.broadcast_to(game.XW1[:nd][None], (nb, nd, widths[0])) if l == 0 else Hv @ game.W[l]
            Hn = np.empty((nb, nd, widths[l]), dtype=np.float64)
            for x in range(nd):
                e0, e1 = ptr[x], ptr[x + 1]
                s, vs, zconst = parts[x]
                mx = m[:, e0:e1]
                # players from constant rows (d = 1 there; the other rows of zconst are zero)
                acc = mx.astype(np.float64) @ zconst[l] if e1 > e0 else np.zeros((nb, widths[l]))
                if vs.size:                                   # players from rows that vary with S
                    us = var_pos[s[vs]]
                    acc += np.einsum("bj,bjh->bh", mx[:, vs] * dm[:, us], Zv[:, us, :])
                Hn[:, x, :] = dm[:, x:x + 1] * (acc + dm[:, x:x + 1] * Zv[:, x, :]) + game.b[l][None, :]
            if l < L - 1:
                Hn = np.maximum(Hn, 0.0)
            Hv = Hn
        out[b0:b0 + nb] = Hv[:, 0, game.cls]
    return out


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
