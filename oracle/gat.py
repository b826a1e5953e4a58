"""The coalition game of a two-layer graph attention network (App. E: the
paper explains a GAT with 8 attention heads on Cora to show that the method
treats the model as a black box).

Test infrastructure: only tests/, the smoke check and the benchmark's CPU
baseline use this module.

A coalition S keeps the edges of S (players are directed edges, as for the
GCN) and every node keeps its self loop.  One GAT layer (Velickovic et al.,
ICLR 2018, with self loops) with H heads of width F maps H to

    Z = H W,  Z_h = the h-th block of F columns,
    e_h(u -> w) = LeakyReLU(a_src,h . Z_h[u] + a_dst,h . Z_h[w])  (slope 0.2),
    alpha_h(u -> w) = softmax of e_h over the edges into w present in S and
                      the self loop w -> w,
    out_h[w] = sum_u alpha_h(u -> w) Z_h[u],

heads concatenated, plus a bias.  The network: layer 1 with H heads, ELU,
layer 2 with one head of width C (the classes); f(S) is one class's output
at the target (a logit).  The softmax is renormalised under each coalition:
only present edges compete.  Two implementations, pinned against each
other: a dense one (attention matrices with absent entries at -inf) and an
edge-list one.
"""
import numpy as np


def _as64(a):
    return np.asarray(a, dtype=np.float64)


def leaky(x, slope=0.2):
    return np.where(x > 0, x, slope * x)


def elu(x):
    return np.where(x > 0, x, np.expm1(np.minimum(x, 0.0)))


def layer_dense(H, present, sub, W, a_src, a_dst, b, slope=0.2, Z=None):
    """One GAT layer with dense attention matrices: A[w, u] = 1 for present
    edges u -> w and for u = w; the softmax runs over each row's ones.  Z,
    if given, is H W (a constant of the target for the first layer)."""
    n = H.shape[0]
    a_src = _as64(a_src).reshape(-1, _as64(a_src).shape[-1])
    heads, F = a_src.shape
    a_dst = _as64(a_dst).reshape(heads, F)
    A = np.eye(n, dtype=bool)
    A[sub["edge_dst"][present], sub["edge_src"][present]] = True
    Z = (H @ _as64(W) if Z is None else Z).reshape(n, heads, F)
    out = np.zeros((n, heads, F))
    for h in range(heads):
        s = Z[:, h, :] @ a_src[h]
        d = Z[:, h, :] @ a_dst[h]
        E = leaky(d[:, None] + s[None, :], slope)
        E = np.where(A, E, -np.inf)
        P = np.exp(E - E.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        out[:, h, :] = P @ Z[:, h, :]
    return out.reshape(n, heads * F) + _as64(b)[None, :]


def layer_edges(H, present, sub, W, a_src, a_dst, b, slope=0.2, Z=None):
    """The same layer over an edge list (present edges and self loops),
    normalised per destination."""
    n = H.shape[0]
    a_src = _as64(a_src).reshape(-1, _as64(a_src).shape[-1])
    heads, F = a_src.shape
    a_dst = _as64(a_dst).reshape(heads, F)
    src = np.concatenate([sub["edge_src"][present], np.arange(n)])
    dst = np.concatenate([sub["edge_dst"][present], np.arange(n)])
    Z = (H @ _as64(W) if Z is None else Z).reshape(n, heads, F)
    s = np.einsum("nhf,hf->nh", Z, a_src)
    d = np.einsum("nhf,hf->nh", Z, a_dst)
    e = leaky(s[src] + d[dst], slope)                       # edges x heads
    mx = np.full((n, heads), -np.inf)
    np.maximum.at(mx, dst, e)
    p = np.exp(e - mx[dst])
    den = np.zeros((n, heads))
    np.add.at(den, dst, p)
    out = np.zeros((n, heads, F))
    np.add.at(out, dst, (p / den[dst])[:, :, None] * Z[src])
    return out.reshape(n, heads * F) + _as64(b)[None, :]


class GatGame:
    """f(S) of a two-layer GAT at the target (local node 0) for class `cls`."""

    def __init__(self, sub, X, params, cls=None, dense=False, slope=0.2):
        self.sub = sub
        self.p = {k: _as64(v) for k, v in params.items()}
        self.H0 = _as64(X)[sub["node_gid"]]
        self.Z1 = self.H0 @ self.p["W1"]          # X W_1 rows: the same for every coalition
        self.cls = cls
        self.layer = layer_dense if dense else layer_edges
        self.slope = slope

    def logits(self, mask):
        present = np.asarray(mask, dtype=bool)
        p = self.p
        H1 = elu(self.layer(self.H0, present, self.sub, p["W1"], p["att_src1"], p["att_dst1"], p["b1"],
                            self.slope, Z=self.Z1))
        H2 = self.layer(H1, present, self.sub, p["W2"], p["att_src2"][None, :], p["att_dst2"][None, :], p["b2"],
                        self.slope)
        return H2[0]

    def __call__(self, mask):
        return float(self.logits(mask)[self.cls])

    def values(self, masks):
        return np.array([self(m) for m in masks], dtype=np.float64)
