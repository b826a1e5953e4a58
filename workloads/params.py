"""Seeded node features and random-init GCN parameters (fp32)."""
import numpy as np


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def binary_features(n, d, density, seed):
    """Bag-of-words-like 0/1 features, Bernoulli(density)."""
    return (_rng(seed).random((n, d), dtype=np.float32) < density).astype(np.float32)


def tfidf_features(n, d, density, seed):
    """Non-negative TF-IDF-like rows: ~density non-zeros drawn from a
    log-normal, each row L1-normalised."""
    rng = _rng(seed)
    nz = rng.random((n, d), dtype=np.float32) < density
    vals = np.exp(rng.normal(0.0, 1.0, size=(n, d))).astype(np.float32)
    x = np.where(nz, vals, np.float32(0.0))
    s = x.sum(axis=1, keepdims=True)
    return (x / np.where(s > 0, s, 1.0)).astype(np.float32)


def gaussian_features(n, d, seed):
    return _rng(seed).standard_normal((n, d), dtype=np.float32)


def glorot_gcn(dims, seed, bias="zero"):
    """Glorot-uniform weights W_l of shape dims[l] x dims[l+1], U(+-sqrt(6/(fan_in+fan_out)));
    biases zero (`bias="zero"`) or U(-0.1, 0.1) (`bias="random"`)."""
    rng = _rng(seed)
    Ws, bs = [], []
    for l in range(len(dims) - 1):
        a = np.sqrt(6.0 / (dims[l] + dims[l + 1]))
        Ws.append(rng.uniform(-a, a, size=(dims[l], dims[l + 1])).astype(np.float32))
        if bias == "zero":
            bs.append(np.zeros(dims[l + 1], dtype=np.float32))
        else:
            bs.append(rng.uniform(-0.1, 0.1, size=dims[l + 1]).astype(np.float32))
    return Ws, bs


def glorot_gat(d, heads, head_dim, classes, seed, bias="zero"):
    """Random-init parameters of a two-layer GAT: layer 1 `heads` heads of
    width `head_dim` (outputs concatenated), layer 2 one head of width
    `classes`.  Weights and attention vectors Glorot-uniform, biases zero or
    U(-0.1, 0.1).  Returned as a dict of fp32 arrays: W1 [d, heads*head_dim],
    att_src1 / att_dst1 [heads, head_dim], b1 [heads*head_dim],
    W2 [heads*head_dim, classes], att_src2 / att_dst2 [classes], b2 [classes]."""
    rng = _rng(seed)
    hf = heads * head_dim

    def glorot(shape, fan_in, fan_out):
        a = np.sqrt(6.0 / (fan_in + fan_out))
        return rng.uniform(-a, a, size=shape).astype(np.float32)

    def b(n):
        if bias == "zero":
            return np.zeros(n, dtype=np.float32)
        return rng.uniform(-0.1, 0.1, size=n).astype(np.float32)

    return dict(W1=glorot((d, hf), d, hf), att_src1=glorot((heads, head_dim), head_dim, 1),
                att_dst1=glorot((heads, head_dim), head_dim, 1), b1=b(hf),
                W2=glorot((hf, classes), hf, classes), att_src2=glorot((classes,), classes, 1),
                att_dst2=glorot((classes,), classes, 1), b2=b(classes))
