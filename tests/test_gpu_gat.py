"""GPU parity of the GAT variant (App. E) against the oracle's GAT game:
coalition values within the y bar (f(empty), f(E_c) and the explained class
exact), pruned coalitions equal to f(empty) exactly, Shapley values within
the phi bar, exhaustive sampling equal to the exact Shapley values of eq. 1."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gat as G
from oracle import sampler, shapley, subgraph, wls
from paper_2401_04829_amd.explainer import GatExplainer
from tests.gpu_util import masks_np, require_gpu, y_tolerance

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _say(*a):
    print(*a, flush=True)


def _cora_gat():
    cfg = W.make_config("cora")
    P = W.glorot_gat(cfg["X"].shape[1], 8, 16, 7, 41, bias="random")   # 8 heads of 16 (App. E)
    return cfg, P


def _small(seed, heads, F, C, n=60, e=200):
    indptr, indices = W.random_digraph(n, e, seed=seed, symmetric=True)
    X = W.gaussian_features(n, 12, seed + 7)
    P = W.glorot_gat(12, heads, F, C, seed + 9, bias="random")
    return indptr, indices, X, P


def _check(ex, indptr, indices, X, P, v, p, seed, rows=None, target_class=-1):
    res = ex.explain(v, p, seed, target_class=target_class)
    torch.cuda.synchronize()
    sub = subgraph.extract(indptr, indices, v, 2)
    M = sub["num_edges"]
    game = G.GatGame(sub, X, P)
    full = game.logits(np.ones(M, bool))
    cls = int(np.argmax(full)) if target_class < 0 else target_class
    game.cls = cls
    f0, f1 = game(np.zeros(M, bool)), float(full[cls])
    assert int(res.cls.item()) == cls
    fef = res.f_empty_full.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(fef - [f0, f1]) <= y_tolerance(np.array([f0, f1]), f0, f1))
    pl = sampler.plan(M, p)
    m, w_ref = sampler.sample(pl, seed, v)
    np.testing.assert_array_equal(masks_np(res.masks), sampler.pack(m))
    k = m.shape[0]
    if rows is None:
        rows = np.arange(k)
    y_ref = game.values(m[rows])
    y = res.y.cpu().numpy().astype(np.float64)
    err = np.abs(y[rows] - y_ref)
    assert (err <= y_tolerance(y_ref, f0, f1)).all(), err.max()
    dead = ~m[:, : int(sub["dst_ptr"][1])].any(axis=1)
    assert np.all(res.y.cpu().numpy()[dead] == res.f_empty_full.cpu().numpy()[0])
    return res, game, m, w_ref, (f0, f1)


@pytest.mark.parametrize("heads,F,C", [(8, 16, 7), (1, 5, 3), (3, 20, 4), (4, 64, 2)])
def test_gat_values_small_graphs(dev, heads, F, C):
    """Every coalition of several targets of random graphs, widths across
    one to four features per lane."""
    indptr, indices, X, P = _small(heads * 100 + F, heads, F, C)
    ex = GatExplainer(indptr, indices, X, P)
    deg = np.diff(indptr)
    for v in np.argsort(-deg)[:3]:
        _say("gat small", heads, F, C, int(v))
        _check(ex, indptr, indices, X, P, int(v), 600, 3)


def test_gat_cora_values_and_phi(dev):
    """Cora-shaped targets, 8 heads of 16 (App. E): sampled coalition values
    within the y bar and phi within the phi bar of the oracle's least squares
    on the oracle's own values."""
    cfg, P = _cora_gat()
    ex = GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)
    for v in cfg["targets"][:3]:
        _say("gat cora", v)
        res, game, m, w, (f0, f1) = _check(ex, cfg["indptr"], cfg["indices"], cfg["X"], P, v, 2000, 7)
        assert int(res.info.item()) == 0
        phi_ref = wls.kernel_shap(m, w, game.values(m), f0, f1)
        phi = res.phi.cpu().numpy().astype(np.float64)
        assert np.abs(phi - phi_ref).max() <= 1e-3 * np.abs(phi_ref).max()


def test_gat_fixed_class(dev):
    cfg, P = _cora_gat()
    ex = GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)
    v = cfg["targets"][5]
    _check(ex, cfg["indptr"], cfg["indices"], cfg["X"], P, v, 1000, 2, rows=np.arange(0, 1000, 7), target_class=3)


def test_gat_exhaustive_equals_exact_shapley(dev):
    """A target with at most 10 players and every coalition sampled: the
    GPU explanation equals eq. 1 on the oracle's GAT game."""
    indptr, indices, X, P = _small(5, 8, 16, 4, n=80, e=120)
    deg = np.diff(indptr)
    ex = GatExplainer(indptr, indices, X, P)
    done = 0
    for v in np.argsort(-deg):
        sub = subgraph.extract(indptr, indices, int(v), 2)
        M = sub["num_edges"]
        if not 3 <= M <= 10:
            continue
        _say("gat exhaustive", int(v), M)
        res = ex.explain(int(v), 2 ** M - 2, 1)
        torch.cuda.synchronize()
        game = G.GatGame(sub, X, P)
        game.cls = int(np.argmax(game.logits(np.ones(M, bool))))
        assert int(res.cls.item()) == game.cls
        codes = np.arange(1 << M)
        table = np.array([game(((codes[i] >> np.arange(M)) & 1).astype(bool)) for i in range(1 << M)])
        exact = shapley.exact_shapley(table, M)
        phi = res.phi.cpu().numpy().astype(np.float64)
        assert np.abs(phi - exact).max() <= 1e-3 * np.abs(exact).max()
        done += 1
        if done == 2:
            break
    assert done > 0


def test_gat_batch_equals_single(dev):
    """gnnshap_gat_explain_batch (App. E through the batched entry points):
    for 12 Cora-shaped targets, with targets of a different fixed class as
    well, every output (masks, weights, coalition values, f(empty), f(E_c),
    class, phi, info) equals the single-target calls' bit for bit, and the
    batch's phi of the first target is within the phi bar of the oracle's
    least squares on the oracle's GAT values."""
    cfg, P = _cora_gat()
    ex = GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)
    targets = [int(v) for v in cfg["targets"][:12]]
    for target_class in (-1, 2):
        _say("gat batch", len(targets), "targets, class", target_class)
        batch = ex.explain_batch(targets, 2000, 7, target_class=target_class)
        torch.cuda.synchronize()
        for i, v in enumerate(targets):
            b = batch[i]
            s = ex.explain(v, 2000, 7, target_class=target_class)
            torch.cuda.synchronize()
            for name in ("masks", "weights", "y", "f_empty_full", "cls", "phi", "info"):
                assert torch.equal(getattr(b, name), getattr(s, name)), (v, target_class, name)
    b = ex.explain_batch(targets[:1], 2000, 7)[0]
    torch.cuda.synchronize()
    sub = subgraph.extract(cfg["indptr"], cfg["indices"], targets[0], 2)
    M = sub["num_edges"]
    game = G.GatGame(sub, cfg["X"], P)
    game.cls = int(np.argmax(game.logits(np.ones(M, bool))))
    assert int(b.cls.item()) == game.cls
    pl = sampler.plan(M, 2000)
    m, w = sampler.sample(pl, 7, targets[0])
    np.testing.assert_array_equal(masks_np(b.masks), sampler.pack(m))
    f0, f1 = game(np.zeros(M, bool)), game(np.ones(M, bool))
    phi_ref = wls.kernel_shap(m, w, game.values(m), f0, f1)
    phi = b.phi.cpu().numpy().astype(np.float64)
    assert np.abs(phi - phi_ref).max() <= 1e-3 * np.abs(phi_ref).max()
