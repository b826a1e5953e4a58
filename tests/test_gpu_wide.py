"""GPU parity of the coalition values of two- and three-layer GCNs with wide
hidden layers on two hops, and three-layer GCNs on three hops (the MFMA
contraction of each layer at the nodes that players enter; for three layers
the dense transform by W_2 between them), against the fp64 oracle game
(Sec. 3.4, GCN of Sec. 4.2).

Bar: |y_gpu - y_ref| <= 1e-4 max(|y_ref|, |f(E_c)|, |f(empty)|); rows
without an in-edge of the target equal the device's f(empty) exactly.
Cases: hidden widths of 3 to 17 feature tiles (one, two and three feature
blocks), two and three layers (layer-2 widths above, equal to and below
layer 1's), in-neighbours with hundreds of players (many 64-player windows
at unaligned offsets), edges between in-neighbours (players whose source
has a coalition-dependent degree), random biases, arbitrary masks with an
odd row count through gnnshap_eval_coalitions, and the sampler's complement
pairs through the single-target and batched explanations (equal bit for
bit).  Several passes over the rows of a three-layer model are covered at
full size (the ogbn-arxiv-shaped targets of the parity tests).  Three hops:
second-hop nodes with many in-edges from the third hop, edges between
first- and second-hop nodes, layer 2 needed only at the target and its
in-neighbours.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gcn, sampler, subgraph
from paper_2401_04829_amd import _lib as L
from paper_2401_04829_amd.explainer import _vp
from tests.gpu_util import explainer_for, masks_np, require_gpu, y_tolerance

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _say(*a):
    print(*a, flush=True)


def _hub_graph(seed, n_nb, n, extra, feat, dims):
    """Node 0 with n_nb in-neighbours (1..n_nb), each with many in-edges of
    its own, a few edges between in-neighbours, and random edges."""
    rng = np.random.default_rng(seed)
    src, dst = [], []
    for x in range(1, n_nb + 1):
        src.append(x)
        dst.append(0)
        deg = int(rng.integers(20, 260))
        s = rng.choice(np.arange(n_nb + 1, n), size=deg, replace=False)
        src.extend(s.tolist())
        dst.extend([x] * deg)
    for _ in range(max(1, n_nb // 2)):                       # triangles through the target
        a, b = rng.choice(np.arange(1, n_nb + 1), size=2, replace=False)
        src.append(int(a))
        dst.append(int(b))
    src.extend(rng.integers(0, n, extra).tolist())
    dst.extend(rng.integers(0, n, extra).tolist())
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, feat, seed + 1)
    Ws, bs = W.glorot_gcn(dims, seed + 2, bias="random")
    return dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=2)


def _ref(cfg, v, target_class=-1):
    sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
    M = sub["num_edges"]
    game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"])
    logits = game.logits(np.ones(M, bool))
    cls = gcn.predicted_class(logits) if target_class < 0 else target_class
    srt = np.sort(logits)[::-1]
    if target_class < 0 and srt[0] - srt[1] < 1e-5 * max(1.0, abs(srt[0])):
        pytest.skip("predicted class is a near tie")
    game.cls = cls
    return sub, game, cls, game(np.zeros(M, bool)), float(logits[cls])


def _check_y(y_gpu, masks_bool, game, f0, f1, fef_dev, deg_v):
    y_ref = game.values(masks_bool)
    err = np.abs(y_gpu.astype(np.float64) - y_ref)
    tol = y_tolerance(y_ref, f0, f1)
    bad = np.flatnonzero(err > tol)
    assert bad.size == 0, f"{bad.size} rows off, worst {err.max():.3e} vs tol {tol[bad[0]]:.3e}"
    pruned = ~masks_bool[:, :deg_v].any(axis=1)
    assert (y_gpu[pruned] == fef_dev[0]).all()


# hidden widths and classes: two-layer, then three-layer models
WIDTHS = [((48,), 5), ((64,), 3), ((128,), 41), ((272,), 7),
          ((48, 64), 5), ((64, 48), 3), ((256, 256), 40), ((80, 272), 7)]


@pytest.mark.parametrize("hid,C", WIDTHS)
def test_wide_arbitrary_masks(dev, hid, C):
    """gnnshap_eval_coalitions on random (not complement-paired) masks, odd k."""
    h = hid[0] if len(hid) == 1 else hid[0] + 3 * hid[-1]   # a seed per model
    cfg = _hub_graph(40 + h, 6, 1500, 800, 24, [24, *hid, C])
    ex = explainer_for(cfg)
    ex.prepare()
    v = 0
    sub_ref, game, cls, f0, f1 = _ref(cfg, v)
    M = sub_ref["num_edges"]
    rng = np.random.default_rng(h)
    k = 301
    dens = rng.uniform(0.02, 0.98, size=(k, 1))
    mb = rng.random((k, M)) < dens
    mb[0] = False
    mb[1] = True
    mb[2, :] = rng.random(M) < 0.5
    mb[2, :sub_ref["dst_ptr"][1]] = False                     # a pruned row
    masks = torch.from_numpy(sampler.pack(mb).view(np.int64)).to(dev)
    sub = ex.extract(v)
    wpr = (M + 63) // 64
    y = torch.empty(k, dtype=torch.float32, device=dev)
    fef = torch.empty(2, dtype=torch.float32, device=dev)
    cl = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_eval_workspace(sub.sg, ex.model, k), dtype=torch.uint8, device=dev)
    _say("wide arbitrary", hid, C, M, k)
    L.gnnshap_eval_coalitions(sub.sg, ex.model, _vp(ex.X), -1, _vp(masks), k, wpr, _vp(y), _vp(fef), _vp(cl),
                              _vp(ws), ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(cl.item()) == cls
    fe = fef.cpu().numpy()
    t0 = y_tolerance(np.array([f0, f1]), f0, f1)
    assert abs(fe[0] - f0) <= t0[0] and abs(fe[1] - f1) <= t0[1]
    _check_y(y.cpu().numpy(), mb, game, f0, f1, fe, sub_ref["dst_ptr"][1])


@pytest.mark.parametrize("hid,C", WIDTHS)
def test_wide_sampled_pairs_single_and_batch(dev, hid, C):
    """The sampler's complement pairs: every row through explain() and through
    explain_batch (bit-identical), against the oracle."""
    h = hid[0] if len(hid) == 1 else hid[0] + 3 * hid[-1]   # a seed per model
    cfg = _hub_graph(70 + h, 9, 2500, 1500, 20, [20, *hid, C])
    ex = explainer_for(cfg)
    ex.prepare()
    targets = [0, 1, 3]
    p, seed = 2000, 123
    singles = []
    for v in targets:
        sub_ref, game, cls, f0, f1 = _ref(cfg, v)
        M = sub_ref["num_edges"]
        if M < 2:
            continue
        _say("wide pairs", hid, C, v, M)
        r = ex.explain(v, p, seed)
        torch.cuda.synchronize()
        pl = sampler.plan(M, p)
        mb, _ = sampler.sample(pl, seed, v)
        np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(mb))
        _check_y(r.y.cpu().numpy(), mb, game, f0, f1, r.f_empty_full.cpu().numpy(), sub_ref["dst_ptr"][1])
        singles.append((v, r.y.clone(), r.phi.clone(), r.f_empty_full.clone()))
    res = ex.explain_batch([v for v, *_ in singles], p, seed)
    torch.cuda.synchronize()
    for t, (v, y1, phi1, fef1) in enumerate(singles):
        e = res[t]
        assert torch.equal(e.y, y1), v
        assert torch.equal(e.f_empty_full, fef1), v
        assert torch.equal(e.phi, phi1), v


def test_wide_odd_k_rejected_for_sampled_entry(dev):
    cfg = _hub_graph(9, 3, 400, 100, 8, [8, 64, 3])
    ex = explainer_for(cfg)
    ex.prepare()
    sub = ex.extract(0)
    M = sub.sg.num_edges
    wpr = (M + 63) // 64
    k = 5
    masks = torch.zeros((k, wpr), dtype=torch.int64, device=dev)
    y = torch.empty(k, dtype=torch.float32, device=dev)
    fef = torch.empty(2, dtype=torch.float32, device=dev)
    ws = torch.empty(L.gnnshap_eval_workspace(sub.sg, ex.model, k), dtype=torch.uint8, device=dev)
    with pytest.raises(L.GnnShapError):
        L.gnnshap_eval_sampled_coalitions(sub.sg, ex.model, _vp(ex.X), -1, _vp(masks), k, wpr, _vp(y), _vp(fef),
                                          None, _vp(ws), ws.numel(), torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("hid,C", [((48,), 5), ((64, 48), 3)])
def test_wide_every_source_in_h1(dev, hid, C):
    """A star (the target and its leaves, edges both ways): every player's
    source is in H_1, so no node lies outside it and the contraction has no
    operand rows; all of layer 1 (and layer 2) comes from the epilogue."""
    n = 40
    src = list(range(1, n)) + [0] * (n - 1)
    dst = [0] * (n - 1) + list(range(1, n))
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, 16, 3)
    Ws, bs = W.glorot_gcn([16, *hid, C], 4, bias="random")
    cfg = dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=2)
    ex = explainer_for(cfg)
    ex.prepare()
    sub_ref, game, cls, f0, f1 = _ref(cfg, 0)
    assert sub_ref["num_nodes"] == sub_ref["dst_ptr"].shape[0] - 1   # no node outside H_1
    M = sub_ref["num_edges"]
    p, seed = 3000, 5
    _say("wide star", hid, C, M)
    r = ex.explain(0, p, seed)
    torch.cuda.synchronize()
    mb, _ = sampler.sample(sampler.plan(M, p), seed, 0)
    np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(mb))
    _check_y(r.y.cpu().numpy(), mb, game, f0, f1, r.f_empty_full.cpu().numpy(), sub_ref["dst_ptr"][1])


def _deep_graph(seed, n_nb, n, extra, feat, dims):
    """Three hops: node 0 with n_nb in-neighbours (1..n_nb), each with two to
    six in-neighbours of its own among the next nodes (the second hop), each
    of those with 20 to 200 in-edges from the rest (the third hop), a few
    edges between first- and second-hop nodes, and random edges."""
    rng = np.random.default_rng(seed)
    src, dst = [], []
    nxt = n_nb + 1
    second = []
    for x in range(1, n_nb + 1):
        src.append(x)
        dst.append(0)
        for _ in range(int(rng.integers(2, 7))):
            src.append(nxt)
            dst.append(x)
            second.append(nxt)
            nxt += 1
    for y in second:
        deg = int(rng.integers(20, 201))
        s = rng.choice(np.arange(nxt, n), size=deg, replace=False)
        src.extend(s.tolist())
        dst.extend([y] * deg)
    near = np.arange(1, nxt)
    for _ in range(len(second) // 2):
        a, b = rng.choice(near, size=2, replace=False)
        src.append(int(a))
        dst.append(int(b))
    src.extend(rng.integers(0, n, extra).tolist())
    dst.extend(rng.integers(0, n, extra).tolist())
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, feat, seed + 1)
    Ws, bs = W.glorot_gcn(dims, seed + 2, bias="random")
    return dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=3)


DEEP = [((64, 64), 3), ((48, 80), 5), ((272, 48), 7)]


@pytest.mark.parametrize("hid,C", DEEP)
def test_wide_three_hops_arbitrary_masks(dev, hid, C):
    """Three layers on three hops through gnnshap_eval_coalitions: random
    masks, odd k, every row against the oracle."""
    cfg = _deep_graph(200 + hid[0] + 3 * hid[1], 6, 6000, 300, 24, [24, *hid, C])
    ex = explainer_for(cfg)
    ex.prepare()
    sub_ref, game, cls, f0, f1 = _ref(cfg, 0)
    M = sub_ref["num_edges"]
    hp = sub_ref["hop_ptr"]
    assert hp[3] > hp[2] + 10 and sub_ref["num_nodes"] > hp[3]    # a real second and third hop
    rng = np.random.default_rng(hid[0])
    k = 201
    mb = rng.random((k, M)) < rng.uniform(0.02, 0.98, size=(k, 1))
    mb[0] = False
    mb[1] = True
    masks = torch.from_numpy(sampler.pack(mb).view(np.int64)).to(dev)
    sub = ex.extract(0)
    wpr = (M + 63) // 64
    y = torch.empty(k, dtype=torch.float32, device=dev)
    fef = torch.empty(2, dtype=torch.float32, device=dev)
    cl = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_eval_workspace(sub.sg, ex.model, k), dtype=torch.uint8, device=dev)
    _say("wide three hops, arbitrary masks", hid, C, M, k)
    L.gnnshap_eval_coalitions(sub.sg, ex.model, _vp(ex.X), -1, _vp(masks), k, wpr, _vp(y), _vp(fef), _vp(cl),
                              _vp(ws), ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(cl.item()) == cls
    fe = fef.cpu().numpy()
    t0 = y_tolerance(np.array([f0, f1]), f0, f1)
    assert abs(fe[0] - f0) <= t0[0] and abs(fe[1] - f1) <= t0[1]
    _check_y(y.cpu().numpy(), mb, game, f0, f1, fe, sub_ref["dst_ptr"][1])


@pytest.mark.parametrize("hid,C", DEEP[:2])
def test_wide_three_hops_pairs_single_and_batch(dev, hid, C):
    """Three layers on three hops, the sampler's complement pairs: explain()
    for three targets against the oracle, explain_batch equal bit for bit
    (5,000 coalitions for 900 to 1,800 players)."""
    cfg = _deep_graph(300 + hid[0] + 3 * hid[1], 3, 4000, 150, 20, [20, *hid, C])
    ex = explainer_for(cfg)
    ex.prepare()
    p, seed = 5000, 29
    singles = []
    for v in (0, 1, 2):
        sub_ref, game, cls, f0, f1 = _ref(cfg, v)
        M = sub_ref["num_edges"]
        if M < 2:
            continue
        _say("wide three hops, pairs", hid, C, v, M)
        r = ex.explain(v, p, seed)
        torch.cuda.synchronize()
        mb, _ = sampler.sample(sampler.plan(M, p), seed, v)
        np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(mb))
        _check_y(r.y.cpu().numpy(), mb, game, f0, f1, r.f_empty_full.cpu().numpy(), sub_ref["dst_ptr"][1])
        assert int(r.info.item()) == 0 and bool(torch.isfinite(r.phi).all()), v
        singles.append((v, r.y.clone(), r.phi.clone(), r.f_empty_full.clone()))
    res = ex.explain_batch([v for v, *_ in singles], p, seed)
    torch.cuda.synchronize()
    for t, (v, y1, phi1, fef1) in enumerate(singles):
        e = res[t]
        assert torch.equal(e.y, y1), v
        assert torch.equal(e.f_empty_full, fef1), v
        assert torch.equal(e.phi, phi1), v


def _wide_hub300():
    """Target 0 with 300 in-neighbours (three in-edges each from outside,
    some edges between them), 512-wide hidden layers: a row of H1 and Z2 for
    the 301 nodes of H_1 and its complement takes 2.5 MB, so the three-layer
    path runs in passes of 256 rows."""
    rng = np.random.default_rng(7)
    n, n_nb = 2000, 300
    src, dst = [], []
    for x in range(1, n_nb + 1):
        src.append(x)
        dst.append(0)
        s = rng.choice(np.arange(n_nb + 1, n), size=3, replace=False)
        src += s.tolist()
        dst += [x] * 3
    for _ in range(20):
        a, b = rng.choice(np.arange(1, n_nb + 1), size=2, replace=False)
        src.append(int(a))
        dst.append(int(b))
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, 16, 8)
    Ws, bs = W.glorot_gcn([16, 512, 512, 6], 9, bias="random")
    return dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=2)


def test_wide_three_layers_several_passes(dev):
    """Three layers over several passes of rows (the last one ragged), with
    arbitrary masks (1,001 rows: passes 256, 256, 256, 233) and with the
    sampler's complement pairs (each pass also writes the complements)."""
    cfg = _wide_hub300()
    ex = explainer_for(cfg)
    ex.prepare()
    sub_ref, game, cls, f0, f1 = _ref(cfg, 0)
    M = sub_ref["num_edges"]
    deg_v = sub_ref["dst_ptr"][1]
    rng = np.random.default_rng(11)
    k = 1001
    mb = rng.random((k, M)) < rng.uniform(0.02, 0.98, size=(k, 1))
    mb[0] = False
    mb[1] = True
    masks = torch.from_numpy(sampler.pack(mb).view(np.int64)).to(dev)
    sub = ex.extract(0)
    wpr = (M + 63) // 64
    y = torch.empty(k, dtype=torch.float32, device=dev)
    fef = torch.empty(2, dtype=torch.float32, device=dev)
    cl = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_eval_workspace(sub.sg, ex.model, k), dtype=torch.uint8, device=dev)
    _say("wide three layers, arbitrary masks", M, k)
    L.gnnshap_eval_coalitions(sub.sg, ex.model, _vp(ex.X), -1, _vp(masks), k, wpr, _vp(y), _vp(fef), _vp(cl),
                              _vp(ws), ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(cl.item()) == cls
    fe = fef.cpu().numpy()
    _check_y(y.cpu().numpy(), mb, game, f0, f1, fe, deg_v)
    p, seed = 2000, 17
    _say("wide three layers, complement pairs", M, p)
    r = ex.explain(0, p, seed)
    torch.cuda.synchronize()
    ms, _ = sampler.sample(sampler.plan(M, p), seed, 0)
    np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(ms))
    _check_y(r.y.cpu().numpy(), ms, game, f0, f1, r.f_empty_full.cpu().numpy(), deg_v)
