"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Bars: subgraph arrays and masks bit-exact; weights equal to the fp32 rounding
of the oracle's fp64 weights; coalition values within 1e-4 of
max(|y|, |f(E_c)|, |f(empty)|); Shapley values within 1e-3 of max|phi|.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gcn, sampler, subgraph, wls, shapley
from tests.gpu_util import (explainer_for, masks_np, require_gpu, sample_on_gpu, y_tolerance)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _say(*a):
    print(*a, flush=True)


def _small_cfg(seed, n, e, dims, hops, bias="random"):
    indptr, indices = W.random_digraph(n, e, seed=seed, symmetric=True)
    X = W.gaussian_features(n, dims[0], seed + 7)
    Ws, bs = W.glorot_gcn(dims, seed + 9, bias=bias)
    return dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=hops)


def _check_subgraph(got, ref):
    assert got.sg.num_nodes == ref["num_nodes"] and got.sg.num_edges == ref["num_edges"]
    assert got.hop_ptr == ref["hop_ptr"].tolist()
    np.testing.assert_array_equal(got.node_gid.cpu().numpy(), ref["node_gid"])
    np.testing.assert_array_equal(got.dst_ptr.cpu().numpy(), ref["dst_ptr"])
    np.testing.assert_array_equal(got.edge_src.cpu().numpy(), ref["edge_src"])
    np.testing.assert_array_equal(got.edge_dst.cpu().numpy(), ref["edge_dst"])
    np.testing.assert_array_equal(got.edge_gid.cpu().numpy(), ref["edge_gid"])


# -- 1. computational graph -----------------------------------------------------------

@pytest.mark.parametrize("hops", [1, 2, 3])
def test_extract_small_graphs_bit_exact(dev, hops):
    for seed in range(3):
        cfg = _small_cfg(seed, 60, 150, [4, 8, 3], hops)
        ex = explainer_for(cfg)
        for v in range(0, 60, 3):
            _say("extract small", seed, hops, v)
            _check_subgraph(ex.extract(v), subgraph.extract(cfg["indptr"], cfg["indices"], v, hops))
        assert int(ex.extract_ws.count_nonzero()) == 0       # workspace left zero-filled


@pytest.mark.parametrize("name", ["tiny", "cora", "pubmed"])
def test_extract_workload_targets_bit_exact(dev, name):
    cfg = W.make_config(name)
    ex = explainer_for(cfg)
    targets = cfg["targets"] if name != "pubmed" else cfg["targets"][:40]
    for v in targets:
        _say("extract", name, v)
        got = ex.extract(v)
        ref = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
        _check_subgraph(got, ref)
        lo, hi = cfg["m_range"]
        assert lo <= ref["num_edges"] <= hi


def test_extract_large_graph_multiblock_path(dev):
    """Graphs above 2^18 nodes take the multi-block extraction kernels."""
    n = 300_000
    indptr, indices = W.random_digraph(n, 1_200_000, seed=77, symmetric=True)
    cfg = dict(indptr=indptr, indices=indices, X=np.zeros((n, 4), np.float32),
               weights=[np.zeros((4, 2), np.float32)], biases=[None], hops=2)
    ex = explainer_for(cfg)
    rng = np.random.default_rng(5)
    for v in rng.integers(0, n, 12):
        for hops in (1, 2, 3):
            _say("extract large", int(v), hops)
            ex.hops = hops
            _check_subgraph(ex.extract(int(v)), subgraph.extract(indptr, indices, int(v), hops))
    assert int(ex.extract_ws.count_nonzero()) == 0


def test_extract_capacity_reports_sizes(dev):
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    v = cfg["targets"][0]
    ref = subgraph.extract(cfg["indptr"], cfg["indices"], v, 2)
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    buf = torch.zeros(16, dtype=torch.int64, device=dev)
    sg = L.gnnshap_subgraph(num_hops=2, cap_nodes=1, cap_edges=1, node_gid=buf.data_ptr(), dst_ptr=buf.data_ptr(),
                            edge_src=buf.data_ptr(), edge_dst=buf.data_ptr(), edge_gid=buf.data_ptr())
    st = L.gnnshap_extract_subgraph(ex.graph, v, sg, _vp(ex.extract_ws), ex.extract_ws.numel(),
                                    torch.cuda.current_stream().cuda_stream)
    assert st == L.ECAPACITY
    assert sg.num_nodes == ref["num_nodes"] and sg.num_edges == ref["num_edges"]
    assert int(buf.count_nonzero()) == 0                      # nothing written
    assert int(ex.extract_ws.count_nonzero()) == 0
    _check_subgraph(ex.extract(v), ref)                       # and the next call still works


# -- 2. sampler ------------------------------------------------------------------------

SAMPLER_CASES = [(2, 2), (3, 4), (5, 30), (8, 254), (12, 4094), (13, 1000), (20, 10000), (57, 2000),
                 (60, 2000), (64, 3000), (65, 1554), (128, 5000), (400, 10000), (1000, 6668),
                 (4000, 25000), (20000, 50000), (30000, 100000)]


@pytest.mark.parametrize("M,p", SAMPLER_CASES)
def test_sampler_bit_exact(dev, M, p):
    seed, stream = 0x5EED0002 + M, 1000 + p
    _say("sample", M, p)
    plan, classes, masks, weights = sample_on_gpu(M, p, seed, stream)
    pl = sampler.plan(M, p)
    k = pl["k"]
    got = masks_np(masks)
    gw = weights.cpu().numpy()
    if M <= 4000:
        ref_m, ref_w = sampler.sample(pl, seed, stream)
        np.testing.assert_array_equal(got, sampler.pack(ref_m))
        np.testing.assert_array_equal(gw, ref_w.astype(np.float32))
    else:
        rng = np.random.default_rng(M)
        rows = np.unique(np.concatenate([rng.integers(0, k, 48), [0, k // 2 - 1, k // 2, k - 1]]))
        ref_m, ref_w = sampler.sample_rows(pl, rows, seed, stream)
        np.testing.assert_array_equal(got[rows], sampler.pack(ref_m))
        np.testing.assert_array_equal(gw[rows], ref_w.astype(np.float32))
        # properties of every row: complement pairing, class sizes
        half = k // 2
        pc = np.unpackbits(got.view(np.uint8), axis=1).sum(axis=1)
        assert (pc[:half] + pc[half:] == M).all()
        np.testing.assert_array_equal(got[:half] & got[half:], 0)


def test_sampler_is_deterministic_and_seeded(dev):
    _, _, m1, _ = sample_on_gpu(300, 4000, 7, 9)
    _, _, m2, _ = sample_on_gpu(300, 4000, 7, 9)
    _, _, m3, _ = sample_on_gpu(300, 4000, 8, 9)
    assert torch.equal(m1, m2)
    assert not torch.equal(m1, m3)


# -- 3. coalition values -----------------------------------------------------------------

def _oracle_game(cfg, sub_ref, cls):
    return gcn.Game(sub_ref, cfg["X"], cfg["weights"], cfg["biases"], cls=cls)


def _check_eval(cfg, v, p, seed, rows=None, target_class=-1, ex=None):
    ex = ex or explainer_for(cfg)
    res = ex.explain(v, p, seed, target_class=target_class)
    torch.cuda.synchronize()
    ref_sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
    M = ref_sub["num_edges"]
    game = _oracle_game(cfg, ref_sub, None)
    full_logits = game.logits(np.ones(M, bool))
    cls = gcn.predicted_class(full_logits) if target_class < 0 else target_class
    game.cls = cls
    f0, f1 = game(np.zeros(M, bool)), float(full_logits[cls])
    srt = np.sort(full_logits)[::-1]
    if target_class < 0 and len(srt) > 1 and srt[0] - srt[1] < 1e-5 * max(1.0, abs(srt[0])):
        pytest.skip("predicted class is a near tie")
    assert int(res.cls.item()) == cls
    fef = res.f_empty_full.cpu().numpy()
    tol0 = y_tolerance(np.array([f0, f1]), f0, f1)
    assert abs(fef[0] - f0) <= tol0[0] and abs(fef[1] - f1) <= tol0[1]
    pl = sampler.plan(M, p)
    k = pl["k"]
    if rows is None:
        rows = np.arange(k)
    ref_m, _ = sampler.sample_rows(pl, rows, seed, v) if len(rows) < k else sampler.sample(pl, seed, v)
    got_m = masks_np(res.masks)[rows]
    np.testing.assert_array_equal(got_m, sampler.pack(ref_m))
    y_ref = game.values(ref_m)
    y_gpu = res.y.cpu().numpy()[rows].astype(np.float64)
    err = np.abs(y_gpu - y_ref)
    tol = y_tolerance(y_ref, f0, f1)
    bad = np.flatnonzero(err > tol)
    assert bad.size == 0, f"target {v}: {bad.size} rows off, worst {err.max():.3e} vs tol {tol[bad[0]]:.3e}"
    # pruned rows hold exactly f(empty) as computed on the device
    deg_v = ref_sub["dst_ptr"][1]
    pruned = ~ref_m[:, :deg_v].any(axis=1)
    assert (y_gpu[pruned] == fef[0]).all()
    return res, game, (f0, f1, cls)


def test_eval_tiny_all_rows(dev):
    cfg = W.make_config("tiny")
    _say("eval tiny")
    _check_eval(cfg, cfg["targets"][0], cfg["p"], cfg["seed"])


@pytest.mark.parametrize("L_hops", [(1, 1), (1, 2), (2, 1), (2, 2), (2, 3), (3, 1), (3, 2), (3, 3)])
def test_eval_small_graphs_layers_and_hops(dev, L_hops):
    nl, hops = L_hops
    dims = [6, 16, 8, 5][:nl] + [4]
    for seed in range(2):
        cfg = _small_cfg(10 + seed, 50, 140, dims, hops)
        for v in range(0, 50, 7):
            M = subgraph.extract(cfg["indptr"], cfg["indices"], v, hops)["num_edges"]
            if M < 2:
                continue
            _say("eval small", nl, hops, seed, v, M)
            _check_eval(cfg, v, 600, 99)


def test_eval_fixed_class_and_wide_layers(dev):
    cfg = _small_cfg(31, 80, 400, [20, 130, 70, 9], 2)
    for v in (1, 5):
        _say("eval wide", v)
        _check_eval(cfg, v, 800, 3, target_class=4)


def test_eval_hub_target_unfused_path(dev):
    """A target with 300 in-neighbours: the two-layer kernel's LDS tables do not
    fit, so the layered kernels run; both must agree with the oracle."""
    n = 400
    src = list(range(1, 301)) + [int(x) for x in np.random.default_rng(3).integers(1, n, 600)]
    dst = [0] * 300 + [int(x) for x in np.random.default_rng(4).integers(1, n, 600)]
    indptr, indices = W.in_csr_from_pairs(n, np.array(src), np.array(dst))
    X = W.gaussian_features(n, 12, 5)
    Ws, bs = W.glorot_gcn([12, 16, 5], 6, bias="random")
    cfg = dict(indptr=indptr, indices=indices, X=X, weights=Ws, biases=bs, hops=2)
    rng = np.random.default_rng(9)
    M = subgraph.extract(indptr, indices, 0, 2)["num_edges"]
    k = sampler.plan(M, 3000)["k"]
    _check_eval(cfg, 0, 3000, 21, rows=np.unique(rng.integers(0, k, 64)))


def test_transform_features_and_unfused_first_layer(dev):
    """gnnshap_transform_features against fp64 numpy, and evaluation with
    X W_1 gathered vs computed from X per call."""
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    ex.prepare()
    torch.cuda.synchronize()
    ref = cfg["X"].astype(np.float64) @ cfg["weights"][0].astype(np.float64)
    got = ex.XW1.cpu().numpy()
    assert np.abs(got - ref).max() <= 1e-5 * max(1.0, np.abs(ref).max())
    v = cfg["targets"][3]
    r1 = ex.explain(v, cfg["p"], cfg["seed"])
    y1 = r1.y.clone()
    ex.model.XW1 = None
    r2 = ex.run(ex.extract(v), r1.plan, r1.classes, -1, v)
    ex.model.XW1 = ex.XW1.data_ptr()
    torch.cuda.synchronize()
    d = (r2.y - y1).abs().max().item()
    assert d <= 1e-5 * max(1.0, y1.abs().max().item())


def test_pipelined_targets_match_sequential(dev):
    """explain_many (extraction on its own stream, targets spread over compute
    streams) gives bit-identical masks, values and phi to explain()."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    targets = cfg["targets"]
    many = ex.explain_many(targets, cfg["p"], cfg["seed"], n_streams=8)
    torch.cuda.synchronize()
    for v, r in zip(targets, many):
        _say("pipelined", v)
        one = ex.explain(v, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
        assert torch.equal(one.masks, r.masks)
        assert torch.equal(one.y, r.y)
        assert torch.equal(one.phi, r.phi)
        assert int(r.info.item()) == 0


def test_eval_cora_all_targets_sampled_rows(dev):
    cfg = W.make_config("cora")
    rng = np.random.default_rng(0)
    for v in cfg["targets"]:
        _say("eval cora", v)
        k = sampler.plan(subgraph.extract(cfg["indptr"], cfg["indices"], v, 2)["num_edges"], cfg["p"])["k"]
        rows = np.unique(np.concatenate([rng.integers(0, k, 40), [0, k - 1]]))
        _check_eval(cfg, v, cfg["p"], cfg["seed"], rows=rows)


def test_eval_pubmed_sampled_rows(dev):
    cfg = W.make_config("pubmed")
    rng = np.random.default_rng(1)
    for v in cfg["targets"][:6]:
        _say("eval pubmed", v)
        k = sampler.plan(subgraph.extract(cfg["indptr"], cfg["indices"], v, 3)["num_edges"], cfg["p"])["k"]
        rows = np.unique(np.concatenate([rng.integers(0, k, 16), [0, k - 1]]))
        _check_eval(cfg, v, cfg["p"], cfg["seed"], rows=rows)


# -- 4. least squares ---------------------------------------------------------------------

def _phi_close(phi_gpu, phi_ref, rel=1e-3):
    scale = np.abs(phi_ref).max()
    err = np.abs(phi_gpu - phi_ref).max()
    assert err <= rel * scale, f"max |phi err| {err:.3e} > {rel:.0e} * {scale:.3e}"


def test_solve_end_to_end_tiny_and_cora(dev):
    for name, targets in (("tiny", None), ("cora", 6)):
        cfg = W.make_config(name)
        for v in (cfg["targets"] if targets is None else cfg["targets"][:targets]):
            _say("solve", name, v)
            res, game, (f0, f1, cls) = _check_eval(cfg, v, cfg["p"], cfg["seed"])
            assert int(res.info.item()) == 0
            pl = sampler.plan(res.plan.num_players, cfg["p"])
            m, w = sampler.sample(pl, cfg["seed"], v)
            phi_ref = wls.kernel_shap(m, w, game.values(m), f0, f1)
            phi = res.phi.cpu().numpy().astype(np.float64)
            _phi_close(phi, phi_ref)
            assert abs(phi.sum() - float(res.f_empty_full[1] - res.f_empty_full[0])) < 1e-4 * max(1.0, abs(f1 - f0))


@pytest.mark.parametrize("M", [2, 3, 5, 8, 10])
def test_solve_exhaustive_equals_exact_shapley(dev, M):
    """Every coalition enumerated: Kernel SHAP = eq. 1 (checked on a synthetic game)."""
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    rng = np.random.default_rng(M)
    table = rng.normal(size=1 << M)
    vals = table.copy()
    exact = shapley.exact_shapley(vals, M)
    p = 2 ** M - 2
    plan, classes, masks, _ = sample_on_gpu(M, p, 1, 2)
    mb, _ = sampler.sample(sampler.plan(M, p), 1, 2)
    np.testing.assert_array_equal(masks_np(masks), sampler.pack(mb))
    codes = (mb * (1 << np.arange(M))).sum(axis=1)
    y = torch.tensor(vals[codes], dtype=torch.float32, device=dev)
    fef = torch.tensor([vals[0], vals[-1]], dtype=torch.float32, device=dev)
    phi = torch.empty(M, dtype=torch.float32, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_solve_workspace(plan), dtype=torch.uint8, device=dev)
    L.gnnshap_solve_wls(plan, classes, _vp(masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(ws), ws.numel(),
                        torch.cuda.current_stream().cuda_stream)
    assert int(info.item()) == 0
    _phi_close(phi.cpu().numpy().astype(np.float64), exact, rel=1e-4)


@pytest.mark.parametrize("M,p", [(20, 10000), (60, 2000), (262, 4000), (263, 4000), (400, 10000), (448, 6000),
                                 (449, 6000), (1000, 6668), (4000, 25000)])
def test_solve_recovers_additive_game(dev, M, p):
    """y = f0 + m.a has phi = a exactly for any determined sample set (sizes on
    both sides of the LDS one-workgroup, global one-workgroup and multi-block
    limits)."""
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    _say("additive", M, p)
    plan, classes, masks, _ = sample_on_gpu(M, p, 5, 6)
    rng = np.random.default_rng(M)
    a = rng.normal(size=M)
    f0 = 0.25
    mo, _ = sampler.sample(sampler.plan(M, p), 5, 6)
    np.testing.assert_array_equal(masks_np(masks), sampler.pack(mo))
    mb = torch.tensor(mo, dtype=torch.float64, device=dev)
    y = (f0 + mb @ torch.tensor(a, device=dev)).float()
    fef = torch.tensor([f0, f0 + a.sum()], dtype=torch.float32, device=dev)
    phi = torch.empty(M, dtype=torch.float32, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_solve_workspace(plan), dtype=torch.uint8, device=dev)
    L.gnnshap_solve_wls(plan, classes, _vp(masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(ws), ws.numel(),
                        torch.cuda.current_stream().cuda_stream)
    assert int(info.item()) == 0
    _phi_close(phi.cpu().numpy().astype(np.float64), a)


# -- 5. full-size workloads ---------------------------------------------------------------

def _unpack_rows(masks, M, r0, r1):
    """Rows [r0, r1) of packed masks as fp64 0/1 on the device (test-side arithmetic)."""
    sh = torch.arange(64, device=masks.device, dtype=torch.int64)
    bits = (masks[r0:r1].unsqueeze(-1) >> sh) & 1
    return bits.reshape(r1 - r0, -1)[:, :M].to(torch.float64)


def _solve_phi(res, y, f0, f1):
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    dev = res.masks.device
    M = res.plan.num_players
    fef = torch.tensor([f0, f1], dtype=torch.float32, device=dev)
    phi = torch.empty(M, dtype=torch.float32, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_solve_workspace(res.plan), dtype=torch.uint8, device=dev)
    L.gnnshap_solve_wls(res.plan, res.classes, _vp(res.masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(ws),
                        ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    return phi.cpu().numpy().astype(np.float64)


def _normal_equation_residual(res, phi, f0, chunk=1024):
    """r = X^T W (y - f0 - X phi) and b = X^T W (y - f0) for the sampled rows
    X and their kernel weights W, in fp64 on the device (test-side
    arithmetic).  The efficiency-constrained least squares optimum has
    r = lambda * 1."""
    M, k = res.plan.num_players, res.plan.num_rows
    dev = res.masks.device
    ph = torch.tensor(phi, dtype=torch.float64, device=dev)
    r = torch.zeros(M, dtype=torch.float64, device=dev)
    b = torch.zeros(M, dtype=torch.float64, device=dev)
    for r0 in range(0, k, chunk):
        r1 = min(k, r0 + chunk)
        X = _unpack_rows(res.masks, M, r0, r1)
        w = res.weights[r0:r1].double()
        yc = res.y[r0:r1].double() - f0
        r += X.T @ (w * (yc - X @ ph))
        b += X.T @ (w * yc)
    return r.cpu().numpy(), b.cpu().numpy()


def _full_size_targets(cfg, picks):
    ms = sorted((W.player_count(cfg["indptr"], cfg["indices"], v, cfg["hops"]), v) for v in cfg["targets"])
    idx = sorted({int(round(x)) for x in np.linspace(0, len(ms) - 1, picks)})
    return [ms[i][1] for i in idx]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,picks", [("arxiv", 3), ("reddit", 2)])
def test_full_size_workload(dev, name, picks):
    """At the full sizes of the two large workloads (2-hop graphs of 5k..30k
    players, 50,000 / 100,000 coalitions): extraction bit-exact, sampled
    masks bit-exact, sampled coalition values within the y bar, and phi
    checked by properties that hold at any size: efficiency, the solved
    normal equations, and exact recovery of an additive game on the same
    coalitions.  These properties do not by themselves bound the phi error
    by the phi bar (that needs the smallest eigenvalue of the system);
    tests/test_gpu_full_phi.py compares phi element-wise with the oracle's
    least squares at the smallest target of each large workload."""
    _say("full size", name, "building the workload")
    cfg = W.make_config(name)
    ex = explainer_for(cfg)
    rng = np.random.default_rng(5)
    for v in _full_size_targets(cfg, picks):
        ref_sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
        M = ref_sub["num_edges"]
        pl = sampler.plan(M, cfg["p"])
        k = pl["k"]
        rows = np.unique(np.concatenate([rng.integers(0, k, 12), [0, 1, k // 2 - 1, k // 2, k - 1]]))
        _say("full size", name, "target", v, "M", M, "k", k)
        res, game, (f0, f1, cls) = _check_eval(cfg, v, cfg["p"], cfg["seed"], rows=rows, ex=ex)
        _check_subgraph(ex.extract(v), ref_sub)
        assert int(res.info.item()) == 0
        phi = res.phi.cpu().numpy().astype(np.float64)
        fef = res.f_empty_full.cpu().numpy().astype(np.float64)
        delta = fef[1] - fef[0]
        assert abs(phi.sum() - delta) <= 1e-4 * max(1.0, abs(delta)) + 1e-3 * np.abs(phi).max()
        # the constrained optimum has X^T W (y - f0 - X phi) = lambda 1: the
        # centred residual of the normal equations must be small against the
        # centred right-hand side (a solved system, not the phi bar itself)
        r, b = _normal_equation_residual(res, phi, fef[0])
        rc, bc = r - r.mean(), b - b.mean()
        assert np.linalg.norm(rc) <= 1e-3 * np.linalg.norm(bc), (np.linalg.norm(rc), np.linalg.norm(bc))
        # an additive game on the same coalitions has phi = a
        a = np.random.default_rng(M).normal(size=M)
        at = torch.tensor(a, dtype=torch.float64, device=res.masks.device)
        y_add = torch.cat([(0.25 + _unpack_rows(res.masks, M, r0, min(k, r0 + 1024)) @ at)
                           for r0 in range(0, k, 1024)]).float()
        _phi_close(_solve_phi(res, y_add, 0.25, 0.25 + a.sum()), a)
        del res, y_add
        torch.cuda.empty_cache()


# -- 6. many targets per launch sequence ----------------------------------------------------

def _same_sub(a, b):
    assert a.sg.num_nodes == b.sg.num_nodes and a.sg.num_edges == b.sg.num_edges and a.sg.num_dst == b.sg.num_dst
    assert a.hop_ptr == b.hop_ptr
    for name in ("node_gid", "dst_ptr", "edge_src", "edge_dst", "edge_gid"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


def test_extract_batch_matches_single(dev):
    """gnnshap_extract_batch gives the single-target arrays, grows on
    ECAPACITY, and leaves the per-target slices of its workspace (its front)
    zero-filled for any batch size."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    ex._cap = [8, 16]                                  # force the capacity retry
    targets = cfg["targets"]
    subs, _ = ex.extract_batch(targets)
    torch.cuda.synchronize()
    for v, sb in zip(targets, subs):
        _say("extract batch", v)
        _check_subgraph(sb, subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"]))
    from paper_2401_04829_amd import _lib as L
    slices = ex._bx[0] * L.gnnshap_extract_workspace(cfg["indptr"].size - 1)
    assert int(ex._bx[1][:slices].count_nonzero()) == 0
    subs2, _ = ex.extract_batch(targets[:7])           # smaller batch on the same workspace
    torch.cuda.synchronize()
    for v, sb in zip(targets[:7], subs2):
        _same_sub(sb, ex.extract(v))
    assert int(ex._bx[1][:slices].count_nonzero()) == 0


@pytest.mark.parametrize("name,count", [("tiny", None), ("cora", None), ("pubmed", 6)])
def test_explain_batch_matches_single(dev, name, count):
    """gnnshap_explain_batch equals the single-target calls bit for bit: masks,
    weights, values, f(empty)/f(E_c), class, phi and info (Cora-shaped targets
    above the one-workgroup solve size and the three-layer PubMed-shaped model
    take the single-target kernels inside the batch)."""
    cfg = W.make_config(name)
    ex = explainer_for(cfg)
    targets = cfg["targets"] if count is None else cfg["targets"][:count]
    many = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    for v, r in zip(targets, many):
        _say("explain batch", name, v, r.plan.num_players)
        one = ex.explain(v, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
        _same_sub(r.sub, one.sub)
        for field in ("masks", "weights", "y", "f_empty_full", "cls", "phi", "info"):
            assert torch.equal(getattr(r, field), getattr(one, field)), field
        assert int(r.info.item()) == 0


def test_explain_batch_against_oracle(dev):
    """Batched results against the oracle on the Cora-shaped workload: sampled
    rows' masks bit-exact, values within the y bar, phi within the phi bar."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    targets = cfg["targets"][:12]
    many = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    for v, r in zip(targets, many):
        _say("batch oracle", v)
        ref_sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
        M = ref_sub["num_edges"]
        game = _oracle_game(cfg, ref_sub, None)
        full_logits = game.logits(np.ones(M, bool))
        cls = gcn.predicted_class(full_logits)
        game.cls = cls
        f0, f1 = game(np.zeros(M, bool)), float(full_logits[cls])
        assert int(r.cls.item()) == cls
        pl = sampler.plan(M, cfg["p"])
        m, w = sampler.sample(pl, cfg["seed"], v)
        np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(m))
        rows = np.unique(rng.integers(0, pl["k"], 32))
        y_ref = game.values(m[rows])
        err = np.abs(r.y.cpu().numpy()[rows].astype(np.float64) - y_ref)
        assert (err <= y_tolerance(y_ref, f0, f1)).all()
        phi_ref = wls.kernel_shap(m, w, game.values(m), f0, f1)
        _phi_close(r.phi.cpu().numpy().astype(np.float64), phi_ref)


def test_explain_batch_stays_inside_its_workspace(dev):
    """Panel-path systems (193-448 players) of different sizes in one batch:
    the batched factorisation launches cover the largest system, and a
    smaller one must ignore the panels past its own.  Targets from the
    largest to the smallest, so that the smallest system's workspace slice
    is the last one: every byte past the size the call asks for stays as it
    was, and the results equal a call in a workspace of exactly that size.
    (A trailing-update workgroup past a system's last panel once wrote a
    64 x 64 block past that system's slice.)"""
    cfg = W.make_config("cora")
    sizes = []
    for v in cfg["targets"]:
        M = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])["num_edges"]
        if 192 < M <= 448:
            sizes.append((M, int(v)))
    sizes.sort(reverse=True)
    assert (sizes[0][0] + 63) // 64 - (sizes[-1][0] + 63) // 64 >= 2   # two panels more in the largest
    targets = [v for _, v in sizes]
    ex = explainer_for(cfg)
    ref = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    ref_phi = [ref[t].phi.clone() for t in range(len(targets))]
    tail = 1 << 20
    seen = {}
    orig = type(ex)._batch_call

    def call(self, sgs, plans, cl, target_class, ptrs, ws):
        need = self._batch_workspace(sgs, plans)
        big = torch.full((need + tail,), 0xA5, dtype=torch.uint8, device=dev)
        st = orig(self, sgs, plans, cl, target_class, ptrs, big)
        torch.cuda.synchronize()
        seen["untouched"] = bool((big[need:] == 0xA5).all().item())
        return st

    type(ex)._batch_call = call
    try:
        res = ex.explain_batch(targets, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
    finally:
        type(ex)._batch_call = orig
    assert seen["untouched"], "the batched call wrote past its workspace"
    for t in range(len(targets)):
        assert int(res[t].info.item()) == 0
        assert torch.equal(res[t].phi, ref_phi[t]), t


def _guard_workspaces(ex, attrs=("ws_sample", "ws_eval", "ws_solve", "ws_batch", "ws_fid"), tail=1 << 20):
    """Replace the explainer's workspace buffers by ones whose every request
    gets a fresh buffer: the bytes asked for filled with 0xFF (NaN in every
    float, -1 in every integer), then `tail` bytes of 0xA5.  Returns a
    function that synchronises and tells whether every tail is untouched
    (and forgets the buffers handed out so far)."""
    from paper_2401_04829_amd import explainer as E
    given = []

    class Guarded(E._Buffer):
        def get(self, nbytes):
            nbytes = max(int(nbytes), 256)
            t = torch.empty(nbytes + tail, dtype=torch.uint8, device=self.device)
            t[:nbytes].fill_(0xFF)
            t[nbytes:].fill_(0xA5)
            given.append((t, nbytes))
            self.t = t
            return t

    for attr in attrs:
        setattr(ex, attr, Guarded(ex.device))

    def tails_untouched():
        torch.cuda.synchronize()
        ok = all(bool((t[k:] == 0xA5).all().item()) for t, k in given)
        given.clear()
        return ok
    return tails_untouched


_FIELDS = ("masks", "weights", "y", "f_empty_full", "cls", "phi", "info")


@pytest.mark.parametrize("name,n", [("tiny", None), ("cora", 40), ("pubmed", 12)])
def test_workspaces_need_no_initialisation(dev, name, n):
    """Every workspace the explainer hands the library (sampling, evaluation,
    least squares, batch) is filled with 0xFF bytes and followed by a 1 MiB
    tail of 0xA5: the batched and the single-target calls give the same bits
    as with ordinary workspaces, so nothing is read before it is written,
    and no tail byte changes."""
    cfg = W.make_config(name)
    targets = list(cfg["targets"])[:n] if n else list(cfg["targets"])
    ex = explainer_for(cfg)
    ref = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    ref1 = [ex.explain(v, cfg["p"], cfg["seed"]) for v in targets[:2]]
    torch.cuda.synchronize()
    exg = explainer_for(cfg)
    tails_untouched = _guard_workspaces(exg)
    _say("guarded workspaces", name, len(targets))
    res = exg.explain_batch(targets, cfg["p"], cfg["seed"])
    assert tails_untouched()
    for t in range(len(targets)):
        for f in _FIELDS:
            assert torch.equal(getattr(res[t], f), getattr(ref[t], f)), (t, f)
    for v, r1 in zip(targets[:2], ref1):
        r = exg.explain(v, cfg["p"], cfg["seed"])
        assert tails_untouched()
        for f in _FIELDS:
            assert torch.equal(getattr(r, f), getattr(r1, f)), (v, f)


def test_gat_and_fidelity_workspaces_need_no_initialisation(dev):
    """As above for the GAT explainer (batched and single-target calls, 12
    Cora-shaped targets) and for the fidelity terms of 8 GCN explanations."""
    from paper_2401_04829_amd.explainer import GatExplainer
    cfg = W.make_config("cora")
    P = W.glorot_gat(cfg["X"].shape[1], 8, 16, 7, 41, bias="random")
    targets = [int(v) for v in cfg["targets"][:12]]
    ex = GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)
    ref = ex.explain_batch(targets, 2000, 7)
    ref1 = ex.explain(targets[0], 2000, 7)
    torch.cuda.synchronize()
    exg = GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)
    tails_untouched = _guard_workspaces(exg)
    _say("guarded workspaces, gat", len(targets))
    res = exg.explain_batch(targets, 2000, 7)
    assert tails_untouched()
    for t in range(len(targets)):
        for f in _FIELDS:
            assert torch.equal(getattr(res[t], f), getattr(ref[t], f)), (t, f)
    r = exg.explain(targets[0], 2000, 7)
    assert tails_untouched()
    for f in _FIELDS:
        assert torch.equal(getattr(r, f), getattr(ref1, f)), f
    # fidelity (eq. 7-8) of GCN explanations, ordinary and guarded workspace
    exf = explainer_for(cfg)
    exps = list(exf.explain_batch(cfg["targets"][:8], cfg["p"], cfg["seed"]))
    terms, avg = exf.fidelity(exps, 0.3, 10)
    torch.cuda.synchronize()
    terms, avg = terms.clone(), avg.clone()
    tails_untouched = _guard_workspaces(exf, attrs=("ws_fid",))
    terms_g, avg_g = exf.fidelity(exps, 0.3, 10)
    assert tails_untouched()
    assert torch.equal(terms_g, terms) and torch.equal(avg_g, avg)


def test_explain_batch_repeated_calls_agree(dev):
    """Repeated batched calls on the same targets give the first call's
    outputs bit for bit, with other device work between them, and equal the
    single-target calls."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    targets = cfg["targets"][:40]
    fields = ("masks", "weights", "y", "f_empty_full", "cls", "phi", "info")
    first = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    ref = [{f: getattr(r, f).clone() for f in fields} for r in first]
    for rep in range(3):
        _say("batch replay", rep)
        noise = torch.randn(1 << 20, device=dev).sum()           # unrelated work in between
        one = ex.explain(targets[rep], cfg["p"], cfg["seed"])
        again = ex.explain_batch(targets, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
        assert torch.isfinite(noise)
        for t, r in enumerate(again):
            for f in fields:
                assert torch.equal(getattr(r, f), ref[t][f]), (rep, t, f)
        for f in fields:
            assert torch.equal(getattr(one, f), ref[rep][f]), (rep, f)


@pytest.mark.gpu
def test_explain_batches_pipelined_equal_batch_calls(dev):
    """The pipelined sequence (each batch's extraction queued before the
    previous batch's explanation) gives every batch exactly what a separate
    explain_batch call gives; batches of different sizes, one repeated, and a
    generator stopped early leaves no extraction pending."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    tg = cfg["targets"]
    batches = [tg[:30], tg[30:45], tg[:30], tg[45:100]]
    fields = ("masks", "weights", "y", "f_empty_full", "cls", "phi", "info")
    refs = []
    for b in batches:
        r = ex.explain_batch(b, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
        refs.append([{f: getattr(e, f).clone() for f in fields} for e in r])
    outs = list(ex.explain_batches(batches, cfg["p"], cfg["seed"], prepare_each=True))
    torch.cuda.synchronize()
    assert len(outs) == len(batches)
    for i, (out, ref) in enumerate(zip(outs, refs)):
        _say("pipelined batch", i, len(batches[i]))
        assert len(out) == len(batches[i])
        for t, e in enumerate(out):
            assert e.target == batches[i][t]
            for f in fields:
                assert torch.equal(getattr(e, f), ref[t][f]), (i, t, f)
    gen = ex.explain_batches(batches, cfg["p"], cfg["seed"])
    next(gen)
    gen.close()                          # the second batch's extraction was queued
    again = ex.explain_batch(batches[1], cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    for t, e in enumerate(again):
        for f in fields:
            assert torch.equal(getattr(e, f), refs[1][t][f]), (t, f)
