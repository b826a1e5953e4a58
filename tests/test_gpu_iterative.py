"""GPU parity of the iterative least-squares solver (Sec. 3.5: large systems
are fitted iteratively) against the fp64 oracle.

The solver switches on above the plan's player threshold (default 5000);
these tests lower it so that systems the oracle solves in seconds take the
iterative path, with and without enumerated classes, with no random rows at
all, and through the batched entry point.  Bar: phi within 1e-3 of max|phi|;
repeated solves and batched calls equal single calls bit for bit.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gcn, sampler, shapley, subgraph, wls
from paper_2401_04829_amd import _lib as L
from paper_2401_04829_amd.explainer import _vp
from tests.gpu_util import explainer_for, masks_np, require_gpu, sample_on_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()




def _say(*a):
    print(*a, flush=True)


def _phi_close(phi_gpu, phi_ref, rel=1e-3):
    scale = np.abs(phi_ref).max()
    err = np.abs(phi_gpu - phi_ref).max()
    assert err <= rel * scale, f"max |phi err| {err:.3e} > {rel:.0e} * {scale:.3e}"


def _solve(dev, plan, classes, masks, y, fef):
    M = plan.num_players
    phi = torch.empty(M, dtype=torch.float32, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(L.gnnshap_solve_workspace(plan), dtype=torch.uint8, device=dev)
    L.gnnshap_solve_wls(plan, classes, _vp(masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(ws), ws.numel(),
                        torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return phi.cpu().numpy().astype(np.float64), int(info.item())


def _oracle_rows(plan, masks_gpu, seed, stream):
    """The oracle's masks and weights for the same plan, seed and stream;
    the GPU's masks must equal them bit for bit."""
    pl = sampler.plan(plan.num_players, plan.num_samples)
    mb, w = sampler.sample(pl, seed, stream)
    np.testing.assert_array_equal(masks_np(masks_gpu), sampler.pack(mb))
    return mb, w


def _game(M, mb, seed):
    """A game with pairwise interactions (not additive, so the fit has a
    residual): v(S) = f0 + sum_i a_i s_i + sum_(i,j) in E b_ij s_i s_j."""
    rng = np.random.default_rng(seed)
    a = rng.normal(size=M)
    pairs = rng.integers(0, M, size=(2 * M, 2))
    b = rng.normal(size=2 * M) * 0.5
    f0 = 0.3

    def v(m):
        m = np.asarray(m, dtype=np.float64)
        return f0 + m @ a + (m[:, pairs[:, 0]] * m[:, pairs[:, 1]]) @ b

    return v, f0, float(v(np.ones((1, M)))[0])


@pytest.mark.parametrize("M,p", [(10, 1022), (20, 10000), (64, 3000), (300, 4000), (701, 6000), (1500, 8000)])
def test_iterative_solve_against_oracle(dev, M, p):
    """Conjugate gradients against the oracle's least squares: every class
    enumerated (no random rows), enumerated and random classes together, and
    random rows only, across one and several mask words and row chunks."""
    _say("iterative", M, p)
    plan, classes, masks, weights = sample_on_gpu(M, p, 11, 12)
    plan.iterative_threshold = 1
    assert L.gnnshap_solve_info(plan) == 3
    mb, w = _oracle_rows(plan, masks, 11, 12)
    v, f0, f1 = _game(M, mb, M)
    yv = v(mb).astype(np.float32).astype(np.float64)   # the values the device gets, in fp32
    y = torch.tensor(yv, dtype=torch.float32, device=dev)
    fef = torch.tensor([f0, f1], dtype=torch.float32, device=dev)
    phi, info = _solve(dev, plan, classes, masks, y, fef)
    assert info == 0
    phi_ref = wls.kernel_shap(mb, w, yv, f0, f1)
    _phi_close(phi, phi_ref)
    delta = float(fef[1] - fef[0])
    assert abs(phi.sum() - delta) <= 1e-5 * max(1.0, abs(delta)) + 1e-6 * np.abs(phi).sum()
    again, _ = _solve(dev, plan, classes, masks, y, fef)
    assert np.array_equal(again, phi), "repeated iterative solves differ"


@pytest.mark.parametrize("M,p", [(449, 6000), (1000, 6668), (2500, 15000), (4000, 25000)])
def test_factored_solve_with_residual_against_oracle(dev, M, p):
    """The multi-block Cholesky path (449 to 5,000 players) on a game with
    pairwise interactions, so that the fit keeps a residual and the weights
    and the right-hand side's centring matter (an additive game hides both):
    phi within the bar of the oracle's least squares on the oracle's masks."""
    _say("factored with residual", M, p)
    plan, classes, masks, _ = sample_on_gpu(M, p, 41, 42)
    assert L.gnnshap_solve_info(plan) == 0
    mb, w = _oracle_rows(plan, masks, 41, 42)
    v, f0, f1 = _game(M, mb, 7 * M)
    yv = v(mb).astype(np.float32).astype(np.float64)
    y = torch.tensor(yv, dtype=torch.float32, device=dev)
    fef = torch.tensor([f0, f1], dtype=torch.float32, device=dev)
    phi, info = _solve(dev, plan, classes, masks, y, fef)
    assert info == 0
    phi_ref = (wls.kernel_shap if M <= 1000 else wls.kernel_shap_normal)(mb, w, yv, float(fef[0]), float(fef[1]))
    _phi_close(phi, phi_ref)


def test_iterative_exhaustive_equals_exact_shapley(dev):
    """All coalitions enumerated: the iterative solve gives the exact Shapley
    values of eq. 1 (brute force over 2^M coalitions)."""
    M = 9
    rng = np.random.default_rng(3)
    vals = rng.normal(size=1 << M)
    exact = shapley.exact_shapley(vals, M)
    plan, classes, masks, _ = sample_on_gpu(M, 2 ** M - 2, 1, 2)
    plan.iterative_threshold = 1
    assert L.gnnshap_solve_info(plan) == 3
    mb, _ = _oracle_rows(plan, masks, 1, 2)
    codes = (mb * (1 << np.arange(M))).sum(axis=1)
    y = torch.tensor(vals[codes], dtype=torch.float32, device=dev)
    fef = torch.tensor([vals[0], vals[-1]], dtype=torch.float32, device=dev)
    phi, info = _solve(dev, plan, classes, masks, y, fef)
    assert info == 0
    _phi_close(phi, exact, rel=1e-4)


@pytest.mark.parametrize("M,p", [(600, 4000), (2500, 12000)])
def test_iterative_matches_factorisation(dev, M, p):
    """The same system through the iterative path and through the Cholesky
    paths agree within the phi bar, and an additive game is recovered."""
    _say("iterative vs direct", M, p)
    plan, classes, masks, _ = sample_on_gpu(M, p, 21, 22)
    mb = torch.tensor(_oracle_rows(plan, masks, 21, 22)[0], dtype=torch.float64, device=dev)
    a = np.random.default_rng(M).normal(size=M)
    y = (0.25 + mb @ torch.tensor(a, device=dev)).float()
    fef = torch.tensor([0.25, 0.25 + a.sum()], dtype=torch.float32, device=dev)
    plan.iterative_threshold = M + 1
    assert L.gnnshap_solve_info(plan) != 3
    direct, info_d = _solve(dev, plan, classes, masks, y, fef)
    plan.iterative_threshold = M - 1
    assert L.gnnshap_solve_info(plan) == 3
    it, info_i = _solve(dev, plan, classes, masks, y, fef)
    assert info_d == 0 and info_i == 0
    _phi_close(it, a)
    _phi_close(it, direct)


def test_iterative_through_explain_batch(dev):
    """Cora-shaped targets with the threshold lowered: the batched call sends
    them to the iterative solver and equals the single-target calls bit for
    bit; phi matches the oracle's least squares on the oracle's own masks and
    coalition values."""
    cfg = W.make_config("cora")
    ex = explainer_for(cfg)
    targets = cfg["targets"][:10]
    ex.iterative_threshold = 40
    many = ex.explain_batch(targets, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    saw_iterative = False
    for v, r in zip(targets, many):
        _say("batch iterative", v, r.plan.num_players)
        saw_iterative |= L.gnnshap_solve_info(r.plan) == 3
        one = ex.explain(v, cfg["p"], cfg["seed"])
        torch.cuda.synchronize()
        for field in ("masks", "y", "f_empty_full", "phi", "info"):
            assert torch.equal(getattr(r, field), getattr(one, field)), field
        assert int(r.info.item()) == 0
        M = r.plan.num_players
        sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
        game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"])
        game.cls = gcn.predicted_class(game.logits(np.ones(M, bool)))
        assert int(r.cls.item()) == game.cls
        pl = sampler.plan(M, cfg["p"])
        mb, w = sampler.sample(pl, cfg["seed"], v)
        np.testing.assert_array_equal(masks_np(r.masks), sampler.pack(mb))
        phi_ref = wls.kernel_shap(mb, w, gcn.values_many(game, mb), game(np.zeros(M, bool)), game(np.ones(M, bool)))
        _phi_close(r.phi.cpu().numpy().astype(np.float64), phi_ref)
    assert saw_iterative


def test_iterative_reports_undetermined_plan(dev):
    """Fewer random rows than M - 1 and no enumerated class: the rows cannot
    determine phi; the iterative path reports info = M + 1, as the
    factorisation reports a failed pivot."""
    M, p = 300, 200
    plan, classes, masks, _ = sample_on_gpu(M, p, 31, 32)
    kr = plan.num_rows // 2 - plan.random_begin
    assert plan.random_begin == 0 and kr < M - 1
    y = torch.randn(plan.num_rows, device=dev)
    fef = torch.tensor([0.0, 1.0], dtype=torch.float32, device=dev)
    plan.iterative_threshold = M - 1
    _, info_it = _solve(dev, plan, classes, masks, y, fef)
    assert info_it == M + 1
    plan.iterative_threshold = M + 1
    _, info_direct = _solve(dev, plan, classes, masks, y, fef)
    assert info_direct > 0
