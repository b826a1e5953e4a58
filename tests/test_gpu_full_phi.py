"""GPU parity of the Shapley values of full-size targets against the oracle's
least squares (eq. 2-3, Sec. 3.5) on the oracle's own coalition values.

The expected values come from tests/golden/make_full_size_phi.py, which runs
only the oracle (pruning, sampler, fp64 GCN game over every coalition, least
squares) on the PubMed-shaped workload's smallest (508 players) and largest
(3,994 players; multi-block Cholesky) targets, the arxiv-shaped workload's
smallest target (7,862 players, 50,000 coalitions, iterative solver) and the
Reddit-shaped workload's smallest target (10,793 players, 100,000
coalitions, iterative solver).  Each case checks: the masks equal the
oracle's bit for bit (SHA-256 of the packed rows), the explained class,
f(empty) and f(E_c) and 64 sampled coalition values within the y bar, and
max |phi_gpu - phi_ref| <= 1e-3 max |phi_ref|, through the single-target
call and through the batched call.
"""
import glob
import hashlib
import os

import numpy as np
import pytest
import torch

import workloads as W
from tests.gpu_util import explainer_for, masks_np, require_gpu, y_tolerance

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CASES = sorted(glob.glob(os.path.join(GOLDEN, "full_size_phi_*.npz")))


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _say(*a):
    print(*a, flush=True)


def _load(path):
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def _check(res, g, name):
    M, k = int(g["M"]), int(g["k"])
    assert res.plan.num_players == M and res.plan.num_rows == k
    assert int(res.info.item()) == 0
    got = np.ascontiguousarray(masks_np(res.masks))
    assert hashlib.sha256(got.tobytes()).hexdigest() == str(g["masks_sha256"]), f"{name}: masks differ"
    f0, f1 = float(g["f_empty"]), float(g["f_full"])
    assert int(res.cls.item()) == int(g["cls"])
    fef = res.f_empty_full.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(fef - [f0, f1]) <= y_tolerance(np.array([f0, f1]), f0, f1))
    y = res.y.cpu().numpy().astype(np.float64)[g["rows"]]
    err = np.abs(y - g["y_rows"])
    assert np.all(err <= y_tolerance(g["y_rows"], f0, f1)), f"{name}: y off by {err.max():.3e}"
    phi = res.phi.cpu().numpy().astype(np.float64)
    ref = g["phi"]
    dphi = np.abs(phi - ref).max()
    scale = np.abs(ref).max()
    _say(name, "M", M, "max|dphi|/max|phi|", dphi / scale)
    assert dphi <= 1e-3 * scale, f"{name}: max|dphi| {dphi:.3e} > 1e-3 * {scale:.3e}"


@pytest.mark.timeout(600)
@pytest.mark.parametrize("path", CASES, ids=[os.path.basename(c)[14:-4] for c in CASES])
def test_full_size_phi_against_oracle(dev, path):
    g = _load(path)
    name, v = str(g["workload"]), int(g["target"])
    _say("full-size phi", name, str(g["label"]), v, "building the workload")
    cfg = W.make_config(name)
    assert v in cfg["targets"]
    assert float(g["top2_gap"]) > 1e-5 * max(1.0, abs(float(g["f_full"])))
    ex = explainer_for(cfg)
    res = ex.explain(v, cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    _check(res, g, f"{name} {v} single")
    phi_single = res.phi.clone()
    del res
    batch = ex.explain_batch([v], cfg["p"], cfg["seed"])
    torch.cuda.synchronize()
    _check(batch[0], g, f"{name} {v} batch")
    assert torch.equal(batch[0].phi, phi_single)

