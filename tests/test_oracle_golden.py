"""The stored full-size expected values (tests/golden/full_size_phi_*.npz,
written by tests/golden/make_full_size_phi.py from the oracle alone): the
four cases are present, each keeps efficiency (sum phi = f(E_c) - f(empty),
eq. 2-3), and the smallest PubMed-shaped case is recomputed here by the
oracle and must match what is stored."""
import glob
import hashlib
import os

import numpy as np

import workloads as W
from oracle import gcn, sampler, subgraph, wls

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(path):
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def test_full_size_cases_present_and_efficient():
    cases = [_load(c) for c in sorted(glob.glob(os.path.join(GOLDEN, "full_size_phi_*.npz")))]
    names = {(str(g["workload"]), str(g["label"])) for g in cases}
    assert names == {("pubmed", "smallest"), ("pubmed", "largest"), ("arxiv", "smallest"), ("reddit", "smallest")}
    for g in cases:
        phi = g["phi"]
        assert phi.shape == (int(g["M"]),)
        delta = float(g["f_full"]) - float(g["f_empty"])
        assert abs(phi.sum() - delta) <= 1e-9 * max(1.0, np.abs(phi).sum())


def test_smallest_pubmed_case_is_the_oracle_output():
    path = glob.glob(os.path.join(GOLDEN, "full_size_phi_pubmed_*.npz"))
    g = [x for x in (_load(p) for p in path) if str(x["label"]) == "smallest"][0]
    cfg = W.make_config("pubmed")
    v = int(g["target"])
    sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
    M = sub["num_edges"]
    assert M == int(g["M"])
    game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"], cls=int(g["cls"]))
    pl = sampler.plan(M, cfg["p"])
    masks, w = sampler.sample(pl, cfg["seed"], v)
    assert hashlib.sha256(np.ascontiguousarray(sampler.pack(masks)).tobytes()).hexdigest() == str(g["masks_sha256"])
    y = gcn.values_many(game, masks)
    np.testing.assert_array_equal(y[g["rows"]], g["y_rows"])
    phi = wls.kernel_shap(masks, w, y, float(g["f_empty"]), float(g["f_full"]))
    np.testing.assert_allclose(phi, g["phi"], rtol=0, atol=1e-12 * np.abs(phi).max())
