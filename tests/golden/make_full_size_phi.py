"""Writes the expected Shapley values of full-size targets, computed by the
oracle alone, for the GPU parity tests (tests/test_gpu_full_phi.py).

    python tests/golden/make_full_size_phi.py [pubmed arxiv reddit]

For each case: the oracle's pruned computational graph (Sec. 3.2), the plan
and every sampled coalition (eq. 4-6, Alg. 2-3), the fp64 GCN value of every
coalition (Sec. 4.2, gcn.values_many) and the constrained least squares of
eq. 2-3 (wls.kernel_shap by SVD up to 600 players, wls.kernel_shap_normal
above).  Stored per case in full_size_phi_<workload>_<target>.npz: phi,
f(empty), f(E_c), the explained class, the SHA-256 of the packed masks (the
GPU's masks must equal them bit for bit) and the values of 64 sampled rows.
Only oracle/ and workloads/ are used; nothing comes from the HIP library.
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import workloads as W  # noqa: E402
from oracle import gcn, sampler, subgraph, wls  # noqa: E402


def cases(name, cfg):
    """(label, target) pairs: the target with the fewest players and, for the
    PubMed-shaped workload, the one with the most (the multi-block solve)."""
    ms = [(subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])["num_edges"], v) for v in cfg["targets"]]
    out = [("smallest", min(ms)[1])]
    if name == "pubmed":
        out.append(("largest", max(ms)[1]))
    return out


def one(name, cfg, v, label):
    t0 = time.time()
    sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
    M = sub["num_edges"]
    game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"])
    logits = game.logits(np.ones(M, bool))
    cls = gcn.predicted_class(logits)
    srt = np.sort(logits)[::-1]
    game.cls = cls
    f0, f1 = game(np.zeros(M, bool)), float(logits[cls])
    pl = sampler.plan(M, cfg["p"])
    masks, w = sampler.sample(pl, cfg["seed"], v)
    t1 = time.time()
    y = gcn.values_many(game, masks)
    t2 = time.time()
    if M <= 600:
        phi, how = wls.kernel_shap(masks, w, y, f0, f1), "lstsq"
    else:
        phi, how = wls.kernel_shap_normal(masks, w, y, f0, f1), "normal"
    t3 = time.time()
    digest = hashlib.sha256(np.ascontiguousarray(sampler.pack(masks)).tobytes()).hexdigest()
    rng = np.random.default_rng(v)
    rows = np.unique(np.concatenate([rng.integers(0, pl["k"], 62), [0, pl["k"] - 1]]))
    path = os.path.join(HERE, f"full_size_phi_{name}_{v}.npz")
    np.savez(path, workload=np.array(name), label=np.array(label), target=np.int64(v), M=np.int64(M),
             k=np.int64(pl["k"]), cls=np.int64(cls), top2_gap=np.float64(srt[0] - srt[1]), f_empty=np.float64(f0),
             f_full=np.float64(f1), phi=phi, solver=np.array(how), masks_sha256=np.array(digest), rows=rows,
             y_rows=y[rows])
    print(f"{name} {label} target {v}: M={M} k={pl['k']} sample {t1 - t0:.1f}s values {t2 - t1:.1f}s "
          f"solve ({how}) {t3 - t2:.1f}s -> {os.path.basename(path)}", flush=True)


def main():
    names = sys.argv[1:] or ["pubmed", "arxiv", "reddit"]
    for name in names:
        t = time.time()
        cfg = W.make_config(name)
        print(f"{name}: inputs in {time.time() - t:.1f}s", flush=True)
        for label, v in cases(name, cfg):
            one(name, cfg, v, label)


if __name__ == "__main__":
    main()
