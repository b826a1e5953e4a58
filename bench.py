"""Benchmark of the GNNShap hot path on one MI355X.

One step = Alg. 1 for every target of the Cora-shaped workload (2,708 nodes,
10,556 directed edges, 2-layer GCN 16 hidden / 7 classes, 100 targets with
20..400 players, 10,000 coalitions each): extract the computational graph,
plan, sample, evaluate every coalition, solve the least squares.  Inputs
(graph, features, weights) are resident in HBM before the timed region.

Prints one JSON line: coalition evaluations per second over the whole job,
explain latency per target (host wall time from extraction to phi on the
host), the dominant kernel's roofline figures and the oracle's CPU rate.
"""
import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="cora")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--streams", type=int, default=8)
    return ap.parse_args()


def cpu_baseline(cfg, seconds):
    """The oracle as it stands, on a bounded sample: whole targets of the same
    workload, one after another, until `seconds` of CPU work have passed."""
    from threadpoolctl import threadpool_limits
    from oracle import explain as oracle_explain
    done_k = 0
    t0 = time.perf_counter()
    n = 0
    with threadpool_limits(limits=1):
        for v in cfg["targets"]:
            r = oracle_explain.explain(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"],
                                       v, cfg["hops"], cfg["p"], cfg["seed"])
            done_k += r["plan"]["k"]
            n += 1
            if time.perf_counter() - t0 >= seconds:
                break
    dt = time.perf_counter() - t0
    return {"value": done_k / dt, "unit": "coalition evals/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} whole targets of the {cfg['name']} workload ({done_k} coalitions, "
                      f"extract+sample+fp64 GCN per coalition+lstsq) in {dt:.1f} s, 1 thread"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; multi-GPU runs are not part of it",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import workloads as W
    from paper_2401_04829_amd.explainer import Explainer

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = W.make_config(args.config)
    ex = Explainer(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"], cfg["hops"], device=dev)
    targets = cfg["targets"]

    def step():
        ex.prepare()                 # X W_1 once per step, shared by every target
        res = ex.explain_many(targets, cfg["p"], cfg["seed"], n_streams=args.streams)
        return sum(r.plan.num_rows for r in res), res

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    total_k = 0
    for _ in range(args.steps):
        k, _ = step()
        total_k += k
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = 1e3 * dt / args.steps

    # explain latency per target: extraction to phi on the host
    lat = []
    for v in targets:
        t1 = time.perf_counter()
        r = ex.explain(v, cfg["p"], cfg["seed"])
        r.phi.cpu()
        lat.append(1e3 * (time.perf_counter() - t1))
    lat_sorted = sorted(lat)
    p90 = lat_sorted[min(len(lat) - 1, int(round(0.9 * (len(lat) - 1))))]

    out = {
        "metric": "masked coalition evals/sec + explain latency per target node (1 GPU)",
        "value": total_k / dt,
        "unit": "coalition evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": f"{args.config}: {len(targets)} targets, {cfg['p']} coalitions each, "
                               f"{cfg['indptr'].size - 1} nodes, {cfg['indices'].size} edges, "
                               f"GCN {cfg['dims']}, {cfg['hops']}-hop"},
        "latency_ms": {"median": statistics.median(lat), "p90": p90, "targets": len(lat)},
        "roofline": None,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
