"""Benchmark of the GNNShap hot path on one MI355X.

One step = Alg. 1 for every target of the Cora-shaped workload (2,708 nodes,
10,556 directed edges, 2-layer GCN 16 hidden / 7 classes, 100 targets with
20..400 players, 10,000 coalitions each): X W_1, extract the computational
graphs, plan, sample, evaluate every coalition, solve the least squares.  By
default the whole batch of targets goes through one launch per step
(gnnshap_extract_batch_launch/_finish + gnnshap_explain_batch), the steps
pipelined: each step's extraction is queued before the previous step's
explanation.  --mode streams runs the single-target calls on several
streams instead.  Inputs (graph, features, weights) are resident in HBM
before the timed region.

Prints one JSON line: coalition evaluations per second over the whole job,
explain latency per target (host wall time from extraction to phi on the
host), the dominant kernel's roofline figures and the oracle's CPU rate.
"""
import argparse
import itertools
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
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="cora")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--mode", choices=["batch", "streams"], default="batch",
                    help="batch: one launch per step for all targets; streams: per-target calls on several streams")
    ap.add_argument("--streams", type=int, default=3)
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="bytes of a plain device copy run before the steps (counter calibration)")
    ap.add_argument("--solver-sweep", action="store_true",
                    help="instead of the step: least-squares solve times, factorisation vs iterative")
    ap.add_argument("--gat", action="store_true",
                    help="instead of the step: explain times of the GAT variant and the GCN, one target at a time")
    return ap.parse_args()


def solver_sweep():
    """Solve times of gnnshap_solve_wls on sampled plans of 6,000-30,000
    players, through the factorisation and through the iterative path
    (Sec. 3.5), on noisy values; one JSON line per case."""
    import torch
    from paper_2401_04829_amd import _lib as L
    from paper_2401_04829_amd.explainer import _vp
    dev = torch.device("cuda:0")
    s = torch.cuda.current_stream().cuda_stream
    for M, p in [(6000, 50000), (12000, 50000), (20000, 50000), (30000, 100000)]:
        plan, classes = L.gnnshap_plan_samples(M, p, 3, 4)
        k, wpr = plan.num_rows, plan.words_per_row
        masks = torch.empty((k, wpr), dtype=torch.int64, device=dev)
        weights = torch.empty(k, dtype=torch.float32, device=dev)
        ws = torch.empty(max(L.gnnshap_sample_workspace(plan), 256), dtype=torch.uint8, device=dev)
        L.gnnshap_sample_coalitions(plan, classes, _vp(masks), _vp(weights), _vp(ws), ws.numel(), s)
        g = torch.Generator(device=dev)
        g.manual_seed(M)
        y = torch.randn(k, generator=g, device=dev)
        fef = torch.tensor([0.1, 0.7], dtype=torch.float32, device=dev)
        res = {}
        for path, thr in (("factorised", M + 1), ("iterative", M - 1)):
            L.gnnshap_set_iterative_threshold(thr)
            phi = torch.empty(M, dtype=torch.float32, device=dev)
            info = torch.empty(1, dtype=torch.int32, device=dev)
            wsol = torch.empty(L.gnnshap_solve_workspace(plan), dtype=torch.uint8, device=dev)
            times = []
            for _ in range(3):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                L.gnnshap_solve_wls(plan, classes, _vp(masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(wsol),
                                    wsol.numel(), s)
                torch.cuda.synchronize()
                times.append(1e3 * (time.perf_counter() - t0))
            res[path] = (min(times), int(info.item()), phi.double())
            del wsol
        L.gnnshap_set_iterative_threshold(5000)
        a, b = res["factorised"][2], res["iterative"][2]
        print(json.dumps({"solver_sweep": {"players": M, "coalitions": p, "random_rows": k // 2 - plan.random_begin,
                                           "factorised_ms": res["factorised"][0], "iterative_ms": res["iterative"][0],
                                           "info": [res["factorised"][1], res["iterative"][1]],
                                           "max_dphi_over_max_phi": float((a - b).abs().max() / a.abs().max())}}))
        del masks, weights, ws, y
        torch.cuda.empty_cache()


def gat_times():
    """Explain times of 100 cora-shaped targets x 10,000 coalitions, one
    target at a time, for the two-layer GAT of App. E (8 heads of 16,
    random-init) and for the GCN of the same workload."""
    import torch
    import workloads as W
    from paper_2401_04829_amd.explainer import Explainer, GatExplainer
    cfg = W.make_config("cora")
    P = W.glorot_gat(cfg["X"].shape[1], 8, 16, len(cfg["weights"][-1][0]), 41)
    for name, ex in (("gat", GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)),
                     ("gcn", Explainer(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"],
                                       cfg["hops"]))):
        best = None
        for _ in range(2):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for v in cfg["targets"]:
                ex.explain(v, cfg["p"], cfg["seed"])
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            best = dt if best is None else min(best, dt)
        print(json.dumps({"explain_one_at_a_time": {"model": name, "targets": len(cfg["targets"]),
                                                    "coalitions": cfg["p"], "ms_total": 1e3 * best,
                                                    "ms_per_target": 1e3 * best / len(cfg["targets"])}}))


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


# Peaks (MI355X): HBM3E 8 TB/s; fp32 VALU without packed-fp32 instructions
# (this build disables them): 256 CUs x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz
# = 78.6 TFLOP/s; 32-bit integer VALU ops at the same issue rate: 39.3 Tops/s.
HBM_PEAK_GBS = 8000.0
VALU_FP32_TFLOPS = 78.6
VALU_INT_TOPS = 39.3
MFMA_FP32_TFLOPS = 157.3


def work_model(kernel, results, dims):
    """Algorithmic work of the timed kernel over one step: (amount, unit, bound, peak).

    k_solve_mid / k_solve_one_batch (one-workgroup solves)
                   M^3/6 (Cholesky) + 2 M^2 (two triangular solves) MACs, 2 flop each
    k_eval_l2, k_eval_rows, k_eval_rows_mx
                   (k/2) M h useful MACs per target (complement pairs cover every
                   player-feature product once) + the layer-1 logit dot products;
                   k_eval_rows_mx runs the contraction on fp32 MFMA, so its roof is
                   the fp32 MFMA peak (the dense 0/1 product it issues is twice the
                   useful count, which is what is reported)
    k_gram         K_R M(M+1)/2 pair counts over the random rows, 1 popcount-AND
                   per 64 rows and pair
    k_sample       k x ceil(M/64) x 8 bytes of masks + 4 k bytes of weights written
    k_rhs_part, k_rhs_tile
                   (k/2) x ceil(M/64) x 8 bytes of masks + 4 k bytes of y read
    (a *_batch kernel does the same work for every target of the batch)
    """
    from paper_2401_04829_amd import _lib
    h = dims[1]
    base = kernel[:-len("_batch")] if kernel.endswith("_batch") else kernel
    tot = 0.0
    for r in results:
        M, k = r.plan.num_players, r.plan.num_rows
        wpr = r.plan.words_per_row
        kr = k // 2 - r.plan.random_begin
        path = _lib.gnnshap_solve_info(r.plan)
        batched = kernel.endswith("_batch")
        if base in ("k_solve_mid", "k_solve_one"):
            if path == 1:
                tot += 2.0 * (M ** 3 / 6.0 + 2.0 * M * M)
        elif base in ("k_eval_l2", "k_eval_rows", "k_eval_rows_mx"):
            n1 = r.sub.sg.hop_ptr[2]
            tot += 2.0 * ((k / 2.0) * M * h + k * n1 * h)
        elif base == "k_gram":
            if not batched or path in (1, 2):
                tot += (kr / 64.0) * M * (M + 1) / 2.0
        elif base == "k_sample":
            tot += k * wpr * 8.0 + 4.0 * k
        elif base in ("k_rhs_part", "k_rhs_tile"):
            if not batched or path in (1, 2):
                tot += (k / 2.0) * wpr * 8.0 + 4.0 * k
    if base in ("k_sample", "k_rhs_part", "k_rhs_tile"):
        return tot, "GB/s", "hbm", HBM_PEAK_GBS
    if base == "k_gram":
        return tot, "Tops/s", "alu", VALU_INT_TOPS
    if base == "k_eval_rows_mx":
        return tot, "TFLOP/s", "mfma", MFMA_FP32_TFLOPS
    return tot, "TFLOP/s", "alu", VALU_FP32_TFLOPS


CANDIDATES = {
    "batch": ["k_eval_rows_mx_batch", "k_eval_rows_batch", "k_solve_one_batch", "k_eval_l2_batch", "k_gram_batch", "k_rhs_tile_batch",
              "k_sample_batch"],
    "streams": ["k_solve_mid", "k_eval_rows_mx", "k_eval_l2", "k_rhs_tile", "k_gram", "k_sample"],
}


def roofline(run, lib, dims, mode, steps=10):
    """Times each candidate kernel with HIP events over `steps` steps run as in
    the timed region, picks the one with the largest total and relates its
    algorithmic work to its average launch duration."""
    import torch
    best = None
    for name in CANDIDATES[mode]:
        lib.gnnshap_timing_begin(name)
        res = run(steps)
        torch.cuda.synchronize()
        ms, n = lib.gnnshap_timing_end()
        if n and (best is None or ms > best[1]):
            best = (name, ms, n, res)
    name, ms, n, res = best
    amount, unit, bound, peak = work_model(name, res, dims)
    amount *= steps
    avg_s = ms / 1e3 / n
    per_launch = amount / n
    scale = 1e9 if unit == "GB/s" else 1e12
    achieved = per_launch / avg_s / scale
    return {"kernel": name, "bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
            "frac": achieved / peak, "traffic": measured_traffic(name), "launches": n,
            "avg_launch_us": 1e3 * ms / n, "work_per_launch": per_launch}


def measured_traffic(kernel):
    """HBM bytes per dispatch from the committed counter summary
    (profiles/hbm_traffic.json: FETCH_SIZE and WRITE_SIZE scaled by a copy of
    known size), or None when the kernel's source changed since then."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel)
        if rec is None:
            return None
        with open(os.path.join(ROOT, rec["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != rec["source_sha256"]:
                return None
        return rec["hbm_bytes_per_dispatch"]
    except (OSError, ValueError, KeyError):
        return None


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
    if args.solver_sweep or args.gat:
        if args.solver_sweep:
            solver_sweep()
        if args.gat:
            gat_times()
        return
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    cfg = W.make_config(args.config)
    print(f"workload {args.config}: inputs generated in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)
    ex = Explainer(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"], cfg["hops"], device=dev)
    targets = cfg["targets"]

    def step():
        ex.prepare()                 # X W_1 once per step, shared by every target
        if args.mode == "batch":
            res = ex.explain_batch(targets, cfg["p"], cfg["seed"])
            return res.total_rows, res
        res = ex.explain_many(targets, cfg["p"], cfg["seed"], n_streams=args.streams)
        return sum(r.plan.num_rows for r in res), res

    if args.copy_probe:
        # a plain device copy of known size, for calibrating HBM byte counters
        n = args.copy_probe // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    def run(steps):
        """`steps` steps; in batch mode pipelined, each batch's extraction queued
        before the previous batch's explanation.  Returns (coalitions done, the
        last step's results)."""
        total, last = 0, None
        if args.mode == "batch":
            for res in ex.explain_batches(itertools.repeat(targets, steps), cfg["p"], cfg["seed"], prepare_each=True):
                total += res.total_rows
                last = res
            return total, last
        for _ in range(steps):
            k, last = step()
            total += k
        return total, last

    run(args.warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    total_k, _ = run(args.steps)
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
                               f"GCN {cfg['dims']}, {cfg['hops']}-hop",
                   "mode": args.mode},
        "latency_ms": {"median": statistics.median(lat), "p90": p90, "targets": len(lat)},
        "roofline": None,
        "cpu_baseline": None,
    }
    if not args.no_roofline:
        from paper_2401_04829_amd import _lib
        out["roofline"] = roofline(lambda n: run(n)[1], _lib, cfg["dims"], args.mode)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
