"""Benchmark of the GNNShap hot path on one MI355X.

One step = Alg. 1 for every target of the Reddit-shaped workload by default
(232,965 nodes, 114.6M directed edges, 602-dim features, 2-layer GCN 128
hidden / 41 classes, 20 targets with 2-hop computational graphs of
10,000-30,000 players, 100,000 coalitions each): X W_1, extract the
computational graphs, plan, sample, evaluate every coalition, solve the least
squares.  The whole batch of targets goes through one launch sequence per
step (gnnshap_extract_batch_launch/_finish + gnnshap_explain_batch), the
steps pipelined: each step's extraction is queued before the previous step's
explanation.  --config names another workload (tiny, cora, pubmed, arxiv);
--mode streams runs the single-target calls on several streams instead.
Inputs (graph, features, weights) are resident in HBM before the timed
region.

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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="reddit")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="wall seconds of oracle work per worker process for cpu_baseline")
    ap.add_argument("--mode", choices=["batch", "streams"], default="batch",
                    help="batch: one launch per step for all targets; streams: per-target calls on several streams")
    ap.add_argument("--streams", type=int, default=3)
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--no-latency", action="store_true",
                    help="skip the single-target latency pass (for counter runs)")
    ap.add_argument("--roofline-steps", type=int, default=2)
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
            plan.iterative_threshold = thr
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
        a, b = res["factorised"][2], res["iterative"][2]
        print(json.dumps({"solver_sweep": {"players": M, "coalitions": p, "random_rows": k // 2 - plan.random_begin,
                                           "factorised_ms": res["factorised"][0], "iterative_ms": res["iterative"][0],
                                           "info": [res["factorised"][1], res["iterative"][1]],
                                           "max_dphi_over_max_phi": float((a - b).abs().max() / a.abs().max())}}))
        del masks, weights, ws, y
        torch.cuda.empty_cache()


def gat_times():
    """Explain times of 100 cora-shaped targets x 10,000 coalitions for the
    two-layer GAT of App. E (8 heads of 16, random-init) and for the GCN of
    the same workload: one target at a time, and the whole batch through the
    batched entry points (gnnshap_gat_explain_batch / gnnshap_explain_batch)."""
    import torch
    import workloads as W
    from paper_2401_04829_amd.explainer import Explainer, GatExplainer
    cfg = W.make_config("cora")
    P = W.glorot_gat(cfg["X"].shape[1], 8, 16, len(cfg["weights"][-1][0]), 41)
    targets = [int(v) for v in cfg["targets"]]
    for name, ex in (("gat", GatExplainer(cfg["indptr"], cfg["indices"], cfg["X"], P)),
                     ("gcn", Explainer(cfg["indptr"], cfg["indices"], cfg["X"], cfg["weights"], cfg["biases"],
                                       cfg["hops"]))):
        for mode in ("one_at_a_time", "batch"):
            best = None
            for _ in range(3):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                if mode == "batch":
                    ex.explain_batch(targets, cfg["p"], cfg["seed"])
                else:
                    for v in targets:
                        ex.explain(v, cfg["p"], cfg["seed"])
                torch.cuda.synchronize()
                dt = time.perf_counter() - t0
                best = dt if best is None else min(best, dt)
            print(json.dumps({"explain_times": {"model": name, "mode": mode, "targets": len(targets),
                                                "coalitions": cfg["p"], "ms_total": 1e3 * best,
                                                "ms_per_target": 1e3 * best / len(targets)}}))


_CPU_CFG = None


def _oracle_worker(job):
    """One worker of the CPU baseline: the oracle on one target's sampled
    rows (extraction, the GCN game, the plan, then per row its Floyd or
    unranked coalition and the fp64 GCN forward) until `seconds` have passed."""
    from threadpoolctl import threadpool_limits
    import numpy as np
    from oracle import gcn, sampler, subgraph
    t_index, seconds = job
    cfg = _CPU_CFG
    v = cfg["targets"][t_index % len(cfg["targets"])]
    t0 = time.perf_counter()
    done = 0
    with threadpool_limits(limits=1):
        sub = subgraph.extract(cfg["indptr"], cfg["indices"], v, cfg["hops"])
        M = sub["num_edges"]
        game = gcn.Game(sub, cfg["X"], cfg["weights"], cfg["biases"])
        game.cls = gcn.predicted_class(game.logits(np.ones(M, bool)))
        pl = sampler.plan(M, cfg["p"])
        rng = np.random.default_rng(1000 + t_index)
        while time.perf_counter() - t0 < seconds:
            rows = rng.integers(0, pl["k"], 4)
            m, _ = sampler.sample_rows(pl, rows, cfg["seed"], v)
            game.values(m)
            done += len(rows)
    return done, time.perf_counter() - t0, M


def cpu_baseline(cfg, seconds):
    """The oracle as it stands on a bounded sample of the same workload, run
    on the host's cores before the GPU is touched: one process per core
    (fork, BLAS limited to one thread each), each on one target's sampled
    rows for `seconds`.  Rate = coalitions evaluated / wall time."""
    import multiprocessing as mp
    import platform
    import numpy as np
    global _CPU_CFG
    _CPU_CFG = cfg
    cores = len(os.sched_getaffinity(0))
    cores = max(1, min(cores, int(os.environ.get("OMP_NUM_THREADS", cores) or cores), 16))
    model = platform.processor()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(cores) as pool:
        res = pool.map(_oracle_worker, [(i, seconds) for i in range(cores)])
    wall = time.perf_counter() - t0
    rows = sum(r[0] for r in res)
    return {"value": rows / wall, "unit": "coalition evals/s", "cores": cores, "kind": "oracle",
            "sample": f"{rows} coalitions of the {cfg['name']} workload's targets (one target per process, "
                      f"{cores} processes x ~{seconds:.0f} s, {wall:.1f} s wall): per target the oracle's extraction, "
                      f"GCN game and plan, per coalition its row of the sampler (Floyd / unranking, sample_rows) "
                      f"and the fp64 GCN forward; the oracle's least squares is not in the sample (it needs every "
                      f"row of a target: minutes per target at the reddit-shaped sizes)",
            "cpu_model": model, "numpy": np.__version__}


# Peaks (MI355X): HBM3E 8 TB/s; fp32 VALU without packed-fp32 instructions
# (the library is compiled without them): 256 CUs x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz
# = 78.6 TFLOP/s; 32-bit integer VALU ops at the same issue rate: 39.3 Tops/s.
HBM_PEAK_GBS = 8000.0
VALU_FP32_TFLOPS = 78.6
VALU_INT_TOPS = 39.3
MFMA_FP32_TFLOPS = 157.3
MFMA_BF16_TFLOPS = 2500.0


def work_model(kernel, results, dims, solves):
    """Algorithmic work of the timed kernel over the timed steps: (amount, unit, bound, peak).

    k_wide_l1      two-layer GCN, wide hidden layer: (k/2) M h useful MACs per target
                   (complement pairs cover every player-feature product once), 2 flop
                   each, run as three bf16 products (the fp32 values split exactly into
                   hi + mid + lo), so 3 x that against the bf16 MFMA peak
    k_eval_rows_mx, k_eval_rows, k_eval_l2
                   the same count; k_eval_rows_mx on fp32 MFMA, the others on VALU
    k_cg_pass_a    per iteration of an iterative solve: the mask words of the random
                   rows kept as bits ((kr - rs) x ceil(M/64) x 8 bytes) + the vector r
                   (8 M) + the product (8 (kr - rs)), and for the rs sparse rows their
                   player lists (4 nnz + 8 (rs + 1)), the entries of r they select
                   (8 nnz) and their products (8 rs)
    k_cg_pass_b    the same words (bit-transposed) + u (8 (kr - rs)) + the product (8 M),
                   and the player-major lists (4 nnz + 8 (M + 1)), the entries of u
                   they select (8 nnz) and their products (8 M)
    k_cg_rows      the pass-A partial products of the bit rows (8 npc (kr - rs), npc
                   taken as ceil(ceil(M/64) / 16)) and u written (8 (kr - rs))
    k_cg_update    five fp64 vectors of M read (R^T u, r, p, s, x) and four written
    k_solve_mid / k_solve_one_batch (one-workgroup solves)
                   M^3/6 (Cholesky) + 2 M^2 (two triangular solves) MACs, 2 flop each
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
    if base.startswith("k_cg_"):
        tot = 0.0
        for M, wpr, kr, iters, rs, nnz in solves:
            bits = (kr - rs) * wpr * 8.0 + 8.0 * M + 8.0 * (kr - rs)
            if base == "k_cg_pass_a":
                tot += iters * (bits + 12.0 * nnz + 16.0 * rs + 8.0)
            elif base == "k_cg_pass_b":
                tot += iters * (bits + 12.0 * nnz + 16.0 * M + 8.0)
            elif base == "k_cg_rows":
                npc = -(-wpr // 16)
                tot += iters * 8.0 * (npc + 1) * (kr - rs)
            elif base == "k_cg_update":
                tot += iters * 72.0 * M
        return tot, "GB/s", "hbm", HBM_PEAK_GBS
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
        elif base == "k_wide_l1":
            tot += 3.0 * 2.0 * (k / 2.0) * M * h
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
    if base == "k_wide_l1":
        return tot, "TFLOP/s", "mfma", MFMA_BF16_TFLOPS
    if base == "k_eval_rows_mx":
        return tot, "TFLOP/s", "mfma", MFMA_FP32_TFLOPS
    return tot, "TFLOP/s", "alu", VALU_FP32_TFLOPS


CANDIDATES = {
    "batch": ["k_cg_pass_a", "k_cg_pass_b", "k_cg_rows", "k_cg_update", "k_wide_l1", "k_eval_rows_mx_batch", "k_eval_rows_batch",
              "k_solve_one_batch", "k_eval_l2_batch", "k_gram_batch", "k_rhs_tile_batch", "k_sample"],
    "streams": ["k_cg_pass_a", "k_cg_pass_b", "k_cg_rows", "k_cg_update", "k_wide_l1", "k_solve_mid", "k_eval_rows_mx", "k_eval_l2",
                "k_rhs_tile", "k_gram", "k_sample"],
}


def roofline(run, lib, dims, mode, steps):
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
        solves = lib.gnnshap_timing_solves()
        if n and (best is None or ms > best[1]):
            best = (name, ms, n, res, solves)
    name, ms, n, res, solves = best
    amount, unit, bound, peak = work_model(name, res, dims, solves)
    if not name.startswith("k_cg_"):
        amount *= steps                          # per-step model, `steps` steps timed
    avg_s = ms / 1e3 / n
    per_launch = amount / n
    scale = 1e9 if unit == "GB/s" else 1e12
    achieved = per_launch / avg_s / scale
    return {"kernel": name, "bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
            "frac": achieved / peak, "traffic": measured_traffic(name), "launches": n,
            "avg_launch_us": 1e3 * ms / n, "work_per_launch": per_launch,
            "iterative_solves": len(solves) if name.startswith("k_cg_") else None}


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
        print(json.dumps({"error": "bench.py runs on one GPU: a share of the targets per GPU is not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import workloads as W

    if args.solver_sweep or args.gat:
        import torch
        assert torch.cuda.is_available(), "bench.py needs a GPU"
        if args.solver_sweep:
            solver_sweep()
        if args.gat:
            gat_times()
        return
    t_gen = time.perf_counter()
    cfg = W.make_config(args.config)
    print(f"workload {args.config}: inputs generated in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)
    # the CPU baseline forks its worker processes before anything touches the GPU
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, args.cpu_seconds)
        print(f"cpu baseline: {cpu['value']:.1f} coalitions/s on {cpu['cores']} cores", file=sys.stderr, flush=True)

    import torch
    from paper_2401_04829_amd.explainer import Explainer
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
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
    print(f"warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    total_k, last = run(args.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = 1e3 * dt / args.steps
    print(f"timed: {args.steps} steps, {ms_per_step:.1f} ms per step", file=sys.stderr, flush=True)
    # every system of the last timed step was solved
    infos = ([int(x) for x in last.info.cpu().tolist()] if args.mode == "batch"
             else [int(r.info.item()) for r in last])
    assert all(i == 0 for i in infos), f"solver info {infos}"

    # explain latency per target: extraction to phi on the host, after one warm-up target
    latency = None
    if not args.no_latency:
        ex.explain(targets[0], cfg["p"], cfg["seed"]).phi.cpu()
        lat = []
        for v in targets:
            t1 = time.perf_counter()
            r = ex.explain(v, cfg["p"], cfg["seed"])
            r.phi.cpu()
            lat.append(1e3 * (time.perf_counter() - t1))
        lat_sorted = sorted(lat)
        p90 = lat_sorted[min(len(lat) - 1, int(round(0.9 * (len(lat) - 1))))]
        latency = {"median": statistics.median(lat), "p90": p90, "targets": len(lat)}
        print("latency pass done", file=sys.stderr, flush=True)

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
        "latency_ms": latency,
        "roofline": None,
        "cpu_baseline": cpu,
    }
    if not args.no_roofline:
        from paper_2401_04829_amd import _lib
        out["roofline"] = roofline(lambda n: run(n)[1], _lib, cfg["dims"], args.mode, args.roofline_steps)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
