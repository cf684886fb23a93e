"""Throughput of the candidate-scoring pass on one MI355X.

A step is one whole scoring pass over a resident pool (the two-objective
workload: m = 256 observations, n = 262144 candidates, d = 10, EHVI over the
observed front, 64-tree feasibility mask, top-4): GP posterior of both
objectives (K*, mean, triangular product, variance), EHVI, forest mask and
top-q, all on the device.  The host fit of the two GPs happens once before the
timed region and is reported on its own (fit_ms).

Prints one JSON line (rank 0).  Also measures the dominant kernel (the fused
posterior) on its own with HIP events on the stream it runs on, for the
roofline figure, and times the CPU oracle on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_FP64_MFMA_TFLOPS = 78.6
PEAK_HBM_GBPS = 8000.0

# HBM traffic of one posterior launch on the two-objective workload (m=256,
# n=262144, d=10, Matern-5/2) per precision, from rocprofv3 FETCH_SIZE /
# WRITE_SIZE passes (calibrated against a plain copy: FETCH_SIZE x 2.0,
# WRITE_SIZE x 1.0), valid only for that workload and the kernel source they
# were taken on.
POSTERIOR_TRAFFIC = {"source_sha1": "2390c5c7a554f5900a4d3815ba24f2cb7a60f96a",
                     "bytes": {"f32": 14046269, "f64": 17451049}}


def posterior_traffic(args):
    if args.config != 3 or args.kernel != "matern52" or args.warp:
        return None
    import hashlib
    src = os.path.join(ROOT, "paper_2408_04323_amd", "csrc", "k_posterior.hip")
    with open(src, "rb") as fh:
        digest = hashlib.sha1(fh.read()).hexdigest()
    if digest == POSTERIOR_TRAFFIC["source_sha1"]:
        return POSTERIOR_TRAFFIC["bytes"][args.dtype]
    return None
METRIC = "candidate configs scored/sec (GP+acq+RF mask) and % roofline, m=256 n=262144"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20,
                    help="untimed passes first: the GPU's clocks take some 10 ms of load to settle")
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="default run only: skip the other workloads timed after the metric (the whole "
                         "suggestion step, three objectives at m=512 n=2^20, the believer, MACE)")
    ap.add_argument("--kernel-loops", type=int, default=20)
    ap.add_argument("--kernel", choices=["matern52", "matern32"], default="matern52",
                    help="covariance of the GPs (matern32 = the paper's own)")
    ap.add_argument("--warp", action="store_true", help="Kumaraswamy input warping (the paper's own)")
    ap.add_argument("--dtype", choices=["f32", "f64"], default="f32",
                    help="precision of the scoring pass (posterior, acquisition, top-q keys); the pool stays "
                         "float32")
    ap.add_argument("--mace", action="store_true",
                    help="one-objective workloads: time the MACE suggestion (posterior, UCB/PI/EI, mask, "
                         "Pareto front, seeded pick) and print its own line")
    ap.add_argument("--suggest", action="store_true",
                    help="time the whole suggestion step (scoot_suggest: hyperparameter search, forest "
                         "training, Sobol pool with known constraints, scoring, pick) on the workload's "
                         "observations and print its own line")
    ap.add_argument("--only", choices=["all", "posterior", "forest", "ehvi", "topq", "pass", "copy"], default="all",
                    help="posterior / forest / ehvi / topq: only that kernel's loop (for profiler "
                         "counters); pass: only the loop of whole scoring passes (every kernel the metric "
                         "times, the fused EHVI and top-q stage 1 included); copy: a plain 1 GiB device copy "
                         "(counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(this build runs on a single GPU; the scoring pass would shard by candidate)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2408_04323_amd as S
    from workloads import make_workload
    from workloads.synth import CONFIGS

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    if args.only == "copy":
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": a.numel() * 4, "copy_bytes_written": b.numel() * 4}))
        return

    if args.suggest:
        return bench_suggest(args)
    if args.config == 5:
        return bench_believer(args)
    if args.mace:
        return bench_mace(args)
    t0 = time.time()
    w = make_workload(args.config, kernel=args.kernel, warp=args.warp)
    gen_s = time.time() - t0
    c = CONFIGS[args.config]
    p, n, m = w["p"], len(w["Xc"]), w["m"]

    # library load and first-call setup happen before the fit is timed
    S.gp_fit(w["X"][:8], w["Y"][:8, 0], w["lengthscale"][0], 1.0, 1e-3).close()
    tf = time.perf_counter()
    warps = w.get("warp")
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                    w["prior_mean"][j], dtype=args.dtype, kernel=args.kernel,
                    warp_a=None if warps is None else warps[0][j], warp_b=None if warps is None else warps[1][j])
           for j in range(p)]
    fit_ms = (time.perf_counter() - tf) * 1e3
    fd = w["forest"]
    forest = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"],
                             fd["tree_offset"], w["d"])
    Xc = torch.as_tensor(w["Xc"]).to(dev)
    bufs = S.PoolBuffers(n, p, w["q"], gps[0].dtype, dev)
    front, n_boxes = S.ehvi_front(w["Y"], w["ref"]) if p > 1 else (np.zeros((0, 1)), 0)
    print(f"[bench] workload {c['name']} m={m} n={n} d={w['d']} p={p} front={len(front)} "
          f"gen {gen_s:.1f}s fit {fit_ms:.1f}ms", file=sys.stderr, flush=True)

    def step():
        S.score_pool(gps, forest, Xc, w["q"], best_y=w["best_y"], xi=w["xi"], Y_obs=w["Y"],
                     ref=w.get("ref"), delta=w["delta"], buffers=bufs)

    def time_loop(fn, loops):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(loops):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / loops  # ms

    # dominant kernel: the fused posterior of one objective, on the stream it runs on
    def post():
        S.posterior(gps[0], Xc, bufs.mu[0], bufs.sigma[0])

    # The clocks take some 10 ms of load to settle (a kernel trace shows the
    # same launch at 224 us cold and 206 us warm): 40 launches first.
    for _ in range(40):
        post()
    if args.only == "posterior":
        ms = time_loop(post, args.kernel_loops)
        print(json.dumps({"posterior_ms": ms}))
        return
    if args.only == "pass":
        step()
        print(json.dumps({"pass_ms": time_loop(step, args.kernel_loops)}))
        return
    if args.only in ("forest", "ehvi", "topq"):
        step()
        fn = {"forest": lambda: S.rf_feasibility(forest, Xc, w["delta"], votes=bufs.votes, mask=bufs.mask),
              "ehvi": lambda: S.acq_ehvi([bufs.mu[j] for j in range(p)], [bufs.sigma[j] for j in range(p)],
                                         w["Y"], w["ref"], out=bufs.acq),
              "topq": lambda: S.suggest_topq(bufs.acq, bufs.mask, w["q"])}[args.only]
        fn()
        print(json.dumps({args.only + "_ms": time_loop(fn, args.kernel_loops)}))
        return
    # Back-to-back launches between one pair of events (an event pair around
    # every launch adds about 10 us of its own between launches).
    post_ms = sorted(time_loop(post, args.kernel_loops) for _ in range(3))[1]

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = e0.elapsed_time(e1) / args.steps
    value = n / (ms_per_step * 1e-3)
    # The median step: 21 more loops of 20 back-to-back passes, each between
    # one event pair (a pair around every single pass would add its own gap,
    # and a short loop would carry the start-up of its first pass).
    reps = sorted(time_loop(step, 20) for _ in range(21))
    median_ms = reps[len(reps) // 2]
    print(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (wall {wall:.3f}s), median {median_ms:.3f}, "
          f"posterior {post_ms:.3f} ms/objective", file=sys.stderr, flush=True)

    # other kernels, for the record
    ehvi_ms = rf_ms = topq_ms = None
    if p > 1:
        ehvi_ms = time_loop(lambda: S.acq_ehvi([bufs.mu[j] for j in range(p)], [bufs.sigma[j] for j in range(p)],
                                               w["Y"], w["ref"], out=bufs.acq), args.kernel_loops)
    rf_ms = time_loop(lambda: S.rf_feasibility(forest, Xc, w["delta"], votes=bufs.votes, mask=bufs.mask),
                      args.kernel_loops)
    topq_ms = time_loop(lambda: S.suggest_topq(bufs.acq, bufs.mask, w["q"]), args.kernel_loops)
    esz = 8 if args.dtype == "f64" else 4
    # Algorithmic HBM bytes per candidate of the other kernels (what each must
    # read and write once): EHVI reads p means and p deviations and writes the
    # score; the forest reads the d features and writes votes (int32) and the
    # mask byte; top-q reads the score and the mask byte.
    hbm = {"ehvi": (2 * p + 1) * esz if p > 1 else None, "forest": 4 * w["d"] + 5, "topq": esz + 1}
    kernels = {}
    for name, ms in (("ehvi", ehvi_ms), ("forest", rf_ms), ("topq", topq_ms)):
        if ms is None:
            continue
        gbs = hbm[name] * n / (ms * 1e-3) / 1e9
        kernels[name] = {"ms_per_call": ms, "bytes_per_candidate": hbm[name], "achieved_GBps": gbs,
                         "hbm_peak_GBps": PEAK_HBM_GBPS, "hbm_frac": gbs / PEAK_HBM_GBPS}
    kernels["note"] = ("one library call each, host-side argument work included; these kernels are bound by "
                       "VALU issue (EHVI), LDS latency (forest) and launch latency (top-q) rather than HBM, so "
                       "hbm_frac is small by design; the VALU and LDS counters are in profiles/")

    # Algorithmic work of the fused posterior per candidate and objective: the
    # triangular product (m^2 flops) and K* with the mean (m (3d + 10) flops;
    # the m square roots and m exponentials are not counted).  On gfx950 the
    # fp32 matrix instructions and the vector ALU share one datapath (measured:
    # they do not overlap), so both draw on the same 157.3 TFLOP/s (78.6 in
    # fp64, for the matrix instructions and the vector ALU alike).
    flops_trsm = m * m
    flops_per_unit = flops_trsm + m * (3 * w["d"] + 10)
    peak = PEAK_FP64_MFMA_TFLOPS if args.dtype == "f64" else PEAK_FP32_MFMA_TFLOPS
    achieved = flops_per_unit * n / (post_ms * 1e-3) / 1e12
    achieved_trsm = flops_trsm * n / (post_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC if (args.config == 3 and args.kernel == "matern52" and not args.warp
                             and args.dtype == "f32") else
        f"candidate configs scored/sec (GP+acq+RF mask), {c['name']}, {args.kernel}{' warped' if args.warp else ''}"
        f"{', fp64' if args.dtype == 'f64' else ''}",
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{c['name']}: m={m} n={n} d={w['d']} p={p} front={len(front)} boxes={n_boxes} "
                        f"kernel={args.kernel}{' warped inputs' if args.warp else ''} "
                        f"trees={c['trees']} depth={c['depth']} q={w['q']}",
            "timed": "posterior x p + acquisition + forest mask + top-q on the device; host GP fit excluded",
            "fit_ms": fit_ms,
            "value_incl_fit": n / ((ms_per_step + fit_ms) * 1e-3),
            "ms_per_step_median": median_ms,
            "median_of": "21 loops of 20 back-to-back passes, one event pair per loop",
            "kernel_ms": {"posterior_per_objective": post_ms},
            "other_kernels": kernels,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": f"posterior_{args.dtype}_kernel (K*, mean, L^-1 K*^T on {args.dtype[1:]}-bit MFMA, variance)",
            "achieved": achieved,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": achieved / peak,
            "traffic": posterior_traffic(args),
            "algorithmic_unit": f"m^2 + m(3d+10) = {flops_per_unit} flops per candidate per objective "
                                f"(triangular product + K* and mean), {n} candidates per launch",
            "frac_triangular_product_only": achieved_trsm / peak,
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    if (not args.no_secondary and args.only == "all" and args.config == 3 and args.kernel == "matern52"
            and not args.warp and args.dtype == "f32"):
        out["secondary"] = secondary_workloads()
    print(json.dumps(out), flush=True)


# The other workloads, each timed by this script in a child process of its own
# after the metric (they are not part of the metric's timed region), so that
# one run of the default command measures them too.
SECONDARY = [
    ("suggest_step", ["--suggest", "--steps", "5", "--warmup", "2"]),
    ("three_objective_pass", ["--config", "4", "--steps", "10", "--warmup", "10", "--kernel-loops", "5",
                              "--no-cpu-baseline", "--no-secondary"]),
    ("believer", ["--config", "5", "--steps", "5", "--warmup", "2"]),
    ("mace", ["--config", "2", "--mace", "--steps", "20", "--warmup", "10"]),
]


def secondary_workloads():
    import subprocess
    res = {}
    for name, extra in SECONDARY:
        print(f"[bench] secondary workload {name}", file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        try:
            r = subprocess.run([sys.executable, "-u", os.path.abspath(__file__)] + extra, stdout=subprocess.PIPE,
                               text=True, timeout=120)
            lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
            if r.returncode != 0 or not lines:
                res[name] = {"error": f"exit status {r.returncode}"}
                continue
            d = json.loads(lines[-1])
            cfg = d.get("config", {})
            e = {"metric": d["metric"], "value": d["value"], "unit": d["unit"], "ms_per_step": d["ms_per_step"],
                 "steps": d["steps"], "warmup": d["warmup"], "workload": cfg.get("workload")}
            if name == "suggest_step":
                e["ms_per_step_host_search"] = cfg.get("ms_per_step_host_search")
                e["picks_match_host_search"] = cfg.get("picks_match_host_search")
            if name == "three_objective_pass":
                e["roofline_frac"] = d.get("roofline", {}).get("frac")
            res[name] = e
        except subprocess.TimeoutExpired:
            res[name] = {"error": "timed out after 120 s"}
        print(f"[bench] secondary workload {name} done in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
              flush=True)
    res["note"] = "each from `python bench.py` with the listed options, run after the metric in a child process"
    res["options"] = {name: " ".join(extra) for name, extra in SECONDARY}
    return res


def bench_believer(args):
    """Workload 5: q sequential Kriging-believer picks over the full pool (one
    suggestion = posterior with V kept, forest mask, then q x (EHVI re-score,
    top-1, V row update, variance downdate)).  Reported on its own line."""
    import numpy as np
    import torch

    import paper_2408_04323_amd as S
    from workloads import make_workload
    from workloads.synth import CONFIGS

    w = make_workload(5)
    c = CONFIGS[5]
    n, p = len(w["Xc"]), w["p"]
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                    w["prior_mean"][j]) for j in range(p)]
    fd = w["forest"]
    forest = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"],
                             fd["tree_offset"], w["d"])
    Xc = torch.as_tensor(w["Xc"]).cuda()
    ws = torch.empty(S.suggest_kb_workspace(gps, n, w["q"]), dtype=torch.uint8, device="cuda")
    for _ in range(args.warmup):
        S.suggest_kb(gps, forest, Xc, w["q"], w["Y"], w["ref"], w["delta"], workspace=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        picks, _ = S.suggest_kb(gps, forest, Xc, w["q"], w["Y"], w["ref"], w["delta"], workspace=ws)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    print(json.dumps({"metric": "believer suggestion (q sequential picks) per second", "value": 1e3 / ms,
                      "unit": "suggestions/s", "ms_per_step": ms, "n_gpus": 1, "steps": args.steps,
                      "warmup": args.warmup, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": f"{c['name']}: m={w['m']} n={n} d={w['d']} p={p} q={w['q']} "
                                             f"trees={c['trees']} depth={c['depth']}",
                                 "picks": picks.tolist(), "workspace_bytes": ws.numel()}}), flush=True)


def bench_mace(args):
    """A one-objective workload scored the paper's SOBO way (Sec. 4.5.1): one
    suggestion = posterior, UCB/PI/EI, forest mask, Pareto front of the three
    scores over the pool, q drawn from it.  Reported on its own line."""
    import torch

    import paper_2408_04323_amd as S
    from workloads import make_workload
    from workloads.synth import CONFIGS

    w = make_workload(args.config)
    c = CONFIGS[args.config]
    if w["p"] != 1:
        print(f"--mace needs a one-objective workload; workload {args.config} has {w['p']}", file=sys.stderr)
        sys.exit(2)
    n, q = len(w["Xc"]), w["q"]
    gp = S.gp_fit(w["X"], w["Y"][:, 0], w["lengthscale"][0], w["signal_var"][0], w["noise_var"][0],
                  w["prior_mean"][0])
    fd = w["forest"]
    forest = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"],
                             fd["tree_offset"], w["d"])
    Xc = torch.as_tensor(w["Xc"]).cuda()
    beta, seed = S.ucb_beta(w["m"] // q), 240804323
    b = S.MaceBuffers(n, q, gp.dtype, Xc.device)
    stream = torch.cuda.current_stream()

    def step():
        S.suggest_mace(gp, forest, Xc, q, w["best_y"], beta, seed, xi=w["xi"], delta=w["delta"], buffers=b)

    def time_loop(fn, loops):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(loops):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / loops

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms = time_loop(step, args.steps)
    n_front = int(b.n_front.cpu()[0])
    kl = args.kernel_loops
    parts = {
        "posterior": time_loop(lambda: S.posterior(gp, Xc, b.mu, b.sigma), kl),
        "scores": time_loop(lambda: S.acq_mace(b.mu, b.sigma, w["best_y"], beta, xi=w["xi"],
                                               out=(b.ucb, b.pi, b.ei)), kl),
        "forest": time_loop(lambda: S.rf_feasibility(forest, Xc, w["delta"], votes=b.votes, mask=b.mask), kl),
        "front": time_loop(lambda: S.pareto_front3(b.ucb, b.pi, b.ei, b.mask, front=b.front), kl),
        "pick": time_loop(lambda: S.random_pick(b.front, seed, q), kl),
    }
    print(json.dumps({"metric": "MACE suggestions (one objective) per second", "value": 1e3 / ms,
                      "unit": "suggestions/s", "candidates_per_s": n / (ms * 1e-3), "ms_per_step": ms, "n_gpus": 1,
                      "steps": args.steps, "warmup": args.warmup, "higher_is_better": True, "dtype": "f32",
                      "data": "synthetic",
                      "config": {"workload": f"{c['name']}: m={w['m']} n={n} d={w['d']} q={q} trees={c['trees']} "
                                             f"depth={c['depth']} beta_t={beta:.4f} (t={w['m'] // q})",
                                 "front_size": n_front, "picks": b.idx.cpu().tolist(), "kernel_ms": parts}}),
          flush=True)


def bench_suggest(args):
    """One SUGGEST of Algorithm 1 on the workload's observations (every draw,
    crashed ones included), the pool as large as the workload's, k = its q.
    Wall time per call (host steps included) with the likelihood search on the
    device (the default) and, for comparison, on the host; and the parts timed
    on their own: hyperparameter search per objective (device and host, one
    at a time and side by side), forest training, pool generation."""
    import numpy as np
    import torch

    import paper_2408_04323_amd as S
    from workloads import make_workload
    from workloads.synth import CONFIGS, levels, sobol_table, space_constraints

    c = CONFIGS[args.config]
    w = make_workload(args.config, with_forest=False)
    d, p, n, k = w["d"], w["p"], len(w["Xc"]), w["q"]
    X_obs, valid = w["X_draws"], w["feasible_draws"].astype(np.uint8)
    Y_obs = np.zeros((len(X_obs), p))
    Y_obs[valid != 0] = w["Y"]
    poly, vinit = sobol_table(d)
    A, b = space_constraints(c)
    space = dict(levels=levels(c), poly=poly, vinit=vinit, A=A, b=b)
    kw = dict(k=k, delta=w["delta"], pool_size=n, n_trees=c["trees"], max_depth=c["depth"], t=max(1, w["m"] // k))

    def call(host_search=False):
        out = S.suggest(X_obs, Y_obs, valid, space, host_search=host_search, **kw)
        torch.cuda.synchronize()
        return out

    for _ in range(args.warmup):
        x, src, theta = call()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        x, src, theta = call()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    call(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        x_h, src_h, theta_h = call(True)
    ms_host = (time.perf_counter() - t0) / args.steps * 1e3

    parts = {}
    ok = valid != 0
    Ys = (Y_obs[ok] - Y_obs[ok].mean(0)) / Y_obs[ok].std(0)
    lo = np.log(np.array([0.01] * d + [0.05, 1e-6]))
    hi = np.log(np.array([10.0] * d + [20.0, 1.0]))
    th0 = np.log(np.array([0.5] * d + [1.0, 1e-3]))
    # the searches alone, one objective at a time and side by side on threads
    # (as the step runs them; on the device each with a stream of its own)
    import threading
    streams = [torch.cuda.Stream() for _ in range(p)]
    for name, fn in (("device", lambda j: S.gp_mle_device(X_obs[ok], Ys[:, j], th0, lo, hi, stream=streams[j].cuda_stream)),
                     ("host", lambda j: S.gp_mle(X_obs[ok], Ys[:, j], th0, lo, hi))):
        # the median of three runs of each (a single run also carries one-off
        # costs such as the first pinned allocations of two threads at once)
        iters, one = [], []
        for j in range(p):
            runs = []
            for _ in range(3):
                t0 = time.perf_counter()
                it = fn(j)[2]
                runs.append((time.perf_counter() - t0) * 1e3)
            iters.append(it)
            one.append(sorted(runs)[1])
        parts[f"mle_{name}_each_objective_alone"] = one
        parts[f"mle_{name}_iterations"] = iters
        runs = []
        for _ in range(3):
            threads = [threading.Thread(target=fn, args=(j,)) for j in range(p)]
            t0 = time.perf_counter()
            for t in threads:
                t.start()
            for t in threads:
                t.join()
            runs.append((time.perf_counter() - t0) * 1e3)
        parts[f"mle_{name}_objectives_side_by_side"] = sorted(runs)[1]
        parts[f"mle_{name}_objectives_side_by_side_runs"] = runs
    t0 = time.perf_counter()
    S.forest_train_create(X_obs, valid.astype(np.float64), c["trees"], c["depth"], seed=0)
    parts["forest_train"] = (time.perf_counter() - t0) * 1e3
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    S.sobol_pool(poly, vinit, levels(c), n, A=A, b=b)
    e0.record(stream)
    for _ in range(10):
        S.sobol_pool(poly, vinit, levels(c), n, A=A, b=b)
    e1.record(stream)
    torch.cuda.synchronize()
    parts["sobol_pool"] = e0.elapsed_time(e1) / 10
    print(json.dumps({"metric": "suggestions (whole SUGGEST step) per second", "value": 1e3 / ms,
                      "unit": "suggestions/s", "ms_per_step": ms, "n_gpus": 1, "steps": args.steps,
                      "warmup": args.warmup, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": f"{c['name']}: {len(X_obs)} observations ({int(ok.sum())} valid) "
                                             f"d={d} p={p} pool={n} k={k} trees={c['trees']} depth={c['depth']}",
                                 "ms_per_step_host_search": ms_host, "parts_ms": parts,
                                 "sources": src.tolist(), "sources_host_search": src_h.tolist(),
                                 "picks_match_host_search": bool(np.array_equal(np.asarray(x), np.asarray(x_h))),
                                 "theta_max_abs_diff_vs_host_search": float(np.max(np.abs(np.asarray(theta) -
                                                                                         np.asarray(theta_h))))}}),
          flush=True)


def cpu_baseline(w, seconds):
    """The oracle as it stands, timed on a bounded sample of the same pool."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle.acquisition import expected_improvement
    from oracle.forest import feasibility_mask, forest_votes
    from oracle.gp import gp_fit, gp_posterior
    from oracle.hypervolume import ehvi, nondominated
    from oracle.select import top_q

    p = w["p"]
    warps = w.get("warp")
    fits = [gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                   w["prior_mean"][j], kernel=w.get("kernel", "matern52"),
                   warp=None if warps is None else (warps[0][j], warps[1][j])) for j in range(p)]
    front = nondominated(w["Y"], w["ref"]) if p > 1 else None
    T = len(w["forest"]["tree_offset"]) - 1
    chunk = 8192
    done = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds and done < len(w["Xc"]):
        Xs = w["Xc"][done:done + chunk]
        X64 = Xs.astype(np.float64)
        mu = np.empty((len(Xs), p))
        sd = np.empty((len(Xs), p))
        for j in range(p):
            mu[:, j], sd[:, j] = gp_posterior(fits[j], X64)
        acq = expected_improvement(mu[:, 0], sd[:, 0], w["best_y"], w["xi"]) if p == 1 else \
            ehvi(mu, sd, front, w["ref"])
        mask = feasibility_mask(forest_votes(w["forest"], Xs), w["delta"], T)
        top_q(acq, mask, w["q"])
        done += len(Xs)
    el = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), None)
    except OSError:
        pass
    return {"value": done / el, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "sample": f"first {done} candidates of the same pool in chunks of {chunk}, {el:.1f}s, fit excluded",
            "cpu_model": model, "os_cpu_count": os.cpu_count(),
            "threads_note": "cores = the BLAS thread count the oracle's triangular solves ran on; the rest of "
                            "the oracle is single-threaded NumPy"}


if __name__ == "__main__":
    main()
