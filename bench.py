"""Benchmark of the TAOT per-step planner on one MI355X.

A step is one pass of the whole hot path over all B problems of a workload:
taot_plan_loads (histogram + marginals) -> taot_sinkhorn_batched (Phase 1) ->
taot_round_schedule (Phases 2 and 3).  Inputs (routing ids, home map, costs,
topology preferences) are generated on the device before the timed region
and stay resident in HBM; outputs and workspaces are preallocated.

Printed: one JSON line.  `value` is the batched Sinkhorn throughput in
problem-iterations per second (B * iters / Sinkhorn time per step, HIP
events on the launch stream); `ms_per_step` is the full planner latency.
The default workload is the R = 256 one (1952 problems of 256 ranks).
"""
import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0                      # MI355X HBM3E
VALU_FMA_PEAK = 256 * 64 * 2.4e9           # fp32 FMA lanes/s without packed math (CU x lanes x clock)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--K", type=int, default=None, help="guest slots per rank (default: the workload's)")
    ap.add_argument("--cpu-sample", type=int, default=32, help="problems in the oracle CPU baseline (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="oracle Sinkhorn passes over the sample repeat until this much time has passed")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (HBM counter calibration)")
    ap.add_argument("--other-steps", type=int, default=3,
                    help="timed steps for the planner latency of workloads 1-4 other than --workload (0: skip)")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--report", default=None, metavar="P1,P2,...",
                    help="plan --workload once and print the planner's four-part report for these "
                         "problems (layers) instead of benchmarking")
    ap.add_argument("--report-file", default=None, help="write the --report text here instead of stdout")
    ap.add_argument("--quality", action="store_true",
                    help="print the plan-quality table of the Phase-2 score ablations on --workload "
                         "(every problem of the batch, no timing) instead of benchmarking")
    ap.add_argument("--hot-rank", action="store_true",
                    help="sweep the hot-rank workloads of the paper's scalability study (EP degree, hot "
                         "fraction, guest slots): plan quality and planner latency per point, instead of "
                         "benchmarking --workload")
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


PLAN_LOADS_SOURCES = ["paper_2608_03676_amd/csrc/loads.hip", "paper_2608_03676_amd/csrc/common.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "plan_loads_workload3_traffic.txt")


def sources_digest(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per plan_loads step from the committed counter summary, or
    None when it is for another workload or the kernels changed since."""
    if workload != 3 or not os.path.exists(TRAFFIC_FILE):
        return None
    fields = {}
    with open(TRAFFIC_FILE) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != sources_digest(PLAN_LOADS_SOURCES):
        return None
    try:
        return float(fields["traffic_bytes_per_step"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib):
    import torch
    n = mib * 2**20 // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4,
                      "launches": 5}), flush=True)


def run_workload(w, K, steps, warmup, dev):
    """Device-generated inputs, preallocated outputs, `warmup` untimed steps,
    then `steps` timed steps (HIP events on the launch stream)."""
    import torch

    import paper_2608_03676_amd as taot
    import workloads as W
    B, R, E, N = w.B, w.R, w.E, w.N
    t0 = time.time()
    ids = W.workload_ids_device(w, dev)
    home_np = W.home_map(w)
    C_np = W.cost_matrix(w)
    Bp_np, Ba_np = taot.topology_pref(C_np)
    home = torch.from_numpy(home_np).to(dev)
    C = torch.from_numpy(C_np).to(dev)
    Bp = torch.from_numpy(Bp_np).to(dev)
    Ba = torch.from_numpy(Ba_np).to(dev)
    torch.cuda.synchronize()
    log(f"[bench] generated {ids.numel() / 1e9:.2f} G ids ({ids.numel() * 4 / 2**30:.1f} GiB) in {time.time() - t0:.1f}s")

    # preallocated outputs and workspaces
    ws = taot.workspace_bytes(B, R, E, K)
    wl = torch.empty(max(ws["plan_loads"], 1), dtype=torch.uint8, device=dev)
    wsk = torch.empty(max(ws["sinkhorn"], 1), dtype=torch.uint8, device=dev)
    wsc = torch.empty(max(ws["round_schedule"], 1), dtype=torch.uint8, device=dev)
    loads = taot.plan_loads(ids, home, E, workspace=wl)
    flow = taot.sinkhorn_batched(loads.supply, loads.demand, C, w.eps, w.iters, workspace=wsk)
    sched = taot.round_schedule(loads.n, loads.spill, loads.spare, loads.excess, loads.alpha, home, flow.T,
                                Bp, Ba, K, w.price_step, 0, workspace=wsc)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        taot.plan_loads(ids, home, E, out=loads, workspace=wl)
        if ev is not None:
            ev[1].record(stream)
        taot.sinkhorn_batched(loads.supply, loads.demand, C, w.eps, w.iters, out=flow, workspace=wsk)
        if ev is not None:
            ev[2].record(stream)
        taot.round_schedule(loads.n, loads.spill, loads.spare, loads.excess, loads.alpha, home, flow.T, Bp, Ba,
                            K, w.price_step, 0, out=sched, workspace=wsc)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup {warmup} done")
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(steps):
        step(events[s])
    end.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / steps
    loads_ms = [e[0].elapsed_time(e[1]) for e in events]
    sk_ms = [e[1].elapsed_time(e[2]) for e in events]
    sch_ms = [e[2].elapsed_time(e[3]) for e in events]
    log(f"[bench] {steps} steps: {ms_step:.3f} ms/step (plan_loads {statistics.mean(loads_ms):.3f}, "
        f"sinkhorn {statistics.mean(sk_ms):.3f}, round_schedule {statistics.mean(sch_ms):.3f} ms)")
    del ids
    return dict(loads=loads, flow=flow, sched=sched, home_np=home_np, C_np=C_np, Bp_np=Bp_np, Ba_np=Ba_np,
                loads_ms=loads_ms, sk_ms=sk_ms, sch_ms=sch_ms, ms_step=ms_step)


def plan_quality_table(w, K, dev):
    """Plan quality of the full score, of its ablations and of row-priority
    matching (round_schedule flags) on one batch: rho before and after the planned moves, replicas
    inside / across nodes (node = rank // 8) and the weighted cost intra +
    3 inter, mean and standard deviation over the batch's problems."""
    import torch

    import paper_2608_03676_amd as taot
    import workloads as W
    B, R, E, N = w.B, w.R, w.E, w.N
    ids = W.workload_ids_device(w, dev)
    home = torch.from_numpy(W.home_map(w)).to(dev)
    C_np = W.cost_matrix(w)
    Bp_np, Ba_np = taot.topology_pref(C_np)
    C, Bp, Ba = (torch.from_numpy(x).to(dev) for x in (C_np, Bp_np, Ba_np))
    loads = taot.plan_loads(ids, home, E)
    flow = taot.sinkhorn_batched(loads.supply, loads.demand, C, w.eps, w.iters)
    del ids
    rho0 = loads.rho.cpu().numpy()
    rows = []
    for name, flags in (("full score", 0), ("no topology term", taot.SCH_NO_TOPO),
                        ("no flow-hint term", taot.SCH_NO_FLOW),
                        ("spill/spare only", taot.SCH_NO_TOPO | taot.SCH_NO_FLOW),
                        ("row priority", taot.SCH_ROW_PRIORITY)):
        sched = taot.round_schedule(loads.n, loads.spill, loads.spare, loads.excess, loads.alpha, home, flow.T,
                                    Bp, Ba, K, w.price_step, 0, flags=flags)
        q = taot.plan_quality(loads.load_r, home, sched, K, ranks_per_node=8, w_inter=3.0)
        torch.cuda.synchronize()
        ra, ni, no, wt = (x.cpu().numpy().astype(float) for x in (q.rho_after, q.intra, q.inter, q.weighted))
        rows.append(dict(variant=name, flags=flags, rho_before=[rho0.mean(), rho0.std()],
                         rho_after=[ra.mean(), ra.std()], intra=[ni.mean(), ni.std()], inter=[no.mean(), no.std()],
                         weighted=[wt.mean(), wt.std()], unfilled=int(sched.unfilled.sum().item())))
    print(f"plan quality, workload {w.index}: {B} problems, R = {R}, K = {K} (mean +- std over problems)")
    print(f"{'variant':<20} {'rho before':>16} {'rho after':>16} {'intra':>14} {'inter':>14} {'intra+3inter':>16} unfilled")
    for r in rows:
        f = lambda v, d=4: f"{v[0]:.{d}f} +- {v[1]:.{d}f}"
        print(f"{r['variant']:<20} {f(r['rho_before']):>16} {f(r['rho_after']):>16} {f(r['intra'], 1):>14} "
              f"{f(r['inter'], 1):>14} {f(r['weighted'], 1):>16} {r['unfilled']}")
    print(json.dumps({"plan_quality": rows, "workload": w.index, "K": K}), flush=True)


HOT_RANK_PANELS = (
    ("EP degree (hot fraction 0.5, K = 2)", [(ep, 0.5, 2) for ep in (4, 8, 16, 32)]),
    ("hot fraction (EP16, K = 2)", [(16, f, 2) for f in (0.3, 0.5, 0.7, 0.9)]),
    ("guest slots per rank (EP16, hot fraction 0.5)", [(16, 0.5, K) for K in (1, 2, 4, 8, 16)]),
)


def hot_rank_sweep(dev, steps, warmup):
    """The three sweeps of the paper's scalability study (Sec. 4.4) on the
    hot-rank workloads, 48 problems per point: the hottest rank's share of
    the load, rho before and after the planned moves, replicas inside and
    across nodes and the weighted cost intra + 3 inter for the full score,
    the weighted cost and rho after without the topology term, rho after
    with row-priority matching, and the planner latency per step (all 48
    problems) from HIP events."""
    import torch

    import paper_2608_03676_amd as taot
    import workloads as W
    out = []
    for title, points in HOT_RANK_PANELS:
        rows = []
        for ep, frac, K in points:
            w = W.llep_workload(ep, frac, K)
            log(f"[hot rank] EP{ep} frac {frac} K={K}")
            run = run_workload(w, K, steps, warmup, dev)
            L, F = run["loads"], run["flow"]
            home = torch.from_numpy(run["home_np"]).to(dev)
            Bp, Ba = (torch.from_numpy(run[x]).to(dev) for x in ("Bp_np", "Ba_np"))
            load = L.load_r.double()
            share = (load.max(1).values / load.sum(1)).cpu().numpy()
            res = dict(ep=ep, frac=frac, K=K, hot_share=float(share.mean()),
                       rho_before=float(L.rho.mean()), ms_per_step=run["ms_step"],
                       us_per_problem=1e3 * run["ms_step"] / w.B)
            for tag, flags in (("", 0), ("_no_topo", taot.SCH_NO_TOPO), ("_row", taot.SCH_ROW_PRIORITY)):
                s = taot.round_schedule(L.n, L.spill, L.spare, L.excess, L.alpha, home, F.T, Bp, Ba, K,
                                        w.price_step, 0, flags=flags)
                q = taot.plan_quality(L.load_r, home, s, K, ranks_per_node=8, w_inter=3.0)
                res["rho_after" + tag] = float(q.rho_after.mean())
                res["intra" + tag] = float(q.intra.double().mean())
                res["inter" + tag] = float(q.inter.double().mean())
                res["weighted" + tag] = float(q.weighted.mean())
                res["unfilled" + tag] = int(s.unfilled.sum())
            rows.append(res)
            del run
            torch.cuda.empty_cache()
        out.append(dict(panel=title, rows=rows))
        print(f"hot-rank sweep, {title}: 48 problems per point, means over the problems")
        print(f"{'EP':>4} {'frac':>5} {'K':>3} {'hot share':>9} {'rho before':>10} {'rho after':>9} {'intra':>6} "
              f"{'inter':>6} {'weighted':>8} | {'no topology: rho after':>22} {'weighted':>8} | "
              f"{'row priority: rho after':>23} | {'planner ms':>10} {'us/problem':>10}")
        for r in rows:
            print(f"{r['ep']:>4} {r['frac']:>5.1f} {r['K']:>3} {r['hot_share']:>9.4f} {r['rho_before']:>10.4f} "
                  f"{r['rho_after']:>9.4f} {r['intra']:>6.1f} {r['inter']:>6.1f} {r['weighted']:>8.1f} | "
                  f"{r['rho_after_no_topo']:>22.4f} {r['weighted_no_topo']:>8.1f} | {r['rho_after_row']:>23.4f} | "
                  f"{r['ms_per_step']:>10.3f} {r['us_per_problem']:>10.1f}")
        print(flush=True)
    print(json.dumps({"hot_rank_sweep": out}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: the planner's problems are independent and "
              f"the library has no multi-GPU path (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2608_03676_amd as taot
    import workloads as W

    dev = torch.device("cuda:0")
    if args.hot_rank:
        hot_rank_sweep(dev, args.steps, args.warmup)
        return
    w = W.WORKLOADS[args.workload]
    K = w.K if args.K is None else args.K
    B, R, E, N = w.B, w.R, w.E, w.N
    if args.quality:
        plan_quality_table(w, K, dev)
        return
    if args.report is not None:
        ids = W.workload_ids_device(w, dev)
        home = torch.from_numpy(W.home_map(w)).to(dev)
        plan = taot.plan_step(ids, home, torch.from_numpy(W.cost_matrix(w)).to(dev), E, w.eps, w.iters, K,
                              price_step=w.price_step)
        torch.cuda.synchronize()
        text = taot.plan_report(plan, home, K, problems=[int(x) for x in args.report.split(",") if x.strip()])
        if args.report_file:
            with open(args.report_file, "w") as fh:
                fh.write(text)
        else:
            sys.stdout.write(text)
        return
    log(f"[bench] workload {w.index}: {w.name}; B={B} R={R} E={E} N={N} iters={w.iters} K={K}")
    run = run_workload(w, K, args.steps, args.warmup, dev)
    loads, flow, sched = run["loads"], run["flow"], run["sched"]
    home_np, C_np, Bp_np, Ba_np = run["home_np"], run["C_np"], run["Bp_np"], run["Ba_np"]
    loads_ms, sk_ms, sch_ms, ms_step = run["loads_ms"], run["sk_ms"], run["sch_ms"], run["ms_step"]

    # ---- algorithmic work of each stage --------------------------------------------
    st_loads = loads.status.cpu().numpy().view(np.uint32)
    st_flow = flow.status.cpu().numpy().view(np.uint32)
    st_sched = sched.status.cpu().numpy().view(np.uint32)
    excess = loads.excess.cpu().numpy()
    spare = loads.spare.cpu().numpy()
    nh = (excess > 0).sum(1).astype(np.int64)
    nc = (spare > 0).sum(1).astype(np.int64)
    support = int((nh * nc).sum())
    rounds = sched.rounds_used.cpu().numpy()
    unfilled = int(sched.unfilled.sum().item())
    # plan_loads bytes: ids read once, n written once and read once by the marginals
    loads_bytes = 4 * B * R * N + 2 * 4 * B * R * E
    sk_fma = 2 * support * w.iters              # one FMA per support entry per half-step
    mean = lambda xs: statistics.mean(xs)
    stage = {
        "plan_loads": {"bound": "hbm", "ms": mean(loads_ms), "achieved": loads_bytes / (mean(loads_ms) * 1e-3) / 1e9,
                       "peak": HBM_PEAK_GBS, "unit": "GB/s", "bytes_per_launch": loads_bytes},
        "sinkhorn": {"bound": "alu", "ms": mean(sk_ms), "achieved": 2 * sk_fma / (mean(sk_ms) * 1e-3) / 1e12,
                     "peak": 2 * VALU_FMA_PEAK / 1e12, "unit": "TFLOP/s", "fma_per_launch": sk_fma,
                     "support_entries": support},
        "round_schedule": {"bound": "latency", "ms": mean(sch_ms), "phase2_inner_mean": float(rounds[:, 0].mean()),
                           "phase3_rounds_mean": float(rounds[:, 1].mean()), "phase3_rounds_max": int(rounds[:, 1].max())},
    }
    for s in stage.values():
        if "peak" in s:
            s["frac"] = s["achieved"] / s["peak"]
    # roofline of the longest stage that has one (the schedule is a chain of
    # dependent rounds: latency, not bandwidth or ALU, bounds it)
    dom_name = max(("plan_loads", "sinkhorn"), key=lambda k: stage[k]["ms"])
    dom = stage[dom_name]
    kernels = {"plan_loads": "histogram_kernel + marginals_kernel (taot_plan_loads)",
               "sinkhorn": "sinkhorn_wave_kernel (taot_sinkhorn_batched)"}
    traffic = measured_traffic(w.index) if dom_name == "plan_loads" else None
    roofline = {"kernel": kernels[dom_name], "bound": dom["bound"], "achieved": dom["achieved"],
                "peak": dom["peak"], "unit": dom["unit"], "frac": dom["frac"], "traffic": traffic}

    value = B * w.iters / (mean(sk_ms) * 1e-3)
    rec = {
        "metric": "batched Sinkhorn problem-iters/s at R=256 + full planner latency (us)/step",
        "value": value, "unit": "problem-iters/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step, "planner_latency_us": ms_step * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (Sinkhorn), int32/int64 (histogram, schedule), f64 (scores)",
        "data": "synthetic (seeded Zipf top-8 routing generated on device)",
        "config": {"workload": f"workload {w.index}: {w.name}", "problems": B, "ranks": R, "experts": E,
                   "ids_per_problem": R * N, "iters": w.iters, "eps": w.eps, "K": K},
        "roofline": roofline,
        "stages": stage,
        "status": {"loads_nonzero": int((st_loads != 0).sum()), "sinkhorn_nonzero": int((st_flow != 0).sum()),
                   "schedule_unfilled": unfilled, "schedule_nonzero": int((st_sched != 0).sum())},
    }

    # ---- planner latency of the other full-size workloads (fewer steps) -------------
    if args.other_steps > 0:
        lat = {str(w.index): {"problems": B, "ranks": R, "ms_per_step": ms_step, "plan_loads_ms": mean(loads_ms),
                              "sinkhorn_ms": mean(sk_ms), "round_schedule_ms": mean(sch_ms)}}
        del run, loads, flow, sched
        torch.cuda.empty_cache()
        for wi in (1, 2, 3, 4):
            if wi == w.index:
                continue
            wo = W.WORKLOADS[wi]
            log(f"[bench] planner latency, workload {wi}: {wo.name}")
            r2 = run_workload(wo, wo.K, args.other_steps, 1, dev)
            lat[str(wi)] = {"problems": wo.B, "ranks": wo.R, "ms_per_step": r2["ms_step"],
                            "plan_loads_ms": mean(r2["loads_ms"]), "sinkhorn_ms": mean(r2["sk_ms"]),
                            "round_schedule_ms": mean(r2["sch_ms"]),
                            "unfilled": int(r2["sched"].unfilled.sum().item())}
            del r2
            torch.cuda.empty_cache()
        rec["planner_latency_by_workload"] = dict(sorted(lat.items()))

    # ---- CPU baseline: the oracle on a bounded sample of the same workload ----------
    if args.cpu_sample > 0:
        rec["cpu_baseline"] = cpu_baseline(w, K, args, home_np, C_np, Bp_np, Ba_np)
    line = json.dumps(rec)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as fh:
            fh.write(line + "\n")


def cpu_baseline(w, K, args, home_np, C_np, Bp_np, Ba_np):
    """The oracle, as it is, on a sample of the workload's problems: ids made
    on the host, plan_loads, then Sinkhorn passes over the sample until
    --cpu-seconds have passed, then Phases 2-3 once."""
    import numpy as np

    import oracle as O
    import workloads as W
    B = w.B
    stride = max(1, B // args.cpu_sample)
    sample = list(range(0, B, stride))[: args.cpu_sample]
    threads = O.max_threads()
    t = time.time()
    parts = []
    for b in sample:  # one problem of ids at a time (OpenMP over ranks; the buffer is reused)
        ids = W.problem_ids_host(w, b)[None]
        parts.append(O.plan_loads(ids, home_np, w.E))
        del ids
    t_gen_loads = time.time() - t
    cat = lambda f: np.concatenate([getattr(x, f) for x in parts])
    excess, spare, spill, alpha, n = cat("excess"), cat("spare"), cat("spill"), cat("alpha"), cat("n")
    a, b, Cd = excess.astype(float), spare.astype(float), C_np.astype(float)
    passes, t_sk = 0, 0.0
    while t_sk < args.cpu_seconds or passes == 0:
        t = time.time()
        Po = O.sinkhorn(a, b, Cd, w.eps, w.iters)
        t_sk += time.time() - t
        passes += 1
    t = time.time()
    se, sa, _ = O.phase2(spill, spare, excess, alpha, home_np, Po.T.astype(np.float32), Bp_np, K)
    O.phase3(n, se, sa, Ba_np, K, w.price_step)
    t_sch = time.time() - t
    used = min(threads, len(sample))
    log(f"[bench] oracle on {len(sample)} problems, {used} threads: ids + plan_loads {t_gen_loads:.1f}s, "
        f"sinkhorn {passes} passes {t_sk:.1f}s, schedule {t_sch:.1f}s")
    return {
        "value": passes * len(sample) * w.iters / t_sk, "unit": "problem-iters/s", "cores": used, "kind": "oracle",
        "sample": f"{len(sample)} of {B} problems (every {stride}th), ids generated on the host; fp64 C oracle "
                  f"Sinkhorn at the full iteration count, {passes} passes over the sample ({t_sk:.1f} s), "
                  f"OpenMP over problems",
        "schedule_s_per_problem": t_sch / len(sample),
    }


if __name__ == "__main__":
    main()
