"""Benchmark of the TAOT per-step planner on one MI355X.

A step is one pass of the whole hot path over all B problems of a workload:
taot_plan_loads (histogram + marginals) -> taot_sinkhorn_batched (Phase 1) ->
taot_round_schedule (Phases 2 and 3).  Inputs (routing ids, home map, costs,
topology preferences) are generated on the device before the timed region
and stay resident in HBM; outputs and workspaces are preallocated.

Printed: one JSON line.  `value` is the batched Sinkhorn throughput in
problem-iterations per second (B * iters / median Sinkhorn call time, HIP
events on the launch stream); `ms_per_step` is the full planner latency.
The default workload is the R = 256 one (1952 problems of 256 ranks); the
planner latency of the other full-size workloads (1, 2, 4) follows, every
stage with its roofline floor and fraction, beside the peak probes (HBM
read, unpacked fp32 FMA, v_exp_f32, LDS read) measured in the same run and
the fp64 oracle timed on the host.
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

HBM_PEAK_GBS = 8000.0                      # MI355X HBM3E (datasheet)
VALU_FMA_PEAK = 256 * 64 * 2.4e9           # fp32 FMA lanes/s without packed math (CU x lanes x clock)
FP32_PUBLISHED_TFLOPS = 157.3              # datasheet fp32 vector peak (needs packed fp32, not used here)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--K", type=int, default=None, help="guest slots per rank (default: the workload's)")
    ap.add_argument("--cpu-sample", type=int, default=32, help="problems in the oracle CPU baseline (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="oracle Sinkhorn passes over the sample repeat until this much time has passed")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (HBM counter calibration)")
    ap.add_argument("--other-steps", type=int, default=10,
                    help="timed steps for the planner latency of workloads 1-4 other than --workload, after "
                         "--warmup untimed ones (0: skip)")
    ap.add_argument("--dense-steps", type=int, default=3,
                    help="timed calls of the dense streamed Sinkhorn (TAOT_SK_DENSE) at the workload-4 shape "
                         "with one cost matrix per problem (0: skip)")
    ap.add_argument("--dense-only", action="store_true", help="only run the dense streamed leg and print it")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--no-peaks", action="store_true", help="skip the peak probes")
    ap.add_argument("--peaks-only", action="store_true", help="only run the peak probes and print them")
    ap.add_argument("--cpu-extrapolate", type=int, default=1,
                    help="time the oracle on one problem of each workload 1-4 and extrapolate its full-step "
                         "latency (0: skip)")
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


# Counter-measured HBM traffic of a stage's kernels, from the committed
# rocprofv3 summaries; used only while the sources they were taken on are
# unchanged (SHA-256 recorded in each summary).
TRAFFIC = {
    "plan_loads": (os.path.join(ROOT, "profiles", "plan_loads_workload3_traffic.txt"), 3,
                   ["paper_2608_03676_amd/csrc/loads.hip", "paper_2608_03676_amd/csrc/common.h"]),
    "sinkhorn": (os.path.join(ROOT, "profiles", "sinkhorn_workload3_traffic.txt"), 3,
                 ["paper_2608_03676_amd/csrc/sinkhorn.hip", "paper_2608_03676_amd/csrc/sk_common.h",
                  "paper_2608_03676_amd/csrc/sk_register.h", "paper_2608_03676_amd/csrc/sk_reg_w2g8.hip",
                  "paper_2608_03676_amd/csrc/common.h"]),
    "dense": (os.path.join(ROOT, "profiles", "sinkhorn_dense_row_workload4_traffic.txt"), 4,
              ["paper_2608_03676_amd/csrc/sk_dense.hip", "paper_2608_03676_amd/csrc/sk_common.h",
               "paper_2608_03676_amd/csrc/common.h"]),
}


def sources_digest(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(stage, workload):
    """HBM bytes per call of a stage from its committed counter summary, or
    None when it is for another workload or the kernels changed since."""
    if stage not in TRAFFIC or workload != TRAFFIC[stage][1]:
        return None
    path, _, sources = TRAFFIC[stage]
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != sources_digest(sources):
        return None
    try:
        return float(fields["traffic_bytes_per_step"])
    except (KeyError, ValueError):
        return None


def gpu_clocks():
    """The GPUs' current shader and memory clock levels and power as the
    amdgpu driver exposes them in sysfs (best effort, read without starting
    another program; None when nothing is readable)."""
    import glob
    out = {}
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        rec = {}
        for name in ("pp_dpm_sclk", "pp_dpm_mclk"):
            try:
                with open(os.path.join(dev, name)) as fh:
                    cur = [l.strip() for l in fh if l.strip().endswith("*")]
                rec[name] = cur[0] if cur else None
            except OSError:
                pass
        for pw in glob.glob(os.path.join(dev, "hwmon", "hwmon*", "power1_*")):
            if pw.endswith(("_average", "_input")):
                try:
                    with open(pw) as fh:
                        rec["power_W"] = int(fh.read().strip()) / 1e6
                except (OSError, ValueError):
                    pass
        if rec:
            out[os.path.basename(os.path.dirname(dev))] = rec
    return out or None


def measure_peaks(dev):
    """Peak probes P1-P4 (libtaot_probes.so), HIP events on the launch stream,
    best of 5 launches after one warm-up: HBM read GB/s, unpacked fp32 FMA/s,
    v_exp_f32/s alone and beside as many FMAs, LDS read bytes/s."""
    import torch
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2608_03676_amd", "libtaot_probes.so"))
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    L.taot_probe_hbm_read.argtypes = [P, SZ, I32, P, P]
    L.taot_probe_fma.argtypes = [I32, I32, P, P]
    L.taot_probe_exp.argtypes = [I32, I32, I32, P, P]
    L.taot_probe_lds.argtypes = [I32, I32, P, P]
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    blocks = 2048  # eight 256-thread workgroups per compute unit
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)

    def best(call):
        call()
        ts = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rc = call()
            b.record(stream)
            torch.cuda.synchronize()
            if rc != 0:
                raise RuntimeError("peak probe launch failed")
            ts.append(a.elapsed_time(b) * 1e-3)
        return min(ts)

    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    t_hbm = best(lambda: L.taot_probe_hbm_read(ctypes.c_void_p(buf.data_ptr()), nbytes, 16384,
                                               ctypes.c_void_p(out.data_ptr()), sp))
    del buf
    it_fma, it_exp, it_lds = 20000, 5000, 20000
    lanes = blocks * 256
    t_fma = best(lambda: L.taot_probe_fma(blocks, it_fma, ctypes.c_void_p(out.data_ptr()), sp))
    t_exp = best(lambda: L.taot_probe_exp(blocks, it_exp, 0, ctypes.c_void_p(out.data_ptr()), sp))
    t_expf = best(lambda: L.taot_probe_exp(blocks, it_exp, 1, ctypes.c_void_p(out.data_ptr()), sp))
    t_lds = best(lambda: L.taot_probe_lds(blocks, it_lds, ctypes.c_void_p(out.data_ptr()), sp))
    fma = lanes * 64.0 * it_fma / t_fma
    exps = lanes * 64.0 * it_exp / t_exp
    exps_f = lanes * 64.0 * it_exp / t_expf
    return {
        "hbm_read_GBs": nbytes / t_hbm / 1e9,
        "fp32_fma_per_s": fma, "fp32_tflops_unpacked": 2 * fma / 1e12,
        "exp_per_s": exps, "exp_to_fma_rate": exps / fma,
        # exp and FMA issued together take 1.5x the exponentials' time when
        # they do not overlap (an exponential occupies two FMA issue slots)
        "exp_with_fma_per_s": exps_f, "exp_plus_fma_time_ratio": t_expf / t_exp,
        "lds_read_Bps": lanes * 8.0 * 16 * it_lds / t_lds,
        "datasheet": {"hbm_GBs": HBM_PEAK_GBS, "fp32_fma_per_s_unpacked": VALU_FMA_PEAK,
                      "fp32_tflops_published": FP32_PUBLISHED_TFLOPS,
                      "lds_Bps_128B_per_clk": 256 * 128 * 2.4e9},
    }


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
    step_ms = [e[0].elapsed_time(e[3]) for e in events]
    log(f"[bench] {steps} steps: {ms_step:.3f} ms/step, median {statistics.median(step_ms):.3f} "
        f"(plan_loads {statistics.median(loads_ms):.3f}, sinkhorn {statistics.median(sk_ms):.3f}, "
        f"round_schedule {statistics.median(sch_ms):.3f} ms, medians)")
    del ids
    return dict(loads=loads, flow=flow, sched=sched, home_np=home_np, C_np=C_np, Bp_np=Bp_np, Ba_np=Ba_np,
                loads_ms=loads_ms, sk_ms=sk_ms, sch_ms=sch_ms, step_ms=step_ms, ms_step=ms_step)


def dense_streamed(dev, steps, warmup):
    """The dense streamed Sinkhorn (TAOT_SK_DENSE: every R x R entry, no
    support compaction) at the workload-4 shape with one cost matrix per
    problem (the fat-tree costs scaled by 1 + 0.01 (b mod 7)), the workload's
    eps and iteration count, marginals from its routing.  HIP events on the
    launch stream around each call.  The row pass reads the stored K~ once
    per iteration (B R^2 fp32) and forms both half-steps' sums from it; the
    floors are that single sweep at 8 TB/s and, for context, the two sweeps
    over C per iteration of the GEMV form (one per half-step)."""
    import numpy as np
    import torch

    import paper_2608_03676_amd as taot
    import workloads as W
    w = W.WORKLOADS[4]
    B, R = w.B, w.R
    ids = W.workload_ids_device(w, dev)
    home = torch.from_numpy(W.home_map(w)).to(dev)
    L = taot.plan_loads(ids, home, w.E)
    del ids
    torch.cuda.empty_cache()
    C0 = torch.from_numpy(W.cost_matrix(w)).to(dev)
    C = torch.stack([C0 * (1.0 + 0.01 * (b % 7)) for b in range(B)]).contiguous()
    wsk = torch.empty(taot.workspace_bytes(B, R, w.E, w.K)["sinkhorn"], dtype=torch.uint8, device=dev)
    out = taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters, taot.SK_DENSE, workspace=wsk)
    for _ in range(warmup):
        taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters, taot.SK_DENSE, out=out, workspace=wsk)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ms = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        taot.sinkhorn_batched(L.supply, L.demand, C, w.eps, w.iters, taot.SK_DENSE, out=out, workspace=wsk)
        e1.record(stream)
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    st = out.status.cpu().numpy().view(np.uint32)
    finite = bool(torch.isfinite(out.T).all().item())
    med = statistics.median(ms)
    per_iter = 4 * B * R * R
    floor = per_iter * w.iters / (HBM_PEAK_GBS * 1e9) * 1e3
    achieved = per_iter * w.iters / (med * 1e-3) / 1e9
    traffic = measured_traffic("dense", 4)
    log(f"[bench] dense streamed, workload-4 shape, per-problem C: {med:.2f} ms for {w.iters} iterations "
        f"({med / w.iters * 1e3:.1f} us/iteration, {achieved:.0f} GB/s of K~)")
    return {"workload": f"workload 4 shape ({B} problems x {R} ranks), one cost matrix per problem "
                        f"(fat-tree costs x (1 + 0.01 (b mod 7))), TAOT_SK_DENSE",
            "iters": w.iters, "eps": w.eps, "ms": statistics.mean(ms), "ms_median": med, "ms_min": min(ms),
            "us_per_iteration": med / w.iters * 1e3, "bound": "hbm", "bytes_per_iteration": per_iter,
            "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "floor_ms": floor, "frac_of_floor": floor / med,
            "two_sweep_floor_ms": 2 * floor, "frac_of_two_sweep_floor": 2 * floor / med,
            "traffic_bytes_per_iteration_row_pass": traffic,
            "status_streamed": int((st == taot.ST_STREAMED).sum()), "status_other": int((st != taot.ST_STREAMED).sum()),
            "plan_finite": finite}


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
    if args.dense_only:
        print(json.dumps({"dense_streamed": dense_streamed(dev, max(args.dense_steps, 1), args.warmup)}), flush=True)
        return
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
    peaks = None
    if not args.no_peaks or args.peaks_only:
        log("[bench] peak probes")
        peaks = measure_peaks(dev)
        log(f"[bench] peaks: {json.dumps(peaks)}")
        if args.peaks_only:
            print(json.dumps({"peaks_measured": peaks}), flush=True)
            return
    clocks_before = gpu_clocks()
    log(f"[bench] workload {w.index}: {w.name}; B={B} R={R} E={E} N={N} iters={w.iters} K={K}")
    run = run_workload(w, K, args.steps, args.warmup, dev)
    rep = stage_report(w, K, run, peaks)
    st = rep["stages"]
    sk = st["sinkhorn"]
    value = B * w.iters / (sk["ms_median"] * 1e-3)

    # the metric's own kernels: taot_sinkhorn_batched (the register kernel
    # and its prepasses), fp32 FMA issue bound
    roofline = {"kernel": "sinkhorn_reg_kernel<2,8> + prepasses (taot_sinkhorn_batched)", "bound": "alu",
                "achieved": sk["achieved"], "peak": sk["peak"], "unit": "TFLOP/s", "frac": sk["frac"],
                "traffic": measured_traffic("sinkhorn", w.index),
                "peak_note": "unpacked fp32 FMA: 256 CU x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz; the published "
                             "157.3 TFLOP/s needs packed fp32, which this build does not use",
                "frac_vs_published_157_3": sk["achieved"] / FP32_PUBLISHED_TFLOPS}
    if peaks:
        roofline["frac_vs_measured_peak"] = sk["achieved"] / peaks["fp32_tflops_unpacked"]
    rec = {
        "metric": "batched Sinkhorn problem-iters/s at R=256 + full planner latency (us)/step",
        "value": value, "unit": "problem-iters/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": run["ms_step"], "planner_latency_us": run["ms_step"] * 1e3,
        "planner_latency_us_median": rep["planner"]["ms_median"] * 1e3,
        "planner_latency_us_min": rep["planner"]["ms_min"] * 1e3,
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (Sinkhorn), int32/int64 (histogram, schedule), f64 (scores)",
        "data": "synthetic (seeded Zipf top-8 routing generated on device)",
        "config": {"workload": f"workload {w.index}: {w.name}", "problems": B, "ranks": R, "experts": E,
                   "ids_per_problem": R * N, "iters": w.iters, "eps": w.eps, "K": K},
        "roofline": roofline,
        "stages": st,
        "planner": rep["planner"],
        "status": rep["status"],
    }
    if peaks:
        rec["peaks_measured"] = peaks

    # ---- planner latency of the other full-size workloads ---------------------------
    gpu_rounds = {w.index: rep["phase3_rounds_mean"]}
    if args.other_steps > 0:
        lat = {str(w.index): dict(problems=B, ranks=R, **rep["summary"], stages=st, planner=rep["planner"],
                                  status=rep["status"])}
        del run
        torch.cuda.empty_cache()
        for wi in (1, 2, 3, 4):
            if wi == w.index:
                continue
            wo = W.WORKLOADS[wi]
            log(f"[bench] planner latency, workload {wi}: {wo.name}")
            r2 = run_workload(wo, wo.K, args.other_steps, args.warmup, dev)
            rep2 = stage_report(wo, wo.K, r2, peaks)
            lat[str(wi)] = dict(problems=wo.B, ranks=wo.R, **rep2["summary"], stages=rep2["stages"],
                                planner=rep2["planner"], status=rep2["status"])
            gpu_rounds[wi] = rep2["phase3_rounds_mean"]
            del r2
            torch.cuda.empty_cache()
        rec["planner_latency_by_workload"] = dict(sorted(lat.items()))
    if args.dense_steps > 0:
        torch.cuda.empty_cache()
        rec["dense_streamed"] = dense_streamed(dev, args.dense_steps, 1)
        torch.cuda.empty_cache()
    rec["clocks"] = {"before": clocks_before, "after": gpu_clocks()}

    # ---- CPU baseline: the oracle on a bounded sample of the same workload ----------
    if args.cpu_sample > 0:
        rec["cpu_baseline"] = cpu_baseline(w, K, args, run_home(w), W.cost_matrix(w))
        if args.cpu_extrapolate:
            rec["cpu_baseline"]["extrapolated"] = cpu_extrapolate(gpu_rounds, rec["cpu_baseline"]["cores"])
    line = json.dumps(rec)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as fh:
            fh.write(line + "\n")


def run_home(w):
    import workloads as W
    return W.home_map(w)


def stage_report(w, K, run, peaks):
    """Per-stage times (mean, median, min over the timed steps), algorithmic
    work, roofline floors and fractions of one workload's planner step:
    plan_loads against HBM (ids read once, n written and read back once),
    the Sinkhorn against the unpacked fp32 FMA issue rate (one FMA per
    support entry per half-step; the plan's HBM write checked too), the
    schedule against the bytes it must move (X and the slots written, the
    plan on the support and the slot experts' counts read: a latency-bound
    chain of rounds, so this floor is far from reach), and the step against
    the sum of the three floors."""
    import numpy as np
    B, R, E, N = w.B, w.R, w.E, w.N
    loads, flow, sched = run["loads"], run["flow"], run["sched"]
    st_loads = loads.status.cpu().numpy().view(np.uint32)
    st_flow = flow.status.cpu().numpy().view(np.uint32)
    st_sched = sched.status.cpu().numpy().view(np.uint32)
    excess = loads.excess.cpu().numpy()
    spare = loads.spare.cpu().numpy()
    nh = (excess > 0).sum(1).astype(np.int64)
    nc = (spare > 0).sum(1).astype(np.int64)
    support = int((nh * nc).sum())
    rounds = sched.rounds_used.cpu().numpy()
    se = sched.slot_expert.cpu().numpy()
    distinct = sum(len(set(row[row >= 0].tolist())) for row in se)
    stats = lambda xs: {"ms": statistics.mean(xs), "ms_median": statistics.median(xs), "ms_min": min(xs)}
    loads_bytes = 4 * B * R * N + 2 * 4 * B * R * E
    sk_fma = 2 * support * w.iters
    sk_bytes = 4 * B * R * R + 2 * 4 * B * R   # plan and potentials written
    sch_bytes = 4 * B * R * R * K + 12 * B * R * K + 4 * support + 4 * R * distinct
    floor = {"plan_loads": loads_bytes / (HBM_PEAK_GBS * 1e9) * 1e3,
             "sinkhorn": max(sk_fma / VALU_FMA_PEAK, sk_bytes / (HBM_PEAK_GBS * 1e9)) * 1e3,
             "round_schedule": sch_bytes / (HBM_PEAK_GBS * 1e9) * 1e3}
    stages = {
        "plan_loads": dict(bound="hbm", **stats(run["loads_ms"]), bytes_per_launch=loads_bytes, peak=HBM_PEAK_GBS,
                           unit="GB/s"),
        "sinkhorn": dict(bound="alu", **stats(run["sk_ms"]), fma_per_launch=sk_fma, support_entries=support,
                         peak=2 * VALU_FMA_PEAK / 1e12, unit="TFLOP/s"),
        "round_schedule": dict(bound="latency", **stats(run["sch_ms"]), bytes_floor=sch_bytes,
                               phase2_inner_mean=float(rounds[:, 0].mean()),
                               phase3_rounds_mean=float(rounds[:, 1].mean()),
                               phase3_rounds_max=int(rounds[:, 1].max())),
    }
    stages["plan_loads"]["achieved"] = loads_bytes / (stages["plan_loads"]["ms_median"] * 1e-3) / 1e9
    stages["sinkhorn"]["achieved"] = 2 * sk_fma / (stages["sinkhorn"]["ms_median"] * 1e-3) / 1e12
    for k in ("plan_loads", "sinkhorn"):
        stages[k]["frac"] = stages[k]["achieved"] / stages[k]["peak"]
    traffic = measured_traffic("plan_loads", w.index)
    stages["plan_loads"]["traffic"] = traffic
    if peaks:
        stages["plan_loads"]["frac_vs_measured_peak"] = stages["plan_loads"]["achieved"] / peaks["hbm_read_GBs"]
        stages["sinkhorn"]["frac_vs_measured_peak"] = stages["sinkhorn"]["achieved"] / peaks["fp32_tflops_unpacked"]
    for k, f in floor.items():
        stages[k]["floor_ms"] = f
        stages[k]["frac_of_floor"] = f / stages[k]["ms_median"]
    step = stats(run["step_ms"])
    planner = dict(**step, floor_ms=sum(floor.values()), frac_of_floor=sum(floor.values()) / step["ms_median"])
    summary = {"ms_per_step": run["ms_step"], "ms_median": step["ms_median"], "ms_min": step["ms_min"],
               "plan_loads_ms": stages["plan_loads"]["ms_median"], "sinkhorn_ms": stages["sinkhorn"]["ms_median"],
               "round_schedule_ms": stages["round_schedule"]["ms_median"],
               "unfilled": int(sched.unfilled.sum().item())}
    status = {"loads_nonzero": int((st_loads != 0).sum()), "sinkhorn_nonzero": int((st_flow != 0).sum()),
              "schedule_unfilled": int(sched.unfilled.sum().item()), "schedule_nonzero": int((st_sched != 0).sum())}
    return {"stages": stages, "planner": planner, "summary": summary, "status": status,
            "phase3_rounds_mean": float(rounds[:, 1].mean())}


def host_cpu():
    """The host's logical CPU count and model name."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "model": model}


def cpu_baseline(w, K, args, home_np, C_np):
    """The oracle, as it is, on a sample of the workload's problems: ids made
    on the host (not timed), plan_loads (histogram ids/s), then Sinkhorn
    passes over the sample until --cpu-seconds have passed, then Phases 2-3
    once."""
    import numpy as np

    import oracle as O
    import workloads as W
    B = w.B
    stride = max(1, B // args.cpu_sample)
    sample = list(range(0, B, stride))[: args.cpu_sample]
    threads = O.max_threads()
    ids = np.stack([W.problem_ids_host(w, b) for b in sample])
    t = time.time()
    Lo = O.plan_loads(ids, home_np, w.E)
    t_loads = time.time() - t
    n_ids = ids.size
    del ids
    a, b, Cd = Lo.excess.astype(float), Lo.spare.astype(float), C_np.astype(float)
    passes, t_sk = 0, 0.0
    while t_sk < args.cpu_seconds or passes == 0:
        t = time.time()
        Po = O.sinkhorn(a, b, Cd, w.eps, w.iters)
        t_sk += time.time() - t
        passes += 1
    Bp_np, Ba_np = O.topology_pref(C_np)
    t = time.time()
    se, sa, _ = O.phase2(Lo.spill, Lo.spare, Lo.excess, Lo.alpha, home_np, Po.T.astype(np.float32), Bp_np, K)
    O.phase3(Lo.n, se, sa, Ba_np, K, w.price_step)
    t_sch = time.time() - t
    used = min(threads, len(sample))
    log(f"[bench] oracle on {len(sample)} problems, {used} threads: plan_loads {t_loads:.2f}s "
        f"({n_ids / t_loads / 1e9:.2f} G ids/s), sinkhorn {passes} passes {t_sk:.1f}s, schedule {t_sch:.1f}s")
    return {
        "value": passes * len(sample) * w.iters / t_sk, "unit": "problem-iters/s", "cores": used, "kind": "oracle",
        "sample": f"{len(sample)} of {B} problems (every {stride}th), ids generated on the host (not timed); fp64 "
                  f"C oracle Sinkhorn at the full iteration count, {passes} passes over the sample ({t_sk:.1f} s), "
                  f"OpenMP over problems",
        "histogram_ids_per_s": n_ids / t_loads,
        "schedule_s_per_problem": t_sch / len(sample),
        "host": host_cpu(), "omp_threads": threads,
    }


def cpu_extrapolate(gpu_rounds, cores):
    """Full-step oracle latency of workloads 1-4, EXTRAPOLATED from one problem
    of each on one thread: plan_loads as timed; the Sinkhorn timed for up to
    20 iterations and scaled to the workload's count; Phase 2 as timed;
    Phase 3 timed for up to 100 rounds and scaled by the mean rounds the GPU
    schedule took; the B problems spread over `cores` threads."""
    import numpy as np

    import oracle as O
    import workloads as W
    out = {}
    for wi in (1, 2, 3, 4):
        w = W.WORKLOADS[wi]
        home, C = W.home_map(w), W.cost_matrix(w)
        ids = W.problem_ids_host(w, 0)[None]
        t = time.time()
        L = O.plan_loads(ids, home, w.E)
        t_loads = time.time() - t
        del ids
        it = min(w.iters, 20)
        t = time.time()
        P = O.sinkhorn(L.excess.astype(float), L.spare.astype(float), C.astype(float), w.eps, it)
        t_sk = (time.time() - t) * w.iters / it
        Bp, Ba = O.topology_pref(C)
        t = time.time()
        se, sa, _ = O.phase2(L.spill, L.spare, L.excess, L.alpha, home, P.T.astype(np.float32), Bp, w.K)
        t_p2 = time.time() - t
        tmax = 100
        t = time.time()
        _, _, rounds, _ = O.phase3(L.n, se, sa, Ba, w.K, w.price_step, t_max=tmax)
        t_p3 = (time.time() - t) / max(int(rounds[0]), 1) * gpu_rounds.get(wi, int(rounds[0]))
        per_problem = t_loads + t_sk + t_p2 + t_p3
        waves = -(-w.B // cores)
        out[str(wi)] = {"extrapolated_ms_per_step": per_problem * waves * 1e3,
                        "per_problem_s": {"plan_loads": t_loads, "sinkhorn": t_sk, "phase2": t_p2, "phase3": t_p3},
                        "note": f"extrapolated: one problem on one thread, x ceil({w.B} / {cores}) problems per "
                                f"thread; Sinkhorn from {it} of {w.iters} iterations, Phase 3 from "
                                f"{int(rounds[0])} rounds scaled to the GPU's mean"}
        log(f"[bench] oracle extrapolation, workload {wi}: {per_problem:.2f} s per problem -> "
            f"{per_problem * waves:.1f} s per step (extrapolated)")
    return out


if __name__ == "__main__":
    main()
