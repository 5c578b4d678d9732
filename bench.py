"""Benchmark: lane-gradient evaluations per second (forward replay + reverse
sweep) on one MI355X, for one of the five synthetic workloads.

A step is one ndvm_grad call (ndvm_grad_many for the program population) that
produces loss[L] and grad[L, P] for a batch of L parameter vectors whose
inputs are already resident in HBM.  Tape production, upload and scheduling
happen before the timed region (reported apart, in the `host` object).  The
default workload is the largest: the Lotka-Volterra RK4 population (1000
steps, 65,536 lanes).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints one JSON line with the metric, a roofline object for the replay
kernel (its launch durations measured with HIP events on the launch stream,
against the algorithmic bytes and flops of one launch) and the CPU oracle
timed on a bounded sample of the same workload (all host threads up to 16,
and one thread).

    python bench.py --sweep [--workload NAME]

prints one JSON line per lane count (powers of two from 2^12 to 2^18) of the
same workload: the lane sweep that shows where a launch fills the GPU.

    python bench.py --flatten --workload exp_decay|random_programs

times the flattened data axis (one lane per parameter vector and data point,
ndvm_grad_points) against the ordinary replay of the same workload.

    python bench.py --calibrate N [--workload NAME] [--steps K]

instead measures calibrations per second: every lane of the workload is one
N-step Adam fit (ndvm_grad + ndvm_adam_step per step, tape uploaded once), as
in the paper's Kalman maximum-likelihood fit (default workload kalman_cv4).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import configs  # noqa: E402

PEAK_FP64 = 78.6e12        # MI355X fp64 vector FLOP/s
PEAK_HBM = 8.0e12          # MI355X HBM3E bytes/s
DEFAULT_WORKLOAD = "lotka_volterra_rk4"

# Doubles of loop-carried state per step and the step count: the values a
# one-level checkpoint of each step must keep for the reverse sweep (the
# predator and prey densities; the filter's state mean and covariance, 4 + 16;
# the logistic state).  The running loss sum needs no checkpoint (its adjoint
# is 1 whatever its value).  The exponential-decay and tree programs are sums
# of independent terms with nothing carried.
STATE_PER_STEP = {"lotka_volterra_rk4": (2, 1000), "kalman_cv4": (20, 200), "logistic_euler": (1, 500),
                  "exp_decay": (0, 0), "random_programs": (0, 0)}
CSRC = os.path.join(ROOT, "paper_2607_03574_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


# every source that decides what the replay kernel does on the GPU (front
# end, validator, scheduler, launch code, kernel)
REPLAY_SOURCES = ("abi.cpp", "common.h", "frontend.cpp", "kernels.hip", "sched.cpp", "sched.h", "slot.h",
                  "slot_exec.h", "tape.cpp")


def kernel_sources_sha256() -> str:
    """Hash of the replay kernel's sources (REPLAY_SOURCES)."""
    h = hashlib.sha256()
    for name in sorted(REPLAY_SOURCES):
        h.update(name.encode() + b"\0")
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def profiled_traffic(workload: str, policy: str = "recompute"):
    """HBM bytes per launch of the replay kernel for `workload` under a save
    policy, from the committed rocprofv3 summary (FETCH_SIZE + WRITE_SIZE, each
    scaled by a copy calibration); None when there is no summary or the kernel
    sources changed since its counters were taken."""
    sha = kernel_sources_sha256()
    for name in sorted(os.listdir(PROFILES)):
        if not (name.startswith(f"ndvm_replay_{workload}_") and name.endswith(".md")):
            continue
        vals = {"policy": "recompute"}
        with open(os.path.join(PROFILES, name)) as f:
            for line in f:
                key, _, val = line.strip().partition(": ")
                if key in ("traffic_bytes_per_launch", "kernel_sources_sha256", "policy"):
                    vals[key] = val
        if vals.get("kernel_sources_sha256") == sha and "traffic_bytes_per_launch" in vals \
                and vals["policy"] == policy:
            return float(vals["traffic_bytes_per_launch"])
    return None


def tape_flops(tape_bytes: bytes) -> float:
    """Algorithmic fp64 operations per lane of one forward + reverse pass over
    the realized trace: forward = one per output element of an elementwise
    op (transcendentals count 1), 2mkn for an m x k by k x n product, 2n for a
    dot; reverse = the flops of the adjoint rules (table tab:adjoints) for
    every op that depends on a parameter."""
    import struct
    (_, n_params, n_obs, n_ops, n_consts, n_aux, loss) = struct.unpack_from("<7I", tape_bytes, 4)
    off = 32 + 8 * n_consts + 4 * n_aux
    ops = [struct.unpack_from("<HBB5I", tape_bytes, off + 24 * k) for k in range(n_ops)]
    active = [False] * n_ops
    fwd = rev = 0.0
    for k, (code, r, c, a, b, cc, d, imm) in enumerate(ops):
        n = r * c
        if code == 0x02:
            active[k] = True
            continue
        if code in (0x01, 0x03):
            continue
        if code == 0x28:   # PACK: data movement only
            continue
        srcs = [a, b] if code in (0x10, 0x11, 0x12, 0x13, 0x1D, 0x20, 0x21, 0x27) else \
            [cc, d] if code == 0x40 else [a]
        active[k] = any(active[s] for s in srcs if s < k)
        ra, ca = ops[a][1], ops[a][2]
        if code == 0x21:
            f = 2.0 * ra * ca * c
            fr = 2 * f
        elif code == 0x20:
            f = 2.0 * ra * ca
            fr = 2 * f
        elif code in (0x23, 0x24, 0x25):
            f, fr = 10.0, 40.0
        elif code in (0x22, 0x29, 0x40):
            f, fr = 0.0, 0.0
        else:
            f, fr = float(n), 2.0 * n
        fwd += f
        if active[k]:
            rev += fr
    return fwd + rev


def build_flattened(name, torch, device):
    """The exponential-decay workload or the program population with the
    data axis flattened into the lanes (ndvm_grad_points: one lane per
    parameter vector and data point, then a fold over the points); one step
    produces the same loss[L] and grad[L, P] per program as the unflattened
    step."""
    import paper_2607_03574_amd as nd
    w = configs.build(name)
    if name == "exp_decay":
        n = w.meta["n_obs_points"]
        terms = [configs.exp_decay_term_program()]
        params = [w.params]
    elif name == "random_programs":
        n = w.meta["n"]
        terms = [configs.tree_term_program(t, c) for t, c in zip(w.meta["trees"], w.n_params_each)]
        params = [np.ascontiguousarray(w.params[q][:, :c]) for q, c in enumerate(w.n_params_each)]
    else:
        raise SystemExit("--flatten takes exp_decay or random_programs")
    pts = torch.tensor(configs.points_of(w.obs, n), device=device)
    t0 = time.perf_counter()
    tapes = [nd.tape_upload(nd.tape_build(t)) for t in terms]
    ps = [torch.tensor(p, device=device) for p in params]
    L = ps[0].shape[0]
    need = max(nd.workspace_bytes_points(t, L, n) for t in tapes)
    host = {"total_host_s": time.perf_counter() - t0, "programs": len(tapes)}
    ws = torch.empty(need, dtype=torch.uint8, device=device)
    outs = [(torch.empty(L, dtype=torch.float64, device=device),
             torch.empty((L, p.shape[1]), dtype=torch.float64, device=device)) for p in ps]

    def step(stream):
        for tape, p, (lo, go) in zip(tapes, ps, outs):
            nd.grad_points(tape, p, pts, 1.0 / n, lo, go, ws, stream)
    meta = dict(programs=len(tapes), lanes_per_program=L, data_points=n, flattened_lanes=L * n)
    return w, step, L * len(tapes), meta, host


POLICIES = {"recompute": 2, "save": 1}   # NDVM_POLICY_RECOMPUTE, NDVM_POLICY_SAVE


def build_inputs(name, torch, device, policy="recompute", branch_skip=False):
    """The workload's device inputs and one step.  Also times the host work
    per program that the lane-gradient rate leaves out: trace production
    (bytecode -> tape), upload (validation, copy) and scheduling for the
    launch's register budget (done once per program and lane count)."""
    import paper_2607_03574_amd as nd
    w = configs.build(name)
    o = torch.tensor(w.obs, device=device)
    p = torch.tensor(w.params, device=device)
    bcs = w.programs if name == "random_programs" else [w.bytecode]
    t0 = time.perf_counter()
    tapes_b = [nd.tape_build(bc) for bc in bcs]
    t1 = time.perf_counter()
    tapes = nd.tape_upload_many(tapes_b, policy=POLICIES[policy] | (nd.BRANCH_SKIP if branch_skip else 0))
    t2 = time.perf_counter()
    if name == "random_programs":
        n_prog, L, P = p.shape
        ws_bytes = nd.workspace_bytes_many(tapes, L)
    else:
        n_prog, (L, P) = 1, p.shape
        ws_bytes = nd.workspace_bytes(tapes[0], L, True)
    t3 = time.perf_counter()
    host = {"trace_us_per_program": (t1 - t0) / n_prog * 1e6, "upload_us_per_program": (t2 - t1) / n_prog * 1e6,
            "schedule_us_per_program": (t3 - t2) / n_prog * 1e6, "total_host_s": t3 - t0, "programs": n_prog,
            "workspace_bytes": int(ws_bytes)}
    ws = torch.empty(max(ws_bytes, 8), dtype=torch.uint8, device=device)
    flops = sum(tape_flops(t) for t in tapes_b) * L
    if name == "random_programs":
        loss = torch.empty((n_prog, L), dtype=torch.float64, device=device)
        grad = torch.zeros((n_prog, L, P), dtype=torch.float64, device=device)

        def step(stream):
            nd.grad_many(tapes, p, o, loss, grad, ws, stream)
        meta = dict(programs=n_prog, lanes_per_program=L)
        return w, step, n_prog * L, flops, meta, (w.programs, w.params, w.n_params_each), host
    tape = tapes[0]
    loss = torch.empty(L, dtype=torch.float64, device=device)
    grad = torch.empty((L, P), dtype=torch.float64, device=device)

    def step(stream):
        nd.grad(tape, p, o, loss, grad, ws, stream)
    meta = dict(lanes=L, params=P, tape_ops=nd.tape_info(tape)["n_ops"])
    return w, step, L, flops, meta, ([w.bytecode], w.params[None], [P]), host


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, progs, budget_s=10.0):
    """The oracle, as it stands, on a bounded sample of the same workload:
    lanes of the benchmark's own parameter population (the first 256 of each
    program, programs in order), repeated until about `budget_s` seconds of
    wall time have been spent with every host thread up to 16 (the host share
    of one GPU), then about a third of that on one thread."""
    import oracle
    bcs, params, nps = progs
    nproc = os.cpu_count() or 1
    threads = max(1, min(nproc, 16))

    def rate(nthreads, budget, lanes):
        t0 = time.perf_counter()
        done, progs_run = 0, 0
        while True:
            for q in range(len(bcs)):
                sub = params[q][:lanes, :nps[q]]
                oracle.run(bcs[q], sub, w.obs, threads=nthreads)
                done += sub.shape[0]
                progs_run = max(progs_run, q + 1)
                if time.perf_counter() - t0 > budget:
                    break
            if time.perf_counter() - t0 > budget:
                break
        dt = time.perf_counter() - t0
        return done / dt, done, dt, progs_run

    lanes = min(params.shape[1], 256)
    v_all, n_all, dt_all, pr_all = rate(threads, budget_s, lanes)
    v_one, n_one, dt_one, pr_one = rate(1, budget_s / 3, min(lanes, 16))
    return dict(value=v_all, unit="lane-gradient evals/s", cores=threads, kind="oracle",
                sample=f"{n_all} lane evaluations (first {lanes} lanes of {pr_all} program(s) of {w.name}, "
                       f"repeated), {dt_all:.1f} s wall on {threads} threads",
                nproc=nproc, cpu_model=cpu_model(), value_1_core=v_one,
                sample_1_core=f"{n_one} lane evaluations (first {min(lanes, 16)} lanes of {pr_one} program(s), "
                              f"repeated), {dt_one:.1f} s wall on 1 thread")


def env_info(torch):
    """What the numbers were measured with."""
    import subprocess
    info = {"gpu": torch.cuda.get_device_name(0), "torch": torch.__version__,
            "hip_runtime": getattr(torch.version, "hip", None)}
    try:
        r = subprocess.run(["git", "-C", ROOT, "rev-parse", "--short=12", "HEAD"], capture_output=True, text=True)
        info["git_commit"] = r.stdout.strip() or None
    except OSError:
        info["git_commit"] = None
    try:
        with open("/opt/rocm/.info/version") as f:
            info["rocm"] = f.read().strip()
    except OSError:
        info["rocm"] = None
    return info


def alg_bytes(name, L, P, n_prog=1):
    """Algorithmic HBM bytes of one launch: parameters read, loss and gradient
    written (8 (2P + 1) per lane), plus a store and a load of every double of
    loop-carried state per step (16 S T per lane)."""
    S, T = STATE_PER_STEP[name]
    return float(n_prog * L * (8 * (2 * P + 1) + 16 * S * T))


def calibration_bench(args):
    """Calibrations per second: all L lanes fitted at once with args.calibrate
    Adam steps each; a timed step is one whole fit of the population."""
    import torch
    import paper_2607_03574_amd as nd
    from paper_2607_03574_amd import torch_api
    name = args.workload if args.workload_given else "kalman_cv4"
    w = configs.build(name)
    if name == "random_programs":
        raise SystemExit("the calibration benchmark takes a single-program workload")
    n_steps, lr = args.calibrate, 1e-6
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    with torch.cuda.stream(stream):
        tape_b = nd.tape_build(w.bytecode)
        tape = nd.tape_upload(tape_b)
        obs = torch.tensor(w.obs, device=device)
        p0 = torch.tensor(w.params, device=device)
        L = p0.shape[0]
        ws = torch.empty(max(nd.workspace_bytes(tape, L, True), 8), dtype=torch.uint8, device=device)
        p = p0.clone()
    torch.cuda.synchronize()

    def fit():
        p.copy_(p0)
        return torch_api.calibrate(tape, p, obs, n_steps, lr, workspace=ws, stream=stream)
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            fit()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        ev0.record(stream)
        for _ in range(args.steps):
            hist = fit()
        ev1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / args.steps
    gpu_s = ev0.elapsed_time(ev1) / 1e3 / args.steps
    flops = tape_flops(tape_b) * L * n_steps
    improved = float((hist[-1] < hist[0]).double().mean().item())
    out = {
        "metric": f"calibrations/sec ({n_steps}-step Adam fits, one per lane) on 1 MI355X",
        "value": L / wall, "unit": "calibrations/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": wall * 1e3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": w.name, "lanes": L, "adam_steps": n_steps, "lr": lr,
                   "lanes_improved": improved},
        "roofline": {"bound": "alu", "achieved": flops / gpu_s / 1e12, "peak": PEAK_FP64 / 1e12,
                     "unit": "TFLOP/s", "frac": flops / gpu_s / PEAK_FP64, "traffic": None,
                     "kernel": "ndvm_replay + ndvm_adam", "kernel_ms": gpu_s * 1e3},
    }
    if not args.no_cpu_baseline:
        from oracle import adam
        lanes = 32
        t0 = time.perf_counter()
        done = 0
        while time.perf_counter() - t0 < 10.0:
            adam.calibrate(w.bytecode, w.params[:lanes], w.obs, n_steps, lr, threads=16)
            done += lanes
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = dict(value=done / dt, unit="calibrations/s", cores=min(os.cpu_count() or 1, 16),
                                   kind="oracle",
                                   sample=f"{done} calibrations ({n_steps} Adam steps each) of the first "
                                          f"{lanes} lanes of {w.name}, {dt:.1f} s wall")
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None, choices=configs.ORDER)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", action="store_true", help="lane sweep 2^12 .. 2^18 of the workload")
    ap.add_argument("--policy", default="recompute", choices=sorted(POLICIES),
                    help="save policy of the reverse sweep: recompute (segment inputs stored, values recomputed) "
                         "or save (every value the adjoint rules read stored)")
    ap.add_argument("--branch-skip", action="store_true",
                    help="tapes uploaded with the BRANCH_SKIP option (waves skip branch arms none of their lanes takes)")
    ap.add_argument("--branch-study", action="store_true",
                    help="branch skipping on programs with heavy arms: lanes ordered by the predicate or "
                         "interleaved, with and without the option")
    ap.add_argument("--walk", action="store_true",
                    help="the device walker (structural walk on the GPU, no tape, no scheduling) on the workload, "
                         "against the scheduled replay, host work included")
    ap.add_argument("--flatten", action="store_true",
                    help="data axis flattened into the lanes (exp_decay, random_programs), against the unflattened step")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the benchmark, run a plain device-to-device copy of this many "
                         "MiB (reference for the FETCH_SIZE / WRITE_SIZE counter scale)")
    ap.add_argument("--calibrate", type=int, default=0, metavar="N",
                    help="measure calibrations/s: every lane is one N-step Adam fit")
    args = ap.parse_args()
    args.workload_given = args.workload is not None
    if args.workload is None:
        args.workload = DEFAULT_WORKLOAD
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 8
        src = torch.ones(n, dtype=torch.float64, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": n * 8, "launches": 3}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the replay runs on one GPU per process; --gpus must be 1 "
                          "(lanes and programs are independent, so several GPUs would each take a slice; not implemented)"}))
        sys.exit(2)
    if args.calibrate:
        return calibration_bench(args)
    import torch
    if args.sweep:
        return sweep(args, torch)
    if args.flatten:
        return flattened_bench(args, torch)
    if args.branch_study:
        return branch_study(args, torch)
    if args.walk:
        return walk_bench(args, torch)
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    with torch.cuda.stream(stream):
        w, step, lanes, flops, meta, progs, host = build_inputs(args.workload, torch, device, args.policy,
                                                                args.branch_skip)
    if args.branch_skip:
        meta["branch_skip"] = True
    torch.cuda.synchronize()
    res = time_steps(torch, stream, step, args.steps, args.warmup)
    kern_s = res["kernel_mean_s"]
    ms_per_step = res["wall_s"] / args.steps * 1e3
    value = lanes / (res["wall_s"] / args.steps)
    if args.workload == "random_programs":
        host["end_to_end_s"] = host["total_host_s"] + kern_s
    B = alg_bytes(args.workload, meta.get("lanes", meta.get("lanes_per_program")), meta.get("params", 0),
                  meta.get("programs", 1)) if args.workload != "random_programs" else \
        float(sum(8 * (2 * P + 1) for P in progs[2]) * meta["lanes_per_program"])
    if args.policy == "save" and args.workload != "random_programs":
        # the save policy needs a store and a load of every value the adjoint
        # rules read: the schedule's checkpoint rows (workspace rows less the
        # trash rows; no spills at these budgets)
        L, P = meta["lanes"], meta["params"]
        rows = host["workspace_bytes"] // (8 * ((L + 63) // 64 * 64)) - 4
        B = float(L * (8 * (2 * P + 1) + 16 * rows))
        meta["saved_doubles_per_lane"] = int(rows)
    roof = roofline(B, flops, kern_s, None if args.branch_skip else profiled_traffic(args.workload, args.policy))
    roof.update(kernel="ndvm_replay", kernel_ms=kern_s * 1e3, kernel_ms_median=res["kernel_median_s"] * 1e3,
                kernel_ms_iqr=res["kernel_iqr_s"] * 1e3)
    out = {
        "metric": "lane-gradient evals/sec (fwd+rev) on 1 MI355X",
        "value": value, "unit": "lane-gradient evals/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": dict(workload=w.name, policy=args.policy, **meta),
        "roofline": roof,
        "host": host,
        "env": env_info(torch),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, progs)
    print(json.dumps(out), flush=True)


def flattened_bench(args, torch):
    """The flattened data axis against the unflattened replay on the same
    workload: lane-grads/s of each (the unflattened figure from a run of the
    ordinary step in the same process)."""
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    with torch.cuda.stream(stream):
        w, step, lanes, meta, host = build_flattened(args.workload, torch, device)
    torch.cuda.synchronize()
    res = time_steps(torch, stream, step, args.steps, args.warmup)
    with torch.cuda.stream(stream):
        _, ustep, ulanes, _, _, _, _ = build_inputs(args.workload, torch, device)
    torch.cuda.synchronize()
    ures = time_steps(torch, stream, ustep, args.steps, args.warmup)
    out = {"metric": "lane-gradient evals/sec (fwd+rev) on 1 MI355X, data axis flattened", "workload": w.name,
           "value": lanes / (res["wall_s"] / args.steps), "unit": "lane-gradient evals/s",
           "ms_per_step": res["wall_s"] / args.steps * 1e3, "kernel_ms_mean": res["kernel_mean_s"] * 1e3,
           "unflattened_value": ulanes / (ures["wall_s"] / args.steps),
           "unflattened_ms_per_step": ures["wall_s"] / args.steps * 1e3,
           "speedup": ures["wall_s"] / res["wall_s"], "dtype": "f64", "data": "synthetic",
           "config": meta, "host": host, "steps": args.steps, "warmup": args.warmup}
    print(json.dumps(out), flush=True)


def walk_bench(args, torch):
    """The device walker on the workload (scalar programs): host work
    (validation, measurement and one copy of the bytecode), the walk's kernel
    time (HIP events over the timed steps) and lane-grads/s, next to the
    scheduled replay's host work (trace, upload, scheduling) and kernel time
    on the same inputs.  One JSON line."""
    import paper_2607_03574_amd as nd
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    w = configs.build(args.workload)
    progs = w.programs if args.workload == "random_programs" else [w.bytecode]
    params = w.params if args.workload == "random_programs" else w.params[None]
    n_prog, L, P = params.shape
    with torch.cuda.stream(stream):
        t0 = time.perf_counter()
        ws = nd.walk_prepare(progs, stream=stream)
        t1 = time.perf_counter()
        need = nd.walk_workspace_bytes(ws, L)
        p = torch.tensor(params, device=device)
        o = torch.tensor(w.obs, device=device)
        work = torch.empty(max(need, 8), dtype=torch.uint8, device=device)
        loss = torch.empty((n_prog, L), dtype=torch.float64, device=device)
        grad = torch.zeros((n_prog, L, P), dtype=torch.float64, device=device)
    torch.cuda.synchronize()

    def step(s):
        nd.walk_grad(ws, p, o, loss, grad, work, s)
    res = time_steps(torch, stream, step, args.steps, args.warmup)
    nd.walk_status(work, stream)
    kern = res["kernel_mean_s"]
    with torch.cuda.stream(stream):
        _, rstep, _, _, _, _, host = build_inputs(args.workload, torch, device)
    torch.cuda.synchronize()
    rres = time_steps(torch, stream, rstep, args.steps, args.warmup)
    out = {"metric": "lane-gradient evals/sec (fwd+rev) on 1 MI355X, device walker", "workload": w.name,
           "value": n_prog * L / (res["wall_s"] / args.steps), "unit": "lane-gradient evals/s",
           "kernel_ms": kern * 1e3, "kernel_ms_median": res["kernel_median_s"] * 1e3,
           "host_prepare_s": t1 - t0, "workspace_bytes": int(need),
           "end_to_end_s": (t1 - t0) + kern,
           "replay_kernel_ms": rres["kernel_mean_s"] * 1e3, "replay_host_s": host["total_host_s"],
           "replay_end_to_end_s": host["total_host_s"] + rres["kernel_mean_s"],
           "dtype": "f64", "data": "synthetic", "programs": n_prog, "lanes_per_program": L,
           "steps": args.steps, "warmup": args.warmup}
    print(json.dumps(out), flush=True)


def branch_study(args, torch):
    """Wave-level branch skipping on tree programs with heavy arms (16,384
    and 65,536 lanes, 128 points): the same lanes ordered by the branch's
    predicate (waves decide alike) or interleaved (every wave runs both
    arms), and populations whose lanes all take one arm, each with and
    without the BRANCH_SKIP option; one JSON line per run."""
    import paper_2607_03574_amd as nd
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    runs = [(c, n_l, o) for n_l in (16384, 65536) for c in range(len(configs.BRANCH_TREES))
            for o in ("sorted", "mixed", "all_then", "all_else")]
    for case, n_lanes, order in runs:
        w = configs.branch_population(case, L=n_lanes, order=order)
        L, P = w.params.shape
        tb = nd.tape_build(w.bytecode)
        for skip in (False, True):
            with torch.cuda.stream(stream):
                tape = nd.tape_upload(tb, policy=nd.POLICY_RECOMPUTE | (nd.BRANCH_SKIP if skip else 0))
                p = torch.tensor(w.params, device=device)
                o = torch.tensor(w.obs, device=device)
                ws = torch.empty(max(nd.workspace_bytes(tape, L, True), 8), dtype=torch.uint8, device=device)
                loss = torch.empty(L, dtype=torch.float64, device=device)
                grad = torch.empty((L, P), dtype=torch.float64, device=device)
            torch.cuda.synchronize()

            def step(s):
                nd.grad(tape, p, o, loss, grad, ws, s)
            res = time_steps(torch, stream, step, args.steps, args.warmup)
            t = res["kernel_mean_s"]
            print(json.dumps({"study": "branch_skip", "case": case, "order": order, "branch_skip": skip,
                              "lanes": L, "points": w.meta["n"], "kernel_ms": t * 1e3,
                              "kernel_ms_median": res["kernel_median_s"] * 1e3,
                              "lane_grads_per_s": L / t}), flush=True)
            del tape, ws


def time_steps(torch, stream, step, steps, warmup):
    """Run `warmup` untimed steps, then `steps` timed ones bracketed by device
    synchronisation; every launch is also bracketed by HIP events on the
    launch stream (the kernel's own duration)."""
    for _ in range(warmup):
        step(stream)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(stream)
    for k in range(steps):
        step(stream)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    d = np.array([evs[k].elapsed_time(evs[k + 1]) / 1e3 for k in range(steps)])
    q1, q3 = np.percentile(d, [25, 75])
    return dict(wall_s=wall, kernel_mean_s=float(d.mean()), kernel_median_s=float(np.median(d)),
                kernel_iqr_s=float(q3 - q1))


def roofline(B, F, t, traffic):
    """Roofline of one launch: the algorithmic bytes B and flops F against
    MI355X's HBM and fp64 vector peaks; the bound is whichever would take
    longer at peak, and frac = that time / the measured time t."""
    t_hbm, t_alu = B / PEAK_HBM, F / PEAK_FP64
    if t_hbm >= t_alu:
        r = {"bound": "hbm", "achieved": B / t / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s"}
    else:
        r = {"bound": "alu", "achieved": F / t / 1e12, "peak": PEAK_FP64 / 1e12, "unit": "TFLOP/s"}
    r["frac"] = r["achieved"] / r["peak"]
    r["traffic"] = traffic
    r.update(alg_bytes_per_launch=B, alg_flops_per_launch=F, t_at_hbm_peak_ms=t_hbm * 1e3,
             t_at_fp64_peak_ms=t_alu * 1e3, alg_frac=max(t_hbm, t_alu) / t,
             fp64_tflops=F / t / 1e12, alg_hbm_gbps=B / t / 1e9,
             counter_hbm_gbps=(traffic / t / 1e9) if traffic else None)
    return r


def sweep(args, torch):
    """Lane sweep of one workload: lane-grads/s and the roofline fraction at
    L = 2^12 .. 2^18 (parameters drawn by the workload's own recipe)."""
    import paper_2607_03574_amd as nd
    name = args.workload
    if name == "random_programs":
        raise SystemExit("the sweep takes a single-program workload")
    device = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=device)
    for e in range(12, 19):
        L = 1 << e
        with torch.cuda.stream(stream):
            w = configs.build(name, L=L)
            tb = nd.tape_build(w.bytecode)
            tape = nd.tape_upload(tb)
            p = torch.tensor(w.params, device=device)
            o = torch.tensor(w.obs, device=device)
            P = p.shape[1]
            ws = torch.empty(max(nd.workspace_bytes(tape, L, True), 8), dtype=torch.uint8, device=device)
            loss = torch.empty(L, dtype=torch.float64, device=device)
            grad = torch.empty((L, P), dtype=torch.float64, device=device)
        torch.cuda.synchronize()

        def step(s):
            nd.grad(tape, p, o, loss, grad, ws, s)
        res = time_steps(torch, stream, step, args.steps, args.warmup)
        t = res["kernel_mean_s"]
        roof = roofline(alg_bytes(name, L, P), tape_flops(tb) * L, t, None)
        print(json.dumps({"workload": name, "lanes": L, "lane_grads_per_s": L / t, "kernel_ms": t * 1e3,
                          "kernel_ms_median": res["kernel_median_s"] * 1e3, "bound": roof["bound"],
                          "frac": roof["frac"], "alg_frac": roof["alg_frac"],
                          "fp64_tflops": roof["fp64_tflops"], "alg_hbm_gbps": roof["alg_hbm_gbps"]}), flush=True)
        del tape, p, ws, loss, grad


if __name__ == "__main__":
    main()
