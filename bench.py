"""Benchmark of the batched route-and-schedule tick on one MI355X.

A step is one tick of the whole hot path over one batch of synthetic input:
im_route (features, policy MLP, masked argmax) then im_schedule (admission,
keys, queue insertion, service, accounting) over every env. Inputs for all
ticks are generated up front and resident in HBM before timing starts.

Prints ONE JSON line (see the keys below). `value` comes from K ticks of
im_tick with events only at the two ends. The same K ticks are then run on an
identical pool with HIP events recorded on the launch stream around every
route and schedule launch; `roofline` is computed for the kernel with the
larger average duration in that pass. `cpu_baseline` is the oracle (plain C++, fp64 policy) timed on the
host cores over a bounded sample of the same workload."""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "env-ticks/s and routed requests/s at 4096 envs; % of HBM/MFMA roofline"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 matrix/vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def algorithmic_flops_per_tick(cfg, n_requests):
    """Minimal policy FLOPs of one tick: per request the MLP without the
    per-env load-statistics columns of layer 1, plus once per env those 4M
    columns (they are shared by every request of the env). A value head adds
    one more output row of the last layer.

    Dual-pathway executor: per request the query half of the semantic layer
    (128 x E_d), the budget head (16), the budget half of the resource layer
    (64 x 16), the merge layer (128 x 192) and the action/value rows (x 128);
    per env the system head (16 x 3M) and the system half of the resource
    layer (64 x 16). The role half of the semantic layer takes n_roles
    distinct inputs and is computed once per pool, not per tick. Matrix
    products only (the LayerNorms add ~6 FLOP per feature)."""
    if cfg.get("net") == "dual":
        Ao = cfg["A"] + (1 if cfg.get("value_head") else 0)
        per_req = 2 * (128 * cfg["embed_dim"] + 16 + 64 * 16 + 128 * 192 + Ao * 128)
        per_env = 2 * (16 * 3 * cfg["M"] + 64 * 16)
        return per_req * n_requests + per_env * cfg["E"]
    widths = list(cfg["widths"])
    if cfg.get("value_head"):
        widths[-1] += 1
    H1 = widths[0]
    per_req = 2 * (cfg["embed_dim"] + 1) * H1
    prev = H1
    for w in widths[1:]:
        per_req += 2 * prev * w
        prev = w
    per_env = 2 * 4 * cfg["M"] * H1
    return per_req * n_requests + per_env * cfg["E"]


def algorithmic_bytes_route(cfg, n_requests, sample=False):
    """Bytes the route step must move: per request its record (q_idx 4 B,
    budget 2 B, role 2 B for the dual-pathway executor), its embedding row
    and its action (4 B; log-prob, entropy and value 4 B each for an RL
    rollout); per env its snapshot row (4M fp32 statistics and M validity
    bytes)."""
    s = 2 if cfg["dtype"] == "bf16" else 4
    per_req = 4 + 2 + cfg["embed_dim"] * s + 4
    if cfg.get("net") == "dual":
        per_req += 2
    if sample:
        per_req += 12
    return per_req * n_requests + (16 * cfg["M"] + cfg["M"]) * cfg["E"]


def algorithmic_bytes_schedule(cfg, n_requests, n_enqueued, n_started):
    """Bytes the schedule step must move: per request its record (budget,
    base_svc, action = 8 B); 16 B per queue entry written at enqueue and read
    at dequeue; per (env, model) its 64 B record and its slots, read and
    written; per env its counters."""
    EM = cfg["E"] * cfg["M"]
    return (8 * n_requests + 16 * (n_enqueued + n_started)
            + EM * 2 * (64 + 16 * cfg["max_slots"] + 8 * 8) + cfg["E"] * 2 * 16)


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2606_11440_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload_tag, src_hash):
    """HBM bytes per launch from a committed rocprofv3 --pmc summary, or None
    when there is none or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_tag}_pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_hash") != src_hash:
        return None
    return d.get("hbm_bytes_per_launch")


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# Worker threads of the oracle baseline: the host cores this process may use,
# at most the 16 a one-GPU share of the host provides.
CPU_SHARE = 16


def cpu_baseline(cfg, W, b, emb_vals, cap, lb, ticks, Q, budget_s=15.0):
    """The oracle on the host cores over a bounded sample of the workload:
    blocks of `envs` consecutive envs, each over the timed ticks, for about
    2/3 of budget_s with every worker thread; then blocks of envs / threads
    envs on one thread for the rest (the single-thread rate)."""
    import oracle
    import workload
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    threads = max(1, min(CPU_SHARE, usable))
    envs = min(cfg["E"], 8 * threads)
    roles = b if cfg.get("net") == "dual" else None

    def run(nthreads, n_envs, seconds):
        """Blocks of n_envs consecutive envs, each over the timed ticks, until
        `seconds` have passed (at least one tick)."""
        t0 = time.perf_counter()
        env_ticks, nreq, blocks, done = 0, 0, 0, 0
        for e0 in range(0, cfg["E"] - n_envs + 1, n_envs):
            o = oracle.Oracle(cfg, W, b, emb_vals, cap[e0:e0 + n_envs], lb, E=n_envs, threads=nthreads,
                              roles=roles)
            blocks += 1
            for a in ticks:
                sub = workload.gen.subset(a, e0, e0 + n_envs)
                o.tick(sub)
                env_ticks += n_envs
                nreq += int(sub["q_idx"].size)
                done += 1
                if time.perf_counter() - t0 > seconds:
                    break
            if time.perf_counter() - t0 > seconds:
                break
        dt = time.perf_counter() - t0
        return env_ticks / dt, nreq / dt, blocks, done, nreq, dt

    v, rq, blocks, done, nreq, dt = run(threads, envs, budget_s * 2 / 3)
    env1 = max(1, envs // threads)
    v1, rq1, blocks1, done1, _, dt1 = run(1, env1, budget_s / 3)
    return {"value": v, "unit": "env-ticks/s", "cores": threads, "kind": "oracle",
            "sample": f"{blocks} block(s) of {envs} envs over the {len(ticks)} timed ticks ({done} env-block "
                      f"ticks, {nreq} requests), {dt:.1f} s wall, {rq:.0f} routed req/s",
            "nproc": os.cpu_count(), "usable_cpus": usable, "cpu_model": cpu_model(),
            "threads_note": f"one oracle worker thread per env block, min({CPU_SHARE}, usable CPUs): "
                            f"{CPU_SHARE} is the host share of one GPU on the machines this runs on",
            "single_thread": {"value": v1, "unit": "env-ticks/s", "routed_req_per_s": rq1,
                              "sample": f"{blocks1} block(s) of {env1} envs, {done1} env-block ticks, "
                                        f"{dt1:.1f} s wall"}}


def mfma_probe(torch, zeros=False):
    """bf16 MFMA throughput of a register-resident 32x32x16 MFMA loop on every
    SIMD (paper_2606_11440_amd/csrc/peak_probe.hip), N(0,1) operands (or
    zeros): the matrix cores' achievable rate on this device with no memory
    traffic."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_11440_amd", "libimprobe.so"))
    lib.im_probe_mfma_bf16.restype = ctypes.c_double
    lib.im_probe_mfma_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_void_p]
    src = (torch.zeros if zeros else torch.randn)(1024, device="cuda", dtype=torch.bfloat16)
    blocks, iters = 1024, 20000
    sink = torch.empty(blocks * 4, device="cuda", dtype=torch.float32)
    st = torch.cuda.current_stream().cuda_stream
    run = lambda: lib.im_probe_mfma_bf16(src.data_ptr(), sink.data_ptr(), blocks, iters, st)  # noqa: E731
    run()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    flops = sum(run() for _ in range(3))
    e.record()
    torch.cuda.synchronize()
    return flops / (s.elapsed_time(e) * 1e-3) / 1e12


def measured_peaks(torch):
    """Achievable peaks on this device: the MFMA probe (random and zero
    operands), a 8192^3 bf16 GEMM (torch.matmul on hipBLASLt) and a 1 GiB
    device copy."""
    mfma_rand = mfma_probe(torch)
    mfma_zero = mfma_probe(torch, zeros=True)
    n = 8192
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        a @ b
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        a @ b
    e.record()
    torch.cuda.synchronize()
    gemm_tflops = 10 * 2 * n ** 3 / (s.elapsed_time(e) * 1e-3) / 1e12
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    s.record()
    for _ in range(5):
        dst.copy_(src)
    e.record()
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * (1 << 30) / (s.elapsed_time(e) * 1e-3) / 1e9
    del a, b, src, dst
    torch.cuda.empty_cache()
    return {"mfma_bf16_tflops_random": mfma_rand, "mfma_bf16_tflops_zero": mfma_zero,
            "bf16_gemm_tflops": gemm_tflops, "copy_gbs_read_plus_write": copy_gbs}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--lam", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch the timed ticks one by one instead of replaying them "
                         "from a captured HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--sample", action="store_true",
                    help="RL-rollout tick: im_route_sample (Gumbel-max sample, log-prob, entropy, "
                         "value head) then im_schedule with the sampled actions")
    ap.add_argument("--blackbox", action="store_true",
                    help="half the models of every env rate-limited blackboxes (dispatch limits "
                         "uniform in [60, 600] per 60-tick window: the congestion feature and the "
                         "backpressure of App. C), and the dual update of lambda (Eq. 7, eta 1e-3, "
                         "lambda_max 1, lambda_0 0.2) after every tick")
    ap.add_argument("--no-peak-probe", action="store_true",
                    help="skip the measured-peak probes (a large bf16 GEMM and a device copy)")
    ap.add_argument("--per-tick", default=None, metavar="FILE",
                    help="write the instrumented pass's route and schedule durations of every "
                         "timed tick (microseconds) to FILE as JSON")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 5 device-to-device copies of MIB MiB (calibrates "
                         "the HBM byte counters of a profiler against a known size)")
    args = ap.parse_args()
    if args.copy_probe:
        import torch
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_per_copy": n, "copies": 5}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1 "
                          "(envs shard across GPUs with no per-tick exchange, see the design notes)"}))
        sys.exit(2)

    import torch

    import paper_2606_11440_amd as P
    import workload

    over = {}
    if args.lam is not None:
        over["lam"] = args.lam
    if args.sample:
        over["value_head"] = True
    cfg = workload.configs.get(args.config, **over)
    T = cfg["T"]
    W_ = args.warmup
    K = args.steps if args.steps is not None else T - W_
    if W_ + K > T:
        over["T"] = W_ + K
        cfg = workload.configs.get(args.config, **over)
        T = cfg["T"]

    # ---- inputs (host generation, then resident in HBM) ----
    t_gen = time.perf_counter()
    if cfg.get("net") == "dual":
        W, b = workload.gen.dual_weights(cfg, args.seed), workload.gen.roles(cfg, args.seed)
    else:
        W, b = workload.gen.weights(cfg, args.seed)
    Q = workload.gen.table_rows(cfg)
    table, emb_vals = workload.gen.embedding(cfg, args.seed, rows=Q)
    cap = workload.gen.capacities(cfg, args.seed)
    lb = workload.gen.logit_bias(cfg)
    counts = workload.gen.counts(cfg, args.seed)
    ticks = [workload.gen.tick(cfg, args.seed, t, counts[t], Q) for t in range(W_ + K)]
    emb_dev = torch.from_numpy(table.view(np.int16) if cfg["dtype"] == "bf16" else table).cuda()
    dev = [P.device_arrivals(a) for a in ticks]
    n_req = [int(a["q_idx"].size) for a in ticks]
    chains = cfg.get("max_steps", 1) > 1
    # chain pools: a tick's rows are its pending calls and its arrivals
    extra = cfg["E"] * cfg["M"] * cfg["max_slots"] if chains else 0
    acts = torch.empty(max(max(n_req), 1) + extra, dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    rl_out = [torch.empty(max(max(n_req), 1) + extra, **f32) for _ in range(3)] if args.sample else None
    bb_limits, lam_dev = [], None
    if args.blackbox:
        rng_bb = np.random.default_rng(args.seed + 7)
        pick = rng_bb.random((cfg["E"], cfg["M"])) < 0.5
        lim = rng_bb.integers(60, 601, size=(cfg["E"], cfg["M"]))
        bb_limits = [(int(e), int(m), int(lim[e, m])) for e, m in zip(*np.nonzero(pick))]
        lam_dev = torch.full((1,), 0.2, dtype=torch.float64, device="cuda")

    def new_pool():
        pl = P.Pool(cfg, W, b, emb_dev, cap, lb)
        for e, m, r in bb_limits:
            pl.set_rpm_limit(e, m, r)
        return pl

    pool = new_pool()

    def route_step(pl, t, st=None, with_schedule=True):
        """One tick: im_tick, or im_route_sample + im_schedule (RL rollout);
        with --blackbox the dual update follows."""
        if args.sample:
            pl.route_sample(dev[t], 1000 + t, acts, *rl_out, stream=st)
            if with_schedule:
                pl.schedule(dev[t], acts, st)
        else:
            pl.tick(dev[t], acts, st)
        if args.blackbox and with_schedule:
            pl.dual_update(1e-3, 1.0, lam_dev, st)
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t_gen

    stream = torch.cuda.current_stream()

    def warm(pl):
        for t in range(W_):
            route_step(pl, t, stream.cuda_stream)
        torch.cuda.synchronize()

    # ---- timed region: K ticks of im_tick, events only at the two ends ----
    warm(pool)
    graph = None
    if not args.eager:
        # The K ticks (two kernels each) are captured into one HIP graph
        # outside the timed region and replayed once inside it: the same
        # kernels on the same inputs, without per-launch host overhead.
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for k in range(K):
                route_step(pool, W_ + k)
        torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    if graph is not None:
        graph.replay()
    else:
        for k in range(K):
            route_step(pool, W_ + k, stream.cuda_stream)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = start.elapsed_time(end)
    assert pool.error() == 0, "device error during the benchmark"
    st = pool.state(0, cfg["E"], with_queues=False)
    pool.close()
    lam_after = None
    if args.blackbox:
        lam_after = float(lam_dev.cpu().item())   # after the warm-up and timed ticks
        lam_dev.fill_(0.2)

    # ---- the same K ticks on an identical pool, HIP events on the launch
    # stream around every route and schedule launch (per-kernel durations;
    # the event records themselves add a gap, so this pass is not the value) ----
    pool2 = new_pool()
    warm(pool2)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    if chains:
        # The rows a chain tick routes (its pending calls and its arrivals) are
        # counted on the device: each tick's count is copied on the stream, after
        # the tick's last event, into a slot of its own and read once after the
        # pass. A host read per tick would drain the stream and put the next
        # tick's launch latency inside its route interval.
        import ctypes
        hip = ctypes.CDLL("libamdhip64.so")
        hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int,
                                       ctypes.c_void_p]
        hip.hipMemcpyAsync.restype = ctypes.c_int
        n_rows_dev = P.im_get_rows(pool2.h).n_rows
        row_counts = torch.zeros(K, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    for k in range(K):
        t = W_ + k
        ev[k][0].record(stream)
        if args.sample:
            route_step(pool2, t, stream.cuda_stream, with_schedule=False)
        else:
            pool2.route(dev[t], acts, None, stream.cuda_stream)
        ev[k][1].record(stream)
        pool2.schedule(dev[t], acts, stream.cuda_stream)
        ev[k][2].record(stream)
        if args.blackbox:
            pool2.dual_update(1e-3, 1.0, lam_dev, stream.cuda_stream)
        if chains:
            rc = hip.hipMemcpyAsync(row_counts.data_ptr() + 4 * k, n_rows_dev, 4, 3,   # device to device
                                    stream.cuda_stream)
            assert rc == 0, f"hipMemcpyAsync failed ({rc})"
    torch.cuda.synchronize()
    if chains:
        for k, n in enumerate(row_counts.cpu().numpy()):
            n_req[W_ + k] = int(n)
    route_ms = [ev[k][0].elapsed_time(ev[k][1]) for k in range(K)]
    sched_ms = [ev[k][1].elapsed_time(ev[k][2]) for k in range(K)]
    assert pool2.error() == 0, "device error during the instrumented pass"
    pool2.close()

    ms_per_step = gpu_ms / K
    env_ticks = cfg["E"] * K
    routed = sum(n_req[W_:W_ + K])
    value = env_ticks / (gpu_ms / 1e3)

    if args.per_tick:
        with open(args.per_tick, "w") as f:
            json.dump({"workload": args.config, "lam": cfg["lam"], "first_tick": W_,
                       "route_us": [x * 1e3 for x in route_ms], "schedule_us": [x * 1e3 for x in sched_ms],
                       "requests": n_req[W_:W_ + K]}, f)

    # ---- rooflines: the dominant kernel ("roofline"), then the other one ----
    route_avg = float(np.mean(route_ms))
    sched_avg = float(np.mean(sched_ms))
    flops = np.mean([algorithmic_flops_per_tick(cfg, n) for n in n_req[W_:W_ + K]])
    peak_f = PEAK_BF16_TFLOPS if cfg["dtype"] == "bf16" else PEAK_F32_TFLOPS
    tag = f"{args.config}_lam{int(cfg['lam'])}" + ("_sample" if args.sample else "") + \
        ("_blackbox" if args.blackbox else "")

    def route_roof():
        # the binding roof of the route step: the larger of its matrix time
        # and its HBM time at nominal peaks
        # the binding roof of the route step: the larger of its matrix time
        # and its HBM time at nominal peaks
        rbytes = np.mean([algorithmic_bytes_route(cfg, n, args.sample) for n in n_req[W_:W_ + K]])
        kname = ("route_sample_" if args.sample else "route_dual_" if cfg.get("net") == "dual" else "route_") + cfg["dtype"]
        traffic = load_traffic("route", tag, source_hash("route.hip"))
        if flops / (peak_f * 1e12) >= rbytes / (PEAK_HBM_GBS * 1e9):
            achieved = flops / (route_avg * 1e-3) / 1e12
            return {"kernel": kname, "bound": "mfma", "achieved": achieved,
                    "peak": peak_f, "unit": "TFLOP/s", "frac": achieved / peak_f,
                    "traffic": traffic, "avg_launch_us": route_avg * 1e3,
                    "algorithmic_per_launch": f"{flops:.4g} FLOP"}
        achieved = rbytes / (route_avg * 1e-3) / 1e9
        return {"kernel": kname, "bound": "hbm", "achieved": achieved,
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                "traffic": traffic, "avg_launch_us": route_avg * 1e3,
                "algorithmic_per_launch": f"{rbytes:.4g} B ({flops:.4g} FLOP)"}

    def schedule_roof():
        # per-tick averages over the ticks that ran (warm-up and timed)
        ran = W_ + K
        enq = int(st["enqueued"].sum())
        sta = int(st["started"].sum())
        byts = algorithmic_bytes_schedule(cfg, routed / K, enq / ran, sta / ran)
        achieved = byts / (sched_avg * 1e-3) / 1e9
        return {"kernel": "schedule", "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                "traffic": load_traffic("schedule", tag, source_hash("schedule.hip")),
                "avg_launch_us": sched_avg * 1e3,
                "algorithmic_per_launch": f"{byts:.4g} B",
                "note": "issue- and latency-bound: one wave per env at 4 waves per SIMD; the HBM "
                        "fraction is reported, not a bound it approaches"}

    roof, roof_other = (route_roof(), schedule_roof()) if route_avg >= sched_avg else \
        (schedule_roof(), route_roof())

    if not args.no_peak_probe:
        mp = measured_peaks(torch)
        roof["measured_peak"] = mp
        if roof["unit"] == "TFLOP/s":
            roof["frac_of_measured"] = roof["achieved"] / mp["mfma_bf16_tflops_random"]
            roof["frac_of_measured_gemm"] = roof["achieved"] / mp["bf16_gemm_tflops"]
        else:
            roof["frac_of_measured"] = roof["achieved"] / mp["copy_gbs_read_plus_write"]

    if cfg.get("net") == "dual":
        net_desc = (f"dual-pathway executor (Sec. 4.2), {cfg['embed_dim']}-d query and role "
                    f"embeddings, {cfg['n_roles']} roles, widths 128/16/16/64/128"
                    + (", value head" if cfg.get("value_head") else ""))
    else:
        net_desc = "MLP " + f"{cfg['feat_dim']}->" + "->".join(map(str, cfg["widths"]))
    line = {
        "metric": METRIC, "value": value, "unit": "env-ticks/s", "n_gpus": 1, "steps": K,
        "warmup": W_, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg["dtype"], "data": "synthetic",
        "config": {"workload": f"{args.config}: {cfg['E']} envs, M={cfg['M']} K={cfg['K']}, "
                               f"lambda={cfg['lam']:g}/tick, qcap {cfg['qcap']}, {net_desc}"
                               f" {cfg['dtype']}, ticks {W_}..{W_ + K - 1} of {T}" +
                               ("; RL rollout: Gumbel-max sampled actions, log-probs, entropies, "
                                "value head" if args.sample else "") +
                               (f"; blackbox models: {len(bb_limits)} of {cfg['E'] * cfg['M']} (env, model) "
                                "pairs rate-limited (60-tick dispatch window, limits uniform in [60, 600]), "
                                "dual update of lambda after every tick" if args.blackbox else ""),
                   "envs": cfg["E"], "requests_per_tick": routed / K, "parallelism": "single GPU",
                   "chains": (f"queries of 1..{cfg['max_steps']} sequential calls (uniform), "
                              "deadlines inherited; requests = calls routed (pending + arrivals)")
                   if chains else None,
                   "launch": "eager" if args.eager else f"one HIP graph of {K} ticks, captured "
                                                        "before the timed region"},
        "routed_req_per_s": routed / (gpu_ms / 1e3),
        "kernels_us": {"route_avg": route_avg * 1e3, "schedule_avg": sched_avg * 1e3,
                       "note": "HIP events around each launch, separate identical pass" + (
                           "; chain pools: each interval also holds a build of the tick's rows "
                           "(im_route and a standalone im_schedule each build them; im_tick once)"
                           if chains else ""),
                       "host_wall_ms_timed": wall * 1e3},
        "roofline": roof,
        "roofline_other_kernel": roof_other,
        "input_gen_s": gen_s,
    }
    if args.blackbox:
        line["lambda_after_timed_ticks"] = lam_after
    if not args.no_cpu_baseline and not args.blackbox:
        line["cpu_baseline"] = cpu_baseline(cfg, W, b, emb_vals, cap, lb, ticks[W_:W_ + K], Q,
                                            args.cpu_seconds)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
