"""Benchmark of the ZeRO P_os+g shard step on one MI355X.

One step = the whole per-rank hot path over one rank's shard: the statistics
kernels (overflow test, sum of squares, clip coefficient), the skip-flag
readback and the fused Adam update that writes the fp16 parameter slice.
Inputs are seeded synthetic shards resident in HBM before timing starts.

Prints ONE JSON line: shard params updated per second (whole job), the step's
HBM rate at 30 algorithmic bytes per parameter, the roofline of the dominant
kernel (the fused update, 28 bytes per parameter, timed with HIP events on its
own stream inside the timed region), and the CPU oracle timed on a bounded
sample of the same workload.

With --optimizer lamb the step is the LAMB shard step over the same shard and
its GPT-2-like layer table (42 algorithmic bytes per parameter: statistics 2,
moments pass 22, apply pass 18); the roofline is the moments pass's.

    python bench.py [--steps K] [--warmup W] [--workload KEY] [--optimizer adam|lamb] [--no-cpu-baseline]
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "shard params updated/sec and achieved HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
STEP_BYTES_PER_PARAM = 30       # grad16 read twice (2+2), master/m/v read+write (24), p16 write (2)
UPDATE_BYTES_PER_PARAM = 28     # the fused update kernel alone
LAMB_STEP_BYTES_PER_PARAM = 42  # statistics 2, moments 14 read + 8 written, apply 12 read + 6 written
LAMB_MOMENTS_BYTES_PER_PARAM = 22
LAMB_APPLY_BYTES_PER_PARAM = 18
DEFAULT_WORKLOAD = "mp16_dp25_100b"
CSRC = os.path.join(ROOT, "paper_1910_02054_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_adam_vec_%s_traffic.txt")   # per workload
LAMB_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_lamb_moments_mp16_dp25_100b_traffic.txt")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("shard_kernels.hpp", "zero_shard.hip")]
LAMB_KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("shard_kernels.hpp", "lamb_kernels.hpp", "zero_lamb.hip")]


def _code_only(text: str) -> str:
    """Source text without comments and blank lines (what the compiler sees of it)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(line.strip() for line in text.splitlines() if line.strip())


def kernel_source_hash() -> str:
    """Hash of the kernels' code and of the production launch policy (the constexpr block of
    zero_shard.hip that fixes block sizes, unrolls, cache policies and occupancy caps);
    comments and layout do not count."""
    h = hashlib.sha256()
    with open(KERNEL_SOURCES[0]) as f:
        h.update(_code_only(f.read()).encode())
    with open(KERNEL_SOURCES[1]) as f:
        host = f.read()
    a, b = host.index("constexpr int kStatsBlock"), host.index("struct Plan {")
    policy = [ln for ln in _code_only(host[a:b]).splitlines() if ln.startswith("constexpr")]
    h.update("\n".join(policy).encode())
    return h.hexdigest()[:16]


def lamb_kernel_source_hash() -> str:
    """Hash of the LAMB kernels' code (with the shared kernel header) and of their
    launch policy (the constexpr block at the top of zero_lamb.hip)."""
    h = hashlib.sha256()
    for path in LAMB_KERNEL_SOURCES[:2]:
        with open(path) as f:
            h.update(_code_only(f.read()).encode())
    with open(LAMB_KERNEL_SOURCES[2]) as f:
        host = f.read()
    a = host.index("constexpr int kLambBlock")
    b = host.index("}  // namespace", a)
    policy = [ln for ln in _code_only(host[a:b]).splitlines() if ln.startswith("constexpr")]
    h.update("\n".join(policy).encode())
    return h.hexdigest()[:16]


def _traffic_from(path, key, source_hash, n):
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    try:
        if kv.get("kernel_source_sha256_16") != source_hash or int(kv["shard_numel"]) != n:
            return None
        return float(kv[key])
    except (KeyError, ValueError):
        return None


def measured_traffic(workload, n):
    """HBM bytes per update launch from the workload's committed counter summary, or None
    when absent, for another shard size, or taken on a different kernel source."""
    return _traffic_from(TRAFFIC_FILE % workload, "update_bytes_per_launch", kernel_source_hash(), n)


def measured_lamb_traffic(n):
    """HBM bytes per LAMB moments launch from the committed counter summary (same rules)."""
    return _traffic_from(LAMB_TRAFFIC_FILE, "moments_bytes_per_launch", lamb_kernel_source_hash(), n)


def _host_cpu():
    """The host's CPU model (from /proc/cpuinfo, if readable) and the cores this process may use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0))}


def cpu_baseline(w, n, theta, m, v, g16, scale, budget_s):
    """The oracle, as it stands, single-threaded on the same shard, 4M-element chunk by chunk
    (each chunk one oracle step: statistics + update), until about budget_s seconds of CPU
    time have been spent (wrapping around the shard if it is done sooner)."""
    import numpy as np
    import oracle
    chunk = 1 << 22
    done, t_used, pos = 0, 0.0, 0
    p16 = np.empty(min(n, chunk), np.uint16)
    while t_used < budget_s:
        b = min(n, pos + chunk)
        th, mm, vv = theta[pos:b].copy(), m[pos:b].copy(), v[pos:b].copy()
        t0 = time.perf_counter()
        oracle.shard_step(g16[pos:b], th, mm, vv, p16[:b - pos], w.lr, w.beta1, w.beta2, w.eps, w.weight_decay,
                          1, scale, w.clip)
        t_used += time.perf_counter() - t0
        done += b - pos
        pos = 0 if b == n else b
    return {"value": done / t_used, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": "%d element-updates of the %d-element shard in 4M-element oracle steps (statistics + "
                      "update), single thread, %.1f s" % (done, n, t_used), **_host_cpu()}


def cpu_baseline_parallel(w, n, theta, m, v, g16, scale, budget_s):
    """The oracle's whole-shard step, unchanged, spread over the host cores this process may
    use: the exact integer statistics of chunks (at most 4M elements) in parallel threads (the oracle is
    C called through ctypes, which releases the interpreter lock), their sum and the shared
    scalars, then the element-wise update of every chunk in parallel with the shared
    multiplier; whole passes over a copy of the shard state until about budget_s seconds."""
    from concurrent.futures import ThreadPoolExecutor
    import numpy as np
    import oracle
    cores = len(os.sched_getaffinity(0))
    chunk = max(1 << 16, min(1 << 22, -(-n // (4 * cores))))  # at least four chunks per thread when n allows
    spans = [(a, min(n, a + chunk)) for a in range(0, n, chunk)]
    cores = min(cores, len(spans))                              # the threads that can have work
    th, mm, vv = theta.copy(), m.copy(), v.copy()
    p16 = np.empty(n, np.uint16)
    hp = oracle.hyper(w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, 1)
    done, t_used, passes = 0, 0.0, 0
    with ThreadPoolExecutor(max_workers=cores) as ex:
        while t_used < budget_s:
            t0 = time.perf_counter()
            parts = list(ex.map(lambda s: oracle.local_stats(g16[s[0]:s[1]]), spans))
            sc = oracle.scalars(sum(q[0] for q in parts), max(q[1] for q in parts), scale, w.clip)
            if not sc.skip:
                list(ex.map(lambda s: oracle.adam(g16[s[0]:s[1]], th[s[0]:s[1]], mm[s[0]:s[1]], vv[s[0]:s[1]],
                                                  p16[s[0]:s[1]], sc.mult, hp), spans))
            t_used += time.perf_counter() - t0
            done += n
            passes += 1
    return {"value": done / t_used, "unit": "params/s", "cores": cores, "kind": "oracle",
            "sample": "%d whole-shard oracle steps of %d elements (exact statistics of all chunks, then the "
                      "update), %d threads, %.1f s" % (passes, n, cores, t_used), **_host_cpu()}


def lamb_cpu_baseline(w, seg, theta, m, v, g16, scale, budget_s):
    """The oracle's LAMB step, as it stands, single-threaded on whole layers of the
    shard in order (a layer's trust ratio needs all of it), until about budget_s
    seconds of CPU time have been spent (wrapping around the shard)."""
    import numpy as np
    import oracle
    done, t_used, k = 0, 0.0, 0
    n_seg = seg.size - 1
    while t_used < budget_s:
        a, b = int(seg[k]), int(seg[k + 1])
        th, mm, vv = theta[a:b].copy(), m[a:b].copy(), v[a:b].copy()
        p16 = np.empty(b - a, np.uint16)
        t0 = time.perf_counter()
        oracle.lamb_step(g16[a:b], th, mm, vv, p16, [0, b - a], w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, 1,
                         scale, w.clip)
        t_used += time.perf_counter() - t0
        done += b - a
        k = (k + 1) % n_seg
    return {"value": done / t_used, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": "%d element-updates over whole layers of the %d-element shard, one oracle LAMB step per "
                      "layer (statistics + moments + exact layer norms + update), single thread, %.1f s"
                      % (done, int(seg[-1]), t_used), **_host_cpu()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle CPU time")
    ap.add_argument("--cpu-parallel-budget", type=float, default=5.0,
                    help="adam only: seconds of the oracle's whole-shard step on all usable host cores "
                         "(reported as cpu_baseline_parallel; 0 = off)")
    ap.add_argument("--step-samples", type=int, default=50,
                    help="after the timed region, time this many further steps one by one with HIP events "
                         "(median, p10, p90 of single steps; 0 = off)")
    ap.add_argument("--profile-every", type=int, default=10,
                    help="time the kernels of one step in this many with HIP events (markers cost GPU time)")
    ap.add_argument("--probe-copy-mib", type=int, default=2048,
                    help="also run the library's copy kernel over this many MiB (counter calibration)")
    ap.add_argument("--optimizer", choices=("adam", "lamb"), default="adam",
                    help="adam: the mixed-precision Adam shard step; lamb: LAMB over the shard's layer table")
    ap.add_argument("--split-phase", action="store_true",
                    help="adam only: each step as zero_shard_stats -> (one rank: the local sum is the global one) "
                         "-> zero_shard_apply, the seam a multi-rank run exchanges 8 bytes at")
    ap.add_argument("--resident", choices=("eager", "graph"), default=None,
                    help="adam only: the resident step (state record and loss scaler on the device, no host "
                         "wait), called eagerly or replayed from a captured HIP graph")
    ap.add_argument("--no-adam-probe", dest="adam_probe", action="store_false",
                    help="adam: skip the update's byte-mix probe (run after the timed steps)")
    ap.add_argument("--no-lamb-probes", dest="lamb_probes", action="store_false",
                    help="lamb only: skip the byte-mix probes of the two passes (run after the timed steps)")
    ap.add_argument("--async-seam", action="store_true",
                    help="with --split-phase: the asynchronous calls (sums in device memory, no host wait; the "
                         "skip flags are checked after the timed region)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the benchmark runs one data-parallel rank on one GPU; --gpus %d is not supported "
              "(the shard step needs no collective on one rank)" % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1910_02054_amd import binding as zb
    from paper_1910_02054_amd import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    w = workloads.WORKLOADS[args.workload]
    lay = zb.zero_partition_layout(w.psi, w.nd, w.rank)
    n = lay.valid_numel
    print("[bench] workload %s n=%d generating inputs" % (w.key, n), file=sys.stderr, flush=True)
    theta, m, v = workloads.initial_state(w, n)
    # two gradient batches, alternated step by step as fresh reduce-scattered gradients would be
    g16s = [workloads.gradients(w, n, k, w.loss_scale) for k in (1, 2)]
    g16 = g16s[0]

    def dev_f32(a):
        return torch.from_numpy(a).to(dev)

    d_theta, d_m, d_v = dev_f32(theta), dev_f32(m), dev_f32(v)
    d_gs = [torch.from_numpy(g.view(np.int16)).to(dev).view(torch.float16) for g in g16s]
    d_p = torch.empty(n, dtype=torch.float16, device=dev)
    stream = torch.cuda.current_stream()
    scaler = zb.Scaler(w.loss_scale)
    lamb = args.optimizer == "lamb"
    seg = plan = None
    if lamb:
        sizes = workloads.model_tensor_sizes(workloads.MODEL_SHAPES[w.key], w.psi)
        seg = workloads.layer_offsets_in(sizes, lay.offset, lay.offset + n)
        plan = zb.LambPlan(seg)

    if args.split_phase and lamb:
        print("bench.py: --split-phase is measured for the Adam step only", file=sys.stderr)
        sys.exit(2)
    if args.async_seam and not args.split_phase:
        print("bench.py: --async-seam needs --split-phase", file=sys.stderr)
        sys.exit(2)
    d_sum = torch.zeros(1, dtype=torch.float64, device=dev)
    d_flags = torch.full((args.warmup + args.steps + max(0, args.step_samples),), -1, dtype=torch.int32,
                         device=dev)
    calls = [0]
    if args.resident and (lamb or args.split_phase):
        print("bench.py: --resident measures the Adam step alone", file=sys.stderr)
        sys.exit(2)
    r_state = graphs = None
    if args.resident:
        r_state = zb.resident_state(dev, w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, w.clip, w.loss_scale,
                                    window=1000)
    if args.resident == "graph":
        # one graph per gradient buffer, replayed alternately; the capture stream gets its workspace
        # (and the arrays their checks) from eager calls on a scratch state first
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        scratch = zb.resident_state(dev, w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, w.clip, w.loss_scale)
        with torch.cuda.stream(cap):
            for d_g in d_gs:
                zb.zero_shard_step_resident(d_g, d_theta, d_m, d_v, d_p, scratch)
        cap.synchronize()
        graphs = []
        for d_g in d_gs:
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=cap):
                zb.zero_shard_step_resident(d_g, d_theta, d_m, d_v, d_p, r_state)
            graphs.append(gr)
        torch.cuda.synchronize()

    # the fused step through the binding's prepared call (arrays and stream resolved once; the
    # library still checks every array on every call), driven by the library's loss scaler
    prepared = zb.ShardStepCall(d_gs, d_theta, d_m, d_v, d_p, w.lr, w.beta1, w.beta2, w.eps, w.weight_decay,
                                w.clip, stream=stream)

    scaled_call = not (args.resident or args.split_phase or lamb)

    def step():
        if scaled_call:
            # one library call per step: the step at the scaler's t and loss scale on gradient
            # buffer t mod 2, then the scaler's update (zero_shard_step_scaled)
            return prepared.scaled(scaler, (scaler.state.applied + 1) & 1)
        d_g = d_gs[scaler.t_next % 2]
        if args.resident == "graph":
            graphs[scaler.t_next % 2].replay()
            scaler.update(False)   # the device record keeps the real schedule; checked after timing
            return 0
        if args.resident == "eager":
            zb.zero_shard_step_resident(d_g, d_theta, d_m, d_v, d_p, r_state, stream=stream)
            scaler.update(False)
            return 0
        if args.async_seam:
            # one rank: the local sum in device memory is the global one; no host wait, so the
            # flag is read after the timed region and t advances as if every step applied
            assert calls[0] < d_flags.numel(), "more async steps than flag slots"
            zb.zero_shard_stats_async(d_g, d_sum, stream=stream)
            zb.zero_shard_apply_async(d_g, d_theta, d_m, d_v, d_p, d_sum, w.lr, w.beta1, w.beta2, w.eps,
                                      w.weight_decay, scaler.t_next, scaler.scale, w.clip,
                                      skipped=d_flags[calls[0]:calls[0] + 1], stream=stream)
            calls[0] += 1
            scaler.update(False)
            return 0
        if args.split_phase:
            local = zb.zero_shard_stats(d_g, stream=stream)
            flag = zb.zero_shard_apply(d_g, d_theta, d_m, d_v, d_p, local, w.lr, w.beta1, w.beta2, w.eps,
                                       w.weight_decay, scaler.t_next, scaler.scale, w.clip, stream=stream)
        elif lamb:
            flag = zb.zero_lamb_step(plan, d_g, d_theta, d_m, d_v, d_p, w.lr, w.beta1, w.beta2, w.eps,
                                     w.weight_decay, scaler.t_next, scaler.scale, w.clip, stream=stream)
        scaler.update(flag)
        return flag

    probe = None
    if args.probe_copy_mib:
        # achievable streaming rate on this GPU: the library's 16-byte copy kernel, timed with
        # events on the stream it runs on (read + write bytes per launch)
        nb = args.probe_copy_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(7)
        dst = torch.empty_like(src)
        for _ in range(3):
            zb.zero_probe_copy(src, dst, nb, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        e0.record(stream)
        for _ in range(reps):
            zb.zero_probe_copy(src, dst, nb, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        cms = e0.elapsed_time(e1) / reps
        probe = {"kernel": "k_probe_copy", "bytes_per_launch": 2 * nb, "ms": cms,
                 "gbps": 2 * nb / (cms * 1e-3) / 1e9}
        del src, dst

    print("[bench] warmup %d" % args.warmup, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    zb.zero_profile_read()
    zb.zero_lamb_profile_read()
    zb.zero_profile_enable(args.profile_every)
    skips = 0
    print("[bench] timing %d steps" % args.steps, file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        skips += step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    zb.zero_profile_enable(False)
    prof = zb.zero_profile_read()
    lprof = zb.zero_lamb_profile_read()
    if args.resident == "graph":
        # replays record no events: the kernels' times come from eager resident steps (the same
        # kernels on the same buffers), on a scratch state record
        zb.zero_profile_enable(1)
        for k in range(20):
            zb.zero_shard_step_resident(d_gs[k % 2], d_theta, d_m, d_v, d_p, scratch, stream=stream)
        torch.cuda.synchronize()
        zb.zero_profile_enable(False)
        prof = zb.zero_profile_read()
    if args.async_seam:
        skips = int((d_flags[:calls[0]] != 0).sum().item())
    if args.resident:
        rs = zb.read_resident_state(r_state)
        skips = int(rs.steps - (rs.t - 1))
    if skips:
        print("bench.py: %d timed steps skipped on overflow; the measurement is invalid" % skips, file=sys.stderr)
        sys.exit(1)

    ms = (t1 - t0) * 1e3 / args.steps
    params_per_s = n / (ms * 1e-3)
    step_q = None
    if args.step_samples > 0:
        # single steps, each bracketed by events on its stream (the markers add a few microseconds
        # of GPU idle per step, so these run a little above ms_per_step of the pipelined region)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.step_samples)]
        extra_skips = 0
        for a, b in evs:
            a.record(stream)
            extra_skips += step()
            b.record(stream)
        torch.cuda.synchronize()
        if args.async_seam:
            extra_skips = int((d_flags[:calls[0]] != 0).sum().item())
        if args.resident:
            rs = zb.read_resident_state(r_state)
            extra_skips = int(rs.steps - (rs.t - 1))
        if extra_skips:
            print("bench.py: a sampled step skipped on overflow; the samples are invalid", file=sys.stderr)
            sys.exit(1)
        qs = np.percentile(np.array([a.elapsed_time(b) for a, b in evs]), [10, 50, 90])
        step_q = {"p10": float(qs[0]), "p50": float(qs[1]), "p90": float(qs[2]), "steps": args.step_samples,
                  "timing": "HIP events around each single step on its stream"}
    if lamb:
        step_gbps = LAMB_STEP_BYTES_PER_PARAM * n / (ms * 1e-3) / 1e9
        k = lprof.steps
        kernel_ms = {"stats_and_finalize": lprof.stats_ms / k, "moments": lprof.moments_ms / k,
                     "layer_sums": lprof.layer_ms / k, "apply": lprof.apply_ms / k, "profiled_steps": k}
        upd_gbps = LAMB_MOMENTS_BYTES_PER_PARAM * n / (kernel_ms["moments"] * 1e-3) / 1e9
        apply_gbps = LAMB_APPLY_BYTES_PER_PARAM * n / (kernel_ms["apply"] * 1e-3) / 1e9
        roof_kernel, traffic = "k_lamb_moments", measured_lamb_traffic(n)
    else:
        step_gbps = STEP_BYTES_PER_PARAM * n / (ms * 1e-3) / 1e9
        kernel_ms = {"stats_and_finalize": prof.stats_ms / prof.steps, "update": prof.update_ms / prof.steps,
                     "profiled_steps": prof.steps}
        upd_gbps = UPDATE_BYTES_PER_PARAM * n / (kernel_ms["update"] * 1e-3) / 1e9
        fused = not (args.resident or args.split_phase)
        if fused and zb.zero_shard_last_step_stats().path == 1:
            # the one-launch small-shard step: statistics and update in one kernel, 28 B/param
            roof_kernel, traffic = "k_small_step", None
        else:
            roof_kernel, traffic = "k_adam_vec", measured_traffic(w.key, n)

    out = {
        "metric": METRIC,
        "value": params_per_s,
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.key, "description": w.description, "psi": w.psi, "nd": w.nd, "rank": w.rank,
                   "shard_numel": n, "parallelism": "one ZeRO P_os+g data-parallel rank (N_d=%d) per GPU" % w.nd},
        "hbm_gbps": step_gbps,
        "hbm_frac_of_peak": step_gbps / HBM_PEAK_GBPS,
        "kernel_ms": kernel_ms,
        "step_ms_quantiles": step_q,
        "roofline": {"bound": "hbm", "kernel": roof_kernel, "achieved": upd_gbps, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": upd_gbps / HBM_PEAK_GBPS,
                     "traffic": traffic},
    }
    if args.resident:
        out["config"].update(path="resident step (device state record and loss scaler, no host wait)" +
                             (", replayed from captured HIP graphs; kernel_ms from 20 eager resident steps"
                              if args.resident == "graph" else ", eager calls"))
    if args.split_phase:
        out["config"].update(path="split phase: zero_shard_stats_async, device-resident global sum, "
                                  "zero_shard_apply_async (no host wait)" if args.async_seam else
                                  "split phase: zero_shard_stats, host-side global sum, zero_shard_apply")
        out["kernel_ms"]["stats_and_finalize"] = None  # timed per apply: only the result-record kernel
    if lamb:
        out["config"].update(optimizer="lamb", layers=int(seg.size - 1))
        out["lamb_apply"] = {"kernel": "k_lamb_apply", "achieved_gbps": apply_gbps,
                             "frac": apply_gbps / HBM_PEAK_GBPS}
    if probe:
        probe["update_frac_of_copy"] = upd_gbps / probe["gbps"]
        out["copy_probe"] = probe
    if not lamb and roof_kernel == "k_adam_vec" and args.adam_probe:
        # the update's byte mix (28 B/param) at its launch shape with trivial arithmetic, in the update's
        # place: each probe launch follows a statistics pass over the gradient, as the update does in
        # a step (so it finds the same part of the gradient in the cache), and is timed alone between
        # two events on the stream, as the profiled updates are.  Runs after every timed step: the
        # probe overwrites the state.
        print("[bench] adam byte-mix probe", file=sys.stderr, flush=True)
        arrs = (d_gs[0], d_theta, d_m, d_v, d_p)
        sums = torch.zeros(1, dtype=torch.float64, device=dev)
        for _ in range(3):
            zb.zero_shard_stats_async(d_gs[0], sums, stream=stream)
            zb.zero_probe_adam_mix(*arrs, stream=stream)
        marks = []
        for _ in range(20):
            zb.zero_shard_stats_async(d_gs[0], sums, stream=stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            zb.zero_probe_adam_mix(*arrs, stream=stream)
            e1.record(stream)
            marks.append((e0, e1))
        torch.cuda.synchronize()
        pms = sum(a.elapsed_time(b) for a, b in marks) / len(marks)
        pg = UPDATE_BYTES_PER_PARAM * n / (pms * 1e-3) / 1e9
        out["adam_probe"] = {"kernel": "k_probe_adam", "probe_ms": pms, "probe_gbps": pg, "update_gbps": upd_gbps,
                             "update_frac_of_probe": upd_gbps / pg,
                             "context": "each launch after a statistics pass over the gradient"}
    if lamb and args.lamb_probes:
        # the byte mixes of the two LAMB passes at their launch shape with trivial arithmetic
        # (after every timed step: the probes overwrite the state), timed with events on the stream
        print("[bench] lamb byte-mix probes", file=sys.stderr, flush=True)
        probes = {}
        for pass_, name, bpp, got in ((0, "moments", LAMB_MOMENTS_BYTES_PER_PARAM, upd_gbps),
                                      (1, "apply", LAMB_APPLY_BYTES_PER_PARAM, apply_gbps)):
            arrs = (d_gs[0], d_theta, d_m, d_v, None) if pass_ == 0 else (None, d_theta, d_m, d_v, d_p)
            for _ in range(3):
                zb.zero_probe_lamb_pass(pass_, *arrs, n=n, stream=stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 20
            e0.record(stream)
            for _ in range(reps):
                zb.zero_probe_lamb_pass(pass_, *arrs, n=n, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            pms = e0.elapsed_time(e1) / reps
            pg = bpp * n / (pms * 1e-3) / 1e9
            probes[name] = {"probe_ms": pms, "probe_gbps": pg, "pass_gbps": got, "pass_frac_of_probe": got / pg}
        out["lamb_probes"] = probes
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        if lamb:
            out["cpu_baseline"] = lamb_cpu_baseline(w, seg, theta, m, v, g16, w.loss_scale, args.cpu_budget)
        else:
            out["cpu_baseline"] = cpu_baseline(w, n, theta, m, v, g16, w.loss_scale, args.cpu_budget)
            if args.cpu_parallel_budget > 0:
                print("[bench] parallel cpu baseline (oracle)", file=sys.stderr, flush=True)
                out["cpu_baseline_parallel"] = cpu_baseline_parallel(w, n, theta, m, v, g16, w.loss_scale,
                                                                     args.cpu_parallel_budget)
    if plan is not None:
        plan.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
