"""Benchmark: one decode step over OPT-shaped decoder-layer linears on one MI355X.

Default workload (the bench line): OPT-6.7B shapes, 32 layers x {QKV [12288,4096],
out [4096,4096], fc1 [16384,4096], fc2 [4096,16384]}, fp16 weights ~N(0, 0.02)
generated from a seeded counter-based generator into pinned host memory, every
linear resident in HBM (CPU fraction 0 from the planner), batch 1, a fresh
x ~N(0, 1) per step already in HBM before the timed region.  A step is
hetegen_decode_step: the four GEMVs of every layer with LayerNorm, value slice,
ReLU and residual fused into them.

Other workloads (--model): opt-13b (layers 0-19 resident, 20-39 streamed from
pinned host with the planner's CPU fraction), opt-30b (all linears in pinned host
memory, planner alpha), opt-66b (bf16, all host, --alpha sweep).  For those the
planner's speeds come from hetegen_probe on this machine, and the JSON line adds the
heterogeneous figures (link and CPU rates, Table-2-style busy fractions).
--placement sched lets the module scheduler (Sec. 4.5) pick the resident linears
under --hbm-budget; --pageable keeps the weights in plain pageable memory, streamed
through the hybrid pin || transfer path (Sec. 4.2-4.3).

The default run (no --model) measures the all-resident OPT-6.7B line above and then,
after freeing it, the same stack at batch 8 in a model created for batch 8 (matrix-core
tiles; `batched` in the same JSON line, 32 steps; --no-batched skips it), the full decode step
at batch 1 with attention over a 512-position KV cache (`kv_step`, 64 decoded tokens after 3 warmup
steps, the paper's end-to-end workload of a 512-token prompt and 64 generated tokens; --no-kv skips it),
and the streamed
half of the metric in the same process (`streamed` in the same JSON line; --no-streamed
skips it): OPT-30B shapes, 48 layers, every linear in
pinned host memory, the planner's CPU fractions refined by the step-level alpha
benchmark, batch 1, 32 steps; the same model with every GPU row streamed (CPU
fraction 0, 2 steps); both against the idle link, one 1 GiB pinned host-to-device copy,
median of 10, measured first.

Prints ONE JSON line.  `value` is the effective weight bandwidth of the whole step
(weight bytes per step / time per step); `ms_per_step` is the decode latency per
token.  `roofline` (all-resident workloads) is the GEMV kernel's algorithmic bytes
per launch (weights, x, bias, y) over its average launch time; every dispatch in
the event-timed region (on the stream the step runs on) is that kernel, so the
average is the region's time over its launches.  Peak: 8 TB/s HBM.
`cpu_baseline` times the oracle (plain C, sequential fp32) on a bounded sample of
the same linears.
"""
import argparse
import ctypes
import hashlib
import json
import mmap
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
OPT = {  # name: (layers, hidden, ffn, dtype, default placement)
    "opt-6.7b": (32, 4096, 16384, 0, "all"),
    "opt-13b": (40, 5120, 20480, 0, "half"),
    "opt-30b": (48, 7168, 28672, 0, "none"),
    "opt-66b": (64, 9216, 36864, 1, "none"),
}
NAMES = ("qkv", "out", "fc1", "fc2")


def shapes(H, F):
    return [(3 * H, H), (H, H), (F, H), (H, F)]


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def kernel_code_sha(path):
    """Hash of a kernel source with comments and blank lines removed (comment edits
    do not change the code the counters were taken on)."""
    lines = []
    for l in open(path).read().splitlines():
        code = l.split("//", 1)[0].rstrip()
        if code:
            lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]


def counter_traffic(model, dt, B):
    """HBM bytes per GEMV launch from the committed counter summary, if it was taken
    on this workload with the current kernel code; else None."""
    name = "gemv_%s_b%d_%s_decode_hbm_counters.md" % ("bf16" if dt == 1 else "f16", B, model.replace("-", ""))
    path = os.path.join(ROOT, "profiles", name)
    src = os.path.join(ROOT, "paper_2403_01164_amd", "csrc", "kernels.hip")
    if not os.path.exists(path):
        return None
    fields = dict(l.split(": ", 1) for l in open(path).read().splitlines() if ": " in l and not l.startswith("#"))
    if fields.get("kernel_code_sha256_16", "").strip() != kernel_code_sha(src):
        return None
    return float(fields["traffic_bytes_per_launch"])



def host_info(torch):
    """Machine the line was measured on: CPU model, cores, NUMA nodes and the GPU's node,
    GPU name and compute units, ROCm / HIP / torch versions (None where unreadable)."""
    def read(path):
        try:
            with open(path) as f:
                return f.read().strip()
        except OSError:
            return None
    cpu, phys = None, set()
    txt = read("/proc/cpuinfo") or ""
    pid = cid = None
    for line in txt.splitlines():
        k, _, v = line.partition(":")
        k, v = k.strip(), v.strip()
        if k == "model name" and cpu is None:
            cpu = v
        elif k == "physical id":
            pid = v
        elif k == "core id":
            cid = v
            phys.add((pid, cid))
    nodes = sorted(int(d[4:]) for d in os.listdir("/sys/devices/system/node")
                   if d.startswith("node") and d[4:].isdigit()) if os.path.isdir("/sys/devices/system/node") else []
    info = {"cpu": cpu, "physical_cores": len(phys) or None, "logical_cpus": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)), "numa_nodes": len(nodes) or None,
            "rocm": read("/opt/rocm/.info/version"), "hip": torch.version.hip, "torch": torch.__version__,
            "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        v = ctypes.c_int(0)
        if hip.hipDriverGetVersion(ctypes.byref(v)) == 0:
            info["hip_driver_version"] = v.value
        if hip.hipRuntimeGetVersion(ctypes.byref(v)) == 0:
            info["hip_runtime_version"] = v.value
    except OSError:
        pass
    info["amdgpu_module"] = read("/sys/module/amdgpu/version")
    try:
        import paper_2403_01164_amd as hg_mod
        info["cpu_share_isa"] = hg_mod.hetegen_cpu_share_isa()
    except Exception:
        pass
    try:
        pr = torch.cuda.get_device_properties(0)
        info["gpu"] = "%s (%s, %d CUs)" % (pr.name, pr.gcnArchName, pr.multi_processor_count)
        bdf = "%04x:%02x:%02x.0" % (pr.pci_domain_id, pr.pci_bus_id, pr.pci_device_id)
        node = read("/sys/bus/pci/devices/%s/numa_node" % bdf)
        info["gpu_pci"] = bdf
        info["gpu_numa_node"] = int(node) if node is not None and node.lstrip("-").isdigit() else None
    except Exception:
        pass
    return info


def single_linear(args, torch, synth, hg):
    """Latency of hetegen_linear on one shape (the single-linear configuration): for each
    CPU fraction and placement, host wall time from the call to the end of the GPU work
    (stream synchronised), median and p10/p90 over the reps; each rep uses the next of
    enough distinct weight copies that they cannot stay in the 256 MB memory-side cache."""
    N, K = (int(v) for v in args.linear.lower().split("x"))
    B, dt = args.batch, 0
    ctx = hg.hetegen_create(0, cpu_threads=args.threads, chunk_bytes=args.chunk_mb << 20, ring_depth=args.ring)
    sptr = torch.cuda.current_stream().cuda_stream
    wb = N * K * 2
    ncopy = max(3, (512 << 20) // wb + 1)
    Wh, Wd = [], []
    bh = hg.hetegen_host_alloc(ctx, N * 2)
    synth.fill_normal_ptr(bh, N, dt, 0, synth.bias_id(0, "qkv"), 0.0, 0.02)
    bd = torch.empty(N, dtype=torch.int16, device="cuda")
    bd.copy_(torch.from_numpy(np.ctypeslib.as_array((ctypes.c_int16 * N).from_address(bh)).copy()))
    for c in range(ncopy):
        w = hg.hetegen_host_alloc(ctx, wb)
        synth.fill_normal_ptr(w, N * K, dt, 0, synth.weight_id(c, "qkv"), 0.0, 0.02)
        Wh.append(w)
        d = torch.empty(N * K, dtype=torch.int16, device="cuda")
        d.copy_(torch.from_numpy(np.ctypeslib.as_array((ctypes.c_int16 * (N * K)).from_address(w)).copy()))
        Wd.append(d)
    x = torch.from_numpy(synth.normal((B, K), dt, 0, synth.act_id(0)).view(np.int16)).cuda()
    y = torch.empty((B, N), dtype=torch.float32, device="cuda")
    probe = hg.hetegen_probe(ctx, Wh[0], N, K, dt, B, 5)
    log("single linear [%d,%d] B=%d: %d weight copies (%.0f MB); probe %s" %
        (N, K, B, ncopy, ncopy * wb / 1e6, {k: round(v / 1e9, 1) for k, v in probe.items()}))
    # fixed costs of a synchronous call that no kernel work removes: the launch round trip
    # (empty kernel + stream synchronisation, timed in C) and this binding's own overhead (the
    # same call refused by its first argument check: ctypes marshalling, no GPU work)
    launch_us = hg.hetegen_probe_launch(ctx, 1000, sptr)
    nb = 20000
    c0 = time.perf_counter()
    for _ in range(nb):
        hg.hetegen_linear_status(ctx, x.data_ptr(), B, K, Wh[0], 0, N, dt, bh, bd.data_ptr(), 2.0, y.data_ptr(),
                                 hg.F32, sptr)
    binding_us = (time.perf_counter() - c0) / nb * 1e6
    log("launch round trip %.2f us, binding %.2f us per call" % (launch_us, binding_us))
    rows = []
    for resident in (True, False):
        for alpha in (0.0, 0.25, 0.5, 1.0):
            def call(c):
                hg.hetegen_linear(ctx, x.data_ptr(), B, K, Wh[c], Wd[c].data_ptr() if resident else 0, N, dt, bh,
                                  bd.data_ptr(), alpha, y.data_ptr(), hg.F32, sptr)
            for c in range(10):
                call(c % ncopy)
            torch.cuda.synchronize()
            ts = []
            for r in range(args.linear_reps):
                t0 = time.perf_counter()
                call((r + 10) % ncopy)
                torch.cuda.synchronize()
                ts.append((time.perf_counter() - t0) * 1e6)
            ts.sort()
            q = lambda f: ts[min(len(ts) - 1, int(f * (len(ts) - 1) + 0.5))]
            n_cpu = min(N, int(np.floor(alpha * N + 0.5)))
            # roofline of the configuration: HBM for resident GPU rows, the link for streamed
            # ones, host reads for CPU rows (Eq. 4 balance when split)
            v_g = HBM_PEAK_GBPS * 1e9 if resident else 1.0 / (1.0 / probe["h2d_Bps"] + 1.0 / probe["hbm_gemv_Bps"])
            if n_cpu == 0:
                work_us, bound = wb / v_g * 1e6, ("hbm" if resident else "h2d")
            elif n_cpu == N:
                work_us, bound = wb / probe["cpu_Bps"] * 1e6, "cpu"
            else:
                work_us = max(n_cpu * K * 2 / probe["cpu_Bps"], (N - n_cpu) * K * 2 / v_g) * 1e6
                bound = "cpu+" + ("hbm" if resident else "h2d")
            # the latency floor: the work at those rates plus the binding and one launch round
            # trip per hand-off (the final synchronisation; with CPU rows also x to the host)
            trips = 1 if n_cpu == 0 else 2
            floor_us = work_us + binding_us + trips * launch_us
            rows.append({"alpha_cpu": alpha, "resident": resident, "median_us": round(q(0.5), 2),
                         "p10_us": round(q(0.1), 2), "p90_us": round(q(0.9), 2),
                         "GBps": round(wb / (q(0.5) * 1e-6) / 1e9, 2), "bound": bound,
                         "work_floor_us": round(work_us, 2), "launch_round_trips": trips,
                         "floor_us": round(floor_us, 2), "frac_of_floor": round(floor_us / q(0.5), 4),
                         "frac_of_work_floor": round(work_us / q(0.5), 4)})
            log("alpha %.2f %s: median %.1f us (p10 %.1f, p90 %.1f), floor %.1f us (%s work %.1f + %d trips)" %
                (alpha, "resident" if resident else "streamed", q(0.5), q(0.1), q(0.9), floor_us, bound, work_us,
                 trips))
    head = rows[0]
    cpu_base = None
    if not args.no_cpu_baseline:
        # the oracle on the same linear and weight copies, with the default OpenMP team and
        # single-threaded, about 3 s each
        import oracle
        xh = synth.normal((B, K), dt, 0, synth.act_id(0))
        yh = np.empty((B, N), np.float32)

        def oracle_rate():
            n, t = 0, 0.0
            while t < 3.0:
                c0 = time.perf_counter()
                oracle.linear_ptr(xh.ctypes.data, K, B, K, Wh[n % ncopy], N, dt, bh, yh)
                t += time.perf_counter() - c0
                n += 1
            return n, t, n * wb / t / 1e9
        gomp = ctypes.CDLL("libgomp.so.1")
        threads = gomp.omp_get_max_threads()
        n_all, t_all, v_all = oracle_rate()
        gomp.omp_set_num_threads(1)
        n_one, t_one, v_one = oracle_rate()
        gomp.omp_set_num_threads(threads)
        cpu_base = {"value": round(wb / (t_all / n_all) / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
                    "sample": "%d calls on the %d weight copies, %.1f s" % (n_all, ncopy, t_all),
                    "us_per_call": round(t_all / n_all * 1e6, 1),
                    "single_thread": {"value": round(v_one, 3), "unit": "GB/s", "us_per_call": round(t_one / n_one * 1e6, 1),
                                      "sample": "%d calls, %.1f s" % (n_one, t_one)}}
        log("oracle: %.2f GB/s on %d threads, %.2f GB/s single-threaded" % (v_all, threads, v_one))
    print(json.dumps({
        "metric": "single-linear latency (us per call, host wall to end of GPU work)",
        "value": head["median_us"], "unit": "us", "n_gpus": 1, "steps": args.linear_reps, "warmup": 10,
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic: seeded N(0,0.02) weights and bias, N(0,1) x",
        "config": {"workload": "single Linear [%d,%d] fp16, batch %d, CPU fractions 0/.25/.5/1, resident and "
                               "streamed; %d weight copies rotated (%.0f MB)" % (N, K, B, ncopy, ncopy * wb / 1e6)},
        "probe_GBps": {k: round(v / 1e9, 2) for k, v in probe.items()},
        "launch_round_trip_us": round(launch_us, 2), "binding_us_per_call": round(binding_us, 2),
        "results": rows, "cpu_baseline": cpu_base, "host": host_info(torch)}))
    for w in Wh:
        hg.hetegen_host_free(ctx, w)
    hg.hetegen_host_free(ctx, bh)
    hg.hetegen_destroy(ctx)

def table2_linear(args, torch, synth, hg):
    """Per-resource busy fractions of one heterogeneous linear, the analogue of Table 2 (Sec. 5.2:
    OPT-13B, the first MLP linear, fc1 [20480, 5120]): at the planner's CPU fraction refined by
    the alpha benchmark of this linear (Sec. 4.4), the share of the linear's wall time during which
    the CPU share runs, the link copies chunks, the pin team stages pageable chunks and the GPU
    runs GEMVs (events around each copy and launch).  Weights pinned, then pageable (the paper's
    setting: its weights are pinned chunk by chunk at run time).  Two weight copies are rotated
    so the CPU share reads DRAM, not cache."""
    N, K = (int(v) for v in args.table2.lower().split("x"))
    B, dt, ncopy = args.batch, 0, 2
    ctx = hg.hetegen_create(0, cpu_threads=args.threads, chunk_bytes=args.chunk_mb << 20, ring_depth=args.ring,
                            pin_threads=args.pin_threads, pin_ring=args.pin_ring)
    s = torch.cuda.current_stream().cuda_stream
    wb = N * K * 2
    Wp, maps, Wq = [], [], []
    for c in range(ncopy):
        w = hg.hetegen_host_alloc(ctx, wb)
        synth.fill_normal_ptr(w, N * K, dt, 0, synth.weight_id(c, "fc1"), 0.0, 0.02)
        Wp.append(w)
        mm = mmap.mmap(-1, wb)
        if hasattr(mm, "madvise") and hasattr(mmap, "MADV_HUGEPAGE"):
            mm.madvise(mmap.MADV_HUGEPAGE)
        maps.append(mm)
        q = ctypes.addressof(ctypes.c_char.from_buffer(mm))
        ctypes.memmove(q, w, wb)
        Wq.append(q)
    bh = hg.hetegen_host_alloc(ctx, N * 2)
    synth.fill_normal_ptr(bh, N, dt, 0, synth.bias_id(0, "fc1"), 0.0, 0.02)
    bd = torch.from_numpy(np.ctypeslib.as_array((ctypes.c_int16 * N).from_address(bh)).copy()).cuda()
    x = torch.from_numpy(synth.normal((B, K), dt, 0, synth.act_id(0)).view(np.int16)).cuda()
    y = torch.empty((B, N), dtype=torch.float32, device="cuda")
    rows = []
    for kind, W in (("pinned", Wp), ("pageable", Wq)):
        pr = hg.hetegen_probe(ctx, W[0], N, K, dt, B, 3, hg.PROBE_CONCURRENT if kind == "pinned" else 0)
        a0 = hg.hetegen_layer_plan([(N, K, dt, 0)], [(pr["cpu_Bps"], pr["h2d_Bps"], pr["hbm_gemv_Bps"],
                                                       pr["pin_Bps"])])[0]
        a1, crossed = hg.hetegen_alpha_benchmark(ctx, x.data_ptr(), B, K, W[0], N, dt, bh, bd.data_ptr(),
                                                 y.data_ptr(), a0, 0.05, 0.01, 2, 2, s)

        def call(i):
            hg.hetegen_linear(ctx, x.data_ptr(), B, K, W[i % ncopy], 0, N, dt, bh, bd.data_ptr(), a1, y.data_ptr(),
                              hg.F32, s)
        for i in range(3):
            call(i)
        torch.cuda.synchronize()
        ts = []
        for i in range(args.table2_reps):
            t0 = time.perf_counter()
            call(i)
            torch.cuda.synchronize()
            ts.append((time.perf_counter() - t0) * 1e3)
        ts.sort()
        hg.hetegen_set_profiling(ctx, 1)
        hg.hetegen_get_profile(ctx, reset=True)
        for i in range(args.table2_reps):
            call(i)
        torch.cuda.synchronize()
        prof = hg.hetegen_get_profile(ctx, reset=True)
        hg.hetegen_set_profiling(ctx, 0)
        wall = prof["wall_ms"]
        n_cpu = min(N, int(np.floor(a1 * N + 0.5)))
        v_com = min(pr["h2d_Bps"], pr["pin_Bps"]) if pr["pin_Bps"] > 0 else pr["h2d_Bps"]
        v_g = 1.0 / (1.0 / v_com + 1.0 / pr["hbm_gemv_Bps"])
        ideal_ms = wb / (pr["cpu_Bps"] + v_g) * 1e3
        row = {"weights": kind, "alpha_cpu_closed_form": round(a0, 4), "alpha_cpu": round(a1, 4),
               "alpha_bench_crossed": crossed, "cpu_rows": n_cpu, "gpu_rows": N - n_cpu,
               "median_ms": round(ts[len(ts) // 2], 3), "p10_ms": round(ts[len(ts) // 10], 3),
               "p90_ms": round(ts[(9 * len(ts)) // 10], 3), "profiled_ms": round(wall / args.table2_reps, 3),
               "eq4_ideal_ms": round(ideal_ms, 3), "frac_of_ideal": round(ideal_ms / ts[len(ts) // 2], 4),
               "busy_frac": {"cpu": round(prof["cpu_ms"] / wall, 4), "io": round(prof["h2d_ms"] / wall, 4),
                             "pin": round(prof["pin_ms"] / wall, 4), "gpu": round(prof["gpu_ms"] / wall, 4)},
               "probe_GBps": {k: round(v / 1e9, 2) for k, v in pr.items()}}
        rows.append(row)
        log("table 2, %s weights: alpha %.4f (closed form %.4f), %.2f ms per call, busy %s" %
            (kind, a1, a0, ts[len(ts) // 2], row["busy_frac"]))
    print(json.dumps({
        "metric": "per-resource busy fraction of one heterogeneous linear (Table 2 analogue)",
        "value": rows[-1]["busy_frac"]["cpu"], "unit": "fraction of the linear's wall time", "n_gpus": 1,
        "steps": args.table2_reps, "warmup": 3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic: seeded N(0,0.02) weights and bias, N(0,1) x",
        "config": {"workload": "one heterogeneous linear [%d,%d] fp16 (OPT-13B fc1 shape), batch %d, planner alpha "
                               "refined by the alpha benchmark; weights pinned, then pageable; %d weight copies "
                               "rotated" % (N, K, B, ncopy)},
        "results": rows, "paper_table2": {"cpu": 0.978, "io": 0.969, "pin": 0.724, "gpu": 0.001},
        "host": host_info(torch)}), flush=True)
    for w in Wp:
        hg.hetegen_host_free(ctx, w)
    hg.hetegen_host_free(ctx, bh)
    hg.hetegen_destroy(ctx)


def mfma_splits(rows, K, cus):
    """Splits of the sum over K in the matrix-core GEMV on a device of `cus` compute units
    (the library's rule: unsplit unless one workgroup per 16-row tile loads the units more
    than 1.15x unevenly; then the fewest splits of at least 32 k-tiles that do not, or the
    most even)."""
    def uneven(wgs):
        return -(-wgs // cus) * cus / wgs
    rt, kt = -(-rows // 16), -(-K // 32)
    best, best_u = 1, uneven(rt)
    if best_u <= 1.15:
        return 1
    g = 2
    while g <= 8 and kt // g >= 32:
        u = uneven(rt * g)
        if u <= 1.15:
            return g
        if u < best_u:
            best, best_u = g, u
        g *= 2
    return best


def ln_partials_on(H):
    """Whether tiled models of hidden size H normalise the inputs of qkv (after layer 0) and
    fc1 from the LayerNorm partials of the out / fc2 before them (the library's rule: H <= 6144
    unless HETEGEN_LN_PARTIALS forces it)."""
    env = os.environ.get("HETEGEN_LN_PARTIALS")
    return {"0": False, "1": True}.get(env, H <= 6144)


def gemv_label(B, H, F, dt, tiled, partials=True, cus=256):
    """GEMV kernels an all-resident eager step at batch B runs (the library's dispatch rules;
    tiled: the step runs the tile-ordered copy of the weights; partials: with LayerNorm
    partials between its matrix-core linears; cus: the device's compute units)."""
    t = "BF16" if dt == 1 else "F16"
    if tiled:
        parts = {}
        for name, (n, k) in zip(NAMES, shapes(H, F)):
            g = mfma_splits(n, k, cus)
            wgs = -(-n // 16) * g
            kmajor = wgs % cus == 0 and wgs // cus <= 4  # the library's tile order rule
            split = ("" if g == 1 else " (K split %d)" % g) + (" k-major" if kmajor else "")
            u = 4 if g > 1 else 8  # tiles per request, no LayerNorm
            if partials and name in ("qkv", "fc1"):
                uln = 8 if (g == 1 and B == 1 and -(-wgs // cus) <= 3) else 4  # with the LayerNorm prologue
                key = "gemv_mfma_kernel<%s,%d,%d,LayerNorm from partials>%s" % (t, B, uln, split)
                parts.setdefault(key, []).append("qkv after layer 0" if name == "qkv" else name)
                if name == "qkv":
                    key = "gemv_mfma_kernel<%s,%d,%d>%s" % (t, B, u, split)
                    parts.setdefault(key, []).append("layer 0's qkv")
                continue
            key = "gemv_mfma_kernel<%s,%d,%d>%s" % (t, B, u, split)
            parts.setdefault(key, []).append(name)
        ni = -(-H // 2048)
        ni = ni if ni <= 5 else 8
        return " + ".join("%s: %s" % (k, ", ".join(v)) for k, v in parts.items()) + \
            " + layernorm_regs_kernel<%s,%d> before %s" % (t, ni, "layer 0's qkv" if partials else "qkv and fc1")
    if B == 1:
        if H % 512 == 0 and H // 512 in (1, 2, 4, 5, 8, 10, 14):
            return "gemv_ln1_kernel<%s,%d> (qkv, fc1) + gemv_x1_kernel<%s,4,1> (out, fc2)" % (t, H // 512, t)
        return "gemv_kernel<%s,1,1,8> (qkv, fc1) + gemv_x1_kernel<%s,4,1> (out, fc2)" % (t, t)
    if B == 2:
        return "gemv_kernel<%s,2,1,8> (qkv, fc1) + gemv_x1_kernel<%s,4,2> (out, fc2)" % (t, t)
    return "gemv_kernel<%s,%d,1,4> (qkv, out, fc1, fc2; LayerNorm fused in qkv and fc1)" % (t, B)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--model", default=None, choices=sorted(OPT),
                    help="one workload (default: the OPT-6.7B all-resident line, followed by the streamed leg "
                         "below unless --no-streamed)")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--max-batch", type=int, default=0,
                    help="largest batch the model is created for (0: --batch); from 2 on its resident weights "
                         "are kept in matrix-core tile order (and row-major too, for batch 1, when both fit)")
    ap.add_argument("--layers", type=int, default=0,
                    help="run only the first N decoder layers (0: all); reported in config")
    ap.add_argument("--placement", choices=("all", "half", "none", "sched"), default=None,
                    help="HBM-resident modules: all, the first half of the layers, none, or the module "
                         "scheduler's choice under --hbm-budget (Sec. 4.5) (default per model)")
    ap.add_argument("--hbm-budget", type=float, default=None,
                    help="GB of HBM for resident weights with --placement sched (default: half the weights)")
    ap.add_argument("--alpha", type=float, default=None,
                    help="fixed CPU fraction for every streamed linear (default: the planner's)")
    ap.add_argument("--alpha-sweep", default=None,
                    help="comma-separated CPU fractions for the streamed linears, each timed after the main "
                         "measurement (e.g. 0,0.1,0.2,0.3,0.4,0.5)")
    ap.add_argument("--sweep-steps", type=int, default=2)
    ap.add_argument("--no-alpha-bench", dest="alpha_bench", action="store_false",
                    help="keep the closed-form CPU fractions (default for streamed linears: refine them with the "
                         "step-level alpha benchmark, Sec. 4.4, and also time the closed-form fractions)")
    ap.add_argument("--threads", type=int, default=0, help="CPU-share threads (0: the OpenMP default count, OMP_NUM_THREADS)")
    ap.add_argument("--pageable", action="store_true",
                    help="weights in plain pageable host memory (transparent huge pages), streamed through the "
                         "hybrid pin || transfer path (Sec. 4.2); biases stay pinned")
    ap.add_argument("--pin-threads", type=int, default=0, help="pin team threads for --pageable (0: library default)")
    ap.add_argument("--pin-ring", type=int, default=0, help="pinned staging buffers for --pageable (0: default)")
    ap.add_argument("--chunk-mb", type=int, default=32)
    ap.add_argument("--ring", type=int, default=8)
    ap.add_argument("--exec", choices=("auto", "persistent", "graph", "eager"), default="auto",
                    help="execution mode of an all-resident step")
    ap.add_argument("--context", type=int, default=0,
                    help="full decode steps with attention over a KV cache holding this many earlier positions "
                         "(synthetic keys/values standing in for a prefill; Sec. 2.1, Eq. 1); 0: the GEMV-only "
                         "step (empty-cache attention)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="end with one plain 256 MiB device-to-device copy, the reference dispatch for "
                         "scaling HBM byte counters")
    ap.add_argument("--linear", default=None, metavar="NxK",
                    help="instead of a decode step: latency of one heterogeneous linear [N,K] (fp16, --batch) at "
                         "CPU fractions 0, .25, .5, 1, resident and streamed, over --linear-reps calls that rotate "
                         "weight copies totalling > 512 MB (prints its own JSON line)")
    ap.add_argument("--linear-reps", type=int, default=200)
    ap.add_argument("--table2", default=None, metavar="NxK",
                    help="instead of a decode step: busy fractions of one heterogeneous linear (Table 2 analogue; "
                         "OPT-13B fc1 is 20480x5120), pinned and pageable weights (prints its own JSON line)")
    ap.add_argument("--table2-reps", type=int, default=20)
    ap.add_argument("--no-streamed", action="store_true",
                    help="default run only: skip the streamed leg (OPT-30B shapes, every linear in pinned host "
                         "memory, planner alpha refined by the step-level benchmark, batch 1)")
    ap.add_argument("--streamed-steps", type=int, default=32, help="timed steps of the streamed leg")
    ap.add_argument("--no-batched", action="store_true",
                    help="default run only: skip the batched leg (the OPT-6.7B stack at batch 8 on the "
                         "matrix-core GEMV, in a model created for batch 8)")
    ap.add_argument("--batched-steps", type=int, default=32, help="timed steps of the batched leg")
    ap.add_argument("--no-kv", action="store_true",
                    help="default run only: skip the kv leg (the OPT-6.7B stack at batch 1 with attention over "
                         "a 512-position KV cache)")
    ap.add_argument("--kv-steps", type=int, default=64, help="timed steps of the kv leg")
    ap.add_argument("--all-streamed-steps", type=int, default=None,
                    help="streamed workloads: also time this many steps with every GPU row streamed (CPU "
                         "fraction 0), against the idle link (default: 2 in the streamed leg, 0 otherwise)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: there is no multi-GPU path (the heterogeneous "
              "linear would shard by output rows across GPUs); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    import paper_2403_01164_amd as hg

    torch.cuda.set_device(0)
    if args.linear:
        single_linear(args, torch, synth, hg)
        return
    if args.table2:
        table2_linear(args, torch, synth, hg)
        return
    # the streamed leg belongs to the default line: no workload option given
    default_run = (args.model is None and args.batch == 1 and not args.layers and args.placement is None and
                   args.context == 0 and not args.pageable and args.alpha is None)
    if args.model is None:
        args.model = "opt-6.7b"
    result = decode_workload(args, torch, synth, hg)
    if default_run and not args.no_batched:
        result["batched"] = batched_leg(args, torch, synth, hg)
    if default_run and not args.no_kv:
        result["kv_step"] = kv_leg(args, torch, synth, hg)
    if default_run and not args.no_streamed:
        result["streamed"] = streamed_leg(args, torch, synth, hg)
    print(json.dumps(result), flush=True)


def kv_leg(args, torch, synth, hg):
    """The full decode step (Sec. 2.1, Eq. 1): the same OPT-6.7B stack at batch 1 with attention
    over a KV cache of 512 earlier positions (synthetic keys and values standing in for a
    prefill), every linear resident."""
    import copy
    a = copy.copy(args)
    a.model, a.batch, a.max_batch, a.layers, a.placement, a.hbm_budget = "opt-6.7b", 1, 0, 0, "all", None
    a.alpha, a.alpha_sweep, a.pageable, a.context, a.exec = None, None, False, 512, "auto"
    a.steps, a.warmup, a.no_cpu_baseline, a.copy_calibration = args.kv_steps, 3, True, False
    log("kv leg: OPT-6.7B shapes, all linears resident, batch 1, 512-position KV cache, %d steps" % a.steps)
    r = decode_workload(a, torch, synth, hg)
    return {"workload": r["config"]["workload"], "context": 512, "steps": r["steps"], "warmup": r["warmup"],
            "ms_per_step": r["ms_per_step"], "step_ms_p10_p50_p90": r.get("step_ms_p10_p50_p90"),
            "kv": r.get("kv"), "roofline": r["roofline"]}


def batched_leg(args, torch, synth, hg):
    """The matrix-core half of the resident path, after the headline line has freed its
    memory: the same OPT-6.7B-shaped stack (32 layers, fp16, every linear resident) in a model
    created for batch 8, stepped at batch 8; tokens per second count all 8 rows."""
    import copy
    a = copy.copy(args)
    a.model, a.batch, a.max_batch, a.layers, a.placement, a.hbm_budget = "opt-6.7b", 8, 8, 0, "all", None
    a.alpha, a.alpha_sweep, a.pageable, a.context, a.exec = None, None, False, 0, "auto"
    a.steps, a.warmup, a.no_cpu_baseline, a.copy_calibration = args.batched_steps, 3, True, False
    log("batched leg: OPT-6.7B shapes, all linears resident, batch 8, %d steps" % a.steps)
    r = decode_workload(a, torch, synth, hg)
    return {"workload": r["config"]["workload"], "batch": 8, "steps": r["steps"], "warmup": r["warmup"],
            "ms_per_step": r["ms_per_step"], "tokens_per_s": round(8 * 1e3 / r["ms_per_step"], 1),
            "step_ms_p10_p50_p90": r.get("step_ms_p10_p50_p90"), "weight_GBps": r["value"],
            "weight_layouts": r["config"].get("weight_layouts"), "roofline": r["roofline"]}


def streamed_leg(args, torch, synth, hg):
    """The streamed half of the metric, after the headline line has freed its memory:
    OPT-30B shapes (48 layers, 59.2 GB of fp16 weights), every linear in pinned host
    memory, CPU fractions from the planner refined by the step-level alpha benchmark,
    batch 1; plus the all-streamed point (CPU fraction 0) and the idle link."""
    import copy
    a = copy.copy(args)
    a.model, a.batch, a.layers, a.placement, a.hbm_budget = "opt-30b", 1, 0, "none", None
    a.alpha, a.alpha_sweep, a.alpha_bench, a.pageable, a.context, a.exec = None, None, True, False, 0, "auto"
    a.steps, a.warmup, a.no_cpu_baseline, a.copy_calibration = args.streamed_steps, 2, True, False
    a.all_streamed_steps = 2 if args.all_streamed_steps is None else args.all_streamed_steps
    log("streamed leg: OPT-30B shapes, all linears in pinned host memory, batch 1, %d steps" % a.steps)
    r = decode_workload(a, torch, synth, hg)
    h = r["hetero"]
    keep = {"workload": r["config"]["workload"], "steps": r["steps"], "warmup": r["warmup"],
            "ms_per_token": r["ms_per_step"], "step_ms_p10_p50_p90": r["step_ms_p10_p50_p90"],
            "weight_GBps": r["value"], "weight_bytes_per_step": r["config"]["weight_bytes_per_step"],
            "roofline": h["roofline"], "ideal_ms_per_step": h["ideal_ms_per_step"],
            "frac_of_ideal": h["frac_of_ideal"], "busy_frac": h["busy_frac"],
            "link_idle_GBps": h["link_idle_GBps"], "h2d_GBps_over_step": h["h2d_GBps_over_step"],
            "cpu_GBps_over_step": h["cpu_GBps_over_step"], "alpha_cpu_by_linear": h["alpha_cpu_by_linear"],
            "probe_GBps": h["probe_GBps"]}
    for k in ("all_streamed", "alpha_benchmark"):
        if k in r:
            keep[k] = r[k]
    return keep


def decode_workload(args, torch, synth, hg):
    """One decode-step workload (args.model, args.batch, placement ...); returns the result dict
    after freeing every buffer it allocated."""
    L, H, F, dt, placement = OPT[args.model]
    L_full = L
    if args.layers:
        L = min(L, args.layers)
    placement = args.placement or placement
    B = args.batch
    ctx = hg.hetegen_create(0, cpu_threads=args.threads, chunk_bytes=args.chunk_mb << 20, ring_depth=args.ring,
                            pin_threads=args.pin_threads, pin_ring=args.pin_ring)
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    res_layers = L if placement == "all" else L // 2 if placement == "half" else 0
    link_idle = None
    if placement != "all":
        # idle host-to-device link, before the weights take the pinned memory: one 1 GiB
        # pinned copy, median of 10 (the denominator of the streamed path's roofline)
        link_idle = hg.hetegen_probe_link(ctx, 1 << 30, 10)
        log("idle link: %.2f GB/s (1 GiB pinned host-to-device copy, median of 10)" % (link_idle / 1e9))

    # ---- synthetic OPT-shaped weights in pinned (or pageable) host memory ----
    t0 = time.time()
    W, b, shp = [], [], []
    maps = []
    for l in range(L):
        for i, (n, k) in enumerate(shapes(H, F)):
            if args.pageable:
                mm = mmap.mmap(-1, n * k * 2)
                if hasattr(mm, "madvise") and hasattr(mmap, "MADV_HUGEPAGE"):
                    mm.madvise(mmap.MADV_HUGEPAGE)
                maps.append(mm)
                w = ctypes.addressof(ctypes.c_char.from_buffer(mm))
            else:
                w = hg.hetegen_host_alloc(ctx, n * k * 2)
            bb = hg.hetegen_host_alloc(ctx, n * 2)
            synth.fill_normal_ptr(w, n * k, dt, 0, synth.weight_id(l, NAMES[i]), 0.0, 0.02)
            synth.fill_normal_ptr(bb, n, dt, 0, synth.bias_id(l, NAMES[i]), 0.0, 0.02)
            W.append(w)
            b.append(bb)
            shp.append((n, k))
    wbytes = sum(n * k * 2 for n, k in shp)
    log("generated %.3f GB of weights in %.1f s" % (wbytes / 1e9, time.time() - t0))

    resident = [1 if (i // 4) < res_layers else 0 for i in range(4 * L)]
    streamed = [i for i in range(4 * L) if not resident[i]]

    # ---- planner: speeds per shape from the probe (streamed linears only) ----
    bws = [(1.0, 1.0, 1.0, 0.0)] * (4 * L)
    probe = {}
    schedule = None
    if streamed:
        last = 4 * (L - 1)
        for m in range(4):
            n, k = shp[last + m]
            t0 = time.time()
            probe[NAMES[m]] = hg.hetegen_probe(ctx, W[last + m], n, k, dt, B, 3, hg.PROBE_CONCURRENT)
            p = probe[NAMES[m]]
            log("probe %s [%d,%d]: V_CPU %.1f GB/s, V_COM %.1f GB/s, V_GPU %.0f GB/s, V_PIN %.1f GB/s (%.1f s)" %
                (NAMES[m], n, k, p["cpu_Bps"] / 1e9, p["h2d_Bps"] / 1e9, p["hbm_gemv_Bps"] / 1e9,
                 p["pin_Bps"] / 1e9, time.time() - t0))
        # the host is shared with other tenants: a probe whose CPU rate falls below 3/4 of the
        # best linear's was slowed while it ran (the shapes' CPU rates differ by far less), so it
        # is taken again, up to twice, keeping the faster result; the planner and the Eq. 4 ideal
        # both read these rates
        for m in range(4):
            for again in range(2):
                best = max(probe[q]["cpu_Bps"] for q in NAMES)
                if probe[NAMES[m]]["cpu_Bps"] >= 0.75 * best:
                    break
                n, k = shp[last + m]
                p = hg.hetegen_probe(ctx, W[last + m], n, k, dt, B, 3, hg.PROBE_CONCURRENT)
                log("probe %s again: V_CPU %.1f GB/s (was %.1f)" %
                    (NAMES[m], p["cpu_Bps"] / 1e9, probe[NAMES[m]]["cpu_Bps"] / 1e9))
                if p["cpu_Bps"] > probe[NAMES[m]]["cpu_Bps"]:
                    probe[NAMES[m]] = p
        bws = [tuple(probe[NAMES[i % 4]][f] for f in ("cpu_Bps", "h2d_Bps", "hbm_gemv_Bps", "pin_Bps"))
               for i in range(4 * L)]
    # fresh input per step, resident in HBM before timing
    nstep = args.warmup + args.steps
    xs = torch.empty((nstep, B, H), dtype=torch.int16, device="cuda")
    for t in range(nstep):
        xs[t] = torch.from_numpy(synth.normal((B, H), dt, 0, synth.act_id(t)).view(np.int16))
    out = torch.empty((2, B, H), dtype=torch.int16, device="cuda")

    if placement == "sched":
        # module scheduler (Sec. 4.5, Eq. 13): T_CPU of each module is its benchmarked time
        # in heterogeneous mode, against the HBM bytes of its resident copy.  A model with
        # every linear heterogeneous at the planned split runs a few steps, and each linear's
        # share of the calling thread's critical path (hetegen_model_linear_ms: its CPU share,
        # the waits around it and the hand-offs) is averaged over them; the fixed cost of a
        # hand-off makes small modules gain more per byte than their CPU time alone says.
        a_all = hg.hetegen_layer_plan([(n, k, dt, 0) for n, k in shp], bws)
        tmp = hg.hetegen_model_create(ctx, L, H, F, dt, W, b, a_all, [0] * (4 * L), max(B, args.max_batch, 1))
        t_het, nb = [0.0] * (4 * L), 3
        for t in range(nb + 1):  # the first step warms up
            hg.hetegen_decode_step(ctx, tmp, xs[t % nstep].data_ptr(), out[0].data_ptr(), B, sptr)
            torch.cuda.synchronize()
            if t > 0:
                t_het = [a + ms * 1e-3 / nb for a, ms in zip(t_het, hg.hetegen_model_linear_ms(tmp, 4 * L))]
        hg.hetegen_model_destroy(ctx, tmp)
        mem = [float(n * k * 2) for n, k in shp]
        budget = args.hbm_budget * 1e9 if args.hbm_budget is not None else sum(mem) / 2
        resident, used = hg.hetegen_module_schedule(t_het, mem, [i // 4 for i in range(4 * L)], budget)
        streamed = [i for i in range(4 * L) if not resident[i]]
        schedule = {"T_is": "benchmarked: each linear's time with every linear heterogeneous, mean of %d steps" % nb,
                    "hbm_budget_GB": round(budget / 1e9, 3), "resident_GB": round(used / 1e9, 3),
                    "resident_modules": sum(resident),
                    "resident_by_linear": {NAMES[m]: sum(resident[m::4]) for m in range(4)},
                    "gain_s_per_GB_mean": {NAMES[m]: round(float(np.mean([t_het[i] / mem[i] * 1e9
                                                                          for i in range(m, 4 * L, 4)])), 5)
                                           for m in range(4)}}
        log("module scheduler: %s" % json.dumps(schedule))
    alpha = hg.hetegen_layer_plan([(n, k, dt, resident[i]) for i, (n, k) in enumerate(shp)], bws)
    if args.alpha is not None:
        alpha = [0.0 if resident[i] else args.alpha for i in range(4 * L)]
    alpha_closed = list(alpha)
    t0 = time.time()
    max_batch = max(B, args.max_batch, 1)
    model = hg.hetegen_model_create(ctx, L, H, F, dt, W, b, alpha, resident, max_batch)
    log("model ready in %.1f s (resident modules %d of %d)" % (time.time() - t0, sum(resident), 4 * L))
    if args.exec != "auto" and not streamed:
        hg.hetegen_model_set_exec(model, {"persistent": hg.EXEC_PERSISTENT, "graph": hg.EXEC_GRAPH,
                                          "eager": hg.EXEC_EAGER}[args.exec])

    P = args.context
    if P > 0:
        # KV cache for positions [0, P + warmup + steps) and those of the extra passes (an alpha
        # sweep, the all-streamed point); positions [0, P) get synthetic keys and values (the
        # same for every layer), step t decodes position P + t
        hd = 128
        kv_len = P + max(nstep, 1 + args.sweep_steps, 1 + (args.all_streamed_steps or 0))
        hg.hetegen_model_kv_create(ctx, model, kv_len, hd)
        kd = torch.from_numpy(synth.normal((B, P, H), dt, 0, 7001).view(np.int16)).cuda()
        vd = torch.from_numpy(synth.normal((B, P, H), dt, 0, 7002).view(np.int16)).cuda()
        for l in range(L):
            hg.hetegen_model_kv_write(ctx, model, l, B, 0, P, kd.data_ptr(), vd.data_ptr(), sptr)
        torch.cuda.synchronize()
        del kd, vd

    def step(t):
        # step t decodes position P + t (KV cache); the extra passes (sweeps, the all-streamed
        # point) reuse the per-step inputs in turn
        if P > 0:
            hg.hetegen_decode_step_kv(ctx, model, xs[t % nstep].data_ptr(), out[t % 2].data_ptr(), B, P + t, sptr)
        else:
            hg.hetegen_decode_step(ctx, model, xs[t % nstep].data_ptr(), out[t % 2].data_ptr(), B, sptr)

    refined = None
    if args.alpha_bench and streamed and args.alpha is None:
        t0 = time.time()
        delta, crossed = hg.hetegen_model_alpha_benchmark(ctx, model, xs[0].data_ptr(), out[0].data_ptr(), B,
                                                          0.08, 0.02, 2, 2, hg.BENCH_WALL, sptr)
        alpha = hg.hetegen_model_get_alpha(model, 4 * L)
        refined = {"delta": round(delta, 4), "crossed": crossed,
                   "alpha_cpu_by_linear": {NAMES[m]: round(alpha[i], 4) for m in range(4)
                                           for i in [next((j for j in streamed if j % 4 == m), None)]
                                           if i is not None}}
        log("step-level alpha benchmark (wall-time objective): delta %+.4f in %.1f s" % (delta, time.time() - t0))

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    hg.hetegen_get_profile(ctx, reset=True)  # host-side counters of the timed steps (no events added)
    wall0 = time.perf_counter()
    e0.record(stream)
    for t in range(args.warmup, nstep):
        step(t)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    tprof = hg.hetegen_get_profile(ctx, reset=True)
    ms_step = e0.elapsed_time(e1) / args.steps
    gbps = wbytes / (ms_step * 1e-3) / 1e9
    log("decode step %.4f ms/token, %.1f GB/s effective (wall %.4f ms/step)" %
        (ms_step, gbps, wall * 1e3 / args.steps))
    # distribution over steps: a second pass with events between consecutive steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for t in range(args.warmup, nstep):
        step(t)
        evs[t - args.warmup + 1].record(stream)
    torch.cuda.synchronize()
    per_step = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    step_pct = [round(per_step[min(len(per_step) - 1, int(q * (len(per_step) - 1) + 0.5))], 5)
                for q in (0.1, 0.5, 0.9)]
    log("per-step ms p10 / p50 / p90: %s" % step_pct)

    if placement == "all":
        desc = "all linears HBM-resident (alpha=0)" + ("" if P > 0 else ", GEMV-only")
    elif placement == "half":
        desc = "layers 0-%d HBM-resident, %d-%d streamed from pinned host" % (res_layers - 1, res_layers, L - 1)
    elif placement == "sched":
        desc = "module scheduler: %d of %d linears HBM-resident (%.2f of %.2f GB budget), rest streamed from " \
               "pinned host" % (sum(resident), 4 * L, schedule["resident_GB"], schedule["hbm_budget_GB"])
    else:
        desc = "all linears in %s host memory, streamed + CPU share" % ("pageable" if args.pageable else "pinned")
    if placement != "all":
        desc += ", %s" % ("alpha=%g" % args.alpha if args.alpha is not None else
                          "planner alpha refined by the step-level alpha benchmark" if refined else "planner alpha")
    if P > 0:
        desc += ", attention over a %d-position KV cache (positions %d-%d decoded)" % (P, P + args.warmup,
                                                                                      P + nstep - 1)
    result = {
        "metric": "decode latency ms/token + effective weight GB/s (frac of HBM/PCIe roofline)",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "ms_per_token": round(ms_step, 5),
        "step_ms_p10_p50_p90": step_pct,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == 1 else "f16",
        "data": "synthetic: seeded N(0,0.02) weights, N(0,1) activations (no checkpoints)",
        "config": {"workload": "%s-shaped decode step, %d layers x {qkv,out,fc1,fc2}, %s, batch %d" %
                               (args.model.upper(), L, desc, B) +
                               ("" if L == L_full else " (first %d of the model's %d layers)" % (L, L_full)),
                   "layers": L, "hidden": H, "ffn": F, "batch": B, "max_batch": max_batch,
                   "weight_bytes_per_step": wbytes,
                   "resident_layers": res_layers, "resident_modules": sum(resident),
                   "parallelism": "single GPU"},
    }
    if schedule:
        result["config"]["schedule"] = schedule
    result["host"] = host_info(torch)

    exec_mode = {1: "persistent", 2: "graph", 3: "eager"}.get(hg.hetegen_model_last_exec(model), "?")
    result["config"]["exec"] = exec_mode
    if P > 0:
        # keys and values read per step (positions 0..pos of every layer), mean over the timed steps
        kv_b = np.mean([2 * L * B * (P + t + 1) * H * 2 for t in range(args.warmup, nstep)])
        result["kv"] = {"context": P, "head_dim": 128, "kv_bytes_per_step": int(kv_b),
                        "tokens_per_s": round(B * 1e3 / ms_step, 2),
                        "weight_plus_kv_GBps": round((wbytes + kv_b) / (ms_step * 1e-3) / 1e9, 1)}
        log("kv: %s" % json.dumps(result["kv"]))
        if not streamed:
            # the step as a whole against HBM: weights, keys and values read once per step
            # (the attention launches are latency-bound; their own times are in the kernel trace)
            ach = (wbytes + kv_b) / (ms_step * 1e-3) / 1e9
            result["roofline"] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                  "frac": round(ach / HBM_PEAK_GBPS, 4), "traffic": None,
                                  "kernel": "whole step: %d GEMV launches + %d attn_kernel launches" % (4 * L, L),
                                  "bytes_per_step": int(wbytes + kv_b)}
    if not streamed and P == 0:
        # dominant kernel: every dispatch of the timed region is the GEMV kernel (LayerNorm,
        # value slice, ReLU and residual are fused into it): one persistent step kernel per
        # step, or one GEMV launch per linear; its average launch time is the event-timed
        # region divided by the launches in it.
        launches = 1 if exec_mode == "persistent" else 4 * L
        avg_us = ms_step * 1e3 / launches
        bytes_per_launch = (wbytes + sum(B * (n + k) * 2 + n * 2 for n, k in shp)) / launches
        achieved = bytes_per_launch / (avg_us * 1e-6) / 1e9
        log("%s: avg %.2f us/launch, %.2f MB/launch -> %.1f GB/s" %
            (exec_mode, avg_us, bytes_per_launch / 1e6, achieved))
        layouts = hg.hetegen_model_layouts(model)
        tiled_used = bool(layouts & hg.LAYOUT_TILED) and (B >= 2 or not layouts & hg.LAYOUT_ROWMAJOR)
        kernel_label = "step_kernel<%s,%d,...>" % ("BF16" if dt == 1 else "F16", B) if exec_mode == "persistent" \
            else gemv_label(B, H, F, dt, tiled_used, ln_partials_on(H),
                            torch.cuda.get_device_properties(0).multi_processor_count)
        result["frac_of_hbm_peak"] = round(gbps / HBM_PEAK_GBPS, 4)
        # achievable read bandwidth of this device (streaming read of 4 GiB), for information
        read_gbps = hg.hetegen_probe_hbm(ctx, 4 << 30, 5) / 1e9
        log("HBM streaming read: %.1f GB/s" % read_gbps)
        # the same weights read by plain streaming reads in the step's launches: the
        # step's floor (launch ramp and drain included)
        read_step_ms = hg.hetegen_model_read_ms(ctx, model, 5, sptr)
        log("plain read of the step's weights in its %d launches: %.4f ms (%.1f GB/s)" %
            (4 * L, read_step_ms, wbytes / (read_step_ms * 1e-3) / 1e9))
        result["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                              "frac": round(achieved / HBM_PEAK_GBPS, 4),
                              "traffic": counter_traffic(args.model, dt, B),
                              "kernel": kernel_label,
                              "avg_launch_us": round(avg_us, 3), "bytes_per_launch": round(bytes_per_launch),
                              "launches_per_step": launches,
                              "hbm_read_achievable_GBps": round(read_gbps, 1),
                              "frac_of_achievable": round(achieved / read_gbps, 4),
                              "read_same_launches_ms": round(read_step_ms, 5),
                              "frac_of_read_same_launches": round(read_step_ms / ms_step, 4)}
        result["config"]["weight_layouts"] = "+".join(n for f, n in ((hg.LAYOUT_ROWMAJOR, "row-major"),
                                                                    (hg.LAYOUT_TILED, "tiled"),
                                                                    (hg.LAYOUT_KMAJOR, "k-major")) if layouts & f)
        if tiled_used and exec_mode != "persistent":
            # the timed region also holds the LayerNorm launches (B x H x 2 bytes read and written
            # each): before layer 0's qkv, or before every qkv and fc1 without the partials; they
            # are not in launches_per_step or bytes_per_launch, so `achieved` understates the
            # GEMV's own rate by their share of the step
            n_ln = 1 if ln_partials_on(H) else 2 * L
            result["roofline"]["region_also_holds"] = "%d layernorm_regs_kernel launch%s per step (%d bytes each)" % (
                n_ln, "" if n_ln == 1 else "es", B * H * 4)
    elif streamed:
        # heterogeneous figures: link and CPU rates, the ideal rate of Eq. 4, busy fractions
        sb = sum(shp[i][0] * shp[i][1] * 2 for i in streamed)
        n_cpu = [min(shp[i][0], int(np.floor(alpha[i] * shp[i][0] + 0.5))) for i in range(4 * L)]
        cpu_b = sum(n_cpu[i] * shp[i][1] * 2 for i in streamed)
        h2d_b = sb - cpu_b
        v_cpu = float(np.mean([p["cpu_Bps"] for p in probe.values()]))
        # Eq. 8: with pageable weights the link side runs at min(V_PIN, V_TRANS)
        v_com = float(np.mean([min(p["h2d_Bps"], p["pin_Bps"]) if p["pin_Bps"] > 0 else p["h2d_Bps"]
                               for p in probe.values()]))
        v_gpu = float(np.mean([p["hbm_gemv_Bps"] for p in probe.values()]))
        v_g = 1.0 / (1.0 / v_com + 1.0 / v_gpu)
        hbm_b = wbytes - sb
        ideal_s = sb / (v_cpu + v_g) + hbm_b / v_gpu
        hg.hetegen_set_profiling(ctx, 1)
        hg.hetegen_get_profile(ctx, reset=True)
        nprof = min(2, args.steps)
        for t in range(nprof):
            step(args.warmup + t)
        torch.cuda.synchronize()
        prof = hg.hetegen_get_profile(ctx, reset=True)
        hg.hetegen_set_profiling(ctx, 0)
        wall_ms = prof["wall_ms"]
        result["hetero"] = {
            "alpha_cpu_by_linear": {NAMES[m]: round(alpha[i], 4) for m in range(4)
                                    for i in [next((j for j in streamed if j % 4 == m), None)] if i is not None},
            "probe_GBps": {k: {f: round(v[f] / 1e9, 2) for f in ("cpu_Bps", "h2d_Bps", "hbm_gemv_Bps", "pin_Bps")}
                           for k, v in probe.items()},
            "streamed_bytes_per_step": sb, "h2d_bytes_per_step": h2d_b, "cpu_bytes_per_step": cpu_b,
            "h2d_GBps_over_step": round(h2d_b / (ms_step * 1e-3) / 1e9, 2),
            "link_idle_GBps": round(link_idle / 1e9, 2),
            "h2d_frac_of_idle_link": round(h2d_b / (ms_step * 1e-3) / link_idle, 4),
            # the planner's V_COM (copies timed while the CPU share runs), for information
            "h2d_frac_of_concurrent_probe": round(h2d_b / (ms_step * 1e-3) / v_com, 4),
            "roofline": {"bound": "pcie", "achieved": round(h2d_b / (ms_step * 1e-3) / 1e9, 2),
                         "peak": round(link_idle / 1e9, 2), "unit": "GB/s",
                         "frac": round(h2d_b / (ms_step * 1e-3) / link_idle, 4), "traffic": None,
                         "kernel": "streamed GPU rows: chunk copies (hipMemcpyAsync on the copy stream)",
                         "achieved_is": "weight bytes streamed host-to-device per step / step time",
                         "peak_is": "idle 1 GiB pinned host-to-device copy, median of 10, same run"},
            "cpu_GBps_over_step": round(cpu_b / (ms_step * 1e-3) / 1e9, 2),
            # host-memory bytes of the step: the CPU share reads its rows once; a streamed row is
            # read once by the DMA from pinned memory, or, from pageable memory, read and written
            # by the pin team first (three passes)
            "host_memory_GBps_over_step": round((cpu_b + h2d_b * (3 if args.pageable else 1)) /
                                                (ms_step * 1e-3) / 1e9, 2),
            "ideal_ms_per_step": round(ideal_s * 1e3, 3),
            "frac_of_ideal": round(ideal_s * 1e3 / ms_step, 4),
            "busy_frac": {"cpu": round(prof["cpu_ms"] / wall_ms, 4), "io": round(prof["h2d_ms"] / wall_ms, 4),
                          "gpu": round(prof["gpu_ms"] / wall_ms, 4), "pin": round(prof["pin_ms"] / wall_ms, 4)},
            "profiled_ms_per_step": round(wall_ms / nprof, 3),
            # the calling thread's time per timed step: CPU shares, waits for their inputs (the
            # GPU work ahead of them, then the hand-off), waits for the link after them, and the
            # rest (enqueueing kernels and copies, the glue between linears)
            "host_ms_per_step": {"cpu_shares": round(tprof["cpu_ms"] / args.steps, 3),
                                 "input_wait": round(tprof["xwait_ms"] / args.steps, 3),
                                 "link_wait": round(tprof["tailwait_ms"] / args.steps, 3),
                                 "enqueue_in_linears": round((tprof["hetlin_ms"] - tprof["cpu_ms"] -
                                                              tprof["xwait_ms"] - tprof["tailwait_ms"]) /
                                                             args.steps, 3),
                                 "outside_linears": round(ms_step - tprof["hetlin_ms"] / args.steps, 3),
                                 "n_cpu_shares": int(tprof["cpu_shares"] // args.steps)},
        }
        if hbm_b > 0:
            # a mixed placement: the HBM-resident rows against 8 TB/s (their GEMVs' event-timed
            # GPU time in the profiled pass), and the rest of the step against the heterogeneous
            # ideal of the streamed bytes (the resident linears run between them, not beside)
            res_ms = prof["res_gpu_ms"] / nprof
            res_b = prof["res_gpu_bytes"] / nprof
            rest_ms = ms_step - res_ms
            str_ideal_ms = sb / (v_cpu + v_g) * 1e3
            result["hetero"]["resident_part"] = {
                "bytes_per_step": int(res_b), "gpu_ms_per_step": round(res_ms, 3),
                "GBps": round(res_b / (res_ms * 1e-3) / 1e9, 1) if res_ms > 0 else None,
                "frac_of_hbm_peak": round(res_b / (res_ms * 1e-3) / (HBM_PEAK_GBPS * 1e9), 4) if res_ms > 0 else None,
                "measured_as": "events around each resident GEMV launch in the profiled pass"}
            result["hetero"]["streamed_part"] = {
                "bytes_per_step": int(sb), "ms_per_step": round(rest_ms, 3),
                "ideal_ms_per_step": round(str_ideal_ms, 3),
                "frac_of_ideal": round(str_ideal_ms / rest_ms, 4) if rest_ms > 0 else None,
                "measured_as": "step time less the resident GEMVs' GPU time"}
        log("hetero: %s" % json.dumps(result["hetero"]))

    n_all = args.all_streamed_steps or 0
    if streamed and n_all > 0:
        # every GPU row streamed (CPU fraction 0 on every host-resident linear): the streamed
        # path alone against the idle link
        hg.hetegen_model_set_alpha(model, [0.0] * (4 * L))
        step(0)
        torch.cuda.synchronize()
        e0.record(stream)
        for t in range(n_all):
            step(1 + t)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_all = e0.elapsed_time(e1) / n_all
        hg.hetegen_model_set_alpha(model, alpha)
        ach = sb / (ms_all * 1e-3) / 1e9
        result["all_streamed"] = {
            "alpha_cpu": 0.0, "steps": n_all, "ms_per_step": round(ms_all, 3),
            "weight_GBps": round(wbytes / (ms_all * 1e-3) / 1e9, 2),
            "roofline": {"bound": "pcie", "achieved": round(ach, 2), "peak": round(link_idle / 1e9, 2), "unit": "GB/s",
                         "frac": round(ach * 1e9 / link_idle, 4), "traffic": None,
                         "achieved_is": "streamed weight bytes per step / step time (every row streamed)",
                         "peak_is": "idle 1 GiB pinned host-to-device copy, median of 10, same run"}}
        log("all streamed: %.1f ms/token, %.2f GB/s over the link (%.3f of the idle link)" %
            (ms_all, ach, ach * 1e9 / link_idle))

    if refined:
        # the same step with the closed-form fractions, for comparison
        hg.hetegen_model_set_alpha(model, alpha_closed)
        step(0)
        torch.cuda.synchronize()
        e0.record(stream)
        for t in range(args.steps):
            step(args.warmup + t)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_closed = e0.elapsed_time(e1) / args.steps
        hg.hetegen_model_set_alpha(model, alpha)
        result["alpha_benchmark"] = dict(refined, ms_per_step_closed_form=round(ms_closed, 3),
                                         ms_per_step_refined=round(ms_step, 3))
        log("closed-form alpha: %.2f ms/token; refined: %.2f ms/token" % (ms_closed, ms_step))

    # ---- latency vs CPU fraction of the streamed linears ----
    if args.alpha_sweep and streamed:
        sweep = []
        for a_s in [float(v) for v in args.alpha_sweep.split(",")]:
            hg.hetegen_model_set_alpha(model, [0.0 if resident[i] else a_s for i in range(4 * L)])
            step(0)
            torch.cuda.synchronize()
            e0.record(stream)
            for t in range(args.sweep_steps):
                step(1 + t)
            e1.record(stream)
            torch.cuda.synchronize()
            ms_a = e0.elapsed_time(e1) / args.sweep_steps
            h2d_a = sum((shp[i][0] - min(shp[i][0], int(np.floor(a_s * shp[i][0] + 0.5)))) * shp[i][1] * 2
                        for i in streamed)
            sweep.append({"alpha_cpu": a_s, "ms_per_step": round(ms_a, 3),
                          "GBps": round(wbytes / (ms_a * 1e-3) / 1e9, 2),
                          "h2d_GBps_over_step": round(h2d_a / (ms_a * 1e-3) / 1e9, 2)})
            log("alpha %.2f: %.2f ms/token, %.1f GB/s, link %.1f GB/s" %
                (a_s, ms_a, wbytes / (ms_a * 1e-3) / 1e9, h2d_a / (ms_a * 1e-3) / 1e9))
        hg.hetegen_model_set_alpha(model, alpha)
        result["alpha_sweep"] = sweep

    # ---- CPU baseline: the oracle on a bounded sample of the same linears ----
    if not args.no_cpu_baseline:
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        budget_s = 15.0
        done_bytes, t_cpu, n_lin = 0, 0.0, 0
        xb = {k: synth.normal((B, k), dt, 0, 99) for k in (H, F)}
        ybuf = {}
        while t_cpu < budget_s and n_lin < 64 * len(shp):
            i = n_lin % len(shp)
            n, k = shp[i]
            y = ybuf.setdefault(n, np.empty((B, n), np.float32))
            c0 = time.perf_counter()
            oracle.linear_ptr(xb[k].ctypes.data, k, B, k, W[i], n, dt, b[i], y)
            t_cpu += time.perf_counter() - c0
            done_bytes += n * k * 2
            n_lin += 1
        result["cpu_baseline"] = {"value": round(done_bytes / t_cpu / 1e9, 3), "unit": "GB/s", "cores": threads,
                                  "kind": "oracle",
                                  "sample": "%d linears in step order (%d per step; %.2f GB of weights), batch %d, "
                                            "%.1f s" % (n_lin, len(shp), done_bytes / 1e9, B, t_cpu),
                                  "ms_per_token_extrapolated": round(t_cpu / done_bytes * wbytes * 1e3, 1)}
        log("oracle: %.3f GB/s on %d threads" % (done_bytes / t_cpu / 1e9, threads))

    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()

    hg.hetegen_model_destroy(ctx, model)
    for p in (b if args.pageable else W + b):
        hg.hetegen_host_free(ctx, p)
    hg.hetegen_destroy(ctx)
    return result


if __name__ == "__main__":
    main()
