"""Benchmark: one decode step over OPT-shaped decoder-layer linears on one MI355X.

Default workload: OPT-6.7B shapes, 32 layers x {QKV [12288,4096], out [4096,4096],
fc1 [16384,4096], fc2 [4096,16384]}, fp16 weights ~N(0, 0.02) generated from a
seeded counter-based generator into pinned host memory, every linear resident in
HBM (CPU fraction 0 from the planner), batch 1, fresh x ~N(0, 1) per step, already
in HBM before the timed region.  A step is hetegen_decode_step: the four GEMVs of
every layer with LayerNorm, value slice, ReLU and residual fused into them.

Prints ONE JSON line.  `value` is the effective weight bandwidth of the whole step
(weight bytes per step / time per step); `ms_per_step` is the decode latency per
token.  `roofline` is the GEMV kernel's algorithmic bytes per launch (weights, x, bias,
y) over its average launch time; every dispatch in the event-timed region (on the
stream the step runs on) is that kernel, so the average is the region's time over
its launches.  Peak: 8 TB/s HBM.  `cpu_baseline` times the
oracle (plain C, sequential fp32) on a bounded sample of the same linears.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
OPT = {  # name: (layers, hidden, ffn, dtype)
    "opt-6.7b": (32, 4096, 16384, 0),
    "opt-13b": (40, 5120, 20480, 0),
    "opt-30b": (48, 7168, 28672, 0),
    "opt-66b": (64, 9216, 36864, 1),
}
NAMES = ("qkv", "out", "fc1", "fc2")


def shapes(H, F):
    return [(3 * H, H), (H, H), (F, H), (H, F)]


def counter_traffic(model, dt, B):
    """HBM bytes per GEMV launch from the committed counter summary, if it was taken
    on this workload with the current kernel source; else None."""
    import hashlib
    name = "gemv_%s_b%d_%s_decode_hbm_counters.md" % ("bf16" if dt == 1 else "f16", B, model.replace("-", ""))
    path = os.path.join(ROOT, "profiles", name)
    src = os.path.join(ROOT, "paper_2403_01164_amd", "csrc", "kernels.hip")
    if not os.path.exists(path):
        return None
    fields = dict(l.split(": ", 1) for l in open(path).read().splitlines() if ": " in l and not l.startswith("#"))
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    if fields.get("kernel_source_sha256_16", "").strip() != sha:
        return None
    return float(fields["traffic_bytes_per_launch"])


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--model", default="opt-6.7b", choices=sorted(OPT))
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="end with one plain 256 MiB device-to-device copy, the reference dispatch for "
                         "scaling HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (the heterogeneous "
              "linear shards by output rows across GPUs, see the design notes); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    import paper_2403_01164_amd as hg

    torch.cuda.set_device(0)
    L, H, F, dt = OPT[args.model]
    B = args.batch
    ctx = hg.hetegen_create(0)
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream

    # ---- synthetic OPT-shaped weights in pinned host memory ----
    t0 = time.time()
    W, b, shp = [], [], []
    for l in range(L):
        for i, (n, k) in enumerate(shapes(H, F)):
            w = hg.hetegen_host_alloc(ctx, n * k * 2)
            bb = hg.hetegen_host_alloc(ctx, n * 2)
            synth.fill_normal_ptr(w, n * k, dt, 0, synth.weight_id(l, NAMES[i]), 0.0, 0.02)
            synth.fill_normal_ptr(bb, n, dt, 0, synth.bias_id(l, NAMES[i]), 0.0, 0.02)
            W.append(w)
            b.append(bb)
            shp.append((n, k))
    wbytes = sum(n * k * 2 for n, k in shp)
    log("generated %.3f GB of weights in %.1f s" % (wbytes / 1e9, time.time() - t0))

    # ---- planner: every linear resident -> CPU fraction 0 ----
    alpha = hg.hetegen_layer_plan([(n, k, dt, 1) for n, k in shp], [(1.0, 1.0, 1.0, 0.0)])
    assert all(a == 0.0 for a in alpha)
    t0 = time.time()
    model = hg.hetegen_model_create(ctx, L, H, F, dt, W, b, alpha, [1] * len(shp), max(B, 1))
    log("uploaded resident weights in %.1f s" % (time.time() - t0))

    # fresh input per step, resident in HBM before timing
    nstep = args.warmup + args.steps
    xs = torch.empty((nstep, B, H), dtype=torch.int16, device="cuda")
    for t in range(nstep):
        xs[t] = torch.from_numpy(synth.normal((B, H), dt, 0, synth.act_id(t)).view(np.int16))
    out = torch.empty((2, B, H), dtype=torch.int16, device="cuda")

    def step(t):
        hg.hetegen_decode_step(ctx, model, xs[t].data_ptr(), out[t % 2].data_ptr(), B, sptr)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    e0.record(stream)
    for t in range(args.warmup, nstep):
        step(t)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = e0.elapsed_time(e1) / args.steps
    gbps = wbytes / (ms_step * 1e-3) / 1e9
    log("decode step %.4f ms/token, %.1f GB/s effective (wall %.4f ms/step)" %
        (ms_step, gbps, wall * 1e3 / args.steps))

    # ---- dominant kernel: every dispatch of the replayed step is the GEMV kernel
    # (LayerNorm, value slice, ReLU and residual are fused into it), so its average
    # launch time is the event-timed region divided by the launches in it.
    launches_per_step = 4 * L
    avg_us = ms_step * 1e3 / launches_per_step
    bytes_per_launch = (wbytes + sum(B * (n + k) * 2 + n * 2 for n, k in shp)) / launches_per_step
    achieved = bytes_per_launch / (avg_us * 1e-6) / 1e9
    log("GEMV: avg %.2f us/launch, %.2f MB/launch -> %.1f GB/s" % (avg_us, bytes_per_launch / 1e6, achieved))

    result = {
        "metric": "decode latency ms/token + effective weight GB/s (frac of HBM/PCIe roofline)",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "ms_per_token": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == 1 else "f16",
        "data": "synthetic: seeded N(0,0.02) weights, N(0,1) activations (no checkpoints)",
        "config": {"workload": "%s-shaped decode step, %d layers x {qkv,out,fc1,fc2}, all linears HBM-resident "
                               "(alpha=0), batch %d, GEMV-only" % (args.model.upper(), L, B),
                   "layers": L, "hidden": H, "ffn": F, "batch": B, "weight_bytes_per_step": wbytes,
                   "alpha": 0.0, "parallelism": "single GPU"},
        "frac_of_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": counter_traffic(args.model, dt, B),
                     "kernel": "gemv_kernel<%s,%d,...>" % ("BF16" if dt == 1 else "F16", B),
                     "avg_launch_us": round(avg_us, 3), "bytes_per_launch": round(bytes_per_launch),
                     "launches_per_step": launches_per_step},
    }

    # ---- CPU baseline: the oracle on a bounded sample of the same linears ----
    if not args.no_cpu_baseline:
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        budget_s = 15.0
        done_bytes, t_cpu, n_lin = 0, 0.0, 0
        xb = {k: synth.normal((B, k), dt, 0, 99) for k in (H, F)}
        ybuf = {}
        i = 0
        while t_cpu < budget_s and i < len(shp):
            n, k = shp[i]
            y = ybuf.setdefault(n, np.empty((B, n), np.float32))
            c0 = time.perf_counter()
            oracle.linear_ptr(xb[k].ctypes.data, k, B, k, W[i], n, dt, b[i], y)
            t_cpu += time.perf_counter() - c0
            done_bytes += n * k * 2
            n_lin += 1
            i += 1
        result["cpu_baseline"] = {"value": round(done_bytes / t_cpu / 1e9, 3), "unit": "GB/s", "cores": threads,
                                  "kind": "oracle",
                                  "sample": "first %d of the %d linears of one step (%.2f GB of weights), "
                                            "batch %d, %.1f s" % (n_lin, len(shp), done_bytes / 1e9, B, t_cpu),
                                  "ms_per_token_extrapolated": round(t_cpu / done_bytes * wbytes * 1e3, 1)}
        log("oracle: %.3f GB/s on %d threads" % (done_bytes / t_cpu / 1e9, threads))

    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()

    hg.hetegen_model_destroy(ctx, model)
    for p in W + b:
        hg.hetegen_host_free(ctx, p)
    hg.hetegen_destroy(ctx)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
