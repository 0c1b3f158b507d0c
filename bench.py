"""Benchmark of the Flash-ABFT attention forward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload dec_l4096]

A step is one fabft_attn_fwd call (Q K^T, online softmax with the fused
checksum, P V, per-row check) over the whole workload, inputs resident in
HBM. Prints one JSON line: attention TFLOP/s with the checksum on (the
value), the checksum-off rate and overhead, the dominant kernel against the
bf16 MFMA roofline, and the fp64 oracle timed on the host as a baseline.

FLOP convention: 4*d per visible (query, key) pair (causal: the visible
triangle only); the same count with the checksum on and off.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_{workload}.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2507_16676_amd", "csrc", "fabft_kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_src_sha() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def make_device_inputs(w, device):
    """Seeded N(0,1) inputs of the workload's shape and recipe, drawn on the
    GPU (the timed path needs no host copy); bf16 round-to-nearest-even."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(w.seed)
    shp_q = (w.B, w.H, w.Lq, w.d)
    shp_k = (w.B, w.H, w.Lk, w.d)
    q = torch.randn(shp_q, generator=g, device=device, dtype=torch.float32)
    k = torch.randn(shp_k, generator=g, device=device, dtype=torch.float32)
    v = torch.randn(shp_k, generator=g, device=device, dtype=torch.float32)
    if w.qk_prescale != 1.0:
        q *= w.qk_prescale
        k *= w.qk_prescale
    if w.peaked_frac > 0:
        n = int(round(w.peaked_frac * w.Lk))
        gc = torch.Generator()
        gc.manual_seed(w.seed + 1)
        for b in range(w.B):
            for h in range(w.H):
                idx = torch.randperm(w.Lk, generator=gc)[:n].to(device)
                k[b, h, idx] *= w.peaked_mult
    return (q.to(torch.bfloat16).contiguous(), k.to(torch.bfloat16).contiguous(),
            v.to(torch.bfloat16).contiguous())


def time_launches(fn, steps, stream):
    """Total and per-launch time (ms) of `steps` calls, HIP events on `stream`."""
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(steps):
        fn()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    return evs[0].elapsed_time(evs[-1]), per


DECODE_SHAPES = [(4, 32, 1, 32768), (4, 32, 16, 32768), (1, 32, 1, 131072), (8, 8, 64, 8192)]


def decode_sweep(d: int = 128, splits=(0, 4, 8, 16, 32, 64), reps: int = 50, shapes=None,
                 warm_ms: float = 100.0):
    """K/V bytes streamed per second for the one-pass forward (nsplit 0) and
    the key-split forward on decode shapes, checksum on, non-causal. Each
    configuration first runs untimed for about `warm_ms` (the GPU clock
    rises only under sustained load), then `reps` launches are timed."""
    import torch
    import paper_2507_16676_amd as F
    import workloads as W
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    for (B, H, Lq, Lk) in (shapes or DECODE_SHAPES):
        w = W.Workload(f"decode_b{B}_h{H}_q{Lq}_k{Lk}", B, H, Lq, Lk, d, False, d ** -0.5)
        q, k, v = make_device_inputs(w, dev)
        kv_bytes = 2 * B * H * Lk * d * 2
        rows = {}
        for ns in splits:
            if ns == 0:
                fn = lambda: F.attn_fwd(q, k, v, causal=False, scale=w.scale)
            else:
                ws = torch.empty(F.splitkv_workspace_bytes(B, H, Lq, d, ns), dtype=torch.uint8,
                                 device=dev)
                fn = (lambda ns=ns, ws=ws: F.attn_fwd_splitkv(q, k, v, causal=False, scale=w.scale,
                                                             nsplit=ns, workspace=ws))
            fn()
            torch.cuda.synchronize()
            t, _ = time_launches(fn, 5, stream)
            for _ in range(max(5, int(warm_ms / max(t / 5, 1e-3)))):
                fn()
            t, _ = time_launches(fn, reps, stream)
            us = 1e3 * t / reps
            rows[f"nsplit_{ns}" if ns else "one_pass"] = {"us": round(us, 1),
                                                          "TB/s": round(kv_bytes / us / 1e6, 3)}
        print(json.dumps({"workload": w.name, "kv_bytes": kv_bytes,
                          "default_nsplit": F.splitkv_default_splits(B, H, Lq, Lk, d),
                          "results": rows}), flush=True)


def copy_probe(mib: int, dev):
    """One device-to-device copy of known size: the calibration launch for
    the HBM byte counters (FETCH_SIZE, WRITE_SIZE) of a profiled run."""
    import torch
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] copy probe: {mib} MiB device-to-device")


def cpu_baseline(w, target_s: float):
    """Time the fp64 oracle on the host for a bounded sample of the workload:
    whole heads (all query rows) of batch entry 0, drawn with the same
    recipe, as many as fit in about `target_s` seconds."""
    import numpy as np
    import oracle
    import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"), default=1)
    except Exception:   # threadpoolctl missing: report the affinity mask
        threads = len(os.sched_getaffinity(0))
    one = w.with_(B=1, H=1)
    inp = W.make_inputs(one)
    q, k, v = inp.as_f32()
    t0 = time.perf_counter()
    oracle.attention(q, k, v, w.causal, w.scale)
    t_head = time.perf_counter() - t0
    n_heads = int(max(1, min(w.B * w.H, math.floor(target_s / max(t_head, 1e-6)))))
    sample = w.with_(B=1, H=n_heads)
    inp = W.make_inputs(sample)
    q, k, v = inp.as_f32()
    t0 = time.perf_counter()
    oracle.attention(q, k, v, w.causal, w.scale)
    dt = time.perf_counter() - t0
    tflops = sample.flops / dt / 1e12
    return {"value": tflops, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n_heads} of {w.B * w.H} heads (b=0, all {w.Lq} rows), "
                      f"{dt:.2f} s, fp64 numpy",
            "seconds": dt, "blas": "numpy BLAS"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="dec_l4096")
    ap.add_argument("--rounds", type=int, default=5,
                    help="interleaved on/off rounds for the overhead figure")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-shape", default=None,
                    help="with --decode-sweep: one shape B,H,Lq,Lk instead of the default set")
    ap.add_argument("--decode-splits", default=None,
                    help="with --decode-sweep: comma-separated split counts (0 = one pass)")
    ap.add_argument("--decode-sweep", action="store_true",
                    help="instead of the benchmark line: time the one-pass and the key-split "
                         "forward on decode shapes (few queries, many keys), one JSON line each")
    ap.add_argument("--weighted", action="store_true",
                    help="also run the weighted second checksum (an extension)")
    ap.add_argument("--score-check", action="store_true",
                    help="also run the score check (an extension; its K-sum pre-pass is timed)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device copy of this size (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the Flash-ABFT forward is a single-GPU kernel "
              "here (heads shard across GPUs with no communication); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2507_16676_amd as F
    F.set_weighted_check(args.weighted)
    if args.decode_sweep:
        kw = {}
        if args.decode_shape:
            kw["shapes"] = [tuple(int(x) for x in args.decode_shape.split(","))]
        if args.decode_splits:
            kw["splits"] = tuple(int(x) for x in args.decode_splits.split(","))
        decode_sweep(**kw)
        if args.copy_probe_mib > 0:
            copy_probe(args.copy_probe_mib, torch.device("cuda:0"))
        return
    import workloads as W

    w = W.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"[bench] workload {w.name}: B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} d{w.d} causal={w.causal}")
    q, k, v = make_device_inputs(w, dev)
    if args.score_check:
        sws = torch.empty(F.score_check_workspace_bytes(w.B, w.H, w.Lk, w.d), dtype=torch.uint8,
                          device=dev)
        F.set_score_check(sws)
    o = torch.empty_like(q)
    resid = torch.empty((w.B, w.H, w.Lq), dtype=torch.float32, device=dev)
    flags = torch.empty((w.B, w.H, w.Lq), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def on():
        F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale, out=(o, resid, flags))

    def off():
        F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale, check=False, out=(o,))

    # fault-free check first: counting the flags waits on the host, and the
    # GPU lowers its clock while idle (the first ~25 launches after such a
    # gap run ~15% slower), so the warmup runs last, right before the timing
    on()
    torch.cuda.synchronize()
    nflag = int((flags != 0).sum())
    for _ in range(args.warmup):
        on()
        off()
    torch.cuda.synchronize()
    log(f"[bench] warmup done; fault-free flagged rows: {nflag}")

    # ---- timed region: exactly `steps` checksum-on steps
    total_ms, per = time_launches(on, args.steps, stream)
    ms = total_ms / args.steps
    flops = w.flops
    tflops = flops / (ms * 1e-3) / 1e12
    avg_launch_ms = sum(per) / len(per)
    log(f"[bench] checksum on: {ms:.4f} ms/step, {tflops:.1f} TFLOP/s")

    # ---- checksum off, and interleaved on/off rounds for the overhead
    ratios, on_ms, off_ms = [], [], []
    k_round = max(3, args.steps // 2)
    for r in range(args.rounds):
        t_on, _ = time_launches(on, k_round, stream)
        t_off, _ = time_launches(off, k_round, stream)
        on_ms.append(t_on / k_round)
        off_ms.append(t_off / k_round)
        ratios.append(t_on / t_off)
    ratios.sort()
    overhead = 100.0 * (ratios[len(ratios) // 2] - 1.0)
    ms_off = sorted(off_ms)[len(off_ms) // 2]
    ms_on_r = sorted(on_ms)[len(on_ms) // 2]
    tflops_off = flops / (ms_off * 1e-3) / 1e12
    log(f"[bench] checksum off: {ms_off:.4f} ms/step, {tflops_off:.1f} TFLOP/s; "
        f"interleaved on {ms_on_r:.4f} ms/step; overhead {overhead:.2f}%")

    # ---- roofline of the dominant kernel (the checksum-on forward; one
    # launch per step)
    achieved = flops / (avg_launch_ms * 1e-3) / 1e12
    traffic = None
    tf = TRAFFIC_FILE.format(workload=w.name)
    if os.path.exists(tf):
        with open(tf) as f:
            t = json.load(f)
        if t.get("kernel_src_sha") == kernel_src_sha():
            traffic = t["bytes_per_launch"]
    roofline = {"bound": "mfma", "achieved": round(achieved, 2),
                "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": (f"fabft::fwd_kernel<{128 if w.d == 96 else w.d}, "
                           f"{str(w.causal).lower()}, true, false, "
                           f"false, false, false>"),
                "avg_launch_ms": round(avg_launch_ms, 5)}

    if args.copy_probe_mib > 0:
        copy_probe(args.copy_probe_mib, dev)

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the fp64 oracle on the host ...")
        cpu = cpu_baseline(w, args.cpu_seconds)
        log(f"[bench] oracle: {cpu['value'] * 1e3:.2f} GFLOP/s on {cpu['cores']} threads "
            f"({cpu['sample']})")

    line = {
        "metric": "attention TFLOP/s (bf16, 1 GPU) + % MFMA peak; checksum overhead %; "
                  "fault-detect rate",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1), drawn on the GPU)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "Lq": w.Lq, "Lk": w.Lk,
                   "d": w.d, "causal": w.causal, "scale": w.scale,
                   "checksum": "on" + ("+weighted" if args.weighted else "")
                               + ("+scores" if args.score_check else "")},
        "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "checksum_off": {"ms_per_step": round(ms_off, 5), "tflops": round(tflops_off, 2)},
        "checksum_overhead_pct": round(overhead, 3),
        "fault_free_flagged_rows": nflag,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
