"""Benchmark of the MI355X 2-simplicial attention hot path (one GPU).

One step = the whole hot path over one batch of synthetic input already
resident in HBM: the forward (O, LSE) and the full backward (Delta, the
query-side kernel for dQ/dK'/dV', the key-side kernel for dK/dV).

Workload (default): B=1, H=16, N=32768, D=128, w1=512, w2=32, bf16, Q and K
rows L2-normalised and scaled by sqrt(D), seed 4 -- the long-context training
shape the headline metric is quoted on.

FLOP convention: forward 4*B*H*N*w1*w2*D, backward 12*B*H*N*w1*w2*D (the six
window contractions S, dP, dV, dK, dQ~, U~, counting the S recompute once);
the masked start of the sequence is not discounted.

Prints one JSON line. Multi-GPU runs are not part of this build: the path runs
on one GPU (sharding would split (batch, head) pairs or the sequence with a
w1-row halo exchange), so --gpus other than 1 exits with a message.
"""

import argparse
import hashlib
import glob
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 FLOP/clk
METRIC = "2-simplicial attn fwd/bwd TFLOP/s and % bf16 MFMA peak at N=32k, w1=512, w2=32"


def source_hash():
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2507_02754_amd", "csrc", "*")))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic(kernel, workload):
    """Per-launch HBM bytes of `kernel` from the committed counter summary, or None
    if there is none or it was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line:
            key, val = line.split(":", 1)
            vals[key.strip()] = val.strip()
    if vals.get("source_sha256") != source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, inputs, target_s):
    """The CPU oracle, as it is, on a bounded sample of the same workload: head
    (0, 0), consecutive queries from the middle of the sequence (full windows),
    forward + backward, until about `target_s` seconds have elapsed."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle as orc

    start = w.N // 2
    lo = start - (w.w1 - 1)
    arrs = [x[0, lo:, 0, :].to("cpu").double().numpy() for x in inputs]
    q0 = w.w1 - 1
    done = 0
    chunk = 64
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < target_s and q0 + done + chunk <= arrs[0].shape[0]:
        qs = range(q0 + done, q0 + done + chunk)
        orc.forward(*arrs[:5], w.w1, w.w2, w.scale, queries=qs)
        orc.backward(*arrs, w.w1, w.w2, w.scale, queries=qs)
        done += chunk
    el = time.perf_counter() - t0
    flops = 16.0 * done * w.w1 * w.w2 * w.D
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {
        "value": flops / el / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
        "sample": f"fwd+bwd of {done} queries (head 0, queries {start}..{start + done - 1}) "
                  f"of {w.name}; {el:.1f} s; nominal 16*w1*w2*D FLOPs per query",
        "host_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long_bf16_n32k")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 1 GiB device-to-device copy first (HBM counter calibration)")
    ap.add_argument("--gqa-kv-heads", type=int, default=0,
                    help="also time the grouped-query forward and backward with this many "
                         "K-side heads (reported under \"gqa\"; not part of the step)")
    ap.add_argument("--fused-main", action="store_true",
                    help="time the fused backward (one S/dP computation, partial sums reduced in order) "
                         "as the step's backward instead of the two-kernel backward")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused-backward section")
    ap.add_argument("--det", action="store_true",
                    help="also time the determinant-logit forward and backward (Section 5) at "
                         "B=1, H=16, N=4096, D=128, w1=512, w2=32 (reported under \"det\")")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs the hot path on one GPU only; multi-GPU sharding "
              "(over (batch, head) or the sequence with a w1-row halo) is not built. "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2507_02754_amd import (load_library, simplicial_attn_bwd_key_side,
                                      simplicial_attn_bwd_fused, simplicial_attn_bwd_fused_reduce,
                                      simplicial_attn_bwd_fused_workspace_size,
                                      simplicial_attn_bwd_preprocess, simplicial_attn_bwd_query_side,
                                      simplicial_attn_bwd_workspace_size, simplicial_attn_fwd,
                                      simplicial_attn_fwd_gqa, simplicial_attn_bwd_gqa,
                                      simplicial_attn_bwd_gqa_workspace_size,
                                      simplicial_attn_det_bwd, simplicial_attn_det_fwd,
                                      simplicial_attn_det_bwd_workspace_size,
                                      simplicial_attn_path_name)
    from paper_2507_02754_amd.workloads import WORKLOADS, make_inputs

    load_library()
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    print(f"[bench] {w.name} B={w.B} H={w.H} N={w.N} D={w.D} w1={w.w1} w2={w.w2} "
          f"fwd={simplicial_attn_path_name(0, w.B, w.N, w.H, w.D, w.w1, w.w2, w.torch_dtype)} "
          f"bwd={simplicial_attn_path_name(1, w.B, w.N, w.H, w.D, w.w1, w.w2, w.torch_dtype)}",
          file=sys.stderr, flush=True)
    inputs_cpu = make_inputs(w)
    q, k, kp, v, vp, do = (x.to(dev) for x in inputs_cpu)
    out = torch.empty_like(q)
    lse = torch.empty((w.B, w.H, w.N), dtype=torch.float32, device=dev)
    dq, dk, dkp, dv, dvp = (torch.empty_like(q) for _ in range(5))
    ws = torch.empty(simplicial_attn_bwd_workspace_size(w.B, w.N, w.H, w.D, w.w1, w.w2, w.torch_dtype),
                     dtype=torch.uint8, device=dev)
    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # The backward exactly as simplicial_attn_bwd runs it, stage by stage (its
    # stage entry points), so that each kernel is timed by HIP events. With
    # --fused-main the step's backward is the fused backward instead.
    fws = simplicial_attn_bwd_fused_workspace_size(w.B, w.N, w.H, w.D, w.w1, w.w2, w.torch_dtype)
    fused = bool(args.fused_main and fws)
    if fused:
        ws = torch.empty(fws, dtype=torch.uint8, device=dev)
        phases = ["fwd", "bwd_preprocess", "bwd_fused", "bwd_reduce"]
    else:
        phases = ["fwd", "bwd_preprocess", "bwd_query_side", "bwd_key_side"]

    def step(ev=None):
        if ev:
            ev[0].record()
        simplicial_attn_fwd(q, k, kp, v, vp, w.w1, w.w2, w.scale, out=out, lse=lse)
        if ev:
            ev[1].record()
        simplicial_attn_bwd_preprocess(out, do, w.w1, w.w2, ws)
        if ev:
            ev[2].record()
        if fused:
            simplicial_attn_bwd_fused(q, k, kp, v, vp, do, lse, w.w1, w.w2, ws, w.scale, grads=(dk, dv))
        else:
            simplicial_attn_bwd_query_side(q, k, kp, v, vp, do, lse, w.w1, w.w2, ws, w.scale,
                                           grads=(dq, dkp, dvp))
        if ev:
            ev[3].record()
        if fused:
            simplicial_attn_bwd_fused_reduce(q, w.w1, w.w2, ws, w.scale, grads=(dq, dkp, dvp))
        else:
            simplicial_attn_bwd_key_side(q, k, kp, v, vp, do, lse, w.w1, w.w2, ws, w.scale,
                                         grads=(dk, dv))
        if ev:
            ev[4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record()
    for i in range(args.steps):
        step(evs[i])
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)
    per = {p: sorted(e[j].elapsed_time(e[j + 1]) for e in evs) for j, p in enumerate(phases)}
    ms = {p: sum(v) / args.steps for p, v in per.items()}
    ms_step = total_ms / args.steps

    def med(v):
        n = len(v)
        return v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2])

    fwd_each = per["fwd"]
    bwd_each = sorted(sum(e[j].elapsed_time(e[j + 1]) for j in (1, 2, 3)) for e in evs)

    unit = float(w.B) * w.H * w.N * w.w1 * w.w2 * w.D
    fwd_flops, bwd_flops = 4 * unit, 12 * unit
    bwd_ms = ms[phases[1]] + ms[phases[2]] + ms[phases[3]]
    value = (fwd_flops + bwd_flops) / (ms_step * 1e-3) / 1e12
    fwd_tf = fwd_flops / (ms["fwd"] * 1e-3) / 1e12
    bwd_tf = bwd_flops / (bwd_ms * 1e-3) / 1e12

    # Roofline of the dominant kernel: algorithmic FLOPs per launch / its time
    # (HIP events on the stream the library launches on). The query-side stage
    # also runs the small chunk-boundary fix-up kernel inside its events.
    qkernel = "bwd_query_kernel" if w.w2 <= 32 else "bwd_q_kernel"
    if fused:
        algo = {  # phase: (kernel, algorithmic FLOPs, executed MFMA FLOPs)
            "fwd": ("fwd_mfma_kernel", 4 * unit, 4 * unit),
            "bwd_fused": ("bwd_fused_kernel", 12 * unit, 12 * unit),  # S, dP, dV, dK, dQ~, U~ once each
        }
    else:
        algo = {
            "fwd": ("fwd_mfma_kernel", 4 * unit, 4 * unit),
            "bwd_query_side": (qkernel, 8 * unit, 8 * unit),   # S recompute, dP, dQ~, U~
            "bwd_key_side": ("bwd_key_kernel", 4 * unit, 8 * unit),  # dV, dK (+ S/dP recompute, not counted)
        }
    dom = max(algo, key=lambda p: ms[p])
    kname, kflops, _ = algo[dom]
    achieved = kflops / (ms[dom] * 1e-3) / 1e12
    kernels = {}
    for p_, (kn, af, ef) in algo.items():
        kernels[kn] = {"ms": round(ms[p_], 4),
                       "algorithmic_tflops": round(af / (ms[p_] * 1e-3) / 1e12, 2),
                       "frac": round(af / (ms[p_] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                       "executed_frac": round(ef / (ms[p_] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    roofline = {"bound": "mfma", "kernel": kname, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": read_traffic(kname, w.name),
                "fwd_frac": round(fwd_flops / (ms["fwd"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "bwd_frac": round(bwd_flops / (bwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                "step_frac": round(value / PEAK_BF16_TFLOPS, 4),
                "kernels": kernels}

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "D": w.D, "w1": w.w1,
                   "w2": w.w2, "seed": w.seed, "inputs": w.note},
        "fwd_ms": round(ms["fwd"], 4),
        "bwd_ms": round(bwd_ms, 4),
        "fwd_tflops": round(fwd_tf, 2),
        "bwd_tflops": round(bwd_tf, 2),
        "fwd_pct_peak": round(100 * fwd_tf / PEAK_BF16_TFLOPS, 2),
        "bwd_pct_peak": round(100 * bwd_tf / PEAK_BF16_TFLOPS, 2),
        "phase_ms": {p: round(ms[p], 4) for p in phases},
        "fwd_ms_median_min": [round(med(fwd_each), 4), round(fwd_each[0], 4)],
        "bwd_ms_median_min": [round(med(bwd_each), 4), round(bwd_each[0], 4)],
        "wall_s_timed": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if fws and not fused and not args.no_fused:
        # The fused backward (same inputs, its own workspace): Delta, the fused
        # kernel, the reduction of its partial sums; HIP events per stage.
        fwsb = torch.empty(fws, dtype=torch.uint8, device=dev)

        def fused_step(ev=None):
            if ev:
                ev[0].record()
            simplicial_attn_bwd_preprocess(out, do, w.w1, w.w2, fwsb)
            if ev:
                ev[1].record()
            simplicial_attn_bwd_fused(q, k, kp, v, vp, do, lse, w.w1, w.w2, fwsb, w.scale, grads=(dk, dv))
            if ev:
                ev[2].record()
            simplicial_attn_bwd_fused_reduce(q, w.w1, w.w2, fwsb, w.scale, grads=(dq, dkp, dvp))
            if ev:
                ev[3].record()

        for _ in range(args.warmup):
            fused_step()
        fev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            fused_step(fev[i])
        torch.cuda.synchronize()
        fst = [sum(e[j].elapsed_time(e[j + 1]) for e in fev) / args.steps for j in range(3)]
        fb = sum(fst)
        result["fused_backward"] = {
            "bwd_ms": round(fb, 4), "preprocess_ms": round(fst[0], 4), "fused_kernel_ms": round(fst[1], 4),
            "reduce_ms": round(fst[2], 4),
            "bwd_tflops": round(bwd_flops / (fb * 1e-3) / 1e12, 2),
            "bwd_frac": round(bwd_flops / (fb * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "fused_kernel_frac": round(12 * unit / (fst[1] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "workspace_bytes": fws,
            "note": "bwd_fused_kernel: S, dP, dV, dK, dQ~, U~ once each (12 units); fused_reduce_kernel adds "
                    "the per-64-key partial sums of dq, dk', dv' in order",
        }
        del fwsb
    if args.gqa_kv_heads:
        # Grouped-query forward + backward at the same query shape, K, K', V, V'
        # taken from the first Hkv heads of the inputs.
        hkv = args.gqa_kv_heads
        kv = [x[:, :, :hkv].contiguous() for x in (k, kp, v, vp)]
        gkv = tuple(torch.empty_like(kv[0]) for _ in range(4))
        gws = torch.empty(simplicial_attn_bwd_gqa_workspace_size(w.B, w.N, w.H, hkv, w.D, w.w1, w.w2,
                                                                 w.torch_dtype),
                          dtype=torch.uint8, device=dev)

        def gqa_step(ev=None):
            if ev:
                ev[0].record()
            simplicial_attn_fwd_gqa(q, *kv, w.w1, w.w2, w.scale, out=out, lse=lse)
            if ev:
                ev[1].record()
            simplicial_attn_bwd_gqa(q, *kv, out, do, lse, w.w1, w.w2, w.scale, grads=(dq, *gkv),
                                    workspace=gws)
            if ev:
                ev[2].record()

        for _ in range(args.warmup):
            gqa_step()
        gev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            gqa_step(gev[i])
        torch.cuda.synchronize()
        gf = sum(e[0].elapsed_time(e[1]) for e in gev) / args.steps
        gb = sum(e[1].elapsed_time(e[2]) for e in gev) / args.steps
        result["gqa"] = {"kv_heads": hkv, "fwd_ms": round(gf, 4), "bwd_ms": round(gb, 4),
                         "fwd_tflops": round(fwd_flops / (gf * 1e-3) / 1e12, 2),
                         "bwd_tflops": round(bwd_flops / (gb * 1e-3) / 1e12, 2),
                         "step_tflops": round((fwd_flops + bwd_flops) / ((gf + gb) * 1e-3) / 1e12, 2)}
        del kv, gkv, gws
    if args.det:
        # Determinant logits (forward and backward on the MFMA kernels): timed
        # on a 4096-token sequence with the windows and head shape of the main
        # workload.
        db, dh, dn = 1, 16, 4096
        g = torch.Generator(device="cpu").manual_seed(11)
        dq_, dk_, dkp_, dv_, dvp_, ddo = (torch.randn((db, dn, dh, w.D), generator=g)
                                          .to(w.torch_dtype).to(dev) for _ in range(6))
        dws = torch.empty(simplicial_attn_det_bwd_workspace_size(db, dn, dh, w.D, w.w1, w.w2,
                                                                 w.torch_dtype),
                          dtype=torch.uint8, device=dev)
        de = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        dsteps = 3
        for it in range(dsteps + 1):  # one warm-up step, then dsteps timed
            if it == 1:
                de[0].record()
            o_, l_ = simplicial_attn_det_fwd(dq_, dk_, dkp_, dv_, dvp_, w.w1, w.w2, w.scale)
            simplicial_attn_det_bwd(dq_, dk_, dkp_, dv_, dvp_, o_, ddo, l_, w.w1, w.w2, w.scale,
                                    workspace=dws)
        de[1].record()
        torch.cuda.synchronize()
        whole = de[0].elapsed_time(de[1]) / dsteps
        # forward / backward split from one more step
        t_f = torch.cuda.Event(enable_timing=True)
        t_b = torch.cuda.Event(enable_timing=True)
        t_e = torch.cuda.Event(enable_timing=True)
        t_f.record()
        o_, l_ = simplicial_attn_det_fwd(dq_, dk_, dkp_, dv_, dvp_, w.w1, w.w2, w.scale)
        t_b.record()
        simplicial_attn_det_bwd(dq_, dk_, dkp_, dv_, dvp_, o_, ddo, l_, w.w1, w.w2, w.scale,
                                workspace=dws)
        t_e.record()
        torch.cuda.synchronize()
        dunit = float(db) * dh * dn * w.w1 * w.w2 * w.D
        result["det"] = {"config": {"B": db, "H": dh, "N": dn, "D": w.D, "w1": w.w1, "w2": w.w2},
                         "step_ms": round(whole, 3), "fwd_ms": round(t_f.elapsed_time(t_b), 3),
                         "bwd_ms": round(t_b.elapsed_time(t_e), 3),
                         "nominal_tflops": round(16 * dunit / (whole * 1e-3) / 1e12, 2),
                         "kernels": "forward and backward: MFMA kernels (w2 <= 32)"}
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, inputs_cpu, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
