"""Benchmark of the K-interval attention hot path on one MI355X.

One step = kia_attn_fwd + kia_attn_bwd over one batch of the GPT-2-124M
attention workload (B8 H12 T1024 d64, causal, fp32; FWM tau = 8, Nearest,
Prob-STE, K = 4, full calibration gradient), inputs resident in HBM before
the timed region. The GPU's clock and power management need tens of ms of
sustained load to settle (from idle, step times rise from 0.61 to 0.74 ms
and fall back to a steady 0.555 ms over about 45 steps), so steps first run
for --settle-ms (reported under "settle"), then the W warm-up steps, then the
K steps are timed as a training loop runs them, then run again with two HIP
events recorded around every kernel on its launch stream, for the
per-kernel durations and the roofline of the dominant kernel. Prints one
JSON line (metric, value in counted TFLOP/s from the first pass, roofline,
and the oracle's CPU time on the same workload).

Counted FLOPs follow the FlashAttention causal convention: 2 GEMM units in
the forward (Q K^T, P V) and 5 in the backward (S recompute, dP, dV, dQ,
dK), each B*H*T^2*d flops. Executed: forward 3 (Q K^T once, P V, and the
O^L product of Prob-STE), bwd_main 3 (dP, dV, dK: the scores' decided
positions are the forward's), bwd_dq 1.

roofline.per_kernel gives the same counted-flop figures for each of the
three MFMA kernels (forward 2 units, bwd_main 3, bwd_dq 1).

--deterministic times the deterministic backward (kia_set_deterministic:
every reduction in a fixed order); config.deterministic records it.

roofline.mfma_probe is the fp32 matrix-core rate this GPU sustains on a
stream of independent MFMAs (kia_mfma_peak_probe) and its shader clock
during that stream: the measured ceiling beside the published peak.

roofline.traffic is the HBM byte count per launch of the dominant kernel
from the rocprofv3 FETCH_SIZE/WRITE_SIZE summaries under profiles/, reported
for the two profiled configurations (the default workload and operator in
fp32; the 1B-scale workload with bf16 inputs and its default operator) and
only while that kernel's sources hash to the profiled version (else null);
roofline.per_kernel gives each MFMA kernel's bytes and GB/s the same way.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

PEAK_FP32_MFMA = 157.3  # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2500.0  # TFLOP/s, MI355X dense bf16 matrix
PEAK_HBM = 8000.0       # GB/s


ROOT = os.path.dirname(os.path.abspath(__file__))
# counter summaries of the profiled configurations, by input type
TRAFFIC = {False: os.path.join(ROOT, "profiles", "traffic_gpt2_124m.md"),
           True: os.path.join(ROOT, "profiles", "traffic_scale_1b_bf16.md")}
PROFILED_WORKLOAD = {False: "gpt2_124m", True: "scale_1b"}
KERNEL_SOURCES = {
    False: {"kia_fwd": ["kia_fwd.hip", "kia_device.hpp", "kia_kernels.hpp"],
            "kia_bwd_main": ["kia_bwd.hip", "kia_device.hpp", "kia_kernels.hpp"],
            "kia_bwd_dq": ["kia_bwd.hip", "kia_device.hpp", "kia_kernels.hpp"]},
    True: {n: ["kia_bf16.hip", "kia_device.hpp", "kia_kernels.hpp"]
           for n in ("kia_fwd", "kia_bwd_main", "kia_bwd_dq")},
}


def mfma_probe(kia, torch, stream):
    """Sustained fp32 matrix-core rate and shader clock on this GPU from
    kia_mfma_peak_probe: 8 workgroups of 4 waves per CU, 2048 rounds of 4
    independent MFMAs each, best of 5 timed launches after one warm-up."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    wg, iters = 8 * cus, 2048
    out = torch.zeros(4, dtype=torch.int64, device="cuda")
    kia.kia_mfma_peak_probe(out, wg, iters, stream)
    best = float("inf")
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        kia.kia_mfma_peak_probe(out, wg, iters, stream)
        b.record(stream)
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b))
    t = out.cpu().tolist()
    flops = wg * 4 * iters * 4 * 4096
    tflops = flops / (best * 1e-3) / 1e12
    return {"tflops": round(tflops, 2), "frac_of_peak": round(tflops / PEAK_FP32_MFMA, 4),
            "clock_ghz": round((t[1] - t[0]) / max(1, t[3] - t[2]) * 0.1, 3),
            "workgroups": wg, "iters": iters}


def profiled_traffic(kernel, b16=False):
    """HBM bytes per launch of `kernel` (bf16-input kernels if b16) from the
    committed counter summary, or None when the kernel's sources changed
    since the counters were taken."""
    try:
        text = open(TRAFFIC[b16]).read()
        table = json.loads(re.search(r"```json\n(.*?)```", text, re.S).group(1))
        entry = table[kernel]
    except (OSError, AttributeError, KeyError, ValueError):
        return None
    if source_hash(kernel, b16) != entry["source_sha256_16"]:
        return None
    return int(entry["bytes_per_launch"])


def source_hash(kernel, b16=False):
    """First 16 hex digits of sha256 over the kernel's sources with comments
    and whitespace removed (a comment edit does not change the kernel)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[b16][kernel]:
        with open(os.path.join(ROOT, "paper_2609_33591_amd", "csrc", name)) as f:
            code = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", "", code)
        h.update("".join(code.split()).encode())
    return h.hexdigest()[:16]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, q, k, v, dO, n_slices=0):
    """The fp64 oracle (test infrastructure) on the workload's first
    n_slices (b,h) slices (all if 0), one fwd+bwd step on the host cores it
    may use; returned in the metric's unit (counted TFLOP/s, scaled to the
    slices timed; 'extrapolated' when not all slices were timed)."""
    import oracle
    oracle.build(force=False)
    B, H, T, d = q.shape
    n = B * H if n_slices <= 0 else min(n_slices, B * H)
    args = [x.double().numpy() for x in (q, k, v)]
    t0 = time.perf_counter()
    oracle.attn_fwd(*args, K=w["K"], calib=w["calib"], tau=w["tau"], recon=w["recon"],
                    causal=True, slices=(0, n))
    oracle.attn_bwd(*args, dO.double().numpy(), K=w["K"], calib=w["calib"], tau=w["tau"],
                    recon=w["recon"], ste=w["ste"], detach=w["detach"], causal=True,
                    slices=(0, n))
    dt = time.perf_counter() - t0
    flops = 7.0 * n * T * T * d
    part = "the whole workload" if n == B * H else \
        f"{n} of the {B * H} (b,h) slices (value extrapolated to the workload's rate)"
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s",
            "cores": oracle.max_threads(), "kind": "oracle",
            "sample": f"{part}, one fwd+bwd step, fp64 C oracle, {dt:.2f} s wall",
            "extrapolated": n < B * H,
            "host": {"affinity_cpus": len(os.sched_getaffinity(0)),
                     "os_cpu_count": os.cpu_count(),
                     "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS"),
                     "cpu_model": cpu_model()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    # the GPU's clock and power management settle only after tens of ms of
    # sustained load (step times 0.61 -> 0.74 -> 0.555 ms over the first ~45
    # steps from idle): before the warm-up steps, steps run until this much
    # time has passed (reported under "settle")
    ap.add_argument("--settle-ms", type=float, default=100.0)
    ap.add_argument("--workload", default="gpt2_124m")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-slices", type=int, default=0,
                    help="time the oracle on this many (b,h) slices only and extrapolate "
                         "(0: all)")
    ap.add_argument("--input-dtype", choices=("f32", "bf16"), default="f32",
                    help="bf16: q, k, v, dO in bf16 through kia_attn_*_bf16 (bf16 MFMA, "
                         "fp32 accumulation)")
    ap.add_argument("--output-dtype", choices=("f32", "bf16"), default="f32",
                    help="bf16 (with --input-dtype bf16): o, dq, dk, dv in bf16 through "
                         "kia_attn_*_bf16o")
    ap.add_argument("--sweep-variant", type=int, default=None,
                    help="variant i (0..17) of the sweep at the bench shape (calibration, "
                         "reconstruction, surrogate, K, detach and seed)")
    ap.add_argument("--recon", default=None,
                    choices=("lerp", "nearest", "softmax", "bf16_exp", "fp8_exp"),
                    help="override the workload's weight function (softmax, bf16_exp, "
                         "fp8_exp: the exponential baselines, fp32 inputs only)")
    ap.add_argument("--calib", default=None, choices=("minmax", "fwm", "resolved"),
                    help="override the workload's calibration")
    ap.add_argument("--probe", action="store_true",
                    help="after the timed steps, time the geometry probe (kia_geometry_probe) "
                         "on the forward's statistics, reported under 'geometry_probe'")
    ap.add_argument("--deterministic", action="store_true",
                    help="time the deterministic backward (kia_set_deterministic: every "
                         "reduction in a fixed order, no split grids)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed steps, run one plain device copy of this many MiB "
                         "(the known-size reference that scales HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the "
              "operator shards over (b, h) with no communication between GPUs",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_33591_amd as kia
    from paper_2609_33591_amd.inputs import WORKLOADS, make_inputs

    from paper_2609_33591_amd.inputs import sweep_variants
    w = dict(WORKLOADS[args.workload])
    if args.sweep_variant is not None:
        w.update(sweep_variants()[args.sweep_variant])
    if args.recon:
        w["recon"] = args.recon
    if args.calib:
        w["calib"] = args.calib
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    K, calib, tau, recon, ste, det = w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"]
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], qk_scale=w["qk_scale"])
    b16 = args.input_dtype == "bf16"
    b16o = args.output_dtype == "bf16"
    if b16o and not b16:
        sys.exit("--output-dtype bf16 needs --input-dtype bf16")
    if b16:
        q, k, v, dO = (x.to(torch.bfloat16) for x in (q, k, v, dO))
    qg, kg, vg, dg = (x.cuda() for x in (q, k, v, dO))
    odt = torch.bfloat16 if b16o else torch.float32
    o = torch.empty(qg.shape, dtype=odt, device="cuda")
    dq, dk, dv = (torch.empty(qg.shape, dtype=odt, device="cuda") for _ in range(3))
    stats = kia.new_stats(B, H, T, d, recon, ste, True, bf16_out=b16o)
    stream = torch.cuda.current_stream()
    if b16o:
        fwd, bwd = kia.kia_attn_fwd_bf16o, kia.kia_attn_bwd_bf16o
    else:
        fwd = kia.kia_attn_fwd_bf16 if b16 else kia.kia_attn_fwd
        bwd = kia.kia_attn_bwd_bf16 if b16 else kia.kia_attn_bwd
    peak = PEAK_BF16_MFMA if b16 else PEAK_FP32_MFMA
    kia.kia_set_deterministic(args.deterministic)

    def step():
        fwd(qg, kg, vg, o, stats, K, calib, tau, recon, ste, det, True, stream)
        bwd(qg, kg, vg, o, dg, stats, dq, dk, dv, K, calib, tau, recon, ste, det, True, stream)

    # clock settle: whole steps, in batches of 10, until settle_ms have passed
    t_set, n_set = time.perf_counter(), 0
    while (time.perf_counter() - t_set) * 1e3 < args.settle_ms:
        for _ in range(10):
            step()
        n_set += 10
        torch.cuda.synchronize()
    settle = {"steps": n_set, "ms": round((time.perf_counter() - t_set) * 1e3, 1)}
    for _ in range(args.warmup):
        step()
    # the K timed steps, as a training loop runs them (no per-launch events)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    # the same K steps again with every kernel bracketed by two events on its
    # launch stream: per-kernel durations for kernel_ms and the roofline (the
    # event records add about 2 us per launch, so this pass is not the value)
    kia.kia_timing_enable(True)
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record(stream)
    for _ in range(args.steps):
        step()
    f1.record(stream)
    torch.cuda.synchronize()
    hooked_ms = f0.elapsed_time(f1)
    kern = {}
    for name in ("kia_fwd", "kia_bwd_pre", "kia_bwd_main", "kia_bwd_dq", "kia_bwd_ties",
                 "kia_bwd_p1", "kia_cast_bf16"):
        ms, n = kia.kia_timing_read(name)
        kern[name] = (ms / n if n else 0.0, n)
    kia.kia_timing_enable(False)

    ms_step = total_ms / args.steps
    unit = B * H * T * T * d  # one counted GEMM unit (causal half, 2 flops/MAC)
    tflops = 7.0 * unit / (ms_step * 1e-3) / 1e12
    # dominant kernel and its algorithmic flops per launch: the forward
    # kernel counts Q K^T and P V (2 units; O^L is executed, not counted),
    # bwd_main dP, dV, dK (3 units), bwd_dq the dQ product (1 unit)
    UNITS = {"kia_fwd": 2, "kia_bwd_main": 3, "kia_bwd_dq": 1}
    default_config = (args.workload == "gpt2_124m" and not b16 and not args.recon
                      and not args.calib and args.sweep_variant is None
                      and not args.deterministic)
    # the counters were taken on the default operator of two configurations:
    # the GPT-2-124M workload in fp32 and the 1B-scale one with bf16 inputs
    profiled = (args.workload == PROFILED_WORKLOAD[b16] and not b16o and not args.recon
                and not args.calib and args.sweep_variant is None and not args.deterministic)
    traffic = {n: profiled_traffic(n, b16) if profiled else None for n in UNITS}
    dom = max(UNITS, key=lambda n: kern[n][0])
    units = UNITS[dom]
    achieved = units * unit / (kern[dom][0] * 1e-3) / 1e12

    def gbs(n):
        return (round(traffic[n] / (kern[n][0] * 1e-3) / 1e9, 1)
                if traffic[n] and kern[n][0] > 0 else None)

    roof = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 3),
            "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic[dom],
            "hbm_gbs": gbs(dom),
            "avg_ms": round(kern[dom][0], 4),
            "flops_per_launch": units * unit,
            # the same figures for each of the three MFMA kernels (the forward
            # and bwd_main take nearly equal times, so either can dominate)
            "per_kernel": {n: {"units": u, "avg_ms": round(kern[n][0], 4),
                               "achieved": round(u * unit / (kern[n][0] * 1e-3) / 1e12, 3),
                               "frac": round(u * unit / (kern[n][0] * 1e-3) / 1e12 / peak, 4),
                               "traffic": traffic[n], "hbm_gbs": gbs(n)}
                           for n, u in UNITS.items() if kern[n][0] > 0}}
    line = {
        "metric": ("K-interval attn fwd+bwd TFLOP/s at B8 H12 T1024 d64 causal; % fp32 MFMA peak"
                   if default_config else
                   f"{'K-interval' if recon in ('lerp', 'nearest') else recon} attn fwd+bwd "
                   f"TFLOP/s at B{B} H{H} T{T} d{d} causal, "
                   f"{'bf16' if b16 else 'fp32'} inputs{', bf16 outputs' if b16o else ''}"),
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": settle,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if b16 else "f32",
        "data": f"synthetic: q,k,v,dO i.i.d. N(0,1) fp32 (CPU torch.Generator seed {w['seed']})"
                f"{', rounded to bf16' if b16 else ''}, resident in HBM before timing",
        "config": {"workload": f"{args.workload} attention", "B": B, "H": H, "T": T, "d": d,
                   "causal": True, "K": K, "calib": calib, "tau": tau, "recon": recon,
                   "ste": ste, "detach": det, "input_dtype": "bf16" if b16 else "f32",
                   "output_dtype": "bf16" if b16o else "f32",
                   "sweep_variant": args.sweep_variant, "deterministic": args.deterministic,
                   "parallelism": "single GPU"},
        "pct_fp32_mfma_peak": round(100 * tflops / PEAK_FP32_MFMA, 2),
        "pct_mfma_peak_of_input_dtype": round(100 * tflops / peak, 2),
        "tokens_per_s": round(B * T / (ms_step * 1e-3), 1),
        "kernel_ms": {n: round(v[0], 4) for n, v in kern.items()},
        "ms_per_step_with_kernel_events": round(hooked_ms / args.steps, 4),
        "roofline": roof,
    }
    if not b16:
        roof["mfma_probe"] = mfma_probe(kia, torch, stream)
    if args.probe:
        # two passes of score sub-tiles per (query, key) pair plus the
        # per-key statistics; counted as 2 GEMM units (Q K^T twice)
        gout = torch.empty((B, H, T, 10), dtype=torch.float32, device="cuda")
        fwd(qg, kg, vg, o, stats, K, calib, tau, recon, ste, det, True, stream)
        kia.kia_geometry_probe(qg, kg, stats, gout, K, calib, tau, recon, True, stream)
        torch.cuda.synchronize()
        kia.kia_timing_enable(True)
        for _ in range(args.steps):
            kia.kia_geometry_probe(qg, kg, stats, gout, K, calib, tau, recon, True, stream)
        ms, n = kia.kia_timing_read("kia_geometry")
        kia.kia_timing_enable(False)
        pms = ms / max(n, 1)
        line["geometry_probe"] = {"avg_ms": round(pms, 4), "launches": n,
                                  "tflops_2units": round(2 * unit / (pms * 1e-3) / 1e12, 3)}
    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, q, k, v, dO, args.cpu_slices)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
