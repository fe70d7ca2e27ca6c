"""Benchmark of the sliced-inference hot path on one MI355X.

Workload (default): ResNet-50-shaped CNN, bf16, batch 8, 3x224x224 inputs,
cut into 4 slices at the stage boundaries, every bottleneck's 3x3 conv (the
resource-dominant op) split into k = 4 sub-slices, autoencoder codecs with
R = 8 at the 3 boundaries.  One step = one pass of the whole hot path over one
batch: the layer profile and the partitioning plan (host), then the sliced
forward pass with boundary encode/decode (device).

Prints one JSON line.  Options: --steps K --warmup W --gpus N (only 1).
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0


def op_flops(m, op):
    """Algorithmic FLOP of a contraction op (2 x multiply-adds), 0 otherwise."""
    T = m.tensors
    out = T[op["out"]]["shape"]
    n_out = 1
    for s in out:
        n_out *= s
    k = op["kind"]
    if k == "conv":
        return 2 * n_out * T[op["inputs"][0]]["shape"][1] * op["kh"] * op["kw"]
    if k == "linear":
        return 2 * n_out * op["nin"]
    return 0


def codec_ratios(m, cuts):
    """Compression ratio per cut: the largest R in 8, 4, 2, 1 that divides the boundary's
    channel count C and leaves C / R a multiple of the 16-byte granule (8 bf16 / 4 fp32)."""
    import synth
    g = 8 if m.dtype == "bf16" else 4
    out = []
    for li in cuts:
        c = synth.boundary_channels(m, li)
        out.append(next((r for r in (8, 4, 2) if c % r == 0 and (c // r) % g == 0), 1))
    return out


def numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


GEMM_SRC = os.path.join(ROOT, "paper_2404_02445_amd", "csrc", "gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_kernel_resnet50_b8_traffic.md")


def gemm_source_hash():
    import hashlib
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def read_counters(path):
    """rocprofv3 --pmc csv -> {dispatch id: (kernel name, value)} for its one counter."""
    import csv
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            out[int(r["Dispatch_Id"])] = (r["Kernel_Name"], float(r["Counter_Value"]))
    return out


# the kernels that run the GEMM ops (conv / linear / AE codec): the implicit-GEMM kernel and the
# patch-staged 3x3 conv
GEMM_KERNELS = ("gemm_kernel", "conv3_halo_kernel")


def summarize_pmc(fetch_csv, write_csv, copy_mib):
    """Markdown summary of per-dispatch HBM-side traffic of the GEMM-op kernels, scaled by the
    counters of a raw copy of known size (copy_mib MiB read and written)."""
    fetch, write = read_counters(fetch_csv), read_counters(write_csv)
    def avg(rows, key):
        keys = key if isinstance(key, tuple) else (key,)
        v = [val for name, val in rows.values() if any(k in name for k in keys)]
        return (sum(v) / len(v), len(v)) if v else (0.0, 0)
    # calibration: the largest copy_kernel dispatch is the known-size copy
    cf = max((val for name, val in fetch.values() if "copy_kernel" in name), default=0.0)
    cw = max((val for name, val in write.values() if "copy_kernel" in name), default=0.0)
    kib = copy_mib * 1024.0
    sf, sw = (kib / cf if cf else float("nan")), (kib / cw if cw else float("nan"))
    gf, n_f = avg(fetch, GEMM_KERNELS)
    gw, n_w = avg(write, GEMM_KERNELS)
    hf, n_h = avg(fetch, "conv3_halo_kernel")
    hw, _ = avg(write, "conv3_halo_kernel")
    rf, n_r = avg(fetch, "splitk_reduce_kernel")
    rw, _ = avg(write, "splitk_reduce_kernel")
    traffic = (gf * sf + gw * sw) * 1024.0
    lines = [
        "# GEMM-op kernels' HBM-side traffic, ResNet-50 bf16 batch 8 (sequential sliced forward)",
        "",
        "Counters: rocprofv3 `FETCH_SIZE` and `WRITE_SIZE` (KiB per dispatch), one pass each,",
        f"scaled by the same counters read for a raw copy of {copy_mib} MiB in the same run.",
        "",
        "| quantity | value |",
        "|---|---|",
        f"| copy calibration: FETCH_SIZE / WRITE_SIZE of the {copy_mib} MiB copy (KiB) | {cf:.1f} / {cw:.1f} |",
        f"| scale factors (read, write) | {sf:.4f} / {sw:.4f} |",
        f"| GEMM-op dispatches, gemm_kernel and conv3_halo_kernel (fetch pass / write pass) | {n_f} / {n_w} |",
        f"| their mean FETCH_SIZE / WRITE_SIZE per dispatch (KiB) | {gf:.1f} / {gw:.1f} |",
        f"| of which conv3_halo_kernel: dispatches, mean FETCH / WRITE (KiB) | {n_h}, {hf:.1f} / {hw:.1f} |",
        f"| splitk_reduce_kernel dispatches, mean FETCH / WRITE (KiB) | {n_r}, {rf:.1f} / {rw:.1f} |",
        f"| traffic per GEMM-op launch (scaled read + write, bytes) | {traffic:.0f} |",
        "",
        "```",
        f"gemm_hip_sha256: {gemm_source_hash()}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        "```",
    ]
    return "\n".join(lines)


def committed_traffic():
    """Traffic per gemm_kernel launch from the committed counter summary, or None when the
    summary is missing or the kernel source has changed since it was taken."""
    try:
        txt = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    kv = dict(l.split(": ", 1) for l in txt.splitlines() if l.startswith(("gemm_hip_sha256:", "traffic_bytes_per_launch:")))
    if kv.get("gemm_hip_sha256") != gemm_source_hash():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def op_bytes(m, op, es):
    """Algorithmic bytes of a contraction op: weights + bias + inputs (incl. residual) + output, once each."""
    T = m.tensors
    b = sum(numel(T[t]["shape"]) for t in op["inputs"]) + numel(T[op["out"]]["shape"])
    if op["kind"] == "conv":
        b += op["cout"] * T[op["inputs"][0]]["shape"][1] * op["kh"] * op["kw"] + op["cout"]
    elif op["kind"] == "linear":
        b += op["nout"] * op["nin"] + op["nout"]
    return b * es


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="workload 1..5 (default 2: ResNet-50, batch 8)")
    ap.add_argument("--codec", choices=["ae", "raw"], default="ae")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-op-timing", action="store_true")
    ap.add_argument("--op-report", action="store_true", help="print per-op times (ms) to stderr")
    ap.add_argument("--pipeline", type=int, default=2, metavar="D",
                    help="run batches through the slice pipeline with D code slots per cut (0: sequential)")
    ap.add_argument("--replicas", type=int, default=0,
                    help="pipeline instances of the sliced model; 0: try 1, 2 and 3 before the timed region "
                         "and keep the fastest (3 instances + torch's stream = 4 hardware queues)")
    ap.add_argument("--stream-per-slice", type=int, default=0, help="1: one stream per slice, 0: one per instance")
    ap.add_argument("--no-graphs", action="store_true",
                    help="launch the pipeline's kernels one by one instead of replaying captured HIP graphs")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run a raw boundary copy of this many MiB per step (counter calibration)")
    ap.add_argument("--plan", choices=["config", "measured"], default="config",
                    help="config: the workload's prescribed cuts and k; measured: Alg. 1 free mode with the "
                         "parallelism search over t_p(l, k) measured on this GPU")
    ap.add_argument("--k-max", type=int, default=4, help="largest sub-slice count of the measured search")
    ap.add_argument("--no-measured-plan", action="store_true",
                    help="skip the measured-profile planning pass (profiler runs: only the step's launches)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the traffic summary from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) "
                         "of this script with --calibrate-copy-mib, and exit")
    args = ap.parse_args()
    if args.summarize_pmc:
        print(summarize_pmc(*args.summarize_pmc, args.calibrate_copy_mib or 64))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(slices and sub-slices run on one device); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2404_02445_amd as P
    import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    m = synth.build(args.config)
    x_host = synth.make_input(m)
    sm = P.SlicedModel(m, device=dev)
    s = m.slicing
    plan_kw = dict(n_slices=s["n_slices"], allowed_cut=s["allowed_cut"], elim_tau=s["elim_tau"],
                   k_override=s["k_override"])
    x = torch.from_numpy(x_host).to(dev)
    # measured-profile planning (Alg. 1 + Eq. 5 over t_p measured here), reported in every run
    if args.no_measured_plan and args.plan == "measured":
        sys.exit("--plan measured needs the measured-profile pass")
    measured = None
    if not args.no_measured_plan:
        mplan, tp, mprof = sm.measured_plan(x, k_max=args.k_max, reps=3)
        measured = {"k_max": args.k_max, "n_slices": mplan.n_slices, "slice_end": mplan.slice_end,
                    "k": mplan.k, "t_tau_ms": round(mplan.t_tau * 1e3, 4),
                    "tp_ms_by_k": [round(sum(r[e] for r in tp) * 1e3, 4) for e in range(args.k_max)]}
    if args.plan == "measured":
        plan = mplan
        prof_fixed = mprof
        plan_kw = dict(elim_tau=0.05, k_max=args.k_max, tp_table=tp, ta_table=[[0.0] * args.k_max for _ in tp])
    else:
        plan = sm.plan()
        prof_fixed = None
    cuts = plan.slice_end[:-1]
    ratios = codec_ratios(m, cuts)
    cw = synth.make_codec_weights(m, cuts, ratio=ratios) if args.codec == "ae" else None
    codecs, keep = sm.codecs(plan, args.codec, cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    stream = torch.cuda.current_stream()
    calib = None
    if args.calibrate_copy_mib:
        nb = args.calibrate_copy_mib << 20
        calib = (torch.empty(nb, dtype=torch.uint8, device=dev), torch.empty(nb, dtype=torch.uint8, device=dev))

    def step():
        prof = prof_fixed or sm.profile()                     # a1-a2: layer profiles (Eq. 1-4)
        pl = P.mopar_plan_slices(prof, **plan_kw)             # a3-a4: HyPAD plan and sub-slice counts
        sm.forward(pl, x, out, codecs, codes, ws)             # a5-a10: sliced forward with codec hand-off
        return pl

    def sequential_run(steps):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(steps):
            step()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        per = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
        return evs[0].elapsed_time(evs[-1]), wall, per

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    pipe = None
    replicas, replica_tuning = args.replicas, None
    if args.pipeline:
        use_graphs = not args.no_graphs and not args.stream_per_slice

        def make_pipe(r):
            pp = sm.pipeline(plan, args.codec, cw, depth=args.pipeline, replicas=r,
                             stream_per_slice=bool(args.stream_per_slice))
            return pp.use_graphs(True) if use_graphs else pp

        def pstep_on(pp):
            prof = prof_fixed or sm.profile()
            pl = P.mopar_plan_slices(prof, **plan_kw)
            pp.submit(x, out)
            return pl

        if replicas == 0:
            # instance count: each candidate warmed up, then timed over a few steps, before
            # (and outside) the timed region
            replica_tuning = {}
            n_try = max(10, min(args.steps, 20))
            for r in (1, 2, 3):
                pp = make_pipe(r)
                for _ in range(max(args.warmup, 5)):
                    pstep_on(pp)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for _ in range(n_try):
                    pstep_on(pp)
                torch.cuda.synchronize()
                replica_tuning[r] = round(m.batch * n_try / (time.perf_counter() - t0), 1)
                del pp
            replicas = max(replica_tuning, key=replica_tuning.get)
        pipe = make_pipe(replicas)

        def pstep():
            return pstep_on(pipe)

        for _ in range(args.warmup):
            pstep()
        torch.cuda.synchronize()

    # --- timed region: exactly K steps ------------------------------------------------
    if pipe is None:
        total_ms, wall, per_step = sequential_run(args.steps)
    else:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            pstep()
        t_host = time.perf_counter() - t0
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        total_ms = wall * 1e3
        seq_ms, _, per_step = sequential_run(args.steps)   # per-batch latency, one at a time
        seq_value = m.batch * args.steps / (seq_ms / 1e3)
    ms_per_step = total_ms / args.steps
    value = m.batch * args.steps / (total_ms / 1e3)
    if pipe is None:
        seq_value = value
        t_host = None

    # planning cost on the host (already inside the steps above, overlapped with the GPU)
    tp0 = time.perf_counter()
    for _ in range(20):
        P.mopar_plan_slices(prof_fixed or sm.profile(), **plan_kw)
    plan_us = (time.perf_counter() - tp0) / 20 * 1e6

    res = {
        "metric": "inferences/s per sliced model at 1 GPU; RD-op MFMA util %; boundary codec GB/s",
        "value": round(value, 2),
        "unit": "inferences/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": m.dtype,
        "data": "synthetic (seeded N(0,1) inputs, random-init weights of the named architecture)",
        "config": {"workload": f"{m.name}: {m.dtype}, batch {m.batch}, {plan.n_slices} slices at "
                               f"{cuts}, RD k={max(plan.k)}, {args.codec} codec"
                               + (f" R={ratios}" if args.codec == "ae" else ""),
                   "batch": m.batch, "slices": plan.n_slices, "k": plan.k, "codec": args.codec},
        "latency_ms": {"p50": round(statistics.median(per_step), 4),
                       "p95": round(float(np.percentile(per_step, 95)), 4)},
        "mode": (f"slice pipeline: {replicas} instance(s) x {plan.n_slices} slices on "
                 f"{len(set(id(s) for s in pipe.streams))} streams, {args.pipeline} code slots per (instance, cut); "
                 f"latency_ms is one batch at a time") if pipe else "sequential: one batch at a time",
        "replicas": replicas if pipe else None,
        "graphs": bool(pipe) and not args.no_graphs and not args.stream_per_slice,
        "replica_tuning_inf_per_s": replica_tuning,
        "wall_s_timed_region": round(wall, 4),
        "sequential_value": round(seq_value, 2),
        "host_plan_us": round(plan_us, 1),
        "host_submit_ms_per_step": round(t_host / args.steps * 1e3, 4) if t_host is not None else None,
        "plan": args.plan,
        "measured_plan": measured,
    }

    # --- per-op timing pass (HIP events on the launch stream, same steps) ----------------
    if not args.no_op_timing:
        sm.set_timing(True)
        n_t = min(args.steps, 20)
        gemm_ms = rd_ms = 0.0
        gemm_fl = rd_fl = 0
        gemm_launches = 0
        gemm_bytes = 0
        es = 2 if m.dtype == "bf16" else 4
        enc_ms = [0.0] * len(cuts)
        dec_ms = [0.0] * len(cuts)
        bw_ms = 0.0
        bw_bytes = 0
        per_op = [0.0] * len(m.ops)
        # AE codec GEMMs (encode and decode of every cut) are gemm_kernel launches too
        codec_fl, codec_bytes = [], []
        for c, li in enumerate(cuts):
            shp = m.tensors[m.layer_output_tid(li)]["shape"]
            ch = synth.boundary_channels(m, li)
            pos = numel(shp) // ch
            ce = ch // ratios[c] if args.codec == "ae" else ch
            codec_fl.append(2 * pos * ch * ce)
            codec_bytes.append((pos * ch + pos * ce + ch * ce + ce) * es)
        for _ in range(n_t):
            step()
            ops_ms, cut_ms = sm.op_times()
            for i, t in enumerate(ops_ms):
                per_op[i] += t / n_t
            for i, op in enumerate(m.ops):
                t = ops_ms[i]
                if op["kind"] in ("conv", "linear"):
                    f = op_flops(m, op)
                    gemm_ms += t
                    gemm_fl += f
                    gemm_bytes += op_bytes(m, op, es)
                    gemm_launches += 1
                    if op.get("rd"):
                        rd_ms += t
                        rd_fl += f
                else:
                    bw_ms += t
                    ins = sum(numel(m.tensors[tt]["shape"]) for tt in op["inputs"])
                    bw_bytes += (ins + numel(m.tensors[op["out"]]["shape"])) * es
            for c, (e, d) in enumerate(cut_ms):
                enc_ms[c] += e
                dec_ms[c] += d
                if args.codec == "ae":
                    gemm_ms += e + d
                    gemm_fl += 2 * codec_fl[c]
                    gemm_bytes += 2 * codec_bytes[c]
                    gemm_launches += 2
        sm.set_timing(False)
        if args.op_report:
            for i, op in enumerate(m.ops):
                sh = m.tensors[op["out"]]["shape"]
                f = op_flops(m, op)
                tf = f / (per_op[i] * 1e-3) / 1e12 if per_op[i] > 0 and f else 0.0
                print(f"op {i:3d} {op['name']:<14} {op['kind']:<9} k={plan.k[op['layer']] if op.get('rd') else 1} "
                      f"out={sh} {per_op[i] * 1e3:8.2f} us {tf:7.1f} TF/s", file=sys.stderr)
        # codec traffic: read the tensor + write the code (encode) and back (decode), weights once
        codec = []
        for c, li in enumerate(cuts):
            shp = m.tensors[m.layer_output_tid(li)]["shape"]
            tb = numel(shp) * es
            r = ratios[c] if args.codec == "ae" else 1
            cbytes = tb // r
            wb = 0
            if args.codec == "ae":
                ch = synth.boundary_channels(m, li)
                wb = (2 * ch * (ch // r) + ch + ch // r) * es
            e_avg, d_avg = enc_ms[c] / n_t, dec_ms[c] / n_t
            codec.append({"cut_after": m.layers[li], "tensor_MB": round(tb / 1e6, 3),
                          "encode_us": round(e_avg * 1e3, 2), "decode_us": round(d_avg * 1e3, 2),
                          "encode_GBs": round((tb + cbytes + wb / 2) / (e_avg * 1e-3) / 1e9, 1),
                          "decode_GBs": round((tb + cbytes + wb / 2) / (d_avg * 1e-3) / 1e9, 1)})
        gemm_avg_ms = gemm_ms / max(gemm_launches, 1)
        achieved = gemm_fl / (gemm_ms * 1e-3) / 1e12
        peak = PEAK_TFLOPS[m.dtype]
        traffic = committed_traffic() if m.name.startswith("resnet50") else None
        res["roofline"] = {
            "bound": "mfma",
            "kernel": "gemm_kernel (conv3_halo_kernel for the patch-staged 3x3 convs): every conv / linear "
                      "op and AE codec GEMM of a step (device time of each launch from its own HIP event "
                      "pair; an op's time also holds the stem's layout conversion and the split-K reduce "
                      "of split ops)",
            "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": round(traffic) if traffic is not None else None,
            "flop_per_launch": round(gemm_fl / max(gemm_launches, 1)),
            "algorithmic_bytes_per_launch": round(gemm_bytes / max(gemm_launches, 1)),
            "avg_launch_us": round(gemm_avg_ms * 1e3, 2),
            "launches_per_step": gemm_launches // n_t,
        }
        res["rd_mfma_util"] = {"achieved_TFLOPs": round(rd_fl / (rd_ms * 1e-3) / 1e12, 2) if rd_ms else None,
                               "frac_of_peak": round(rd_fl / (rd_ms * 1e-3) / 1e12 / peak, 4) if rd_ms else None,
                               "rd_ms_per_step": round(rd_ms / n_t, 4)}
        res["codec"] = codec
        # ideal step time: every op (and codec GEMM) at its own roofline, max(FLOP / P, bytes / B)
        B = PEAK_HBM_GBS * 1e9
        ideal_s = 0.0
        rd_ideal_s = 0.0
        for op in m.ops:
            f = op_flops(m, op)
            if op["kind"] in ("conv", "linear"):
                by = op_bytes(m, op, es)
            else:
                by = (sum(numel(m.tensors[t]["shape"]) for t in op["inputs"]) + numel(m.tensors[op["out"]]["shape"])) * es
            t_op = max(f / (peak * 1e12), by / B)
            ideal_s += t_op
            if op.get("rd"):
                rd_ideal_s += f / min(peak * 1e12, f / by * B)
        if args.codec == "ae":
            for c in range(len(cuts)):
                ideal_s += 2 * max(codec_fl[c] / (peak * 1e12), codec_bytes[c] / B)
        res["ideal_step"] = {"ms": round(ideal_s * 1e3, 4),
                             "frac_of_sequential_p50": round(ideal_s * 1e3 / res["latency_ms"]["p50"], 4)}
        if rd_ms:
            res["rd_mfma_util"]["attainable_frac"] = round(rd_ideal_s * 1e3 / (rd_ms / n_t), 4)
        res["bandwidth_ops"] = {"ms_per_step": round(bw_ms / n_t, 4),
                                "GBs": round(bw_bytes / (bw_ms * 1e-3) / 1e9, 1) if bw_ms else None}
        res["gemm_ms_per_step"] = round(gemm_ms / n_t, 4)

    # --- boundary codec in isolation, cold cache (a 512 MB write between runs evicts the
    #     256 MB Infinity Cache), against a raw copy of the same tensor ------------------
    if args.codec == "ae" and not args.no_op_timing:
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        raw = P.make_codec("raw")
        iso = []
        for c, li in enumerate(cuts):
            shp = list(m.tensors[m.layer_output_tid(li)]["shape"])
            gshape = [shp[0]] + shp[2:] + [shp[1]] if len(shp) == 4 else shp      # NHWC on the device
            tdt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
            xt = torch.randn(gshape, device=dev).to(tdt)
            yt = torch.empty_like(xt)
            code = torch.empty(P.mopar_boundary_code_bytes(codecs[c], shp, m.dtype), dtype=torch.uint8, device=dev)
            rawbuf = torch.empty_like(xt)

            def cold(fn, reps=5):
                ts = []
                for _ in range(reps):
                    scratch.fill_(1)
                    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a0.record(stream)
                    fn()
                    a1.record(stream)
                    torch.cuda.synchronize()
                    ts.append(a0.elapsed_time(a1))
                return statistics.median(ts)
            t_enc = cold(lambda: P.mopar_boundary_encode(codecs[c], shp, m.dtype, xt, code))
            t_dec = cold(lambda: P.mopar_boundary_decode(codecs[c], shp, m.dtype, code, yt))
            t_raw = cold(lambda: P.mopar_boundary_encode(raw, shp, m.dtype, xt, rawbuf))
            tb = numel(shp) * es
            e_gbs = (tb + code.numel()) / (t_enc * 1e-3) / 1e9
            d_gbs = (tb + code.numel()) / (t_dec * 1e-3) / 1e9
            r_gbs = 2 * tb / (t_raw * 1e-3) / 1e9
            iso.append({"cut_after": m.layers[li], "encode_GBs": round(e_gbs, 1), "decode_GBs": round(d_gbs, 1),
                        "raw_copy_GBs": round(r_gbs, 1), "encode_frac_of_8TBs": round(e_gbs / PEAK_HBM_GBS, 3),
                        "decode_frac_of_8TBs": round(d_gbs / PEAK_HBM_GBS, 3),
                        "encode_frac_of_raw": round(e_gbs / r_gbs, 3), "decode_frac_of_raw": round(d_gbs / r_gbs, 3)})
        res["codec_isolated_cold"] = iso
        del scratch

    if calib is not None:   # known-size raw copies: the reference for HBM counter scaling
        raw = P.make_codec("raw")
        n = calib[0].numel() // 2
        for _ in range(3):
            P.mopar_boundary_encode(raw, (n,), "bf16", calib[0], calib[1])
        torch.cuda.synchronize()

    # --- CPU baseline: the oracle on a bounded sample of the same workload -------------
    if not args.no_cpu_baseline:
        import oracle
        cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        os.environ.setdefault("OMP_NUM_THREADS", str(cores))
        oracle.lib()
        done = 0
        t0 = time.perf_counter()
        while True:
            oracle.forward(m, x_host, k=plan.k, cuts=cuts, codecs=cw, sample=[done % m.batch])
            done += 1
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        el = time.perf_counter() - t0
        cpu_model = ""
        try:
            cpu_model = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name"))
        except (OSError, StopIteration):
            pass
        res["cpu_baseline"] = {"value": round(done / el, 4), "unit": "inferences/s", "cores": cores,
                               "nproc": len(os.sched_getaffinity(0)), "cpu_model": cpu_model,
                               "kind": "oracle",
                               "sample": f"{done} single-image forward(s) of the same sliced workload "
                                         f"(same plan, codecs and weights), {el:.1f} s"}
    print(json.dumps(res))


if __name__ == "__main__":
    main()
