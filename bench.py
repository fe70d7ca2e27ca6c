"""Benchmark of the sliced-inference hot path on one MI355X.

Headline workload (default ``--config 5``, the largest of the five): the 2-layer
LSTM language model, bf16, batch 64 x 128 tokens, cut into 3 slices (embedding /
LSTM / projection), the 1024 -> 32000 vocabulary projection (the
resource-dominant op) split into k = 8 sub-slices, autoencoder codecs with
R = 8 at both boundaries.  One step = one pass of the whole hot path over one
batch: the layer profile and the partitioning plan (host; the batch runs the
plan computed in its step), then the sliced forward pass with boundary
encode / decode (device).

The line also carries ``per_config``: the same measurement, shorter, for the
other four workloads (tiny VGG, ResNet-50, VGG-16, BERT-base).

Prints one JSON line.  Options: --steps K --warmup W --gpus N (only 1).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0
METRIC = "inferences/s per sliced model at 1 GPU; RD-op MFMA util %; boundary codec GB/s"
HEADLINE_CFG = 5
CSRC = os.path.join(ROOT, "paper_2404_02445_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


def numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


def codec_ratio(c):
    """R = 8 (the smallest ratio the paper studies) when it divides C, else 4, 2 or 1."""
    return next((r for r in (8, 4, 2) if c % r == 0), 1)


# ---------------------------------------------------------------------------
# algorithmic work of an op (FLOP of its contractions; bytes of weights, inputs
# and outputs, each moved once)
# ---------------------------------------------------------------------------

def op_flops(m, op):
    T = m.tensors
    out = T[op["out"]]["shape"]
    k = op["kind"]
    if k == "conv":
        return 2 * numel(out) * T[op["inputs"][0]]["shape"][1] * op["kh"] * op["kw"]
    if k == "linear":
        return 2 * numel(out) * op["nin"]
    if k == "lstm":
        b, t, h = out
        return 2 * b * t * 4 * h * (T[op["inputs"][0]]["shape"][2] + h)
    if k == "attention":
        b, s, f = out
        return 4 * b * s * s * f
    return 0


def op_bytes(m, op, es):
    T = m.tensors
    ins = 0
    for t in op["inputs"]:
        ins += numel(T[t]["shape"]) * (4 if T[t]["dtype"] in ("f32", "i32") else es)
    b = ins + numel(T[op["out"]]["shape"]) * es
    for key in ("w", "b", "g", "beta", "w_tok", "w_pos", "w_type", "table", "w_ih", "w_hh", "b_ih", "b_hh"):
        if key in op:
            b += m.weights[op[key]].size * es
    return b


GEMM_KINDS = ("conv", "linear", "lstm")        # run on gemm_kernel / conv3_halo_kernel


def rd_names(m, rd):
    names = [m.ops[i]["name"] for i in rd]
    return ", ".join(names) if len(names) <= 3 else f"{len(names)} ops ({names[0]} ... {names[-1]})"


# ---------------------------------------------------------------------------
# profiler summaries (rocprofv3 output of this script) and the committed traffic
# ---------------------------------------------------------------------------

def source_hash():
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


_DEMANGLED = {}


def _demangle(name):
    """Readable kernel name.  This library's kernels (namespace mopar, integer / bool / type template
    arguments) are decoded here; other names go through c++filt."""
    import re
    mm = re.match(r"_ZN5mopar(\d+)", name)
    if mm:
        n = int(mm.group(1))
        base = name[len(mm.group(0)):len(mm.group(0)) + n]
        rest = name[len(mm.group(0)) + n:]
        args = []
        if rest.startswith("I"):
            body = rest[1:]
            while body and not body.startswith("E"):
                if body.startswith("DF16b"):
                    args.append("bf16"); body = body[5:]
                elif body.startswith("f"):
                    args.append("float"); body = body[1:]
                else:
                    t = re.match(r"L([ib])(\d+)E", body)
                    if not t:
                        break
                    args.append(("true" if t.group(2) == "1" else "false") if t.group(1) == "b" else t.group(2))
                    body = body[t.end():]
        return base + (f"<{', '.join(args)}>" if args else "")
    if not name.startswith("_Z"):
        return name
    if name not in _DEMANGLED:
        import subprocess
        try:
            _DEMANGLED[name] = subprocess.run(["c++filt", name], capture_output=True, text=True,
                                              timeout=10).stdout.strip() or name
        except (OSError, subprocess.SubprocessError):
            _DEMANGLED[name] = name
    return _DEMANGLED[name]


def _short(name):
    """Kernel name without its argument list (template arguments kept).  rocprofv3's csv names
    spell bf16 template arguments as "bool _Accum"; they are written back as bf16."""
    name = _demangle(name).replace("(anonymous namespace)::", "").replace("bool _Accum", "bf16")
    depth, out = 0, []
    for i, ch in enumerate(name):
        if ch == "(" and depth == 0 and out:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).replace("void ", "").replace("mopar::", "")


def _rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def summarize_trace(path, title, cmd, min_share=0.002):
    """Markdown: per (kernel, grid, stream) dispatch count and mean / median duration from a
    rocprofv3 kernel-trace csv (groups below `min_share` of all kernel time folded into one row)."""
    groups = {}
    for r in _rows(path):
        key = (_short(r["Kernel_Name"]), int(r.get("Grid_Size", r.get("Grid_Size_X", 0)) or 0),
               int(r.get("Workgroup_Size", r.get("Workgroup_Size_X", 0)) or 0), int(r.get("Stream_Id", 0) or 0))
        groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    total = sum(sum(v) for v in groups.values())
    lines = [f"# {title}", "", "Command (from the repository root, on the GPU box):", "", "```", cmd, "```", "",
             f"Source hash of `csrc/`: `{source_hash()}`.  Durations in microseconds, grouped by kernel, "
             f"grid size (threads) and HIP stream; share = the group's fraction of all kernel time.", "",
             "| kernel | grid | block | stream | dispatches | mean us | median us | share |",
             "|---|---|---|---|---|---|---|---|"]
    rest_n, rest_t = 0, 0.0
    for key, v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        if sum(v) / total < min_share:
            rest_n += len(v)
            rest_t += sum(v)
            continue
        lines.append(f"| `{key[0]}` | {key[1]} | {key[2]} | {key[3]} | {len(v)} | {statistics.fmean(v):.2f} | "
                     f"{statistics.median(v):.2f} | {sum(v) / total:.3f} |")
    if rest_n:
        lines.append(f"| (other groups) | | | | {rest_n} | | | {rest_t / total:.3f} |")
    return "\n".join(lines)


def summarize_pmc(paths, title, cmd, copy_mib, grid_of_interest=None):
    """Markdown: per (kernel, grid) mean of each counter from rocprofv3 --pmc csv files, and the
    HBM traffic of the dispatches of interest scaled by the counters of a raw copy of known size."""
    vals = {}
    names = []
    for path in paths:
        for r in _rows(path):
            cn = r["Counter_Name"]
            if cn not in names:
                names.append(cn)
            key = (_short(r["Kernel_Name"]), int(r.get("Grid_Size", 0) or 0))
            vals.setdefault(key, {}).setdefault(cn, []).append(float(r["Counter_Value"]))
    lines = [f"# {title}", "", "Commands (from the repository root, on the GPU box; one counter pass each):", "",
             "```", cmd, "```", "", f"Source hash of `csrc/`: `{source_hash()}`.  Mean counter value per dispatch.",
             "", "| kernel | grid | " + " | ".join(names) + " |", "|---|---|" + "---|" * len(names)]
    for key, d in sorted(vals.items(), key=lambda kv: kv[0]):
        lines.append(f"| `{key[0]}` | {key[1]} | " + " | ".join(
            f"{statistics.fmean(d[n]):.1f}" if n in d else "" for n in names) + " |")
    out = {}
    if "FETCH_SIZE" in names and "WRITE_SIZE" in names:
        copies = [d for k, d in vals.items() if "copy_kernel" in k[0] and "FETCH_SIZE" in d and "WRITE_SIZE" in d]
        cf = max((max(d["FETCH_SIZE"]) for d in copies), default=0.0)
        cw = max((max(d["WRITE_SIZE"]) for d in copies), default=0.0)
        kib = copy_mib * 1024.0
        sf, sw = (kib / cf if cf else float("nan")), (kib / cw if cw else float("nan"))
        lines += ["", f"Copy calibration: a raw copy of {copy_mib} MiB reads FETCH_SIZE {cf:.1f} KiB and "
                      f"WRITE_SIZE {cw:.1f} KiB: scale factors {sf:.4f} (read), {sw:.4f} (write)."]
        if grid_of_interest:
            # the dispatches of interest: comma-separated grid sizes and / or kernel-name substrings;
            # the traffic per launch is their dispatch-weighted mean
            # Each selector is [name][@grid][#mfma]: a kernel-name part, a grid size, and an exact
            # SQ_INSTS_MFMA count that keeps only the dispatches of one op when several ops share a
            # kernel and grid (the passes are separate runs of one deterministic sequence, so the
            # i-th dispatch of a group is the same op in every pass).  Selectors are separated by
            # "|"; the traffic is the mean over every selected dispatch.
            sel = [x.strip() for x in str(grid_of_interest).split("|") if x.strip()]

            def parse(x):
                x, _, mf = x.partition("#")
                name, at, grid = x.rpartition("@")
                if not at:
                    name, grid = (x, "") if not x.isdigit() else ("", x)
                return name, (int(grid) if grid else None), (float(mf) if mf else None)
            tot, cnt = 0.0, 0
            for x in sel:
                name, grid, mf = parse(x)
                for key, d in vals.items():
                    if (name and name not in key[0]) or (grid is not None and key[1] != grid):
                        continue
                    if "FETCH_SIZE" not in d or "WRITE_SIZE" not in d:
                        continue
                    idx = range(min(len(d["FETCH_SIZE"]), len(d["WRITE_SIZE"])))
                    if mf is not None:
                        idx = [i for i in idx if i < len(d.get("SQ_INSTS_MFMA", [])) and d["SQ_INSTS_MFMA"][i] == mf]
                    for i in idx:
                        tot += (d["FETCH_SIZE"][i] * sf + d["WRITE_SIZE"][i] * sw) * 1024.0
                        cnt += 1
            if cnt:
                out = {"traffic_bytes_per_launch": round(tot / cnt), "dispatches": cnt}
            lines += ["", "```", f"source_hash: {source_hash()}",
                      f"grid: {grid_of_interest}",
                      f"dispatches: {out.get('dispatches', 0)}",
                      f"traffic_bytes_per_launch: {out.get('traffic_bytes_per_launch', 'nan')}", "```"]
    return "\n".join(lines)


def committed_traffic(workload):
    """HBM traffic per launch of the workload's dominant kernel from its committed counter summary
    (profiles/<kernel>_<workload>_traffic.md) and the dispatches it covers, or (None, None) when
    missing or taken on other sources."""
    try:
        files = [f for f in os.listdir(PROFILES) if f.endswith(f"_{workload}_traffic.md")]
    except OSError:
        return None, None
    for f in files:
        kv = {}
        for line in open(os.path.join(PROFILES, f)).read().splitlines():
            if ": " in line and line.split(": ", 1)[0] in ("source_hash", "traffic_bytes_per_launch", "grid", "scope"):
                kv[line.split(": ", 1)[0]] = line.split(": ", 1)[1]
        if kv.get("source_hash") == source_hash():
            try:
                return float(kv["traffic_bytes_per_launch"]), kv.get("scope")
            except (KeyError, ValueError):
                return None, None
    return None, None


# ---------------------------------------------------------------------------
# one workload
# ---------------------------------------------------------------------------

WORKLOAD_TAG = {1: "tinyvgg_b1", 2: "resnet50_b8", 3: "vgg16_b16", 4: "bertbase_b32", 5: "lstmlm_b64"}


def cpu_model():
    """The host CPU's model name, as the kernel reports it (None where it does not)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def run_config(cfg, args, headline):
    import numpy as np
    import torch

    import paper_2404_02445_amd as P
    import synth

    dev = "cuda:0"
    steps, warmup = (args.steps, args.warmup) if headline else (args.config_steps, max(2, min(args.warmup, 5)))
    m = synth.build(cfg)
    x_host = synth.make_input(m)
    sm = P.SlicedModel(m, device=dev)
    s = m.slicing
    plan_kw = dict(n_slices=s["n_slices"], allowed_cut=s["allowed_cut"], elim_tau=s["elim_tau"],
                   k_override=s["k_override"])
    x = torch.from_numpy(x_host).to(dev)
    es = 2 if m.dtype == "bf16" else 4
    peak = PEAK_TFLOPS[m.dtype]
    log(f"cfg {cfg}: {m.name} built and loaded")

    measured = None
    if headline and not args.no_measured_plan:
        # on a stream of its own, so that a kernel trace tells its launches (every sub-slice
        # count up to k_max) from the timed ones on the default stream
        mstream = torch.cuda.Stream(device=dev)
        mstream.wait_stream(torch.cuda.current_stream(dev))
        mplan, tp, _ = sm.measured_plan(x, k_max=args.k_max, reps=3, stream=mstream)
        torch.cuda.synchronize(dev)
        measured = {"k_max": args.k_max, "n_slices": mplan.n_slices, "slice_end": mplan.slice_end,
                    "k": mplan.k, "t_tau_ms": round(mplan.t_tau * 1e3, 4),
                    "tp_ms_by_k": [round(sum(r[e] for r in tp) * 1e3, 4) for e in range(args.k_max)]}
    plan = sm.plan()
    cuts = plan.slice_end[:-1]
    ratios = [codec_ratio(synth.boundary_channels(m, li)) for li in cuts]
    cw = synth.make_codec_weights(m, cuts, ratio=ratios) if args.codec == "ae" else None
    codecs, keep = sm.codecs(plan, args.codec, cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    ref_out = sm.alloc_output()
    stream = torch.cuda.current_stream()

    def plan_step():
        """a1-a4 on the host: layer profiles (Eq. 1-4), then the HyPAD plan and sub-slice counts."""
        return P.mopar_plan_slices(sm.profile(), **plan_kw)

    def same_plan(a, b):
        return a.slice_end == b.slice_end and a.k == b.k

    def seq_step(out):
        pl = plan_step()
        if not same_plan(pl, plan):
            raise RuntimeError("the step's plan differs from the plan the buffers were sized for")
        sm.forward(pl, x, out, codecs, codes, ws)

    for _ in range(warmup):
        seq_step(ref_out)
    torch.cuda.synchronize()

    # --- slice pipeline: R instances x D code slots; each (instance, slot) writes its own output
    depth = args.pipeline
    pipe, replicas, tuning = None, args.replicas, None

    def make_pipe(r):
        return sm.pipeline(plan, args.codec, cw, depth=depth, replicas=r, stream_per_slice=False).use_graphs(True)

    def pstep(pp, outs, i):
        """One step through the pipeline: the step's own plan, then batch i into output slot i mod
        (instances x slots).  (A plan that changed would need a pipeline built for it; with a fixed
        model it never changes, and the check makes the planning result part of the step.)"""
        pl = plan_step()
        if not same_plan(pl, plan):
            raise RuntimeError("the step's plan differs from the pipeline's")
        pp.submit(x, outs[i % len(outs)])

    if depth:
        if replicas == 0:
            # Each instance count is tried on two sets of streams, and the timed region runs the
            # fastest pipeline itself, on the streams it was measured on: the runtime places
            # streams on a few hardware queues in creation order, and two instances whose streams
            # share a queue run one after the other (no faster than one batch at a time).
            tuning, cands = {}, {}
            n_try = max(6, min(steps, 20))
            for r, tag in ((1, "1"), (2, "2"), (3, "3"), (2, "2b"), (3, "3b")):
                pp = make_pipe(r)
                po = [sm.alloc_output() for _ in range(r * depth)]
                for i in range(max(warmup, 3)):
                    pstep(pp, po, i)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for i in range(n_try):
                    pstep(pp, po, i)
                torch.cuda.synchronize()
                tuning[tag] = round(m.batch * n_try / (time.perf_counter() - t0), 1)
                cands[tag] = (r, pp, po)
            best = max(tuning, key=tuning.get)
            replicas, pipe, outs = cands.pop(best)
            del cands, pp, po
        else:
            pipe = make_pipe(replicas)
            outs = [sm.alloc_output() for _ in range(replicas * depth)]
        for i in range(warmup):
            pstep(pipe, outs, i)
        torch.cuda.synchronize()

    # --- timed region: exactly K steps ---------------------------------------------------
    log(f"cfg {cfg}: timed region, {steps} steps, {replicas} instance(s)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if pipe is not None:
        for i in range(steps):
            pstep(pipe, outs, warmup + i)
    else:
        for _ in range(steps):
            seq_step(ref_out)
    t_host = time.perf_counter() - t0
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / steps
    value = m.batch * steps / wall

    # --- every pipelined output against the sequential forward of the same input, bitwise ----
    check = None
    if pipe is not None:
        seq_step(ref_out)
        torch.cuda.synchronize()
        check = all(torch.equal(o, ref_out) for o in outs)
        if not check:
            raise RuntimeError(f"config {cfg}: a pipelined output differs from the sequential forward")

    # --- one batch at a time: latency -----------------------------------------------------
    n_lat = max(5, min(steps, 20))
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(n_lat):
        seq_step(ref_out)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [evs[i].elapsed_time(evs[i + 1]) for i in range(n_lat)]
    seq_value = m.batch / (statistics.median(per) / 1e3)

    # --- the same, with RAW codecs (a bit copy of each boundary tensor): what the AE codec saves
    #     or costs against handing the tensor over as it is ------------------------------------
    raw_codec = None
    if args.codec == "ae":
        rcodecs, rkeep = sm.codecs(plan, "raw")
        rcodes = sm.alloc_codes(plan, rcodecs)
        rout = sm.alloc_output()
        for _ in range(2):
            sm.forward(plan, x, rout, rcodecs, rcodes, ws)
        revs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
        torch.cuda.synchronize()
        revs[0].record(stream)
        for i in range(n_lat):
            sm.forward(plan, x, rout, rcodecs, rcodes, ws)
            revs[i + 1].record(stream)
        torch.cuda.synchronize()
        rper = [revs[i].elapsed_time(revs[i + 1]) for i in range(n_lat)]
        raw_codec = {"sequential_value": round(m.batch / (statistics.median(rper) / 1e3), 2),
                     "latency_ms": {"p50": round(statistics.median(rper), 4),
                                    "p95": round(float(np.percentile(rper, 95)), 4)},
                     "code_bytes_per_batch": int(sum(b.numel() * b.element_size() for b in rcodes))}
        del rcodes, rout, rkeep

    flop_step = sum(op_flops(m, op) for op in m.ops)
    codec_fl, codec_by = [], []
    for c, li in enumerate(cuts):
        shp = m.tensors[m.layer_output_tid(li)]["shape"]
        ch = synth.boundary_channels(m, li)
        pos = numel(shp) // ch
        ce = ch // ratios[c] if args.codec == "ae" else ch
        codec_fl.append(2 * pos * ch * ce if args.codec == "ae" else 0)
        codec_by.append((pos * ch + pos * ce + (ch * ce + ce if args.codec == "ae" else 0)) * es)
    flop_step += 2 * sum(codec_fl)

    res = {
        "workload": f"{m.name}: {m.dtype}, batch {m.batch}, {plan.n_slices} slices at {cuts}, "
                    f"RD k={max(plan.k)}, {args.codec} codec" + (f" R={ratios}" if args.codec == "ae" else ""),
        "value": round(value, 2), "unit": "inferences/s", "ms_per_step": round(ms_per_step, 4),
        "steps": steps, "warmup": warmup, "dtype": m.dtype, "batch": m.batch,
        "slices": plan.n_slices, "k": plan.k,
        "latency_ms": {"p50": round(statistics.median(per), 4), "p95": round(float(np.percentile(per, 95)), 4)},
        "sequential_value": round(seq_value, 2),
        "raw_codec": raw_codec,
        "mode": (f"slice pipeline: {replicas} instance(s) x {plan.n_slices} slices, one stream each, HIP graphs "
                 f"replayed, {depth} code slots and {replicas * depth} output buffers per (instance, slot); "
                 f"latency_ms is one batch at a time") if pipe is not None else "sequential",
        "replica_tuning_inf_per_s": tuning,
        "pipeline_outputs_equal_sequential": check,
        "wall_s_timed_region": round(wall, 4),
        "host_submit_ms_per_step": round(t_host / steps * 1e3, 4),
        "timed_region_roofline": {
            "flop_per_step": flop_step,
            "achieved_TFLOPs": round(flop_step / (ms_per_step * 1e-3) / 1e12, 2),
            "frac_of_peak": round(flop_step / (ms_per_step * 1e-3) / 1e12 / peak, 4)},
    }
    if measured is not None:
        res["measured_plan"] = measured

    # --- per-op device time (each kernel's own HIP event pair, on the launch stream) ---------
    log(f"cfg {cfg}: {value:.1f} inferences/s; per-op timing")
    sm.set_timing(True)
    n_t = max(3, min(steps, 10))
    per_op = [0.0] * len(m.ops)
    enc_ms, dec_ms = [0.0] * len(cuts), [0.0] * len(cuts)
    for _ in range(n_t):
        seq_step(ref_out)
        ops_ms, cut_ms = sm.op_times()
        for i, t in enumerate(ops_ms):
            per_op[i] += max(t, 0.0) / n_t
        for c, (e, d) in enumerate(cut_ms):
            enc_ms[c] += e / n_t
            dec_ms[c] += d / n_t
    sm.set_timing(False)
    if args.op_report:
        for i, op in enumerate(m.ops):
            f = op_flops(m, op)
            tf = f / (per_op[i] * 1e-3) / 1e12 if per_op[i] > 0 and f else 0.0
            print(f"cfg {cfg} op {i:3d} {op['name']:<14} {op['kind']:<10} "
                  f"k={plan.k[op['layer']] if op.get('rd') else 1} {per_op[i] * 1e3:9.2f} us {tf:7.1f} TF/s",
                  file=sys.stderr)

    gemm_ms = sum(per_op[i] for i, op in enumerate(m.ops) if op["kind"] in GEMM_KINDS)
    gemm_fl = sum(op_flops(m, op) for op in m.ops if op["kind"] in GEMM_KINDS)
    if args.codec == "ae":
        gemm_ms += sum(enc_ms) + sum(dec_ms)
        gemm_fl += 2 * sum(codec_fl)
    rd = [i for i, op in enumerate(m.ops) if op.get("rd")]
    rd_ms = sum(per_op[i] for i in rd)
    rd_fl = sum(op_flops(m, m.ops[i]) for i in rd)
    rd_by = sum(op_bytes(m, m.ops[i], es) for i in rd)
    B = PEAK_HBM_GBS * 1e9
    rd_roof_s = sum(max(op_flops(m, m.ops[i]) / (peak * 1e12), op_bytes(m, m.ops[i], es) / B) for i in rd)
    rd_hbm = rd_fl / rd_by < peak * 1e12 / B          # below the ridge: HBM-bound
    # the roofline of the dominant kernel: the RD op (one launch per RD op holds all k sub-slices)
    rd_launch_us = rd_ms / len(rd) * 1e3
    if rd_hbm:
        achieved = rd_by / len(rd) / (rd_launch_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        achieved = rd_fl / len(rd) / (rd_launch_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4)}
    roof["traffic"], scope = committed_traffic(WORKLOAD_TAG[cfg])
    if scope:
        roof["traffic_scope"] = scope
    roof.update({
        "kernel": "the RD ops' launches (gemm_kernel; conv3_halo_kernel for patch-staged 3x3 convs), one "
                  "launch per RD op holding its k sub-slices: " + rd_names(m, rd),
        "launches_per_step": len(rd), "flop_per_launch": rd_fl // len(rd),
        "algorithmic_bytes_per_launch": rd_by // len(rd), "avg_launch_us": round(rd_launch_us, 2),
        "attainable_frac": round(rd_roof_s / (rd_ms * 1e-3), 4),
        "timing": "HIP event pair per kernel on its launch stream, sequential passes over the same steps"})
    res["roofline"] = roof
    res["rd_mfma_util"] = {"achieved_TFLOPs": round(rd_fl / (rd_ms * 1e-3) / 1e12, 2),
                           "frac_of_peak": round(rd_fl / (rd_ms * 1e-3) / 1e12 / peak, 4),
                           "attainable_frac": round(rd_roof_s / (rd_ms * 1e-3), 4),
                           "rd_ms_per_step": round(rd_ms, 4)}
    res["gemm_ops"] = {"achieved_TFLOPs": round(gemm_fl / (gemm_ms * 1e-3) / 1e12, 2),
                       "frac_of_peak": round(gemm_fl / (gemm_ms * 1e-3) / 1e12 / peak, 4),
                       "ms_per_step": round(gemm_ms, 4)}
    other = [i for i, op in enumerate(m.ops) if op["kind"] not in GEMM_KINDS]
    bw_ms = sum(per_op[i] for i in other)
    bw_by = sum(op_bytes(m, m.ops[i], es) for i in other)
    res["other_ops"] = {"ms_per_step": round(bw_ms, 4), "GBs": round(bw_by / (bw_ms * 1e-3) / 1e9, 1) if bw_ms else None,
                        "kinds": sorted({m.ops[i]["kind"] for i in other})}
    ideal = sum(max(op_flops(m, op) / (peak * 1e12), op_bytes(m, op, es) / B) for op in m.ops)
    ideal += sum(2 * max(f / (peak * 1e12), b / B) for f, b in zip(codec_fl, codec_by))
    res["ideal_step"] = {"ms": round(ideal * 1e3, 4), "frac_of_sequential_p50": round(ideal * 1e3 / statistics.median(per), 4)}
    codec = []
    for c, li in enumerate(cuts):
        tb = numel(m.tensors[m.layer_output_tid(li)]["shape"]) * es
        codec.append({"cut_after": m.layers[li], "tensor_MB": round(tb / 1e6, 3),
                      "encode_us": round(enc_ms[c] * 1e3, 2), "decode_us": round(dec_ms[c] * 1e3, 2),
                      "encode_GBs": round(codec_by[c] / (enc_ms[c] * 1e-3) / 1e9, 1) if enc_ms[c] else None,
                      "decode_GBs": round(codec_by[c] / (dec_ms[c] * 1e-3) / 1e9, 1) if dec_ms[c] else None})
    res["codec"] = codec

    # --- the codec in isolation, cold cache (a 512 MB write evicts the 256 MB Infinity Cache),
    #     beside a raw copy of the same tensor ----------------------------------------------
    if args.codec == "ae" and not args.no_cold_codec:
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        raw = P.make_codec("raw")
        iso = []
        tdt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
        for c, li in enumerate(cuts):
            shp = list(m.tensors[m.layer_output_tid(li)]["shape"])
            gshape = [shp[0]] + shp[2:] + [shp[1]] if len(shp) == 4 else shp
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

    if args.calibrate_copy_mib:         # a raw copy of known size: the reference for counter scaling
        raw = P.make_codec("raw")
        nb = args.calibrate_copy_mib << 20
        a, b = torch.empty(nb, dtype=torch.uint8, device=dev), torch.empty(nb, dtype=torch.uint8, device=dev)
        for _ in range(3):
            P.mopar_boundary_encode(raw, (nb // 2,), "bf16", a, b)
        torch.cuda.synchronize()
        del a, b

    # --- CPU baseline: the oracle on a bounded sample of the same workload ----------------------
    budget = args.cpu_seconds if headline else args.config_cpu_seconds
    if not args.no_cpu_baseline and budget > 0:
        log(f"cfg {cfg}: oracle CPU baseline, {budget} s")
        import oracle
        cores = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
        os.environ.setdefault("OMP_NUM_THREADS", str(cores))
        oracle.lib()
        done = 0
        t0 = time.perf_counter()
        while True:
            oracle.forward(m, x_host, k=plan.k, cuts=cuts, codecs=cw, sample=[done % m.batch])
            done += 1
            if time.perf_counter() - t0 >= budget:
                break
        el = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(done / el, 4), "unit": "inferences/s", "cores": cores,
                               "kind": "oracle", "cpu": cpu_model(),
                               "sample": f"{done} single-{'image' if cfg <= 3 else 'sequence'} forward(s) of the "
                                         f"same sliced workload (same plan, codecs and weights), {el:.1f} s"}
    if pipe is not None:
        pipe.synchronize()
    del pipe, sm, ws, codes, codecs, keep
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=HEADLINE_CFG,
                    help="headline workload 1..5 (default 5, the largest: the LSTM LM, batch 64 x 128)")
    ap.add_argument("--no-per-config", action="store_true", help="measure the headline workload only")
    ap.add_argument("--config-steps", type=int, default=10, help="timed steps of each per_config workload")
    ap.add_argument("--codec", choices=["ae", "raw"], default="ae")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle CPU-baseline budget, headline")
    ap.add_argument("--config-cpu-seconds", type=float, default=3.0, help="oracle CPU-baseline budget, per config")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold-codec", action="store_true")
    ap.add_argument("--op-report", action="store_true", help="print per-op times to stderr")
    ap.add_argument("--pipeline", type=int, default=2, metavar="D",
                    help="code slots per (instance, cut) of the slice pipeline (0: one batch at a time)")
    ap.add_argument("--replicas", type=int, default=0,
                    help="pipeline instances; 0: try 1, 2 and 3 before the timed region, keep the fastest")
    ap.add_argument("--k-max", type=int, default=8, help="largest sub-slice count of the measured-profile plan")
    ap.add_argument("--no-measured-plan", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run a raw copy of this many MiB (counter calibration for --pmc runs)")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("CSV", "TITLE", "CMD"),
                    help="print a markdown summary of a rocprofv3 kernel-trace csv and exit")
    ap.add_argument("--summarize-pmc", nargs="+", metavar="ARG",
                    help="TITLE CMD COPY_MIB SELECT CSV...: markdown summary of rocprofv3 --pmc csv files, and "
                         "exit; SELECT = '|'-separated [kernel-name part][@grid][#SQ_INSTS_MFMA] selectors of the "
                         "dispatches whose mean HBM traffic per launch is reported (0: none)")
    args = ap.parse_args()
    if args.summarize_trace:
        print(summarize_trace(*args.summarize_trace))
        return
    if args.summarize_pmc:
        title, cmd, mib, grid, *paths = args.summarize_pmc
        print(summarize_pmc(paths, title, cmd, int(mib), grid if grid not in ("", "0") else None))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: every GPU box of this setup has one, and the sliced path runs "
              "its slices and sub-slices on that one device; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    head = run_config(args.config, args, headline=True)
    per = {}
    if not args.no_per_config:
        for cfg in (1, 2, 3, 4, 5):
            if cfg != args.config:
                r = run_config(cfg, args, headline=False)
                per[WORKLOAD_TAG[cfg]] = r
                print(f"per-config {cfg} done: {r['value']} inferences/s", file=sys.stderr, flush=True)
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "inferences/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic (seeded inputs and random-init weights of the named architecture)",
        "config": {"workload": head["workload"], "batch": head["batch"], "slices": head["slices"], "k": head["k"],
                   "codec": args.codec},
        "roofline": head.pop("roofline"),
        "cpu_baseline": head.pop("cpu_baseline", None),
    }
    for k in ("workload", "value", "unit", "ms_per_step", "steps", "warmup", "dtype", "batch", "slices", "k"):
        head.pop(k, None)
    out.update(head)
    out["per_config"] = per
    print(json.dumps(out))


if __name__ == "__main__":
    main()
