"""Oracle of the service profile and of the hybrid partitioning (HyPAD) -- TEST INFRASTRUCTURE.

Plain Python in float64, following Sec. III-B (operator -> layer -> service
profile, Eq. 1-4) and Sec. III-C (Eq. 5-6, node/edge elimination and
Algorithm 1).  Where the printed algorithm is garbled, the reading used is
stated at the function.

Sums are taken in a fixed, stated order so that a second implementation
following the same order reproduces every double bit for bit.
"""
from __future__ import annotations

import itertools
import math
from dataclasses import dataclass, field

INF = math.inf

# Roofline constants for the analytic operator profile (MI355X published peaks).
PEAK_FLOPS = {"bf16": 2.5e15, "f32": 157.3e12}
PEAK_BYTES = 8.0e12
DTYPE_BYTES = {"bf16": 2, "f32": 4, "i32": 4}


# ---------------------------------------------------------------------------
# Sub-slice ranges (Sec. III-C: eta equal-size sub-slices)
# ---------------------------------------------------------------------------

def subslice_range(n: int, k: int, j: int):
    """Output range [lo, hi) of sub-slice j when n outputs are split k ways.

    Equal sizes when k divides n; otherwise the first n mod k ranges hold one
    extra element (reading of 'equal-size' for a ragged n).
    """
    if not (1 <= k <= n and 0 <= j < k):
        raise ValueError("need 1 <= k <= n and 0 <= j < k")
    q, r = divmod(n, k)
    return j * q + min(j, r), (j + 1) * q + min(j + 1, r)


# ---------------------------------------------------------------------------
# Service profile (Sec. III-B)
# ---------------------------------------------------------------------------

def _numel(shape):
    n = 1
    for s in shape:
        n *= int(s)
    return n


def op_profile(model, op):
    """Operator profile (m_i, t_i): memory = bytes of parameters + inputs + output;
    time = max(FLOP / peak, bytes / HBM bandwidth) -- an analytic stand-in for the
    learned operator predictor of Sec. III-B (which needs production traces).

    FLOP counts only the contractions (conv, linear, attention, LSTM); every
    other op is priced by its bytes.  Returns (mem_bytes, time_s, flop).
    """
    dt = model.dtype
    T = model.tensors
    pb = 0
    for key in ("w", "b", "g", "beta", "w_tok", "w_pos", "w_type", "table", "w_ih", "w_hh", "b_ih", "b_hh"):
        if key in op:
            pb += _numel(model.weights[op[key]].shape) * DTYPE_BYTES[dt]
    ib = sum(_numel(T[t]["shape"]) * DTYPE_BYTES[T[t]["dtype"]] for t in op["inputs"])
    k = op["kind"]
    out_shape = T[op["out"]]["shape"]
    if k == "conv":             # a branch writing part of a concatenated tensor counts its own channels
        out_shape = (out_shape[0], op["cout"], out_shape[2], out_shape[3])
    ob = _numel(out_shape) * DTYPE_BYTES[T[op["out"]]["dtype"]]
    in_shape = T[op["inputs"][0]]["shape"]
    if k == "conv":
        flop = 2 * _numel(out_shape) * in_shape[1] * op["kh"] * op["kw"]
    elif k == "linear":
        flop = 2 * _numel(out_shape) * op["nin"]
    elif k == "attention":
        b, s, f = out_shape
        flop = 4 * b * s * s * f
    elif k == "lstm":
        b, t, h = out_shape
        flop = 2 * b * t * 4 * h * (in_shape[2] + h)
    else:
        flop = 0
    mem = float(pb + ib + ob)
    time = max(float(flop) / PEAK_FLOPS[dt], mem / PEAK_BYTES)
    return mem, time, flop


def node_outputs(model):
    """The tensor leaving each planning node (the output of its last op)."""
    return [[o for o in model.ops if o["layer"] == l][-1]["out"] for l in range(len(model.layers))]


def crossing_tensors(model, j):
    """Tensors a cut after node j carries (Sec. III-C, edge elimination): every node
    output of a node <= j that an op of a node > j reads -- after the nodes between
    them are merged, the edges from one side to the other are parallel edges, merged
    into one whose size is the sum of these tensors.  Ascending tensor id."""
    outs = node_outputs(model)
    src = {t: l for l, t in enumerate(outs) if l <= j}
    read_later = {t for o in model.ops if o["layer"] > j for t in o["inputs"]}
    return sorted(t for t in src if t in read_later)


@dataclass
class LayerProfile:
    mem_bytes: float
    time_s: float
    out_bytes: float
    rd_width: int


def dominant_ops(mems, frac):
    """Dominant operators of a layer (Sec. III-B): the ops sorted by memory footprint,
    largest first (reading of 'ascending ... top n': the top n by size), ties by
    position, and the shortest such prefix whose footprint reaches frac of the
    layer's total (the total summed in op order, the prefix in sorted order).
    Returns the selected indices in op order."""
    total = 0.0
    for m in mems:
        total = total + m
    order = sorted(range(len(mems)), key=lambda i: (-mems[i], i))
    acc, chosen = 0.0, []
    for i in order:
        acc = acc + mems[i]
        chosen.append(i)
        if acc >= frac * total:
            break
    return sorted(chosen)


def layer_profiles(model, dominant=None):
    """Layer profiles M_l, t_l (Eq. 1-3) and the service profile vectors (Eq. 4).

    Ops with branch 0 form the sequential chain (Eq. 1): M_c = max m_i,
    t_c = sum t_i.  Ops with branch b >= 1 at position p form parallel branches
    (Eq. 2): M_b = max_p sum_b m_bp, t_b = sum_p max_b t_bp.  The layer is the
    hybrid of Eq. 3: M = max(M_c, M_b), t = t_c + t_b (an empty part counts 0).
    Sums run in op order (chain), branch order (per position) and position
    order (over positions).  rd_width is the smallest output width among the
    layer's resource-dominant ops (0 when it has none).
    With ``dominant`` = f (0.8 in the paper), only the layer's dominant operators
    (dominant_ops) enter the aggregation; rd_width and out_bytes are unchanged.
    """
    out = []
    for li in range(len(model.layers)):
        all_ops = [o for o in model.ops if o["layer"] == li]
        ops = all_ops
        if dominant is not None:
            keep = dominant_ops([op_profile(model, o)[0] for o in all_ops], dominant)
            ops = [all_ops[i] for i in keep]
        mc, tc = 0.0, 0.0
        pos_m, pos_t = {}, {}
        for o in ops:
            m, t, _ = op_profile(model, o)
            if o["branch"] == 0:
                mc = max(mc, m)
                tc = tc + t
        for p in sorted({o["pos"] for o in ops if o["branch"] > 0}):
            at = sorted([o for o in ops if o["branch"] > 0 and o["pos"] == p], key=lambda o: o["branch"])
            s_m, mx_t = 0.0, 0.0
            for o in at:
                m, t, _ = op_profile(model, o)
                s_m = s_m + m
                mx_t = max(mx_t, t)
            pos_m[p], pos_t[p] = s_m, mx_t
        mb = max(pos_m.values()) if pos_m else 0.0
        tb = 0.0
        for p in sorted(pos_t):
            tb = tb + pos_t[p]
        if li + 1 < len(model.layers):      # the cut after this node: every crossing tensor
            ob = 0.0
            for t in crossing_tensors(model, li):
                ob = ob + float(_numel(model.tensors[t]["shape"]) * DTYPE_BYTES[model.tensors[t]["dtype"]])
        else:
            T = model.tensors[all_ops[-1]["out"]]
            ob = float(_numel(T["shape"]) * DTYPE_BYTES[T["dtype"]])
        widths = [o["cout"] if o["kind"] == "conv" else o["nout"] for o in all_ops if o.get("rd")]
        out.append(LayerProfile(max(mc, mb), tc + tb, ob, min(widths) if widths else 0))
    return out


# ---------------------------------------------------------------------------
# Hybrid partitioning (Sec. III-C, Eq. 5-6, Algorithm 1)
# ---------------------------------------------------------------------------

@dataclass
class PlanOpts:
    n_slices: int = 0                   # 0: the DP chooses the count; > 0: exactly this many
    allowed_cut: list | None = None     # n-1 flags (cut after node j); None: all, after elimination
    elim_tau: float = 0.05              # node-elimination threshold; < 0 disables
    c_m: float = 1.0                    # cost per unit of memory and time (Eq. 6)
    c_n: float = 1.0                    # cost per unit of transfer time (Eq. 6)
    bw: float = 8.0e12                  # boundary bandwidth, bytes/s
    ratio: list | None = None           # per cut position (n-1), compression ratio; None: 1
    k_max: int = 1
    lambda_bytes: float = 0.0           # eta <= M_g / lambda when > 0
    tp_table: list | None = None        # [n][k_max] measured t_p(l, eta); None: analytic
    ta_table: list | None = None        # [n][k_max] measured t_a(l, eta); None: 0
    k_override: list | None = None      # per node, > 0 forces k
    uniform: bool = False               # the Uniform variant: n_slices slices of equal node counts


@dataclass
class Plan:
    n_slices: int
    slice_end: list                     # last node (0-based) of each slice
    k: list                             # per node
    cost: float
    t_tau: float
    t_unsplit: float
    latency_ok: bool
    allowed: list = field(default_factory=list)


class Infeasible(Exception):
    pass


def eliminate(M, tau):
    """Node elimination (Sec. III-C): node j is merged with node j+1 -- no cut between
    them -- when |M_j - M_{j+1}| / M_j <= tau.  Reading: the original adjacent
    footprints are compared, denominator M_j, in one pass; merging never changes a
    node's own footprint, so the fixpoint loop of Algorithm 1 ends after one pass.
    Edge elimination (merging parallel edges, sizes summed) is the identity on a
    chain of single-input single-output nodes.
    Returns n-1 flags: 1 = a cut after node j remains allowed.
    """
    n = len(M)
    if tau < 0:
        return [1] * (n - 1)
    return [0 if abs(M[j] - M[j + 1]) / M[j] <= tau else 1 for j in range(n - 1)]


def cost_cal(prof, opts, i, j):
    """Compute cost of slice i..j (1-based, inclusive) in Eq. 6: c_m * (M_g * sum t),
    with M_g = max M_l over the slice (the slice is sized for its peak layer) and the
    sum taken in ascending l."""
    mx = 0.0
    st = 0.0
    for l in range(i, j + 1):
        mx = max(mx, prof[l - 1].mem_bytes)
        st = st + prof[l - 1].time_s
    return opts.c_m * (mx * st)


def t_comm(prof, opts, j):
    """Transfer time of the boundary after node j (1-based, j < n): (bytes / ratio) / bw."""
    r = 1.0 if opts.ratio is None else float(opts.ratio[j - 1])
    return (prof[j - 1].out_bytes / r) / opts.bw


def cost_com(prof, opts, j, n):
    """Communication cost of a slice ending at node j (Eq. 6): c_n * t_c; none after the last node."""
    return 0.0 if j == n else opts.c_n * t_comm(prof, opts, j)


def plan_slices(prof, opts: PlanOpts) -> Plan:
    """HyPAD (Algorithm 1) on a chain of n planning nodes.

    Step 1, graph simplification: node elimination when no cut set is prescribed.
    Step 2, the DP over split points.  Reading of the garbled indices: with nodes
    1..n, dp[0] = 0 and for j = 1..n, i = 1..j (ascending, cut before i allowed)
      dp[j] = min(dp[j], dp[i-1] + (cal(i, j) + com(j)))   -- strict '<' keeps the
    smallest i on ties (longest last slice).  With a fixed slice count K the same
    recurrence runs over dp[s][j], s = 1..K.  The backtrack follows the stored
    argmin (no floating-point equality test).
    Step 3, parallelism: for each slice g, eta ranges over 1..eta_max (eta_max =
    k_max, and <= floor(M_g / lambda) when lambda > 0); the eta minimising
    sum_{l in g} (t_p(l, eta) + t_a(l, eta)) (Eq. 5; strict '<': smallest eta on
    ties) is given to the slice's RD nodes; other nodes get 1.  Without measured
    tables t_p = t_l and t_a = 0.  A positive k_override wins.
    Latency (second constraint of Eq. 6): t_tau of Eq. 5 with the chosen k and the
    cut transfer times, compared with the unsplit sum of t_l; reported only.
    """
    n = len(prof)
    if n < 1:
        raise ValueError("empty profile")
    if opts.allowed_cut is not None:
        allowed = [1 if a else 0 for a in opts.allowed_cut]
        if len(allowed) != n - 1:
            raise ValueError("allowed_cut must have n-1 entries")
    else:
        allowed = eliminate([p.mem_bytes for p in prof], opts.elim_tau)

    def cut_ok(i):          # may a slice start at node i (1-based)?
        return i == 1 or allowed[i - 2] == 1

    K = opts.n_slices
    if K < 0 or K > n:
        raise Infeasible("n_slices out of range")
    if opts.uniform:
        # the Uniform partitioning of the evaluation (Sec. IV): the same number of
        # slices, each with the same number of nodes -- node counts as array_split
        # gives them (the first n mod K slices one node longer); no elimination
        if K == 0:
            raise ValueError("the uniform variant needs n_slices > 0")
        q, r = divmod(n, K)
        ends, e = [], -1
        for s_ in range(K):
            e += q + (1 if s_ < r else 0)
            ends.append(e)
        cost = plan_cost(prof, opts, ends)
        allowed = [1] * (n - 1)
        ends.reverse()
    elif K == 0:
        dp = [INF] * (n + 1)
        arg = [0] * (n + 1)
        dp[0] = 0.0
        for j in range(1, n + 1):
            for i in range(1, j + 1):
                if not cut_ok(i) or dp[i - 1] == INF:
                    continue
                v = dp[i - 1] + (cost_cal(prof, opts, i, j) + cost_com(prof, opts, j, n))
                if v < dp[j]:
                    dp[j], arg[j] = v, i
        ends = []
        j = n
        while j > 0:
            ends.append(j - 1)
            j = arg[j] - 1
        cost = dp[n]
    else:
        dp = [[INF] * (n + 1) for _ in range(K + 1)]
        arg = [[0] * (n + 1) for _ in range(K + 1)]
        dp[0][0] = 0.0
        for s in range(1, K + 1):
            for j in range(s, n + 1):
                for i in range(s, j + 1):
                    if (s == 1) != (i == 1):
                        continue
                    if not cut_ok(i) or dp[s - 1][i - 1] == INF:
                        continue
                    v = dp[s - 1][i - 1] + (cost_cal(prof, opts, i, j) + cost_com(prof, opts, j, n))
                    if v < dp[s][j]:
                        dp[s][j], arg[s][j] = v, i
        if dp[K][n] == INF:
            raise Infeasible("fewer allowed cuts than n_slices - 1")
        ends = []
        j, s = n, K
        while j > 0:
            ends.append(j - 1)
            j, s = arg[s][j] - 1, s - 1
        cost = dp[K][n]
    ends.reverse()

    # step 3: parallelism per slice
    k = [1] * n
    kmax = max(1, opts.k_max)

    def tp(l, e):
        return prof[l].time_s if opts.tp_table is None else opts.tp_table[l][e - 1]

    def ta(l, e):
        return 0.0 if opts.ta_table is None else opts.ta_table[l][e - 1]

    start = 0
    for end in ends:
        mg = max(prof[l].mem_bytes for l in range(start, end + 1))
        emax = kmax
        if opts.lambda_bytes > 0:
            emax = min(emax, int(math.floor(mg / opts.lambda_bytes)))
        emax = max(1, emax)
        best, best_e = INF, 1
        for e in range(1, emax + 1):
            tot = 0.0
            for l in range(start, end + 1):
                ee = e if prof[l].rd_width > 0 else 1
                tot = tot + (tp(l, ee) + ta(l, ee))
            if tot < best:
                best, best_e = tot, e
        for l in range(start, end + 1):
            if prof[l].rd_width > 0:
                k[l] = min(best_e, prof[l].rd_width)
        start = end + 1
    if opts.k_override is not None:
        for l in range(n):
            if opts.k_override[l] > 0:
                if prof[l].rd_width == 0 or opts.k_override[l] > prof[l].rd_width:
                    raise ValueError("k_override on a node without a wide enough RD op")
                if opts.k_override[l] > max(1, opts.k_max) and (opts.tp_table is not None or opts.ta_table is not None):
                    raise ValueError("k_override beyond k_max: the measured tables stop at k_max")
                k[l] = int(opts.k_override[l])

    t_tau = 0.0
    for l in range(n):
        t_tau = t_tau + (tp(l, k[l]) + ta(l, k[l]))
    for e in ends[:-1]:
        t_tau = t_tau + t_comm(prof, opts, e + 1)
    t_unsplit = 0.0
    for l in range(n):
        t_unsplit = t_unsplit + prof[l].time_s
    return Plan(len(ends), ends, k, cost, t_tau, t_unsplit, t_tau <= t_unsplit, allowed)


def plan_cost(prof, opts, ends):
    """Objective of Eq. 6 for the slices ending at ``ends`` (0-based), summed left to right."""
    n = len(prof)
    tot, start = 0.0, 1
    for e in ends:
        j = e + 1
        tot = tot + (cost_cal(prof, opts, start, j) + cost_com(prof, opts, j, n))
        start = j + 1
    return tot


def brute_force_plan(prof, opts: PlanOpts):
    """Enumerate every admissible cut set; return (min cost, list of optimal slice_end lists)."""
    n = len(prof)
    allowed = (list(opts.allowed_cut) if opts.allowed_cut is not None
               else eliminate([p.mem_bytes for p in prof], opts.elim_tau))
    positions = [j for j in range(n - 1) if allowed[j]]
    sizes = range(len(positions) + 1) if opts.n_slices == 0 else [opts.n_slices - 1]
    best, arg = INF, []
    for r in sizes:
        if r > len(positions):
            continue
        for cs in itertools.combinations(positions, r):
            ends = list(cs) + [n - 1]
            c = plan_cost(prof, opts, ends)
            if c < best:
                best, arg = c, [ends]
            elif c == best:
                arg.append(ends)
    return best, arg
