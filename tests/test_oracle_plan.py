"""Pins for the oracle's service profile (Eq. 1-4) and partitioner (Eq. 5-6, Algorithm 1).

* Eq. 1-3 on hand-worked chain / branch / hybrid layers.
* Node elimination against its definition on constructed footprints.
* The DP against exhaustive enumeration of every admissible cut set.
* The tie rule, the parallelism search and the latency check on hand cases.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import plan as P
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def LP(m, t, ob=1.0, rd=0):
    return P.LayerProfile(float(m), float(t), float(ob), rd)


# ---- Eq. 1-3 ------------------------------------------------------------------

def _mini_model(ops_spec):
    """One layer whose ops are given as (branch, pos, mem_bytes, time) via fake linears."""
    m = synth.Model(name="mini", dtype="bf16", batch=1)
    m.layers = ["L"]
    m.tensors = [dict(shape=(1,), dtype="bf16")]
    for i, (br, pos, mem, t) in enumerate(ops_spec):
        m.tensors.append(dict(shape=(1,), dtype="bf16"))
        m.ops.append(dict(kind="fake", layer=0, branch=br, pos=pos, inputs=[0], out=i + 1, mem=mem, t=t))
    return m


@pytest.fixture
def fake_profiles(monkeypatch):
    monkeypatch.setattr(P, "op_profile", lambda model, op: (float(op["mem"]), float(op["t"]), 0))


def test_eq1_chain(fake_profiles):
    m = _mini_model([(0, 1, 10, 1.0), (0, 2, 30, 2.0), (0, 3, 20, 4.0)])
    p = P.layer_profiles(m)[0]
    assert (p.mem_bytes, p.time_s) == (30.0, 7.0)          # max m, sum t


def test_eq2_branches(fake_profiles):
    # branch 1: (5, t=1) (8, t=2) (4, t=1); branch 2: (6, t=3) at position 1 only
    m = _mini_model([(1, 1, 5, 1.0), (1, 2, 8, 2.0), (1, 3, 4, 1.0), (2, 1, 6, 3.0)])
    p = P.layer_profiles(m)[0]
    # positions: M = [5+6, 8, 4] -> 11 ; t = max(1,3) + 2 + 1 = 6
    assert (p.mem_bytes, p.time_s) == (11.0, 6.0)


def test_eq3_hybrid(fake_profiles):
    m = _mini_model([(0, 1, 20, 1.0), (1, 1, 5, 2.0), (2, 1, 7, 5.0), (1, 2, 9, 1.0)])
    p = P.layer_profiles(m)[0]
    # chain: M_c = 20, t_c = 1; branches: M_b = max(5+7, 9) = 12, t_b = 5 + 1 = 6
    assert (p.mem_bytes, p.time_s) == (20.0, 7.0)


def test_op_profile_closed_form_conv():
    m = synth.build(2, batch=1, hw=32, blocks=(1, 1, 1, 1), widths=(8, 8, 8, 8), n_cls=4)
    stem = m.ops[0]
    mem, t, flop = P.op_profile(m, stem)
    # conv 7x7/2, 3 -> 8 channels, 32x32 -> 16x16, batch 1
    assert flop == 2 * 8 * 16 * 16 * 3 * 49
    params = (8 * 3 * 49 + 8) * 2
    assert mem == params + 3 * 32 * 32 * 4 + 8 * 16 * 16 * 2
    assert t == max(flop / 2.5e15, mem / 8e12)


def test_resnet_block_uses_branch_topology():
    m = synth.build(2, batch=1, hw=32, blocks=(1, 1, 1, 1), widths=(8, 8, 8, 8), n_cls=4)
    ops = [o for o in m.ops if o["layer"] == 1]
    prof = {o["name"]: P.op_profile(m, o) for o in ops}
    a, b, c, sc = (prof[f"s1b1.{s}"] for s in "abc") if False else (prof["s1b1.a"], prof["s1b1.b"],
                                                                       prof["s1b1.c"], prof["s1b1.sc"])
    lp = P.layer_profiles(m)[1]
    assert lp.mem_bytes == max(a[0] + sc[0], b[0], c[0])
    assert lp.time_s == ((0.0 + max(a[1], sc[1])) + b[1]) + c[1]
    assert lp.rd_width == 8


# ---- elimination --------------------------------------------------------------

def test_paper_constants():
    g = json.load(open(GOLDEN))
    assert P.PlanOpts().elim_tau == g["node_elimination_threshold"]["value"]


def test_elimination_definition():
    assert P.eliminate([100.0] * 6, 0.05) == [0] * 5                 # all equal: everything merges
    alt = [100.0, 110.0, 100.0, 110.0, 100.0]
    assert P.eliminate(alt, 0.05) == [1] * 4                          # +-10 %: nothing merges
    assert P.eliminate([100.0, 105.0, 200.0], 0.05) == [0, 1]         # exactly 5 %: merged
    assert P.eliminate([100.0, 105.0001, 200.0], 0.05) == [1, 1]
    assert P.eliminate([100.0, 95.0], 0.05) == [0]                    # |M_j - M_j+1| / M_j
    assert P.eliminate([100.0, 100.0], -1) == [1]


# ---- DP vs brute force ----------------------------------------------------------

def _rand_prof(rng, n):
    return [LP(rng.uniform(1, 100), rng.uniform(0.1, 10), rng.uniform(1, 1000), int(rng.integers(0, 2)) * 64)
            for _ in range(n)]


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 11])
def test_dp_equals_brute_force(n):
    rng = np.random.default_rng(100 + n)
    for trial in range(60):
        prof = _rand_prof(rng, n)
        ratio = [float(rng.choice([1, 8, 64])) for _ in range(n - 1)]
        allowed = None if trial % 3 else [int(v) for v in rng.integers(0, 2, n - 1)]
        tau = -1.0 if trial % 2 else 0.05
        for K in [0] + list(range(1, n + 1)):
            opts = P.PlanOpts(n_slices=K, allowed_cut=allowed, elim_tau=tau, c_m=1.0, c_n=rng.uniform(0, 5),
                              bw=rng.uniform(10, 1000), ratio=ratio)
            best, args = P.brute_force_plan(prof, opts)
            if best == math.inf:
                with pytest.raises(P.Infeasible):
                    P.plan_slices(prof, opts)
                continue
            pl = P.plan_slices(prof, opts)
            assert pl.cost == best
            assert P.plan_cost(prof, opts, pl.slice_end) == best
            assert pl.slice_end in args
            if K:
                assert pl.n_slices == K
            cuts = pl.slice_end[:-1]
            assert all(pl.allowed[c] for c in cuts)


def test_tie_rule_longest_last_slice():
    prof = [LP(1.0, 1.0) for _ in range(6)]
    opts = P.PlanOpts(n_slices=0, elim_tau=-1, c_n=0.0)
    assert P.plan_slices(prof, opts).slice_end == [5]                 # one slice: all plans tie at 6
    opts.n_slices = 3
    assert P.plan_slices(prof, opts).slice_end == [0, 1, 5]           # smallest start for each later slice


def test_dp_prefers_cut_between_dissimilar_layers():
    prof = [LP(10, 1), LP(10, 1), LP(10, 1), LP(1000, 1), LP(1000, 1)]
    pl = P.plan_slices(prof, P.PlanOpts(n_slices=0, elim_tau=-1, c_n=0.0))
    assert pl.slice_end == [2, 4]                                     # 10*3 + 1000*2 beats 1000*5


def test_prescribed_cuts_give_unique_plan():
    for cfg in (2, 4, 5):
        m = synth.build(cfg)
        prof = P.layer_profiles(m)
        s = m.slicing
        pl = P.plan_slices(prof, P.PlanOpts(n_slices=s["n_slices"], allowed_cut=s["allowed_cut"],
                                            k_override=s["k_override"]))
        want = [j for j, a in enumerate(s["allowed_cut"]) if a] + [len(m.layers) - 1]
        assert pl.slice_end == want
        assert pl.k == [k if k else 1 for k in s["k_override"]]


def test_infeasible_slice_count():
    prof = [LP(1, 1) for _ in range(4)]
    with pytest.raises(P.Infeasible):
        P.plan_slices(prof, P.PlanOpts(n_slices=3, allowed_cut=[1, 0, 0]))
    with pytest.raises(P.Infeasible):
        P.plan_slices(prof, P.PlanOpts(n_slices=5))


# ---- parallelism search, latency ------------------------------------------------

def test_parallelism_analytic_gives_one():
    prof = [LP(10, 1, rd=64), LP(10, 1, rd=0), LP(50, 2, rd=32)]
    pl = P.plan_slices(prof, P.PlanOpts(n_slices=1, k_max=8))
    assert pl.k == [1, 1, 1]


def test_parallelism_table_minimum_and_ties():
    prof = [LP(10, 1, rd=64), LP(10, 1, rd=0), LP(50, 2, rd=32)]
    tp = [[4.0, 3.0, 1.0, 2.0], [1.0, 1.0, 1.0, 1.0], [4.0, 3.0, 1.0, 2.0]]
    pl = P.plan_slices(prof, P.PlanOpts(n_slices=1, k_max=4, tp_table=tp))
    assert pl.k == [3, 1, 3]
    tie = [[2.0, 1.0, 1.0, 1.0], [1.0] * 4, [2.0, 1.0, 1.0, 1.0]]
    assert P.plan_slices(prof, P.PlanOpts(n_slices=1, k_max=4, tp_table=tie)).k == [2, 1, 2]
    # lambda caps eta at floor(M_g / lambda) = floor(50 / 20) = 2
    assert P.plan_slices(prof, P.PlanOpts(n_slices=1, k_max=4, tp_table=tp, lambda_bytes=20.0)).k == [2, 1, 2]
    # aggregation time pushes the optimum back
    ta = [[0.0, 0.0, 5.0, 5.0], [0.0] * 4, [0.0, 0.0, 5.0, 5.0]]
    assert P.plan_slices(prof, P.PlanOpts(n_slices=1, k_max=4, tp_table=tp, ta_table=ta)).k == [2, 1, 2]


def test_latency_check_hand_case():
    prof = [LP(10, 1.0, ob=80.0), LP(10, 2.0, ob=40.0), LP(10, 3.0, ob=8.0)]
    opts = P.PlanOpts(n_slices=2, allowed_cut=[1, 0], bw=10.0, ratio=[8, 1])
    pl = P.plan_slices(prof, opts)
    assert pl.slice_end == [0, 2]
    assert pl.t_tau == 6.0 + (80.0 / 8) / 10.0
    assert pl.t_unsplit == 6.0
    assert pl.latency_ok is False
    pl2 = P.plan_slices(prof, P.PlanOpts(n_slices=1))
    assert pl2.t_tau == 6.0 and pl2.latency_ok is True


def test_cfg1_plan_three_slices_and_rd_split():
    m = synth.build(1)
    s = m.slicing
    pl = P.plan_slices(P.layer_profiles(m), P.PlanOpts(n_slices=3, elim_tau=s["elim_tau"],
                                                        k_override=s["k_override"]))
    assert pl.n_slices == 3
    assert pl.k[m.layers.index("conv6")] == 2
    assert sum(pl.k) == len(m.layers) + 1


# --- dominant operators (Sec. III-B) and the Uniform variant (Sec. IV) -------------

def test_dominant_ops_is_smallest_set_reaching_the_share():
    # brute force: the selected set has the fewest ops of any subset whose footprint
    # reaches 80 % of the total, and it consists of the largest ops (ties by position)
    import itertools
    rng = np.random.default_rng(11)
    for trial in range(300):
        n = int(rng.integers(1, 8))
        mems = [float(v) for v in rng.integers(1, 6, n) * (10.0 ** rng.integers(0, 3, n))]
        frac = [0.8, 0.5, 1.0, 0.95][trial % 4]
        got = P.dominant_ops(mems, frac)
        total = sum(mems)
        need = min(len(c) for r in range(1, n + 1) for c in itertools.combinations(range(n), r)
                   if sum(mems[i] for i in c) >= frac * total - 1e-9 * total)
        assert len(got) == need
        cut = sorted(mems, reverse=True)[need - 1]
        assert all(mems[i] >= cut for i in got)
        assert got == sorted(got)


def test_dominant_ops_hand_cases():
    assert P.dominant_ops([50, 30, 15, 5], 0.8) == [0, 1]
    assert P.dominant_ops([5, 15, 30, 50], 0.8) == [2, 3]
    assert P.dominant_ops([10, 10, 10, 10], 0.8) == [0, 1, 2, 3]
    assert P.dominant_ops([10, 10, 10, 10], 0.5) == [0, 1]          # ties: earlier positions first
    assert P.dominant_ops([7], 0.8) == [0]


def test_layer_profile_from_dominant_ops(fake_profiles):
    # chain of four ops with memories 50, 30, 15, 5 and times 1, 2, 4, 8:
    # dominant (80 %) = first two -> M = 50, t = 3; all ops -> M = 50, t = 15
    m = _mini_model([(0, 1, 50, 1.0), (0, 2, 30, 2.0), (0, 3, 15, 4.0), (0, 4, 5, 8.0)])
    p = P.layer_profiles(m, dominant=0.8)[0]
    assert (p.mem_bytes, p.time_s) == (50.0, 3.0)
    q = P.layer_profiles(m)[0]
    assert (q.mem_bytes, q.time_s) == (50.0, 15.0)
    # branches: dominant ops are 9 (b1, pos 2) and 7 (b2, pos 1) and 5 (b1 pos 1): total 25, 80 % = 20
    m = _mini_model([(1, 1, 5, 2.0), (2, 1, 7, 5.0), (1, 2, 9, 1.0), (1, 3, 4, 3.0)])
    p = P.layer_profiles(m, dominant=0.8)[0]
    # kept: 9, 7, 5 (21 >= 20); positions: 1 -> 5 + 7 = 12 (t max 5), 2 -> 9 (t 1)
    assert (p.mem_bytes, p.time_s) == (12.0, 6.0)


@pytest.mark.parametrize("n,K", [(7, 3), (10, 4), (5, 5), (6, 1), (13, 4)])
def test_uniform_variant_sizes_and_cost(n, K):
    rng = np.random.default_rng(n * 10 + K)
    prof = _rand_prof(rng, n)
    u = P.plan_slices(prof, P.PlanOpts(n_slices=K, uniform=True))
    sizes = [len(c) for c in np.array_split(np.arange(n), K)]          # numpy's equal split
    assert np.diff([-1] + u.slice_end).tolist() == sizes
    # the DP's optimum over the same slice count can only be cheaper
    best, _ = P.brute_force_plan(prof, P.PlanOpts(n_slices=K, elim_tau=-1.0))
    assert best <= u.cost
    assert u.cost == P.plan_cost(prof, P.PlanOpts(), u.slice_end)
    with pytest.raises(ValueError):
        P.plan_slices(prof, P.PlanOpts(n_slices=0, uniform=True))
