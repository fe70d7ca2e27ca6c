"""Measured-profile planning (Alg. 1 free mode + the parallelism search of Eq. 5
fed by t_p(l, eta) measured on the GPU): the table, the plan the library derives
from it (equal to the oracle planner's on the same numbers), and a forward pass
under that plan against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import plan as OP
from helpers import SMALL, TOL, codec_ratios, rel_err

P = pytest.importorskip("paper_2404_02445_amd")
pytestmark = pytest.mark.gpu


def _np(t):
    a = t.float().cpu().numpy()
    return a.transpose(0, 3, 1, 2) if a.ndim == 4 else a


@pytest.mark.parametrize("cfg", [1, 2, 4, 6])
def test_measured_plan_matches_oracle_planner_and_runs(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    x_host = synth.make_input(m)
    x = torch.from_numpy(x_host).cuda()
    sm = P.SlicedModel(m)
    k_max = 4
    plan, tp, prof = sm.measured_plan(x, k_max=k_max, reps=3)
    tp = np.asarray(tp)
    n = len(m.layers)
    assert tp.shape == (n, k_max)
    assert np.all(np.isfinite(tp)) and np.all(tp > 0)
    # the library's plan over the measured numbers equals the oracle planner's, bit for bit
    want = OP.plan_slices([OP.LayerProfile(*p) for p in prof],
                          OP.PlanOpts(elim_tau=0.05, k_max=k_max, tp_table=tp.tolist(),
                                      ta_table=[[0.0] * k_max for _ in range(n)]))
    assert plan.slice_end == want.slice_end and plan.k == want.k
    assert plan.cost == want.cost and plan.t_tau == want.t_tau
    # every slice's eta is the smallest argmin of its measured time over the RD nodes' widths
    rdw = [p[3] for p in prof]
    lo = 0
    for end in plan.slice_end:
        nodes = range(lo, end + 1)
        ks = {plan.k[l] for l in nodes if rdw[l] > 0}
        assert len(ks) <= 1
        if ks:
            eta = ks.pop()
            tot = [sum(tp[l][e - 1] for l in nodes) for e in range(1, k_max + 1)]
            assert eta == 1 + int(np.argmin(tot))
        lo = end + 1
    # the model runs under the measured plan and matches the oracle under the same plan
    cuts = plan.slice_end[:-1]
    cw = synth.make_codec_weights(m, cuts, ratio=codec_ratios(m, cuts)) if cuts else None
    codecs, keep = sm.codecs(plan, "ae", cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    sm.forward(plan, x, out, codecs, codes, ws)
    torch.cuda.synchronize()
    ref = oracle.forward(m, x_host, k=plan.k, cuts=cuts, codecs=cw)
    assert rel_err(_np(out), ref) <= TOL[m.dtype]


def test_measure_restores_timing_state_and_rejects_bad_arguments():
    m = synth.build(1, **SMALL[1])
    sm = P.SlicedModel(m)
    x = torch.from_numpy(synth.make_input(m)).cuda()
    sm.set_timing(True)
    tp = sm.measure(x, k_max=2, reps=1)
    assert len(tp) == len(m.layers) and all(len(r) == 2 for r in tp)
    n = len(m.layers)
    plan = P.make_plan(n, [n - 1], [1] * n)
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    sm.forward(plan, x, out, None, None, ws)
    ops, _ = sm.op_times()              # timing is still on after the measurement
    assert all(t >= 0 for t in ops)
    sm.set_timing(False)
    with pytest.raises(P.MoparError):
        sm.measure(x, k_max=0)
    with pytest.raises(P.MoparError):
        sm.measure(x, k_max=2, reps=0)


def test_uniform_and_dominant_plans_run_on_the_branching_model():
    # Uniform variant (same slice count as the DP, equal node counts) on the Inception-style
    # model, from the dominant-operator profile; every cut carries one tensor
    m = synth.build(6, **SMALL[6])
    x_host = synth.make_input(m)
    sm = P.SlicedModel(m)
    prof = sm.profile(dominant=0.8)
    mopar = P.mopar_plan_slices(prof, n_slices=0, k_max=2)
    uni = P.mopar_plan_slices(prof, n_slices=mopar.n_slices, uniform=True, k_max=2)
    want = OP.plan_slices([OP.LayerProfile(*p) for p in prof],
                          OP.PlanOpts(n_slices=mopar.n_slices, uniform=True, k_max=2))
    assert (uni.slice_end, uni.k, uni.cost) == (want.slice_end, want.k, want.cost)
    assert mopar.cost <= uni.cost
    for plan in (mopar, uni):
        cuts = plan.slice_end[:-1]
        cw = synth.make_codec_weights(m, cuts, ratio=codec_ratios(m, cuts)) if cuts else None
        codecs, keep = sm.codecs(plan, "ae", cw)
        codes = sm.alloc_codes(plan, codecs)
        ws = sm.alloc_workspace(plan)
        out = sm.alloc_output()
        sm.forward(plan, torch.from_numpy(x_host).cuda(), out, codecs, codes, ws)
        torch.cuda.synchronize()
        ref = oracle.forward(m, x_host, k=plan.k, cuts=cuts, codecs=cw)
        assert rel_err(_np(out), ref) <= TOL[m.dtype]
