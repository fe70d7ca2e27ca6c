"""Slice pipeline across requests (one stream and workspace per slice, a ring of
boundary code buffers): every pipelined batch must equal the sequential
forward of the same input bit for bit, whatever the ring depth."""
import numpy as np
import pytest
import torch

import synth
from tests.helpers import SMALL, codec_ratios

pytestmark = pytest.mark.gpu
P = pytest.importorskip("paper_2404_02445_amd")


@pytest.mark.parametrize("cfg,depth,replicas,per_slice", [(2, 1, 1, True), (2, 3, 1, True), (4, 2, 1, True),
                                                          (5, 2, 1, True), (1, 2, 1, True), (2, 2, 3, False),
                                                          (4, 1, 2, True)])
def test_pipelined_batches_equal_sequential_bitwise(cfg, depth, replicas, per_slice):
    m = synth.build(cfg, **SMALL[cfg])
    sm = P.SlicedModel(m)
    plan = sm.plan()
    cuts = plan.slice_end[:-1]
    cw = synth.make_codec_weights(m, cuts, ratio=codec_ratios(m, cuts))
    n_batches = 2 * depth * replicas + 3
    xs = [torch.from_numpy(synth.make_input(m, seed=500 + i)).cuda() for i in range(n_batches)]
    # sequential reference through mopar_model_forward
    codecs, keep = sm.codecs(plan, "ae", cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    ref = []
    for x in xs:
        o = sm.alloc_output()
        sm.forward(plan, x, o, codecs, codes, ws)
        ref.append(o)
    torch.cuda.synchronize()
    pipe = sm.pipeline(plan, "ae", cw, depth=depth, replicas=replicas, stream_per_slice=per_slice)
    outs = [sm.alloc_output() for _ in xs]
    torch.cuda.synchronize()
    for x, o in zip(xs, outs):
        pipe.submit(x, o)
    pipe.synchronize()
    for i, (a, b) in enumerate(zip(outs, ref)):
        assert torch.equal(a, b), f"batch {i} differs from the sequential forward"
    assert not all(torch.equal(outs[0], o) for o in outs[1:]), "inputs should give different outputs"


def test_pipeline_rejects_bad_arguments():
    m = synth.build(2, **SMALL[2])
    sm = P.SlicedModel(m)
    plan = sm.plan()
    with pytest.raises(P.MoparError):
        sm.pipeline(plan, "ae", synth.make_codec_weights(m, plan.slice_end[:-1]), depth=0)


@pytest.mark.gpu
@pytest.mark.parametrize("cfg,replicas", [(1, 2), (2, 2), (4, 1), (6, 2)])
def test_pipeline_graph_replays_equal_sequential_bitwise(cfg, replicas):
    """Graph replay: several replays of each captured (slot, input, output) graph, with the
    program's own eager work and host synchronisations between them; every replay's output
    must equal the sequential forward of its input bit for bit."""
    m = synth.build(cfg, **SMALL[cfg])
    sm = P.SlicedModel(m)
    plan = sm.plan()
    cuts = plan.slice_end[:-1]
    cw = synth.make_codec_weights(m, cuts, ratio=codec_ratios(m, cuts))
    xs = [torch.from_numpy(synth.make_input(m, seed=700 + i)).cuda() for i in range(2)]
    codecs, keep = sm.codecs(plan, "ae", cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    ref = []
    for x in xs:
        o = sm.alloc_output()
        sm.forward(plan, x, o, codecs, codes, ws)
        ref.append(o)
    torch.cuda.synchronize()
    pipe = sm.pipeline(plan, "ae", cw, depth=2, replicas=replicas, stream_per_slice=False).use_graphs(True)
    outs = [sm.alloc_output() for _ in xs]
    scratch = torch.randn(1 << 16, device="cuda")
    for rnd in range(4):
        for i, (x, o) in enumerate(zip(xs, outs)):
            o.zero_()
            torch.cuda.synchronize()
            pipe.submit(x, o)
            pipe.synchronize()
            scratch.mul_(1.0001).add_(0.5)          # eager work between replays
            torch.cuda.synchronize()
            assert torch.equal(o, ref[i]), f"replay round {rnd}, input {i} differs from the sequential forward"
    pipe.use_graphs(False)
    for i, (x, o) in enumerate(zip(xs, outs)):
        o.zero_()
        pipe.submit(x, o)
        pipe.synchronize()
        assert torch.equal(o, ref[i])


@pytest.mark.gpu
def test_pipeline_graphs_need_one_stream_per_instance():
    m = synth.build(2, **SMALL[2])
    sm = P.SlicedModel(m)
    plan = sm.plan()
    pipe = sm.pipeline(plan, "ae", synth.make_codec_weights(m, plan.slice_end[:-1],
                                                             ratio=codec_ratios(m, plan.slice_end[:-1])),
                       depth=2, replicas=1, stream_per_slice=True)
    with pytest.raises(P.MoparError, match="UNSUPPORTED"):
        pipe.use_graphs(True)
