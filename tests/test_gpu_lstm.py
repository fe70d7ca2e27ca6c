"""The LSTM recurrence on the GPU.

bf16 layers whose hidden size is a multiple of 16 (up to 1024) run the whole
recurrence in one launch; others run one GEMM per step.  Both are checked
against the oracle; so are stacked layers, whose outputs must not depend on the
schedule (the same bits with per-op timing, with the no-allocation forward, and
with a slice cut between the layers).  The one-launch kernel lets any resident block compute a tile whose owner
is not running; the tests force that from the host (hooks make some blocks exit
at once, or start late) and require the same output bits, and run two models
concurrently on two streams.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.helpers import TOL, rel_err
from paper_2404_02445_amd._lib import STATIC_WORKSPACE_BYTES

pytestmark = pytest.mark.gpu
P = pytest.importorskip("paper_2404_02445_amd")


def lstm_model(b, t, e, h, seed=3, layers=1, w=0.3, nodes=False):
    """An embedding and `layers` stacked LSTM layers (each its own planning node if `nodes`)."""
    bld = synth._Builder("lstm", "bf16", b, seed)
    ids = bld.tensor((b, t), "i32")
    bld.new_layer("L0")
    x = bld.embed(ids, b * t, e, "src", -1.0, 1.0)
    for i in range(layers):
        if nodes:
            bld.new_layer(f"L{i + 1}")
        x = bld.lstm(x, h, f"lstm{i}", -w, w)
    return bld.finish(x, 1), np.arange(b * t, dtype=np.int32).reshape(b, t)


def forward(m, ids, stream=None):
    sm = P.SlicedModel(m)
    plan = P.make_plan(1, [0], [1])
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    x = torch.from_numpy(ids).cuda()
    if stream is not None:                  # weights and ids were uploaded on torch's stream
        stream.wait_stream(torch.cuda.current_stream())
    sm.forward(plan, x, out, None, None, ws, stream=stream)
    return out, (sm, ws, x)


def canon(t):
    return t.float().cpu().numpy()


@pytest.mark.parametrize("b,t,e,h,w", [
    (37, 6, 64, 48, 0.3),       # ragged batch group (37 = 2 x 16 + 5), K padded to a whole MFMA step
    (17, 1, 16, 32, 0.3),       # a single step
    (64, 5, 128, 256, 0.3),
    (5, 9, 1024, 1024, 0.3),    # the LSTM LM's hidden size: 32 weight fragments per lane
    (3, 4, 24, 40, 0.3),        # hidden size off the 16-unit tile: one GEMM per step
    (2, 7, 8, 16, 0.3),         # the smallest hidden size: one gate slice, one tile per batch group
    (1, 4096, 8, 16, 0.3),      # the longest sequence of one launch
    (1, 4097, 8, 16, 0.3),      # one step more: one GEMM per step
    # the input projection (16384 x 256 x 4096, float32 out) on 256 x 256 tiles; recurrent weights
    # small enough that the 1024-step recurrence contracts (with weights of +-0.3 at this hidden
    # size it is chaotic, and rounding differences grow until any two implementations disagree)
    (16, 1024, 256, 1024, 0.03),
])
def test_lstm_recurrence_parity(b, t, e, h, w):
    m, ids = lstm_model(b, t, e, h, w=w)
    y, _ = forward(m, ids)
    torch.cuda.synchronize()
    assert rel_err(canon(y), oracle.forward(m, ids)) <= TOL["bf16"]


@pytest.mark.parametrize("absent", [2, 3, 7])
def test_tiles_of_blocks_that_never_run_are_computed_by_others(absent):
    m, ids = lstm_model(40, 12, 64, 256, layers=2)
    ref, _ = forward(m, ids)
    torch.cuda.synchronize()
    os.environ["MOPAR_TEST_LSTM_ABSENT"] = str(absent)
    try:
        got, _ = forward(m, ids)
        torch.cuda.synchronize()
    finally:
        del os.environ["MOPAR_TEST_LSTM_ABSENT"]
    assert torch.equal(got, ref)
    assert rel_err(canon(got), oracle.forward(m, ids)) <= TOL["bf16"]


@pytest.mark.parametrize("late_us", [1000, 5000])
def test_owners_that_start_late_take_over_from_helpers(late_us):
    # the owners of every third gate slice start late: others compute those tiles' first steps
    # (their cell state left in memory), then each owner claims the steps still free and goes on
    m, ids = lstm_model(40, 40, 64, 256, layers=2)
    ref, _ = forward(m, ids)
    torch.cuda.synchronize()
    os.environ["MOPAR_TEST_LSTM_LATE_US"] = str(late_us)
    try:
        got, _ = forward(m, ids)
        torch.cuda.synchronize()
    finally:
        del os.environ["MOPAR_TEST_LSTM_LATE_US"]
    assert torch.equal(got, ref)
    assert rel_err(canon(got), oracle.forward(m, ids)) <= TOL["bf16"]


def test_two_layers_running_concurrently_on_two_streams():
    m, ids = lstm_model(64, 24, 256, 512, layers=2)
    ref, _ = forward(m, ids)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    keep = []
    outs = []
    for rep in range(3):
        for s in (s1, s2):
            o, k = forward(m, ids, stream=s)
            outs.append(o)
            keep.append(k)
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o, ref)


STACKED = [
    (37, 6, 64, 48, 2),      # ragged batch groups (37 = 2 x 16 + 5)
    (2, 7, 8, 16, 2),        # the smallest hidden size
    (64, 40, 128, 256, 3),   # three layers
    (40, 50, 64, 256, 2),
    (5, 9, 1024, 1024, 2),   # the LSTM LM's widths
    (64, 128, 1024, 1024, 2),  # the LSTM LM's layers
]


@pytest.mark.parametrize("b,t,e,h,layers", STACKED)
def test_stacked_layers_parity_and_schedule_independence(b, t, e, h, layers):
    m, ids = lstm_model(b, t, e, h, layers=layers, nodes=True, w=0.1 if t < 64 else 0.05)
    n = len(m.layers)
    sm = P.SlicedModel(m)
    x = torch.from_numpy(ids).cuda()
    whole = P.make_plan(n, [n - 1], [1] * n)
    ws = sm.alloc_workspace(whole)
    ref = oracle.forward(m, ids)

    def run(plan, timing=False, static=False):
        out = sm.alloc_output()
        sm.set_timing(timing)
        try:
            if plan.n_slices == 1 and static:
                sm.forward_static(plan, x, out)
            elif plan.n_slices == 1:
                sm.forward(plan, x, out, None, None, ws)
            else:
                codecs, keep = sm.codecs(plan, "raw")
                codes = sm.alloc_codes(plan, codecs)
                sm.forward(plan, x, out, codecs, codes, sm.alloc_workspace(plan))
            torch.cuda.synchronize()
        finally:
            sm.set_timing(False)
        return out

    y = run(whole)
    assert rel_err(canon(y), ref) <= TOL["bf16"]
    assert torch.equal(run(whole), y), "not deterministic"
    assert torch.equal(run(whole, timing=True), y), "one after the other (per-op timing) differs"
    if sm.workspace_bytes(whole) <= STATIC_WORKSPACE_BYTES:
        assert torch.equal(run(whole, static=True), y), "the no-allocation forward differs"
    every_cut = P.make_plan(n, list(range(n)), [1] * n)   # a slice per layer, raw codecs
    assert torch.equal(run(every_cut), y), "a slice cut between the layers changes the bits"


@pytest.mark.parametrize("absent", [2, 3])
def test_stacked_layers_with_absent_blocks(absent):
    # blocks of both layers never run; the rest compute their tiles
    m, ids = lstm_model(64, 20, 256, 512, layers=2)
    ref, _ = forward(m, ids)
    torch.cuda.synchronize()
    os.environ["MOPAR_TEST_LSTM_ABSENT"] = str(absent)
    try:
        got, _ = forward(m, ids)
        torch.cuda.synchronize()
    finally:
        del os.environ["MOPAR_TEST_LSTM_ABSENT"]
    assert torch.equal(got, ref)
