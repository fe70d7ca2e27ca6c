"""Skip edges across planning nodes (Sec. III-C, edge elimination): a cut carries every
tensor crossing it, the layer profile's cut size is their sum, and each crossing tensor
has its own codec and code buffer.  CPU checks of the oracle and the library's host
logic, GPU checks of the sliced forward and the pipeline on a model whose cuts carry up
to three tensors."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import plan as OP
from tests.helpers import SMALL, TOL, boundary_codecs, rel_err

P = pytest.importorskip("paper_2404_02445_amd")


def _np(t):
    a = t.float().cpu().numpy()
    return a.transpose(0, 3, 1, 2) if a.ndim == 4 else a


def test_crossing_sets_and_cut_sizes_hand_worked():
    m = synth.build(7, **SMALL[7])
    outs = OP.node_outputs(m)            # stem, c1, c2, c3, cat, head
    x0, x1, x2, x3, cat = outs[:5]
    got = [OP.crossing_tensors(m, j) for j in range(5)]
    assert got == [[x0], [x0, x1], [x0, x1, x2], [x1, x3], [cat]]
    b = 3 * 16 * 16 * 2                  # bytes per 16-channel plane of the batch, bf16
    prof = OP.layer_profiles(m)
    assert [p.out_bytes for p in prof[:5]] == [16 * b, 32 * b, 48 * b, 32 * b, 32 * b]
    # a chain model's cut size is the node output (one edge per cut)
    c = synth.build(2, **SMALL[2])
    assert all(OP.crossing_tensors(c, j) == [OP.node_outputs(c)[j]] for j in range(len(c.layers) - 1))


@pytest.mark.parametrize("cfg", [1, 2, 4, 5, 6, 7])
def test_library_cut_tensors_equal_oracle(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    sm = P.SlicedModel(m, device="cpu")
    for j in range(len(m.layers) - 1):
        assert sm.cut_tensors(j) == OP.crossing_tensors(m, j)
    got = sm.profile()
    want = OP.layer_profiles(m)
    assert [g[2] for g in got] == [w.out_bytes for w in want]
    with pytest.raises(P.MoparError):
        sm.cut_tensors(len(m.layers) - 1)


def test_reading_an_inner_tensor_of_an_earlier_node_is_rejected():
    # only a node's output may leave it: point a later node at a tensor made inside an
    # earlier node (the 1x1 reducer of an Inception branch) and creation must fail
    import ctypes
    from paper_2404_02445_amd import _lib as L
    m = synth.build(6, **SMALL[6])
    tens, ops, blob = P.binding._pack(m)
    host = np.zeros(blob.size, dtype=np.uint8)

    def create(ops_arr):
        d = L.ModelDesc()
        d.dtype = L.MOPAR_BF16
        d.n_tensors, d.tensors = len(m.tensors), ctypes.cast(tens, ctypes.POINTER(L.TensorDesc))
        d.n_ops, d.ops = len(m.ops), ctypes.cast(ops_arr, ctypes.POINTER(L.Op))
        d.n_layers, d.input, d.output = len(m.layers), m.input_tid, m.output_tid
        h = ctypes.c_void_p()
        st = P.lib().mopar_model_create(ctypes.byref(d), host.ctypes.data_as(ctypes.c_void_p), blob.size,
                                        ctypes.byref(h))
        if st == 0:
            P.lib().mopar_model_destroy(h)
        return st

    assert create(ops) == 0
    reducer = [i for i, o in enumerate(m.ops) if o["layer"] == 2 and o["name"].endswith(".b2r")][0]
    later = [i for i, o in enumerate(m.ops) if o["layer"] == 3 and o["name"].endswith(".b2r")][0]
    bad = (L.Op * len(m.ops))(*ops)
    bad[later].in0 = m.ops[reducer]["out"]
    assert create(bad) != 0


def _run(m, x, plan, kind, cw, sm=None):
    sm = sm or P.SlicedModel(m)
    codecs, keep = sm.codecs(plan, kind, cw)
    codes = sm.alloc_codes(plan, codecs)
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    sm.forward(plan, torch.from_numpy(x).cuda(), out, codecs, codes, ws)
    torch.cuda.synchronize()
    return out


@pytest.mark.gpu
@pytest.mark.parametrize("cuts", [[1, 3], [2], [0, 1, 2, 3, 4]])
def test_multi_tensor_cuts_forward(cuts):
    m = synth.build(7, **SMALL[7])
    x = synth.make_input(m)
    n = len(m.layers)
    sm = P.SlicedModel(m)
    k = [1] * n
    k[2] = 2                                   # the RD conv in two sub-slices
    plan = P.make_plan(n, cuts + [n - 1], k)
    tids, cw = boundary_codecs(m, cuts)
    assert sm.boundary_tensors(plan) == tids
    y = _run(m, x, plan, "ae", cw, sm)
    ref = oracle.forward(m, x, k=k, cuts=cuts, codecs=cw)
    assert rel_err(_np(y), ref) <= TOL[m.dtype]
    # raw hand-off of every crossing tensor == the unsliced model, bit for bit
    y0 = _run(m, x, P.make_plan(n, [n - 1], k), "raw", None, sm)
    yr = _run(m, x, plan, "raw", None, sm)
    assert torch.equal(y0, yr)


@pytest.mark.gpu
def test_multi_tensor_cuts_pipeline_equals_sequential():
    m = synth.build(7, **SMALL[7])
    x = torch.from_numpy(synth.make_input(m)).cuda()
    n = len(m.layers)
    sm = P.SlicedModel(m)
    cuts = [1, 2, 3]
    k = [1] * n
    k[2] = 2
    plan = P.make_plan(n, cuts + [n - 1], k)
    tids, cw = boundary_codecs(m, cuts)
    ref = _run(m, synth.make_input(m), plan, "ae", cw, sm)
    pipe = sm.pipeline(plan, "ae", cw, depth=2, replicas=2)
    outs = [sm.alloc_output() for _ in range(5)]
    for o in outs:
        pipe.submit(x, o)
    pipe.synchronize()
    for o in outs:
        assert torch.equal(o, ref)
