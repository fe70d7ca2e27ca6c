"""Host-side checks of the HIP library (no GPU): it loads, exports every symbol
of include/mopar.h, and its host logic (planner, profile, sub-slice ranges,
validation) agrees with the oracle bit for bit.  No kernel is launched."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synth
from oracle import plan as OP
from helpers import SMALL

SMALL6 = SMALL[6]

P = pytest.importorskip("paper_2404_02445_amd")
from paper_2404_02445_amd import _lib as L  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_header_symbol():
    hdr = open(os.path.join(ROOT, "include", "mopar.h")).read()
    names = set(re.findall(r"^\s*(?:int|void|const char\*)\s+(mopar_\w+)\s*\(", hdr, re.M))
    assert len(names) >= 13
    assert names == set(L.SIGNATURES)
    lib = P.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert b"gfx950" in lib.mopar_version()


def test_subslice_range_matches_oracle():
    for n in [1, 5, 16, 64, 301, 4096]:
        for k in range(1, min(n, 9) + 1):
            for j in range(k):
                assert P.mopar_subslice_range(n, k, j) == oracle.subslice_range(n, k, j)
    for bad in [(4, 5, 0), (4, 0, 0), (4, 2, 2), (4, 2, -1)]:
        with pytest.raises(P.MoparError):
            P.mopar_subslice_range(*bad)


def _rand_prof(rng, n):
    return [(rng.uniform(1, 100), rng.uniform(0.1, 10), rng.uniform(1, 1000), int(rng.integers(0, 3)) * 32)
            for _ in range(n)]


@pytest.mark.parametrize("n", [1, 2, 4, 7, 12, 21])
def test_planner_bitwise_equal_to_oracle(n):
    rng = np.random.default_rng(n)
    for trial in range(40):
        prof = _rand_prof(rng, n)
        lp = [OP.LayerProfile(*p) for p in prof]
        kmax = int(rng.integers(1, 5))
        kw = dict(n_slices=int(rng.integers(0, n + 1)), elim_tau=[-1.0, 0.05, 0.3][trial % 3],
                  c_m=float(rng.uniform(0.5, 2)), c_n=float(rng.uniform(0, 3)), bw=float(rng.uniform(1, 100)),
                  ratio=[float(rng.choice([1, 8, 64])) for _ in range(n - 1)] if trial % 2 else None,
                  k_max=kmax, lambda_bytes=float(rng.choice([0.0, 20.0])))
        if trial % 4 == 1:
            kw["allowed_cut"] = [int(v) for v in rng.integers(0, 2, n - 1)]
        if trial % 5 == 2:
            kw["tp_table"] = rng.uniform(0.1, 5, (n, kmax)).tolist()
            kw["ta_table"] = rng.uniform(0, 1, (n, kmax)).tolist()
        opts = OP.PlanOpts(**{k: v for k, v in kw.items() if k != "bw"}, bw=kw["bw"])
        try:
            want = OP.plan_slices(lp, opts)
        except OP.Infeasible:
            with pytest.raises(P.MoparError) as ei:
                P.mopar_plan_slices(prof, **kw)
            assert ei.value.status == L.MOPAR_E_INFEASIBLE
            continue
        got = P.mopar_plan_slices(prof, **kw)
        assert got.slice_end == want.slice_end
        assert got.k == want.k
        assert got.cost == want.cost and got.t_tau == want.t_tau and got.t_unsplit == want.t_unsplit
        assert got.latency_ok == want.latency_ok


def test_planner_error_paths():
    prof = [(10.0, 1.0, 5.0, 0), (20.0, 1.0, 5.0, 64)]
    with pytest.raises(P.MoparError) as e:
        P.mopar_plan_slices(prof, k_override=[2, 0])        # k on a node without an RD op
    assert e.value.status == L.MOPAR_E_ARG
    with pytest.raises(P.MoparError) as e:
        P.mopar_plan_slices(prof, k_override=[0, 65])       # wider than the RD op
    assert e.value.status == L.MOPAR_E_ARG
    with pytest.raises(P.MoparError) as e:
        P.mopar_plan_slices(prof, n_slices=2, allowed_cut=[0])
    assert e.value.status == L.MOPAR_E_INFEASIBLE
    with pytest.raises(P.MoparError):
        P.mopar_plan_slices([(0.0, 1.0, 1.0, 0)])           # zero memory footprint
    with pytest.raises(P.MoparError):
        P.mopar_plan_slices(prof, bw=0.0)
    assert P.mopar_plan_slices(prof, n_slices=2).slice_end == [0, 1]


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6, 7])
def test_model_profile_and_plan_equal_oracle(cfg):
    kw = {} if cfg != 3 else dict(batch=2, hw=64)
    m = synth.build(cfg, **kw)
    sm = P.SlicedModel(m, device="cpu")          # create validates and plans; nothing runs
    got = sm.profile()
    want = OP.layer_profiles(m)
    assert [tuple(g) for g in got] == [(w.mem_bytes, w.time_s, w.out_bytes, w.rd_width) for w in want]
    s = m.slicing
    pl = sm.plan()
    po = OP.plan_slices(want, OP.PlanOpts(n_slices=s["n_slices"], allowed_cut=s["allowed_cut"],
                                          elim_tau=s["elim_tau"], k_override=s["k_override"]))
    assert (pl.slice_end, pl.k, pl.cost, pl.t_tau) == (po.slice_end, po.k, po.cost, po.t_tau)
    assert sm.workspace_bytes(pl) > 0


def test_model_create_validation_errors():
    m = synth.build(1)
    tens, ops, blob = P.binding._pack(m)
    host = np.zeros(blob.size, dtype=np.uint8)

    def create(ops_arr, n_layers=len(m.layers), wbytes=blob.size, output=m.output_tid):
        d = L.ModelDesc()
        d.dtype = L.MOPAR_F32
        d.n_tensors, d.tensors = len(m.tensors), ctypes.cast(tens, ctypes.POINTER(L.TensorDesc))
        d.n_ops, d.ops = len(m.ops), ctypes.cast(ops_arr, ctypes.POINTER(L.Op))
        d.n_layers, d.input, d.output = n_layers, m.input_tid, output
        h = ctypes.c_void_p()
        st = P.lib().mopar_model_create(ctypes.byref(d), host.ctypes.data_as(ctypes.c_void_p), wbytes,
                                        ctypes.byref(h))
        if st == 0:
            P.lib().mopar_model_destroy(h)
        return st

    assert create(ops) == 0
    bad = (L.Op * len(m.ops))(*ops)
    bad[1].w = blob.size                           # weight offset past the blob
    assert create(bad) == L.MOPAR_E_ARG
    bad = (L.Op * len(m.ops))(*ops)
    bad[0].n_out = 17                              # output shape no longer matches
    assert create(bad) == L.MOPAR_E_SHAPE
    bad = (L.Op * len(m.ops))(*ops)
    bad[3].in0 = bad[5].out                        # reads a tensor before it is produced
    assert create(bad) == L.MOPAR_E_ARG
    bad = (L.Op * len(m.ops))(*ops)
    bad[2].rd = 1                                  # a pool cannot be an RD op
    assert create(bad) == L.MOPAR_E_ARG
    assert create(ops, n_layers=len(m.layers) + 1) == L.MOPAR_E_ARG
    assert create(ops, wbytes=16) == L.MOPAR_E_ARG
    assert b"op" in P.lib().mopar_last_error()


def test_gemm_operand_of_2gib_rejected_at_create():
    """A GEMM operand of 2 GiB or more (here a 1x1 conv's input image batch) is rejected when
    the model is created, before anything could be enqueued."""
    bld = synth._Builder("big", "bf16", 1, 7)
    x = bld.tensor((1, 8, 16384, 16384), "f32")
    bld.new_layer("L0")
    y = bld.conv(x, 8, 1, 1, 0, "none", "c")
    m = bld.finish(y, 1)
    tens, ops, blob = P.binding._pack(m)
    host = np.zeros(blob.size, dtype=np.uint8)
    d = L.ModelDesc()
    d.dtype = L.MOPAR_BF16
    d.n_tensors, d.tensors = len(m.tensors), ctypes.cast(tens, ctypes.POINTER(L.TensorDesc))
    d.n_ops, d.ops = len(m.ops), ctypes.cast(ops, ctypes.POINTER(L.Op))
    d.n_layers, d.input, d.output = len(m.layers), m.input_tid, m.output_tid
    h = ctypes.c_void_p()
    st = P.lib().mopar_model_create(ctypes.byref(d), host.ctypes.data_as(ctypes.c_void_p), blob.size, ctypes.byref(h))
    assert st == L.MOPAR_E_UNSUPPORTED
    assert b"2 GiB" in P.lib().mopar_last_error()


def test_plan_model_mismatch_rejected():
    m = synth.build(1)
    sm = P.SlicedModel(m, device="cpu")
    bad = P.make_plan(len(m.layers), [3, 9], [1] * len(m.layers))
    bad.raw.k[2] = 2                               # k > 1 on a pool node
    with pytest.raises(P.MoparError):
        sm.workspace_bytes(bad)
    bad2 = P.make_plan(len(m.layers), [5, 4, 9], [1] * len(m.layers))
    with pytest.raises(P.MoparError):
        sm.workspace_bytes(bad2)


def test_codec_code_bytes_host_only():
    raw = P.make_codec("raw")
    assert P.mopar_boundary_code_bytes(raw, (8, 256, 56, 56), "bf16") == 8 * 256 * 56 * 56 * 2
    ae = L.Codec()
    ae.kind, ae.c, ae.c_code, ae.w_enc, ae.w_dec = L.CODEC_AE, 256, 32, 16, 16   # non-null dummies
    assert P.mopar_boundary_code_bytes(ae, (8, 256, 56, 56), "bf16") == 8 * 32 * 56 * 56 * 2
    assert P.mopar_boundary_code_bytes(ae, (32, 128, 256), "bf16") == 32 * 128 * 32 * 2
    ae.c = 128
    with pytest.raises(P.MoparError):
        P.mopar_boundary_code_bytes(ae, (8, 256, 56, 56), "bf16")
    # widths off the 16-byte granule run on the vector-ALU codec kernel: accepted
    ae.c, ae.c_code = 16, 2
    assert P.mopar_boundary_code_bytes(ae, (1, 16, 32, 32), "f32") == 32 * 32 * 2 * 4
    ae.c, ae.c_code = 12, 3
    assert P.mopar_boundary_code_bytes(ae, (2, 7, 12), "bf16") == 2 * 7 * 3 * 2
    ae.c_code = 0
    with pytest.raises(P.MoparError):
        P.mopar_boundary_code_bytes(ae, (2, 7, 12), "bf16")


def test_pipeline_workspace_and_validation_host_only():
    m = synth.build(2)
    sm = P.SlicedModel(m, device="cpu")
    pl = sm.plan()
    n = ctypes.c_size_t()
    assert P.lib().mopar_pipeline_workspace_bytes(sm.handle, ctypes.byref(pl.raw), 3, ctypes.byref(n)) == 0
    per = (sm.workspace_bytes(pl) + 255) // 256 * 256
    assert n.value == per * pl.n_slices * 3
    h = ctypes.c_void_p()
    streams = (ctypes.c_void_p * (3 * pl.n_slices))()
    # depth 0, replicas 0 and a too-small workspace are rejected before any device call
    st = P.lib().mopar_pipeline_create(sm.handle, ctypes.byref(pl.raw), None, 1, 0, streams, None, 0, None,
                                       ctypes.byref(h))
    assert st == L.MOPAR_E_ARG
    st = P.lib().mopar_pipeline_create(sm.handle, ctypes.byref(pl.raw), None, 0, 2, streams, None, 0, None,
                                       ctypes.byref(h))
    assert st == L.MOPAR_E_ARG
    st = P.lib().mopar_pipeline_create(sm.handle, ctypes.byref(pl.raw), None, 3, 2, streams, None, 0, None,
                                       ctypes.byref(h))
    assert st == L.MOPAR_E_WORKSPACE


def test_measure_argument_checks_host_only():
    m = synth.build(1)
    sm = P.SlicedModel(m, device="cpu")
    tab = (ctypes.c_double * (len(m.layers) * 4))()
    dummy = ctypes.c_void_p(16)           # never dereferenced: the checks come first
    for k_max, reps, src in [(0, 1, dummy), (65, 1, dummy), (4, 0, dummy), (4, 1, None)]:
        st = P.lib().mopar_model_measure(sm.handle, k_max, reps, src, dummy, dummy, 1 << 30, None, tab)
        assert st == L.MOPAR_E_ARG
    st = P.lib().mopar_model_measure(sm.handle, 4, 1, dummy, dummy, None, 0, None, tab)
    assert st == L.MOPAR_E_WORKSPACE or sm.workspace_bytes(P.make_plan(len(m.layers), [len(m.layers) - 1],
                                                                        [1] * len(m.layers))) == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_dominant_profile_equals_oracle(cfg):
    kw = {} if cfg != 3 else dict(batch=2, hw=64)
    m = synth.build(cfg, **kw)
    sm = P.SlicedModel(m, device="cpu")
    for frac in (0.8, 0.5):
        got = sm.profile(dominant=frac)
        want = OP.layer_profiles(m, dominant=frac)
        assert [tuple(g) for g in got] == [(w.mem_bytes, w.time_s, w.out_bytes, w.rd_width) for w in want]
    with pytest.raises(P.MoparError):
        sm.profile(dominant=0.0)


def test_uniform_plan_bitwise_equal_to_oracle():
    rng = np.random.default_rng(7)
    for trial in range(60):
        n = int(rng.integers(1, 16))
        prof = _rand_prof(rng, n)
        K = int(rng.integers(1, n + 1))
        kmax = int(rng.integers(1, 4))
        kw = dict(n_slices=K, uniform=True, k_max=kmax, ratio=[float(rng.choice([1, 8])) for _ in range(n - 1)])
        want = OP.plan_slices([OP.LayerProfile(*p) for p in prof], OP.PlanOpts(**kw))
        got = P.mopar_plan_slices(prof, **kw)
        assert (got.slice_end, got.k, got.cost, got.t_tau) == (want.slice_end, want.k, want.cost, want.t_tau)
    with pytest.raises(P.MoparError):
        P.mopar_plan_slices([(1.0, 1.0, 1.0, 0)], n_slices=0, uniform=True)


def test_concatenating_writers_validated():
    m = synth.build(6, **SMALL6)
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
    writers = [i for i, o in enumerate(m.ops) if "out_off" in o]
    first, second = writers[0], writers[1]
    bad = (L.Op * len(m.ops))(*ops)
    bad[second].out_off += 1                      # a gap / overlap between branches
    assert create(bad) == L.MOPAR_E_ARG
    bad = (L.Op * len(m.ops))(*ops)
    bad[first].out_off = 0
    bad[first].n_out += 8                         # writes past the next branch's channels
    assert create(bad) != 0


def _create_error(build):
    """Status of model creation for the model `build` makes (None when accepted)."""
    b = synth._Builder("v", "bf16", 2, 9)
    y = build(b)
    m = b.finish(y, n_slices=1, k_by_layer={})
    try:
        P.SlicedModel(m, device="cpu")
    except P.MoparError as e:
        return e.status
    return None


def test_model_create_checks_what_the_kernels_assume():
    def stem(b, c):
        x = b.tensor((2, 3, 12, 12), "f32")
        b.new_layer("stem")
        return b.conv(x, c, 3, 1, 1, "relu", "stem", bn_fold=True)

    def pool(c):
        def f(b):
            x = stem(b, c)
            b.new_layer("pool")
            return b.maxpool(x, 3, 2, 1, "pool")
        return f

    def conv_after(c):
        def f(b):
            x = stem(b, c)
            b.new_layer("c1")
            return b.conv(x, 16, 3, 1, 1, "relu", "c1", bn_fold=True)
        return f

    def concat(offsets, head=True):
        def f(b):
            x = stem(b, 16)
            b.new_layer("cat")
            out = b.tensor((2, 32, 12, 12))
            for i, (c, off) in enumerate(offsets):
                b.conv(x, c, 1, 1, 0, "relu", f"b{i}", bn_fold=True, branch=i + 1, pos=1, into=(out, off))
            if not head:
                return out
            b.new_layer("head")
            return b.conv(out, 8, 1, 1, 0, "none", "head", bn_fold=True)
        return f

    # 16-byte channel groups (8 bf16): pools and conv inputs off the granule are refused
    assert _create_error(pool(16)) is None
    assert _create_error(pool(12)) == L.MOPAR_E_UNSUPPORTED
    assert _create_error(conv_after(24)) is None
    assert _create_error(conv_after(20)) == L.MOPAR_E_UNSUPPORTED
    # concatenation writers: any offset, but in channel order and covering every channel
    assert _create_error(concat([(13, 0), (19, 13)])) is None
    assert _create_error(concat([(19, 13), (13, 0)])) == L.MOPAR_E_ARG
    assert _create_error(concat([(13, 0), (16, 16)])) == L.MOPAR_E_ARG
    # the output must come from the last op, not from a concatenation's first writer
    assert _create_error(concat([(13, 0), (19, 13)], head=False)) == L.MOPAR_E_ARG


def test_k_override_beyond_measured_tables_refused_by_both_planners():
    """A forced sub-slice count above k_max has no measured t_p / t_a: both planners refuse it
    (the library used to read past the tables; found by the sanitizer run)."""
    prof = [(1e6, 1e-4, 1e3, 64)] * 3
    tp = [[1e-4, 2e-4]] * 3
    with pytest.raises(P.MoparError, match="ARG"):
        P.mopar_plan_slices(prof, k_max=2, tp_table=tp, k_override=[0, 4, 0])
    with pytest.raises(ValueError):
        OP.plan_slices([OP.LayerProfile(*p) for p in prof],
                       OP.PlanOpts(k_max=2, tp_table=tp, k_override=[0, 4, 0]))
    # without tables the analytic t_p applies to any k
    assert P.mopar_plan_slices(prof, k_max=2, k_override=[0, 4, 0]).k[1] == 4


def test_split_k_factor_never_exceeds_what_the_reduce_handles():
    # the split-K reduce keeps every split's partial in flight at once, for at most 16 splits;
    # the factor the executor asks for (a host function of the library) must stay in 1..16, a
    # power of two, and above 1 only for long K loops (at least 24 stages of 64 bf16 / 32 fp32)
    fn = getattr(L.lib(), "_ZN5mopar11gemm_splitsEliiii")
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    for dtype, bk in ((L.MOPAR_BF16, 64), (L.MOPAR_F32, 32)):
        for M in (1, 16, 63, 64, 392, 1568, 25088, 1 << 20):
            for N in (1, 16, 100, 4096, 32000):
                for K in (1, 64, 1535, 1536, 4608, 25088, 1 << 20):
                    s = fn(M, N, K, dtype, 0)
                    assert 1 <= s <= 16 and s & (s - 1) == 0, (M, N, K, s)
                    if (K + bk - 1) // bk < 24:
                        assert s == 1, (M, N, K, s)
                    assert fn(M, N, K, dtype, 1) == 1   # the LSTM epilogue never splits
