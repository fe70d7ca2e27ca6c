"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Floating-point outputs must be within the per-tensor relative error
max|gpu - ref| / max|ref| <= 2e-2 (bf16) or 1e-4 (fp32); sub-sliced kernels
must equal the unsplit kernel bit for bit; a sliced model with raw codecs must
equal the unsliced model bit for bit; the raw codec round-trips bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.helpers import SMALL, TOL, boundary_codecs, codec_ratios, rel_err

pytestmark = pytest.mark.gpu

P = pytest.importorskip("paper_2404_02445_amd")


def _np(t):
    """Device tensor -> numpy in canonical order (rank-4 tensors are stored channels-last)."""
    if t.dim() == 4:
        t = P.boundary_to_canonical(t.reshape(-1), tuple(t.shape))
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def run_gpu(m, x, plan, codec="raw", codec_w=None, repeat=1):
    sm = P.SlicedModel(m)
    ws = sm.alloc_workspace(plan)
    codecs, keep = sm.codecs(plan, codec, codec_w)
    codes = sm.alloc_codes(plan, codecs)
    xin = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    outs = []
    for _ in range(repeat):
        out = sm.alloc_output()
        sm.forward(plan, xin, out, codecs, codes, ws)
        torch.cuda.synchronize()
        outs.append(out)
    return (outs if repeat > 1 else outs[0]), codes, sm


def plan_of(m, sm=None, **kw):
    sm = sm or P.SlicedModel(m)
    return sm.plan(**kw)


# ---------------------------------------------------------------------------
# single operators (small models built around the op under test)
# ---------------------------------------------------------------------------

def conv_model(dtype, n, c, hw, cout, k, stride, pad, act="relu", residual=False, pre=False, seed=5):
    b = synth._Builder("conv", dtype, n, seed)
    x = b.tensor((n, c, hw, hw), "f32")
    b.new_layer("L0")
    if pre:   # an internal conv first, so the op under test reads a channels-last activation
        x = b.conv(x, c, 1, 1, 0, "none", "pre", bn_fold=True)
    res = None
    if residual:
        ho = (hw + 2 * pad - k) // stride + 1
        res = b.conv(x, cout, 1, 1, 0, "none", "sc", bn_fold=True) if (ho == hw) else None
        if res is None:
            res = b.conv(x, cout, 1, stride, 0, "none", "sc", bn_fold=True)
    y = b.conv(x, cout, k, stride, pad, act, "conv", res=res, bn_fold=True, rd=True)
    return b.finish(y, n_slices=1, k_by_layer={})


CONV_CASES = [
    # dtype, n, c, hw, cout, k, stride, pad, residual, pre
    ("bf16", 2, 3, 37, 64, 7, 2, 3, False, False),    # stem-like, padded channels, ragged M
    ("bf16", 2, 3, 30, 40, 3, 1, 1, False, False),    # first layer 3x3: ragged tiles and columns
    ("bf16", 1, 64, 19, 48, 3, 1, 1, True, True),     # 3x3, residual, ragged N tile (patch-staged)
    ("bf16", 2, 128, 20, 64, 3, 1, 1, False, True),   # patch-staged 3x3: two channel chunks, ragged tiles
    ("bf16", 1, 64, 16, 120, 3, 1, 1, True, True),    # patch-staged 3x3: whole tiles, ragged sub-slices
    ("bf16", 2, 192, 12, 40, 3, 1, 1, True, True),    # patch-staged, two chunk buffers: an odd chunk count
    ("bf16", 2, 256, 14, 256, 3, 1, 1, True, True),   # ResNet-50's stage-3 3x3 (four chunks)
    ("bf16", 1, 512, 7, 512, 3, 1, 1, True, True),    # stage 4: eight chunks, a 7 x 7 image in one ragged tile
    ("bf16", 2, 32, 14, 96, 3, 2, 1, True, True),     # strided 3x3
    ("bf16", 1, 128, 9, 256, 1, 1, 0, True, True),    # 1x1 wide
    ("bf16", 3, 16, 11, 20, 1, 2, 0, False, True),    # strided 1x1, N=20
    ("f32", 1, 3, 17, 16, 3, 1, 1, False, False),     # fp32 path
    ("f32", 2, 16, 9, 36, 3, 1, 1, True, True),
]


@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "-".join(map(str, c)))
def test_conv_parity_and_subslice_bitwise(case):
    dt, n, c, hw, cout, k, st, pad, residual, pre = case
    m = conv_model(dt, n, c, hw, cout, k, st, pad, residual=residual, pre=pre)
    x = synth.random_tensor((n, c, hw, hw), "f32", seed=11)
    ref = oracle.forward(m, x)
    plan1 = P.make_plan(1, [0], [1])
    y1, _, _ = run_gpu(m, x, plan1)
    assert rel_err(_np(y1), ref) <= TOL[dt]
    for ks in (2, 3, 4):
        if ks > cout:
            continue
        yk, _, _ = run_gpu(m, x, P.make_plan(1, [0], [ks]))
        assert torch.equal(yk, y1), f"k={ks} differs from the unsplit kernel"


def concat_model(dtype, n, hw, seed=6):
    """A stem conv to 64 channels, then one parallel node whose three branches write side by
    side into an 80-channel tensor at channel offsets 0, 13 and 64: a 1x1 conv (13 outputs),
    the RD 3x3 conv (51 outputs, stride 1, padding 1, 64 input channels -- the patch-staged
    kernel in bf16) and a 1x1 conv (16 outputs).  Offset 13 leaves the 3x3 branch's rows
    unaligned to a vector of four elements.  A 1x1 head conv reads the concatenation."""
    b = synth._Builder("concat", dtype, n, seed)
    x = b.tensor((n, 3, hw, hw), "f32")
    b.new_layer("stem")
    x = b.conv(x, 64, 3, 1, 1, "relu", "stem", bn_fold=True)
    b.new_layer("cat")
    out = b.tensor((n, 80, hw, hw))
    b.conv(x, 13, 1, 1, 0, "relu", "b1", bn_fold=True, branch=1, pos=1, into=(out, 0))
    b.conv(x, 51, 3, 1, 1, "relu", "b2", bn_fold=True, branch=2, pos=1, rd=True, into=(out, 13))
    b.conv(x, 16, 1, 1, 0, "none", "b3", bn_fold=True, branch=3, pos=1, into=(out, 64))
    b.new_layer("head")
    y = b.conv(out, 24, 1, 1, 0, "none", "head", bn_fold=True)
    return b.finish(y, n_slices=1, k_by_layer={})


@pytest.mark.parametrize("dt,n,hw", [("bf16", 2, 18), ("bf16", 1, 16), ("f32", 2, 9)])
def test_concat_at_unaligned_channel_offsets(dt, n, hw):
    m = concat_model(dt, n, hw)
    x = synth.random_tensor((n, 3, hw, hw), "f32", seed=12)
    ref = oracle.forward(m, x)
    y1, _, _ = run_gpu(m, x, P.make_plan(3, [2], [1, 1, 1]))
    assert rel_err(_np(y1), ref) <= TOL[dt]
    for ks in (2, 3, 4):
        yk, _, _ = run_gpu(m, x, P.make_plan(3, [2], [1, ks, 1]))
        assert torch.equal(yk, y1), f"k={ks} differs from the unsplit kernel"


def seq_input_model(dtype, b, s, f, seed=3, scale=1.0):
    """Model whose first op produces an arbitrary [B,S,F] activation: an embedding of ids
    0..B*S-1 into a table of random rows."""
    bld = synth._Builder("seq", dtype, b, seed)
    ids = bld.tensor((b, s), "i32")
    bld.new_layer("L0")
    x = bld.embed(ids, b * s, f, "src", -1.0, 1.0)
    bld.m.weights["src.table"] = synth.random_tensor((b * s, f), dtype, seed=seed + 100, scale=scale)
    return bld, x


def seq_ids(b, s):
    return np.arange(b * s, dtype=np.int32).reshape(b, s)


@pytest.mark.parametrize("dt,b,s,k,nout,act,res,ksub", [
    ("bf16", 3, 45, 136, 200, "gelu", False, 4),   # ragged M, N; K not a multiple of 64
    ("bf16", 2, 64, 768, 3072, "none", True, 4),
    ("bf16", 16, 1, 1024, 512, "relu", False, 8),  # M = 16 (fc-like)
    ("bf16", 1, 5, 64, 10, "none", False, 1),      # N = 10
    ("f32", 2, 7, 36, 44, "relu", True, 2),
    # few rows: K split across the waves of a block, with split-K and a K tail (2000 = 31*64 + 16)
    ("bf16", 16, 1, 2000, 96, "relu", False, 3),
    # split-K summed in the GEMM launch (k = 1) against the separate reduce launch (k = 100 sub-slices
    # need more arrival counters than the op's slot holds): bitwise equal
    ("bf16", 16, 1, 2000, 200, "relu", False, 100),
    # M = 40: the 64x64 and 64x16 K-split tiles (k = 1 vs k = 4) must agree bit for bit
    ("bf16", 5, 8, 1504, 70, "gelu", True, 4),
    ("f32", 4, 4, 700, 33, "none", True, 2),
    # products with at least 1024 tiles of 256 x 256 run on the 32 x 32 MFMA kernel, every
    # sub-slice launch included: 8192 x 256 x 8192 against 1024-column sub-slices
    ("bf16", 16, 512, 256, 8192, "none", False, 8),
    # ragged M (33 tile rows), N and K (312 = 4 x 64 + 56) with residual and GELU, against
    # 500-column sub-slices
    ("bf16", 3, 2743, 312, 8000, "gelu", True, 16),
    # the persistent launch with groups of four columns cut by the sub-slice edge (2 x 4001
    # columns: element stores)
    ("bf16", 4, 2048, 256, 8002, "none", False, 2),
    # BERT-base's FFN1 (4096 x 768 -> 3072, GELU) in its four 768-column sub-slices
    ("bf16", 32, 128, 768, 3072, "gelu", False, 4),
])
def test_linear_parity_and_subslice_bitwise(dt, b, s, k, nout, act, res, ksub):
    bld, x = seq_input_model(dt, b, s, k)
    if res:
        r = bld.linear(x, nout, "none", "r", "rand")
        y = bld.linear(x, nout, act, "lin", "rand", res=r, rd=True)
    else:
        y = bld.linear(x, nout, act, "lin", "rand", rd=True)
    m = bld.finish(y, 1)
    ids = seq_ids(b, s)
    ref = oracle.forward(m, ids)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    assert rel_err(_np(y1), ref) <= TOL[dt]
    yk, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [ksub]))
    assert torch.equal(yk, y1)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("k,st,pad", [(2, 2, 0), (3, 2, 1)])
def test_maxpool_and_avgpool(dt, k, st, pad):
    b = synth._Builder("pool", dt, 2, 9)
    x = b.tensor((2, 16, 15, 15), "f32")
    b.new_layer("L0")
    x = b.conv(x, 32, 3, 1, 1, "none", "c", bn_fold=True)
    p = b.maxpool(x, k, st, pad, "p")
    y = b.avgpool(p, "a")
    m = b.finish(y, 1)
    xx = synth.random_tensor((2, 16, 15, 15), "f32", seed=4)
    _, env, _, _ = oracle.forward(m, xx, keep=True)
    sm = P.SlicedModel(m)
    plan = P.make_plan(1, [0], [1])
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    sm.forward(plan, torch.from_numpy(xx).cuda(), out, None, None, ws)
    torch.cuda.synchronize()
    assert rel_err(_np(out), env[m.output_tid]) <= TOL[dt]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_avgpool_ragged_channels(dt):
    # channel counts that are not a whole number of 16-byte chunks take the per-channel path
    b = synth._Builder("pool", dt, 2, 9)
    x = b.tensor((3, 16, 9, 9), "f32")
    b.new_layer("L0")
    x = b.conv(x, 20, 3, 1, 1, "relu", "c", bn_fold=True)
    y = b.avgpool(x, "a")
    m = b.finish(y, 1)
    xx = synth.random_tensor((3, 16, 9, 9), "f32", seed=5)
    _, env, _, _ = oracle.forward(m, xx, keep=True)
    sm = P.SlicedModel(m)
    plan = P.make_plan(1, [0], [1])
    ws = sm.alloc_workspace(plan)
    out = sm.alloc_output()
    sm.forward(plan, torch.from_numpy(xx).cuda(), out, None, None, ws)
    torch.cuda.synchronize()
    assert rel_err(_np(out), env[m.output_tid]) <= TOL[dt]


def test_layernorm_with_residual():
    bld, x = seq_input_model("bf16", 3, 33, 768)
    r = bld.linear(x, 768, "none", "r", "rand")
    y = bld.layernorm(x, "ln", 1e-12, res=r, rand=True)
    m = bld.finish(y, 1)
    ids = seq_ids(3, 33)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    assert rel_err(_np(y1), oracle.forward(m, ids)) <= TOL["bf16"]


@pytest.mark.parametrize("dt,seq,heads", [("bf16", 128, 12), ("bf16", 37, 2), ("bf16", 1, 1), ("bf16", 64, 3),
                                           ("bf16", 65, 2), ("bf16", 100, 4), ("f32", 40, 2)])
def test_attention(dt, seq, heads):
    # bf16 runs on the matrix cores (64-query tiles, keys padded to 32 and masked), f32 on
    # the vector units; sequence lengths cover one key, whole and partial query tiles
    bld, x = seq_input_model(dt, 2, seq, 3 * 64 * heads, scale=1.5)
    y = bld.attention(x, heads, "att")
    m = bld.finish(y, 1)
    ids = seq_ids(2, seq)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    assert rel_err(_np(y1), oracle.forward(m, ids)) <= TOL[dt]


def test_embed_bert():
    bld = synth._Builder("emb", "bf16", 2, 21)
    ids = bld.tensor((2, 50), "i32")
    bld.new_layer("L0")
    y = bld.embed_bert(ids, 97, 64, 2, 768, "e", 1e-12, std=1.0)
    m = bld.finish(y, 1)
    x = np.random.default_rng(1).integers(0, 97, size=(2, 50)).astype(np.int32)
    y1, _, _ = run_gpu(m, x, P.make_plan(1, [0], [1]))
    assert rel_err(_np(y1), oracle.forward(m, x)) <= TOL["bf16"]


def test_embed_gather_bitwise():
    bld, x = seq_input_model("bf16", 4, 17, 64)
    m = bld.finish(x, 1)
    ids = seq_ids(4, 17)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    np.testing.assert_array_equal(_np(y1), oracle.forward(m, ids))


def test_embed_ids_out_of_range_clamped():
    """Ids outside [0, V) read the nearest table row (documented in the header), never past it."""
    bld, x = seq_input_model("bf16", 2, 5, 64)
    m = bld.finish(x, 1)
    v = 2 * 5
    ids = np.array([[0, -3, 4, v, v + 1000], [-(1 << 30), 9, 1, 2, (1 << 31) - 1]], dtype=np.int32)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    table = np.asarray(m.weights["src.table"])
    want = table[np.clip(ids, 0, v - 1)]
    np.testing.assert_array_equal(_np(y1), want.astype(np.float32))


@pytest.mark.parametrize("b,t,e,h", [(3, 7, 64, 64), (64, 4, 128, 256), (2, 3, 24, 40), (37, 5, 32, 72)])
def test_lstm(b, t, e, h):
    bld, x = seq_input_model("bf16", b, t, e)
    y = bld.lstm(x, h, "lstm", -0.3, 0.3)
    m = bld.finish(y, 1)
    ids = seq_ids(b, t)
    y1, _, _ = run_gpu(m, ids, P.make_plan(1, [0], [1]))
    assert rel_err(_np(y1), oracle.forward(m, ids)) <= TOL["bf16"]


# ---------------------------------------------------------------------------
# boundary codec
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt,shape", [("bf16", (2, 64, 7, 9)), ("bf16", (3, 11, 96)), ("f32", (2, 16, 5, 5))])
def test_codec_raw_roundtrip_bitwise(dt, shape):
    x = torch.from_numpy(synth.random_tensor(shape, dt, seed=2)).to("cuda", P.binding.TORCH_DTYPE[dt])
    cd = P.make_codec("raw")
    nbytes = P.mopar_boundary_code_bytes(cd, shape, dt)
    assert nbytes == x.numel() * x.element_size()
    code = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    P.mopar_boundary_encode(cd, shape, dt, x, code)
    P.mopar_boundary_decode(cd, shape, dt, code, y)
    torch.cuda.synchronize()
    assert torch.equal(code, x.view(-1).view(torch.uint8))
    assert torch.equal(y, x)


@pytest.mark.parametrize("dt,shape,ratio", [("bf16", (2, 256, 7, 9), 8), ("bf16", (3, 13, 768), 8),
                                            ("bf16", (1, 1024, 3, 5), 8), ("f32", (2, 32, 5, 6), 4),
                                            # code widths off the 16-byte granule (vector-ALU layers):
                                            # the tiny VGG's 16-channel boundary at R = 8
                                            ("f32", (1, 16, 16, 16), 8), ("bf16", (2, 9, 24), 8),
                                            ("bf16", (1, 12, 5, 3), 4)])
def test_codec_ae_parity(dt, shape, ratio):
    c = shape[1] if len(shape) == 4 else shape[-1]
    w = synth.random_codec_weights(c, c // ratio, dt, seed=7)
    x_can = synth.random_tensor(shape, dt, seed=8)
    code_ref = oracle.ae_encode(x_can, w["w_enc"], w["b_enc"], dt)
    y_ref = oracle.ae_decode(code_ref, w["w_dec"], w["b_dec"], dt)
    # physical layout: channels-last for images
    x_phys = x_can.transpose(0, 2, 3, 1) if len(shape) == 4 else x_can
    tdt = P.binding.TORCH_DTYPE[dt]
    x = torch.from_numpy(np.ascontiguousarray(x_phys)).to("cuda", tdt)
    dev = [torch.from_numpy(w[k]).to("cuda", tdt) for k in ("w_enc", "b_enc", "w_dec", "b_dec")]
    cd = P.make_codec("ae", c, c // ratio, *dev)
    nbytes = P.mopar_boundary_code_bytes(cd, shape, dt)
    assert nbytes * ratio == x.numel() * x.element_size()
    code = torch.empty(nbytes // x.element_size(), dtype=tdt, device="cuda")
    y = torch.empty_like(x)
    P.mopar_boundary_encode(cd, shape, dt, x, code)
    P.mopar_boundary_decode(cd, shape, dt, code, y)
    torch.cuda.synchronize()
    cshape = (shape[0], shape[2], shape[3], c // ratio) if len(shape) == 4 else shape[:-1] + (c // ratio,)
    code_gpu = code.float().cpu().numpy().reshape(cshape)     # physical layout, transposed below
    y_gpu = y.float().cpu().numpy().reshape(x_phys.shape)
    if len(shape) == 4:
        code_gpu = code_gpu.transpose(0, 3, 1, 2)
        y_gpu = y_gpu.transpose(0, 3, 1, 2)
    assert rel_err(code_gpu, code_ref) <= TOL[dt]
    # decode checked on the GPU's own code, so encode error does not count twice
    y_from_gpu_code = oracle.ae_decode(code_gpu, w["w_dec"], w["b_dec"], dt)
    assert rel_err(y_gpu, y_from_gpu_code) <= TOL[dt]
    assert rel_err(y_gpu, y_ref) <= 2 * TOL[dt]


def test_codec_errors_enqueue_nothing():
    cd = P.make_codec("ae", 64, 8)        # null weights
    with pytest.raises(P.MoparError):
        P.mopar_boundary_code_bytes(cd, (1, 64, 2, 2), "bf16")
    cd2 = P.make_codec("raw")
    with pytest.raises(P.MoparError):
        P.mopar_boundary_code_bytes(cd2, (1, 0, 2, 2), "bf16")


# ---------------------------------------------------------------------------
# whole models (shrunken workloads)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6, 7])
def test_small_model_sliced_ae_parity(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    sm = P.SlicedModel(m)
    plan = sm.plan()
    s = m.slicing
    po = oracle.plan_slices(oracle.layer_profiles(m), oracle.PlanOpts(
        n_slices=s["n_slices"], allowed_cut=s["allowed_cut"], elim_tau=s["elim_tau"], k_override=s["k_override"]))
    assert (plan.slice_end, plan.k) == (po.slice_end, po.k)
    cuts = plan.slice_end[:-1]
    tids, cw = boundary_codecs(m, cuts)
    assert tids == sm.boundary_tensors(plan)
    ref = oracle.forward(m, x, k=plan.k, cuts=cuts, codecs=cw)
    y, _, _ = run_gpu(m, x, plan, "ae", cw)
    assert rel_err(_np(y), ref) <= TOL[m.dtype]


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6, 7])
def test_small_model_raw_slicing_and_subslicing_bitwise(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    sm = P.SlicedModel(m)
    plan = sm.plan()
    n = len(m.layers)
    unsliced = P.make_plan(n, [n - 1], [1] * n)
    y0, _, _ = run_gpu(m, x, unsliced)
    ys, _, _ = run_gpu(m, x, plan, "raw", repeat=2)
    assert torch.equal(ys[0], y0), "sliced + sub-sliced (raw codec) differs from the unsliced model"
    assert torch.equal(ys[1], ys[0]), "not deterministic"
    assert rel_err(_np(y0), oracle.forward(m, x)) <= TOL[m.dtype]


def test_slice_forward_chain_equals_model_forward():
    m = synth.build(2, **SMALL[2])
    x = synth.make_input(m)
    sm = P.SlicedModel(m)
    plan = sm.plan()
    ws = sm.alloc_workspace(plan)
    cur = torch.from_numpy(x).cuda()
    for s in range(plan.n_slices):
        shp = m.tensors[m.layer_output_tid(plan.slice_end[s])]["shape"]
        out = torch.empty(shp, dtype=torch.bfloat16, device="cuda")
        sm.slice_forward(plan, s, cur, out, ws)
        cur = out
    torch.cuda.synchronize()
    y, _, _ = run_gpu(m, x, plan, "raw")
    assert torch.equal(cur, y)


# ---------------------------------------------------------------------------
# full-size workloads, checked on sampled batch rows (every op is independent
# across the batch, so the oracle computes just those rows)
# ---------------------------------------------------------------------------

FULL_SAMPLES = {1: [0], 2: [0, 7], 3: [5], 4: [31], 5: [63]}


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_full_size_sampled_parity(cfg):
    m = synth.build(cfg)
    x = synth.make_input(m)
    sm = P.SlicedModel(m)
    plan = sm.plan()
    cuts = plan.slice_end[:-1]
    cw = synth.make_codec_weights(m, cuts, ratio=codec_ratios(m, cuts))
    y, _, _ = run_gpu(m, x, plan, "ae", cw)
    yg = _np(y)
    assert np.isfinite(yg).all()
    rows = FULL_SAMPLES[cfg]
    ref = oracle.forward(m, x, k=plan.k, cuts=cuts, codecs=cw, sample=rows)
    assert rel_err(yg[rows], ref) <= TOL[m.dtype]
