"""CPU oracle for MOPAR's sliced inference (arXiv 2404.02445) -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never calls it, and it
shares no code with the GPU library: the layer math lives in ``oracle.c``
(plain loops, double accumulation), the profile and the planner in
``plan.py`` (plain Python).  Inputs come from ``synth``, which holds no
arithmetic of the method.

What is computed here, and where the paper defines it:

* layer math of the evaluated services (VGG, ResNet, BERT, LSTM; Sec. II-A,
  Sec. IV): textbook definitions, see ``oracle.c``;
* horizontal sub-slicing of a resource-dominant operator into k equal-size
  sub-slices along its output channels / features, each holding a share of
  the parameters, aggregated by concatenation (Sec. III-C, the hybrid
  strategy pi_P and the aggregation time t_a of Eq. 5);
* vertical slicing at split points (Sec. III-C, pi_S), with the slice
  boundary passed through the codec of Sec. III-D (autoencoder: one encoder
  layer at the end of slice s, one decoder layer at the start of slice s+1;
  or a raw byte copy when no compression is used).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .plan import (subslice_range, layer_profiles, plan_slices, brute_force_plan, crossing_tensors,  # noqa: F401
                   PlanOpts, Plan)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

RND = {"none": 0, "f32": 1, "bf16": 2}
ACT = {"none": 0, "relu": 1, "gelu": 2}


def build_lib(force: bool = False) -> str:
    """Compile ``oracle.c`` with gcc (IEEE semantics: no contraction, no fast-math)."""
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                               "-shared", "-fPIC", src, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build_lib()
        _lib = ctypes.CDLL(_LIB_PATH)
        D, I64, I, P = ctypes.c_double, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
        _lib.or_round1.restype = D
        _lib.or_round1.argtypes = [D, I]
        _lib.or_round.argtypes = [P, I64, I]
        _lib.or_conv2d.argtypes = [P, I64, I64, I64, I64, P, P, I64, I64, I64, I64, I64, P, I, I, P]
        _lib.or_maxpool2d.argtypes = [P, I64, I64, I64, I64, I64, I64, I64, P]
        _lib.or_avgpool_global.argtypes = [P, I64, I64, I64, I64, I, P]
        _lib.or_linear.argtypes = [P, I64, I64, P, P, I64, P, I, I, P]
        _lib.or_layernorm.argtypes = [P, P, I64, I64, P, P, D, I, P]
        _lib.or_attention.argtypes = [P, I64, I64, I64, I64, D, I, P]
        _lib.or_embed_bert.argtypes = [P, I64, I64, P, P, P, I64, P, P, D, I, P]
        _lib.or_embed.argtypes = [P, I64, P, I64, P]
        _lib.or_lstm.argtypes = [P, I64, I64, I64, I64, P, P, P, P, I, P]
        _lib.or_ae_apply.argtypes = [P, I64, I64, I64, P, P, I64, I, P]
    return _lib


def _d(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------------------
# Layer routines (canonical layouts; see oracle.c for the definitions)
# ---------------------------------------------------------------------------

def round_to(x, dtype):
    """Round every element to the storage type ('none' | 'f32' | 'bf16'), RNE."""
    x = _d(x).copy()
    lib().or_round(_p(x), x.size, RND[dtype])
    return x


def conv2d(x, w, b, stride, pad, act="none", res=None, rnd="none"):
    x, w = _d(x), _d(w)
    b = None if b is None else _d(b)
    n, c, h, wd = x.shape
    co, ci, kh, kw = w.shape
    assert ci == c
    ho, wo = (h + 2 * pad - kh) // stride + 1, (wd + 2 * pad - kw) // stride + 1
    y = np.empty((n, co, ho, wo))
    r = None if res is None else _d(res)
    lib().or_conv2d(_p(x), n, c, h, wd, _p(w), _p(b), co, kh, kw, stride, pad, _p(r), ACT[act], RND[rnd], _p(y))
    return y


def maxpool2d(x, k, stride, pad):
    x = _d(x)
    n, c, h, w = x.shape
    ho, wo = (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1
    y = np.empty((n, c, ho, wo))
    lib().or_maxpool2d(_p(x), n, c, h, w, k, stride, pad, _p(y))
    return y


def avgpool_global(x, rnd="none"):
    x = _d(x)
    n, c, h, w = x.shape
    y = np.empty((n, c))
    lib().or_avgpool_global(_p(x), n, c, h, w, RND[rnd], _p(y))
    return y


def linear(x, w, b, act="none", res=None, rnd="none"):
    """y = act(x W^T + b + res) over the last axis of x (an image batch is flattened NCHW)."""
    x, w = _d(x), _d(w)
    if x.ndim == 4:
        x = x.reshape(x.shape[0], -1)
    lead, k = x.shape[:-1], x.shape[-1]
    nout = w.shape[0]
    assert w.shape[1] == k
    m = int(np.prod(lead))
    y = np.empty(tuple(lead) + (nout,))
    r = None if res is None else _d(res)
    lib().or_linear(_p(x), m, k, _p(w), _p(None if b is None else _d(b)), nout, _p(r), ACT[act], RND[rnd], _p(y))
    return y


def layernorm(x, g, beta, eps, res=None, rnd="none"):
    x = _d(x)
    f = x.shape[-1]
    y = np.empty_like(x)
    r = None if res is None else _d(res)
    lib().or_layernorm(_p(x), _p(r), x.size // f, f, _p(_d(g)), _p(_d(beta)), eps, RND[rnd], _p(y))
    return y


def attention(qkv, heads, scale, rnd="none"):
    qkv = _d(qkv)
    b, s, f3 = qkv.shape
    f = f3 // 3
    y = np.empty((b, s, f))
    lib().or_attention(_p(qkv), b, s, heads, f // heads, scale, RND[rnd], _p(y))
    return y


def embed_bert(ids, tok, pos, typ, g, beta, eps, rnd="none"):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    b, s = ids.shape
    f = tok.shape[1]
    y = np.empty((b, s, f))
    lib().or_embed_bert(_p(ids), b, s, _p(_d(tok)), _p(_d(pos)), _p(_d(typ)), f, _p(_d(g)), _p(_d(beta)),
                        eps, RND[rnd], _p(y))
    return y


def embed(ids, table):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    table = _d(table)
    f = table.shape[1]
    y = np.empty(ids.shape + (f,))
    lib().or_embed(_p(ids), ids.size, _p(table), f, _p(y))
    return y


def lstm(x, w_ih, w_hh, b_ih, b_hh, rnd="none"):
    x = _d(x)
    b, t, e = x.shape
    hd = w_hh.shape[1]
    y = np.empty((b, t, hd))
    lib().or_lstm(_p(x), b, t, e, hd, _p(_d(w_ih)), _p(_d(w_hh)), _p(_d(b_ih)), _p(_d(b_hh)), RND[rnd], _p(y))
    return y


def _as_ncl(x):
    """View a boundary tensor as [N][C][L]: images NCHW -> L = H*W; sequences [.., F] -> L = 1."""
    if x.ndim == 4:
        n, c, h, w = x.shape
        return x.reshape(n, c, h * w)
    return x.reshape(-1, x.shape[-1], 1)


def ae_encode(x, w_enc, b_enc, rnd="none"):
    """Encoder of the boundary autoencoder (Sec. III-D): a 1x1 linear layer over channels."""
    return _ae(x, w_enc, b_enc, rnd)


def ae_decode(code, w_dec, b_dec, rnd="none"):
    """Decoder of the boundary autoencoder (Sec. III-D): a 1x1 linear layer back to C channels."""
    return _ae(code, w_dec, b_dec, rnd)


def _ae(x, w, b, rnd):
    x = _d(x)
    v = np.ascontiguousarray(_as_ncl(x))
    n, cin, l = v.shape
    cout = w.shape[0]
    assert w.shape[1] == cin
    y = np.empty((n, cout, l))
    lib().or_ae_apply(_p(v), n, cin, l, _p(_d(w)), _p(_d(b)), cout, RND[rnd], _p(y))
    if x.ndim == 4:
        return y.reshape(x.shape[0], cout, x.shape[2], x.shape[3])
    return y.reshape(x.shape[:-1] + (cout,))


# ---------------------------------------------------------------------------
# Operators, sub-slicing and the sliced model forward
# ---------------------------------------------------------------------------

def run_op(model, op, env, w_rows=None, rnd=None):
    """Evaluate one op of ``model`` (a ``synth.Model``) on tensors in ``env``.

    ``w_rows = (lo, hi)`` restricts the op to output channels / features
    lo..hi-1 using only those rows of its weight and bias: one horizontal
    sub-slice holding its share of the parameters (Sec. III-C, pi_P).
    ``rnd``: storage rounding of the op's output ('none' keeps every value in
    double); None rounds to the model dtype, as the library stores it.
    """
    W = model.weights
    rnd = model.dtype if rnd is None else rnd
    k = op["kind"]
    ins = [env[t] for t in op["inputs"]]
    lo, hi = w_rows if w_rows is not None else (None, None)

    def rows(name):
        a = W[name]
        return a if w_rows is None else a[lo:hi]

    def res_rows(r):
        if r is None or w_rows is None:
            return r
        return r[:, lo:hi] if r.ndim == 4 else r[..., lo:hi]

    res = ins[1] if len(ins) > 1 else None
    if k == "conv":
        return conv2d(ins[0], rows(op["w"]), rows(op["b"]), op["stride"], op["pad"], op["act"],
                      res_rows(res), rnd)
    if k == "linear":
        return linear(ins[0], rows(op["w"]), rows(op["b"]), op["act"], res_rows(res), rnd)
    assert w_rows is None, "only conv / linear ops are sub-sliced"
    if k == "maxpool":
        return maxpool2d(ins[0], op["k"], op["stride"], op["pad"])
    if k == "avgpool":
        return avgpool_global(ins[0], rnd)
    if k == "layernorm":
        return layernorm(ins[0], W[op["g"]], W[op["beta"]], op["eps"], res, rnd)
    if k == "attention":
        return attention(ins[0], op["heads"], op["scale"], rnd)
    if k == "embed_bert":
        return embed_bert(ins[0], W[op["w_tok"]], W[op["w_pos"]], W[op["w_type"]], W[op["g"]], W[op["beta"]],
                          op["eps"], rnd)
    if k == "embed":
        return embed(ins[0], W[op["table"]])
    if k == "lstm":
        return lstm(ins[0], W[op["w_ih"]], W[op["w_hh"]], W[op["b_ih"]], W[op["b_hh"]], rnd)
    raise ValueError(k)


def out_width(model, op):
    """Size of the dimension a sub-slice splits: output channels (conv) or features (linear)."""
    return op["cout"] if op["kind"] == "conv" else op["nout"]


def run_op_sliced(model, op, env, k, rnd=None):
    """The k-way sub-sliced operator: sub-slice j computes its own output range with its own
    rows of the parameters; the k partial outputs are concatenated (the aggregation of Eq. 5)."""
    n = out_width(model, op)
    parts = [run_op(model, op, env, subslice_range(n, k, j), rnd) for j in range(k)]
    axis = 1 if parts[0].ndim == 4 else -1
    return np.concatenate(parts, axis=axis)


def forward(model, x, k=None, cuts=(), codecs=None, sample=None, keep=False, rnd=None):
    """Sliced forward pass of ``model`` on input ``x`` (canonical layout).

    k       -- per planning node, the sub-slice count of its RD ops (None: all 1)
    cuts    -- planning-node indices after which the model is cut into slices
    codecs  -- per cut: None (raw byte hand-off) or a dict of autoencoder weights
    sample  -- optional batch indices; every op is independent across the batch,
               so the result is exactly those rows of the full-batch result
    keep    -- also return every tensor, every code and every boundary tensor before encoding
    rnd     -- storage rounding of every stored tensor: None (the model dtype, as the library
               stores them) or 'none' (exact double arithmetic throughout, for pinning the
               op dispatch against library routines without rounding noise)

    The boundary tensor of a cut is encoded at the end of the slice and
    decoded at the start of the next (Sec. III-D); raw hand-off returns the
    same values.
    """
    if sample is not None:
        x = x[np.asarray(sample)]
    rnd = model.dtype if rnd is None else rnd
    t_in = model.tensors[model.input_tid]
    if t_in["dtype"] == "i32":
        env = {model.input_tid: np.ascontiguousarray(x, dtype=np.int32)}
    else:
        env = {model.input_tid: round_to(x, rnd)}
    cuts = list(cuts)
    if codecs is None:
        codecs = [None] * sum(len(crossing_tensors(model, c)) for c in cuts)
    codes, bounds = {}, {}
    for li in range(len(model.layers)):
        for op in [o for o in model.ops if o["layer"] == li]:
            kk = 1 if k is None else int(k[li])
            if op.get("rd") and kk > 1:
                res = run_op_sliced(model, op, env, kk, rnd)
            else:
                res = run_op(model, op, env, None, rnd)
            if "out_off" in op:
                # a branch of a parallel node: its channels of the concatenated node output
                full = env.get(op["out"])
                if full is None:
                    full = np.zeros((res.shape[0],) + tuple(model.tensors[op["out"]]["shape"][1:]), dtype=res.dtype)
                    env[op["out"]] = full
                full[:, op["out_off"]:op["out_off"] + res.shape[1]] = res
            else:
                env[op["out"]] = res
        if li in cuts:
            # every tensor crossing the cut goes through its own codec (cut-major, ascending id)
            ci = cuts.index(li)
            base = sum(len(crossing_tensors(model, c)) for c in cuts[:ci])
            for q, tid in enumerate(crossing_tensors(model, li)):
                cd = codecs[base + q]
                bounds[(li, tid)] = env[tid]
                if cd is None:
                    code = env[tid].copy()
                    env[tid] = code.copy()
                else:
                    code = ae_encode(env[tid], cd["w_enc"], cd["b_enc"], rnd)
                    env[tid] = ae_decode(code, cd["w_dec"], cd["b_dec"], rnd)
                codes[(li, tid)] = code
                if tid == model.layer_output_tid(li):
                    bounds[li], codes[li] = bounds[(li, tid)], code
    y = env[model.output_tid]
    if keep:
        return y, env, codes, bounds
    return y
