"""Python binding of libmopar: the C entry points under the same names, plus a
``SlicedModel`` helper that turns a model description into the library's
descriptor and weight blob and owns the device buffers (torch is used only
for device memory and streams).

Marshalling done here (no arithmetic of the method):
* weights are re-laid out into the layouts documented in include/mopar.h
  (conv [Co][kh][kw][Cs] channels-last with zero channel padding; linear
  columns of a flattened image in (h, w, c) order; LSTM rows interleaved by
  hidden unit) and stored as their bf16 / float32 bit patterns;
* tensors cross the boundary as raw device pointers plus logical shapes.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib as L
from ._lib import check, lib

DTYPE = {"f32": L.MOPAR_F32, "bf16": L.MOPAR_BF16, "i32": L.MOPAR_I32}
TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_ptr(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------------------
# plain C entry points
# ---------------------------------------------------------------------------

def mopar_subslice_range(n, k, j):
    lo, hi = L.c_i32(), L.c_i32()
    check(lib().mopar_subslice_range(n, k, j, ctypes.byref(lo), ctypes.byref(hi)))
    return lo.value, hi.value


@dataclass
class PlanResult:
    n_slices: int
    slice_end: list
    k: list
    cost: float
    t_tau: float
    t_unsplit: float
    latency_ok: bool
    raw: L.Plan = None
    _keep: tuple = ()


def _profiles_array(profiles):
    arr = (L.LayerProfile * len(profiles))()
    for i, p in enumerate(profiles):
        if isinstance(p, L.LayerProfile):
            arr[i] = p
        else:
            arr[i].mem_bytes, arr[i].time_s, arr[i].out_bytes, arr[i].rd_width = (
                float(p[0]), float(p[1]), float(p[2]), int(p[3]))
    return arr


def mopar_plan_slices(profiles, n_slices=0, allowed_cut=None, elim_tau=0.05, c_m=1.0, c_n=1.0, bw=8.0e12,
                      ratio=None, k_max=1, lambda_bytes=0.0, tp_table=None, ta_table=None, k_override=None,
                      uniform=False):
    """HyPAD partitioning in the library.  ``profiles``: sequence of (mem, time, out_bytes, rd_width)."""
    n = len(profiles)
    prof = _profiles_array(profiles)
    o = L.PlanOpts()
    o.n_slices, o.k_max, o.elim_tau, o.c_m, o.c_n, o.bw_Bps = n_slices, k_max, elim_tau, c_m, c_n, bw
    o.lambda_bytes = lambda_bytes
    o.uniform = 1 if uniform else 0
    keep = []
    if allowed_cut is not None:
        a = (ctypes.c_uint8 * max(1, n - 1))(*[1 if v else 0 for v in allowed_cut])
        o.allowed_cut = ctypes.cast(a, ctypes.POINTER(ctypes.c_uint8))
        keep.append(a)
    if ratio is not None:
        a = (L.c_f64 * max(1, n - 1))(*[float(v) for v in ratio])
        o.ratio = ctypes.cast(a, ctypes.POINTER(L.c_f64))
        keep.append(a)
    for name, tab in (("tp_table", tp_table), ("ta_table", ta_table)):
        if tab is not None:
            flat = [float(v) for row in tab for v in row]
            a = (L.c_f64 * len(flat))(*flat)
            setattr(o, name, ctypes.cast(a, ctypes.POINTER(L.c_f64)))
            keep.append(a)
    if k_override is not None:
        a = (L.c_i32 * n)(*[int(v) for v in k_override])
        o.k_override = ctypes.cast(a, ctypes.POINTER(L.c_i32))
        keep.append(a)
    ends = (L.c_i32 * n)()
    ks = (L.c_i32 * n)()
    p = L.Plan()
    p.n_layers, p.slice_end, p.k = n, ctypes.cast(ends, ctypes.POINTER(L.c_i32)), ctypes.cast(ks, ctypes.POINTER(L.c_i32))
    check(lib().mopar_plan_slices(prof, n, ctypes.byref(o), ctypes.byref(p)))
    return PlanResult(p.n_slices, list(ends[:p.n_slices]), list(ks[:n]), p.cost, p.t_tau, p.t_unsplit,
                      bool(p.latency_ok), p, (ends, ks))


def make_plan(n_layers, slice_end, k):
    """A plan built by hand (e.g. a prescribed cut set), in the library's struct."""
    ends = (L.c_i32 * n_layers)(*slice_end)
    ks = (L.c_i32 * n_layers)(*k)
    p = L.Plan()
    p.n_layers, p.n_slices = n_layers, len(slice_end)
    p.slice_end, p.k = ctypes.cast(ends, ctypes.POINTER(L.c_i32)), ctypes.cast(ks, ctypes.POINTER(L.c_i32))
    return PlanResult(len(slice_end), list(slice_end), list(k), 0.0, 0.0, 0.0, True, p, (ends, ks))


def tensor_desc(shape, dtype):
    d = L.TensorDesc()
    d.dtype = DTYPE[dtype] if isinstance(dtype, str) else dtype
    d.rank = len(shape)
    for i, s in enumerate(shape):
        d.dims[i] = int(s)
    return d


def make_codec(kind, c=0, c_code=0, w_enc=None, b_enc=None, w_dec=None, b_dec=None):
    cd = L.Codec()
    cd.kind = {"raw": L.CODEC_RAW, "ae": L.CODEC_AE}[kind] if isinstance(kind, str) else kind
    cd.c, cd.c_code = c, c_code
    cd.w_enc, cd.b_enc, cd.w_dec, cd.b_dec = _ptr(w_enc), _ptr(b_enc), _ptr(w_dec), _ptr(b_dec)
    return cd


def mopar_boundary_code_bytes(codec, shape, dtype):
    n = ctypes.c_size_t()
    check(lib().mopar_boundary_code_bytes(ctypes.byref(codec), ctypes.byref(tensor_desc(shape, dtype)),
                                          ctypes.byref(n)))
    return n.value


def mopar_boundary_encode(codec, shape, dtype, x, code, stream=None):
    check(lib().mopar_boundary_encode(ctypes.byref(codec), ctypes.byref(tensor_desc(shape, dtype)), _ptr(x),
                                      _ptr(code), _stream_ptr(stream)))


def mopar_boundary_decode(codec, shape, dtype, code, y, stream=None):
    check(lib().mopar_boundary_decode(ctypes.byref(codec), ctypes.byref(tensor_desc(shape, dtype)), _ptr(code),
                                      _ptr(y), _stream_ptr(stream)))


# ---------------------------------------------------------------------------
# weight packing (layouts of include/mopar.h)
# ---------------------------------------------------------------------------

def _as_bytes(a, dtype):
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        return (a.view(np.uint32) >> 16).astype(np.uint16).tobytes()
    return a.tobytes()


class _Blob:
    def __init__(self, dtype):
        self.dtype, self.parts, self.size = dtype, [], 0

    def add(self, arr):
        off = self.size
        b = _as_bytes(arr, self.dtype)
        self.parts.append((off, b))
        self.size = (off + len(b) + 255) // 256 * 256
        return off

    def to_device(self, device):
        host = np.zeros(max(self.size, 16), dtype=np.uint8)
        for off, b in self.parts:
            host[off:off + len(b)] = np.frombuffer(b, dtype=np.uint8)
        return torch.from_numpy(host).to(device)


def _interleave_gates(a, hidden):
    """[4H, ...] with gate blocks i,f,g,o -> row 4u+g holds gate g of unit u."""
    return np.ascontiguousarray(a.reshape((4, hidden) + a.shape[1:]).swapaxes(0, 1).reshape(a.shape))


def _pack(model):
    """Descriptor arrays and weight blob for a ``synth.Model``."""
    dt = model.dtype
    epc = 8 if dt == "bf16" else 4
    blob = _Blob(dt)
    W = model.weights
    tens = (L.TensorDesc * len(model.tensors))()
    for i, t in enumerate(model.tensors):
        tens[i] = tensor_desc(t["shape"], t["dtype"])
    ops = (L.Op * len(model.ops))()
    for i, op in enumerate(model.ops):
        o = ops[i]
        o.layer, o.branch, o.pos, o.rd = op["layer"], op["branch"], op["pos"], 1 if op.get("rd") else 0
        o.in0 = op["inputs"][0]
        o.in1 = op["inputs"][1] if len(op["inputs"]) > 1 else -1
        o.out = op["out"]
        o.w = o.b = o.w2 = o.w3 = o.w4 = o.w5 = -1
        k = op["kind"]
        in_shape = model.tensors[o.in0]["shape"]
        if k == "conv":
            o.kind, o.act = L.OP_CONV, L.ACT[op["act"]]
            o.kh, o.kw, o.stride, o.pad, o.n_out = op["kh"], op["kw"], op["stride"], op["pad"], op["cout"]
            o.out_off = op.get("out_off", 0)
            w = W[op["w"]]
            c = w.shape[1]
            cs = c if c % epc == 0 else (c + epc - 1) // epc * epc
            wp = np.zeros((w.shape[0], w.shape[2], w.shape[3], cs), dtype=np.float32)
            wp[..., :c] = w.transpose(0, 2, 3, 1)
            o.w, o.b = blob.add(wp), blob.add(W[op["b"]])
        elif k == "linear":
            o.kind, o.act, o.n_out = L.OP_LINEAR, L.ACT[op["act"]], op["nout"]
            w = W[op["w"]]
            if len(in_shape) == 4:
                _, c, h, wd = in_shape
                w = w.reshape(w.shape[0], c, h, wd).transpose(0, 2, 3, 1).reshape(w.shape[0], -1)
            o.w, o.b = blob.add(w), blob.add(W[op["b"]])
        elif k == "maxpool":
            o.kind, o.kh, o.kw, o.stride, o.pad = L.OP_MAXPOOL, op["k"], op["k"], op["stride"], op["pad"]
        elif k == "avgpool":
            o.kind = L.OP_AVGPOOL
        elif k == "layernorm":
            o.kind, o.eps = L.OP_LAYERNORM, op["eps"]
            o.w, o.b = blob.add(W[op["g"]]), blob.add(W[op["beta"]])
        elif k == "attention":
            o.kind, o.heads, o.scale = L.OP_ATTENTION, op["heads"], op["scale"]
        elif k == "embed_bert":
            o.kind, o.eps = L.OP_EMBED_BERT, op["eps"]
            tok, pos, typ = W[op["w_tok"]], W[op["w_pos"]], W[op["w_type"]]
            o.rows[0], o.rows[1], o.rows[2] = tok.shape[0], pos.shape[0], typ.shape[0]
            o.w, o.w2, o.w3 = blob.add(tok), blob.add(pos), blob.add(typ)
            o.w4, o.w5 = blob.add(W[op["g"]]), blob.add(W[op["beta"]])
        elif k == "embed":
            o.kind = L.OP_EMBED
            tab = W[op["table"]]
            o.rows[0] = tab.shape[0]
            o.w = blob.add(tab)
        elif k == "lstm":
            h = op["hidden"]
            o.kind, o.n_out = L.OP_LSTM, h
            o.w = blob.add(_interleave_gates(W[op["w_ih"]], h))
            o.w2 = blob.add(_interleave_gates(W[op["w_hh"]], h))
            o.b = blob.add(_interleave_gates(W[op["b_ih"]], h))
            o.w3 = blob.add(_interleave_gates(W[op["b_hh"]], h))
        else:
            raise ValueError(k)
    return tens, ops, blob


def boundary_to_canonical(x, shape):
    """View a physical boundary tensor (NHWC for images) in canonical (NCHW) order."""
    if len(shape) == 4:
        n, c, h, w = shape
        return x.reshape(n, h, w, c).permute(0, 3, 1, 2)
    return x.reshape(shape)


class SlicedModel:
    """A model loaded into the library: weights on the device, descriptor, profile, plan, buffers."""

    def __init__(self, model, device="cuda"):
        self.spec = model
        self.device = device
        self.dtype = model.dtype
        self._tens, self._ops, blob = _pack(model)
        self.weights = blob.to_device(device)
        d = L.ModelDesc()
        d.dtype = DTYPE[model.dtype]
        d.n_tensors, d.tensors = len(model.tensors), ctypes.cast(self._tens, ctypes.POINTER(L.TensorDesc))
        d.n_ops, d.ops = len(model.ops), ctypes.cast(self._ops, ctypes.POINTER(L.Op))
        d.n_layers, d.input, d.output = len(model.layers), model.input_tid, model.output_tid
        self._desc = d
        h = ctypes.c_void_p()
        check(lib().mopar_model_create(ctypes.byref(d), _ptr(self.weights), self.weights.numel(), ctypes.byref(h)))
        self.handle = h
        self.n_layers = len(model.layers)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value and L._lib is not None:
            L._lib.mopar_model_destroy(h)
            self.handle = None

    # -- planning -----------------------------------------------------------
    def profile(self, dominant=None):
        """Layer profiles (Eq. 1-4); ``dominant`` = f builds them from each node's dominant
        operators (mopar_model_profile_dominant), None from every op."""
        arr = (L.LayerProfile * self.n_layers)()
        if dominant is None:
            check(lib().mopar_model_profile(self.handle, arr))
        else:
            check(lib().mopar_model_profile_dominant(self.handle, float(dominant), arr))
        return [(p.mem_bytes, p.time_s, p.out_bytes, p.rd_width) for p in arr]

    def plan(self, **opts):
        """Plan with the model's slicing options (overridable by keyword)."""
        s = dict(self.spec.slicing)
        kw = dict(n_slices=s["n_slices"], allowed_cut=s["allowed_cut"], elim_tau=s["elim_tau"],
                  k_override=s["k_override"])
        kw.update(opts)
        return mopar_plan_slices(self.profile(), **kw)

    def cut_tensors(self, node):
        """mopar_model_cut_tensors: tensor ids a cut after ``node`` carries."""
        cnt = L.c_i32()
        check(lib().mopar_model_cut_tensors(self.handle, node, None, 0, ctypes.byref(cnt)))
        arr = (L.c_i32 * max(cnt.value, 1))()
        check(lib().mopar_model_cut_tensors(self.handle, node, arr, cnt.value, ctypes.byref(cnt)))
        return list(arr[:cnt.value])

    def boundary_tensors(self, plan):
        """Tensor ids handed over at the plan's cuts: cut-major, ascending id within a cut."""
        return [t for e in plan.slice_end[:-1] for t in self.cut_tensors(e)]

    def cut_tensor_shapes(self, plan):
        return [self.spec.tensors[t]["shape"] for t in self.boundary_tensors(plan)]

    # -- buffers ------------------------------------------------------------
    def workspace_bytes(self, plan):
        n = ctypes.c_size_t()
        check(lib().mopar_model_workspace_bytes(self.handle, ctypes.byref(plan.raw), ctypes.byref(n)))
        return n.value

    def alloc_workspace(self, plan):
        return torch.empty(max(self.workspace_bytes(plan), 16), dtype=torch.uint8, device=self.device)

    def alloc_output(self):
        t = self.spec.tensors[self.spec.output_tid]
        return torch.empty(t["shape"], dtype=TORCH_DTYPE[t["dtype"]], device=self.device)

    def codecs(self, plan, kind="ae", weights=None):
        """Codec structs (and their device weights) for the plan's cuts; ``weights`` from
        ``synth.make_codec_weights``.  Returns (ctypes array, device tensors kept alive)."""
        n = len(self.boundary_tensors(plan))
        arr = (L.Codec * max(n, 1))()
        keep = []
        for s in range(n):
            if kind == "raw":
                arr[s] = make_codec("raw")
                continue
            w = weights[s]
            dev = [torch.from_numpy(np.ascontiguousarray(w[key])).to(self.device, TORCH_DTYPE[self.dtype])
                   for key in ("w_enc", "b_enc", "w_dec", "b_dec")]
            keep += dev
            arr[s] = make_codec("ae", w["c"], w["c_code"], *dev)
        return arr, keep

    def alloc_codes(self, plan, codecs):
        bufs = []
        for s, shape in enumerate(self.cut_tensor_shapes(plan)):
            n = mopar_boundary_code_bytes(codecs[s], shape, self.dtype)
            bufs.append(torch.empty(max(n, 16), dtype=torch.uint8, device=self.device))
        return bufs

    # -- execution ------------------------------------------------------------
    def forward(self, plan, x, out, codecs=None, code_bufs=None, ws=None, stream=None):
        bufs = list(code_bufs or [])
        cb = (ctypes.c_void_p * max(len(bufs), 1))(*[b.data_ptr() for b in bufs])
        cod = codecs if codecs is not None else (L.Codec * 1)()
        check(lib().mopar_model_forward(self.handle, ctypes.byref(plan.raw), cod, _ptr(x), _ptr(out), cb,
                                        _ptr(ws), 0 if ws is None else ws.numel(), _stream_ptr(stream)))
        return out

    def forward_static(self, plan, x, out, codecs=None, code_bufs=None, stream=None):
        """mopar_model_forward_static: the same forward with the library's static workspace (for
        callers that cannot allocate; see include/mopar.h)."""
        bufs = list(code_bufs or [])
        cb = (ctypes.c_void_p * max(len(bufs), 1))(*[b.data_ptr() for b in bufs])
        cod = codecs if codecs is not None else (L.Codec * 1)()
        check(lib().mopar_model_forward_static(self.handle, ctypes.byref(plan.raw), cod, _ptr(x), _ptr(out), cb,
                                               _stream_ptr(stream)))
        return out

    # -- cross-request slice pipeline ---------------------------------------------
    def pipeline(self, plan, codec="ae", codec_weights=None, depth=2, replicas=1, stream_per_slice=True):
        """A ``SlicePipeline``: ``replicas`` instances of the sliced model; each instance runs
        its slices on one stream per slice, or on a single stream when ``stream_per_slice`` is False."""
        return SlicePipeline(self, plan, codec, codec_weights, depth, replicas, stream_per_slice)

    # -- measurement -----------------------------------------------------------
    def set_timing(self, enable=True):
        check(lib().mopar_model_set_timing(self.handle, 1 if enable else 0))

    def op_times(self):
        """Per-slot milliseconds of the last timed forward: (op times, [(encode, decode) per cut])."""
        n = L.c_i32()
        check(lib().mopar_model_timing_slots(self.handle, ctypes.byref(n)))
        arr = (L.c_f32 * n.value)()
        check(lib().mopar_model_op_times(self.handle, arr, n.value))
        nops = len(self.spec.ops)
        ops = list(arr[:nops])
        cuts = [(arr[nops + 2 * c], arr[nops + 2 * c + 1]) for c in range((n.value - nops) // 2)]
        return ops, [c for c in cuts if c[0] >= 0 or c[1] >= 0]

    def measure(self, x, k_max=4, reps=3, ws=None, out=None, stream=None):
        """mopar_model_measure: t_p(l, eta) in seconds, a list of n_layers rows of k_max values."""
        n = self.n_layers
        if ws is None:
            ws = self.alloc_workspace(make_plan(n, [n - 1], [1] * n))
        if out is None:
            out = self.alloc_output()
        tab = (L.c_f64 * (n * k_max))()
        check(lib().mopar_model_measure(self.handle, k_max, reps, _ptr(x), _ptr(out), _ptr(ws), ws.numel(),
                                        _stream_ptr(stream), tab))
        return [list(tab[l * k_max:(l + 1) * k_max]) for l in range(n)]

    def measured_plan(self, x, k_max=4, reps=3, stream=None, **opts):
        """Plan from the measured profile: each node's time t_l := t_p(l, 1) measured, the
        parallelism search over t_p(l, eta) (t_a = 0).  Returns (plan, t_p table)."""
        tp = self.measure(x, k_max=k_max, reps=reps, stream=stream)
        prof = [(mem, tp[l][0], ob, rdw) for l, (mem, _, ob, rdw) in enumerate(self.profile())]
        kw = dict(elim_tau=0.05)
        kw.update(opts)
        plan = mopar_plan_slices(prof, k_max=k_max, tp_table=tp, ta_table=[[0.0] * k_max for _ in tp], **kw)
        return plan, tp, prof

    def slice_forward(self, plan, s, x, out, ws, stream=None):
        check(lib().mopar_slice_forward(self.handle, ctypes.byref(plan.raw), s, _ptr(x), _ptr(out), _ptr(ws),
                                        ws.numel(), _stream_ptr(stream)))
        return out


class SlicePipeline:
    """Owns the streams, workspace, code-buffer ring and library handle of a slice pipeline."""

    def __init__(self, sm, plan, codec, codec_weights, depth, replicas=1, stream_per_slice=True):
        self.sm, self.plan = sm, plan
        self.replicas = replicas
        self._submitted = 0
        S = plan.n_slices
        self.streams = []
        for _ in range(replicas):
            if stream_per_slice:
                self.streams += [torch.cuda.Stream(device=sm.device) for _ in range(S)]
            else:
                st = torch.cuda.Stream(device=sm.device)
                self.streams += [st] * S
        self.codecs, self._keep = sm.codecs(plan, codec, codec_weights)
        n = ctypes.c_size_t()
        check(lib().mopar_pipeline_workspace_bytes(sm.handle, ctypes.byref(plan.raw), replicas, ctypes.byref(n)))
        self.ws = torch.empty(max(n.value, 16), dtype=torch.uint8, device=sm.device)
        self.codes = []
        for _ in range(replicas * depth):
            self.codes += sm.alloc_codes(plan, self.codecs)
        sp = (ctypes.c_void_p * len(self.streams))(*[s.cuda_stream for s in self.streams])
        cb = (ctypes.c_void_p * max(len(self.codes), 1))(*[b.data_ptr() for b in self.codes])
        h = ctypes.c_void_p()
        # the library keeps no pointer to these host arrays after create
        check(lib().mopar_pipeline_create(sm.handle, ctypes.byref(plan.raw), self.codecs, replicas, depth, sp,
                                          _ptr(self.ws), self.ws.numel(), cb, ctypes.byref(h)))
        self.handle = h

    def submit(self, x, out):
        """Enqueue one batch.  Batch i runs on instance i mod replicas (the library's rule):
        that instance's first stream waits for the work torch's current stream has queued so
        far (which produced ``x``), and both tensors are marked in use by the instance's streams
        so the caching allocator does not hand their memory out before the batch has run."""
        rep = self._submitted % self.replicas
        S = self.plan.n_slices
        first, last = self.streams[rep * S], self.streams[rep * S + S - 1]
        first.wait_stream(torch.cuda.current_stream(first.device))
        check(lib().mopar_pipeline_submit(self.handle, _ptr(x), _ptr(out)))
        self._submitted += 1
        x.record_stream(first)
        out.record_stream(last)
        return out

    def use_graphs(self, enable=True):
        """Replay captured HIP graphs for later submits (needs one stream per instance)."""
        if not enable:
            self.synchronize()
        check(lib().mopar_pipeline_use_graphs(self.handle, 1 if enable else 0))
        return self

    def synchronize(self):
        for s in self.streams:
            s.synchronize()

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value and L._lib is not None:
            try:
                self.synchronize()
            finally:
                L._lib.mopar_pipeline_destroy(h)
                self.handle = None
