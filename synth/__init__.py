"""Seeded synthetic workloads: model structures, weights, inputs and codec weights.

This module only draws numbers and records shapes. It holds none of the
method's arithmetic (no layer math, no profiles, no planning, no codec): the
CPU oracle and the GPU library each implement those on their own, and both
consume exactly the arrays produced here.

Conventions
-----------
* Every tensor is described in the canonical (PyTorch) layout: images NCHW,
  sequences [B, S, F], token ids int32 [B, S].
* Weights are canonical too: conv [C_out][C_in][kh][kw], linear [out][in],
  LSTM W_ih [4H][E] / W_hh [4H][H] with gate blocks in i, f, g, o order.
* RNG is ``numpy.random.Generator(PCG64(seed))``; values are drawn in
  float64 in forward order (weight, then bias), cast to float32 and, for
  bf16 models, rounded to the nearest bf16 (ties to even).  Arrays are
  returned as float32 holding those values.
* Seeds: weights 1000 + cfg, inputs 2000 + cfg, codec weights 3000 + cfg.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F32, BF16, I32 = "f32", "bf16", "i32"


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); return float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).copy()
    nan = np.isnan(a)
    out[nan] = a[nan]
    return out


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """The upper 16 bits of float32 values that are already bf16 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


@dataclass
class Model:
    name: str
    dtype: str                      # storage / compute type of activations and weights
    batch: int
    tensors: list = field(default_factory=list)   # dict(shape=tuple, dtype=str)
    ops: list = field(default_factory=list)       # dict, see _Builder
    layers: list = field(default_factory=list)    # planning-node names, in order
    weights: dict = field(default_factory=dict)   # name -> float32 array (canonical layout)
    input_tid: int = 0
    output_tid: int = -1
    slicing: dict = field(default_factory=dict)   # n_slices, allowed_cut, elim_tau, k_override
    cfg: int = 0
    codec_ratio: int = 8

    def layer_output_tid(self, layer: int) -> int:
        """Tensor leaving planning node ``layer`` (output of its last op)."""
        return [op for op in self.ops if op["layer"] == layer][-1]["out"]


class _Builder:
    def __init__(self, name, dtype, batch, seed, cfg=0):
        self.m = Model(name=name, dtype=dtype, batch=batch, cfg=cfg)
        self.rng = np.random.Generator(np.random.PCG64(seed))
        self.layer = -1

    # -- bookkeeping -------------------------------------------------------
    def tensor(self, shape, dtype=None):
        self.m.tensors.append(dict(shape=tuple(int(s) for s in shape), dtype=dtype or self.m.dtype))
        return len(self.m.tensors) - 1

    def shape(self, tid):
        return self.m.tensors[tid]["shape"]

    def new_layer(self, name):
        self.m.layers.append(name)
        self.layer = len(self.m.layers) - 1

    def store(self, name, arr64):
        a = np.asarray(arr64, dtype=np.float64).astype(np.float32)
        if self.m.dtype == BF16:
            a = to_bf16_values(a)
        self.m.weights[name] = np.ascontiguousarray(a)
        return name

    def op(self, **kw):
        kw.setdefault("branch", 0)
        kw.setdefault("pos", len([o for o in self.m.ops if o["layer"] == self.layer]) + 1)
        kw.setdefault("rd", False)
        kw["layer"] = self.layer
        self.m.ops.append(kw)
        return kw["out"]

    # -- initialisers ------------------------------------------------------
    def he(self, shape, fan_in):
        return self.rng.standard_normal(shape) * math.sqrt(2.0 / fan_in)

    def normal(self, shape, std):
        return self.rng.standard_normal(shape) * std

    def uniform(self, shape, lo, hi):
        return self.rng.uniform(lo, hi, size=shape)

    # -- op constructors ---------------------------------------------------
    def conv(self, x, cout, k, stride, pad, act, name, res=None, bn_fold=False, **kw):
        n, c, h, w = self.shape(x)
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        wt = self.he((cout, c, k, k), c * k * k)
        if bn_fold:
            gamma = self.uniform((cout,), 0.8, 1.2)
            beta = self.normal((cout,), 0.1)
            mean = self.normal((cout,), 0.1)
            var = self.uniform((cout,), 0.5, 1.5)
            scale = gamma / np.sqrt(var + 1e-5)
            wt = wt * scale[:, None, None, None]
            bias = beta - mean * scale
        else:
            bias = np.zeros(cout)
        self.store(name + ".w", wt)
        self.store(name + ".b", bias)
        into = kw.pop("into", None)          # (tensor, channel offset): fill part of a concatenation
        if into is None:
            out = self.tensor((n, cout, ho, wo))
        else:
            out, off = into
            on, oc, oh, ow = self.shape(out)
            assert (on, oh, ow) == (n, ho, wo) and off + cout <= oc
            kw["out_off"] = off
        ins = [x] + ([res] if res is not None else [])
        return self.op(kind="conv", name=name, inputs=ins, out=out, cout=cout, kh=k, kw=k,
                       stride=stride, pad=pad, act=act, w=name + ".w", b=name + ".b", **kw)

    def inception(self, x, c1, c3r, c3, c5r, c5, cp, name, rd=False):
        """Four parallel branches over x -- 1x1; 1x1 -> 3x3; 1x1 -> 5x5; 3x3 max pool ->
        1x1 -- written side by side into one concatenated tensor (Eq. 2 topology)."""
        n, _, h, w = self.shape(x)
        out = self.tensor((n, c1 + c3 + c5 + cp, h, w))
        self.conv(x, c1, 1, 1, 0, "relu", name + ".b1", bn_fold=True, branch=1, pos=1, into=(out, 0))
        t = self.conv(x, c3r, 1, 1, 0, "relu", name + ".b2r", bn_fold=True, branch=2, pos=1)
        self.conv(t, c3, 3, 1, 1, "relu", name + ".b2", bn_fold=True, branch=2, pos=2, rd=rd, into=(out, c1))
        t = self.conv(x, c5r, 1, 1, 0, "relu", name + ".b3r", bn_fold=True, branch=3, pos=1)
        self.conv(t, c5, 5, 1, 2, "relu", name + ".b3", bn_fold=True, branch=3, pos=2, into=(out, c1 + c3))
        t = self.maxpool(x, 3, 1, 1, name + ".b4p", branch=4, pos=1)
        return self.conv(t, cp, 1, 1, 0, "relu", name + ".b4", bn_fold=True, branch=4, pos=2,
                         into=(out, c1 + c3 + c5))

    def maxpool(self, x, k, stride, pad, name, **kw):
        n, c, h, w = self.shape(x)
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        out = self.tensor((n, c, ho, wo))
        return self.op(kind="maxpool", name=name, inputs=[x], out=out, k=k, stride=stride, pad=pad, **kw)

    def avgpool(self, x, name, **kw):
        n, c, _, _ = self.shape(x)
        out = self.tensor((n, c))
        return self.op(kind="avgpool", name=name, inputs=[x], out=out, **kw)

    def linear(self, x, nout, act, name, init, res=None, **kw):
        shp = self.shape(x)
        if len(shp) == 4:                       # flatten NCHW -> [N, C*H*W]
            lead, nin = (shp[0],), shp[1] * shp[2] * shp[3]
        else:
            lead, nin = shp[:-1], shp[-1]
        if init == "he":
            wt, bias = self.he((nout, nin), nin), np.zeros(nout)
        elif init == "bert":
            wt, bias = self.normal((nout, nin), 0.02), np.zeros(nout)
        elif init == "lstm":
            wt = self.uniform((nout, nin), -0.05, 0.05)
            bias = self.uniform((nout,), -0.05, 0.05)
        elif init == "rand":
            wt = self.normal((nout, nin), 1.0 / math.sqrt(nin))
            bias = self.normal((nout,), 0.5)
        else:
            raise ValueError(init)
        self.store(name + ".w", wt)
        self.store(name + ".b", bias)
        out = self.tensor(tuple(lead) + (nout,))
        ins = [x] + ([res] if res is not None else [])
        return self.op(kind="linear", name=name, inputs=ins, out=out, nout=nout, nin=nin, act=act,
                       w=name + ".w", b=name + ".b", **kw)

    def layernorm(self, x, name, eps, res=None, rand=False, **kw):
        f = self.shape(x)[-1]
        if rand:
            self.store(name + ".g", self.uniform((f,), 0.5, 1.5))
            self.store(name + ".beta", self.normal((f,), 0.2))
        else:
            self.store(name + ".g", np.ones(f))
            self.store(name + ".beta", np.zeros(f))
        out = self.tensor(self.shape(x))
        ins = [x] + ([res] if res is not None else [])
        return self.op(kind="layernorm", name=name, inputs=ins, out=out, eps=eps,
                       g=name + ".g", beta=name + ".beta", **kw)

    def attention(self, qkv, heads, name, **kw):
        b, s, f3 = self.shape(qkv)
        f = f3 // 3
        out = self.tensor((b, s, f))
        return self.op(kind="attention", name=name, inputs=[qkv], out=out, heads=heads,
                       head_dim=f // heads, scale=1.0 / math.sqrt(f // heads), **kw)

    def embed_bert(self, ids, vocab, max_pos, n_types, f, name, eps, std=0.02, **kw):
        b, s = self.shape(ids)
        self.store(name + ".tok", self.normal((vocab, f), std))
        self.store(name + ".pos", self.normal((max_pos, f), std))
        self.store(name + ".type", self.normal((n_types, f), std))
        self.store(name + ".g", np.ones(f))
        self.store(name + ".beta", np.zeros(f))
        out = self.tensor((b, s, f))
        return self.op(kind="embed_bert", name=name, inputs=[ids], out=out, vocab=vocab, f=f, eps=eps,
                       w_tok=name + ".tok", w_pos=name + ".pos", w_type=name + ".type",
                       g=name + ".g", beta=name + ".beta", **kw)

    def embed(self, ids, vocab, f, name, lo, hi, **kw):
        b, s = self.shape(ids)
        self.store(name + ".table", self.uniform((vocab, f), lo, hi))
        out = self.tensor((b, s, f))
        return self.op(kind="embed", name=name, inputs=[ids], out=out, vocab=vocab, f=f,
                       table=name + ".table", **kw)

    def lstm(self, x, hidden, name, lo, hi, **kw):
        b, t, e = self.shape(x)
        self.store(name + ".w_ih", self.uniform((4 * hidden, e), lo, hi))
        self.store(name + ".w_hh", self.uniform((4 * hidden, hidden), lo, hi))
        self.store(name + ".b_ih", self.uniform((4 * hidden,), lo, hi))
        self.store(name + ".b_hh", self.uniform((4 * hidden,), lo, hi))
        out = self.tensor((b, t, hidden))
        return self.op(kind="lstm", name=name, inputs=[x], out=out, hidden=hidden,
                       w_ih=name + ".w_ih", w_hh=name + ".w_hh", b_ih=name + ".b_ih",
                       b_hh=name + ".b_hh", **kw)

    def finish(self, out_tid, n_slices, cuts_after=None, elim_tau=0.05, k_by_layer=None):
        m = self.m
        m.output_tid = out_tid
        n = len(m.layers)
        allowed = None
        if cuts_after is not None:
            allowed = [1 if j in set(cuts_after) else 0 for j in range(n - 1)]
        k_override = [0] * n
        for layer, k in (k_by_layer or {}).items():
            k_override[layer] = k
        m.slicing = dict(n_slices=n_slices, allowed_cut=allowed, elim_tau=elim_tau, k_override=k_override)
        return m


# ---------------------------------------------------------------------------
# The five workloads.  Keyword arguments shrink them for fast tests; the
# defaults are the full-size configurations.
# ---------------------------------------------------------------------------

def tiny_vgg(batch=1, hw=32, chans=(16, 16, 32, 32, 64, 64), n_cls=10, k_rd=2, seed=1001):
    """Tiny VGG-style CNN, fp32: six 3x3 convs (+ReLU), 2x2/2 max-pool after each pair, FC."""
    bld = _Builder("tiny_vgg", F32, batch, seed, cfg=1)
    x = bld.tensor((batch, 3, hw, hw), F32)
    rd_layer = None
    for i, c in enumerate(chans):
        bld.new_layer(f"conv{i + 1}")
        rd = i == len(chans) - 1          # conv6: the largest conv (FLOP tie broken by bytes, then index)
        x = bld.conv(x, c, 3, 1, 1, "relu", f"conv{i + 1}", rd=rd)
        if rd:
            rd_layer = bld.layer
        if i % 2 == 1:
            bld.new_layer(f"pool{i // 2 + 1}")
            x = bld.maxpool(x, 2, 2, 0, f"pool{i // 2 + 1}")
    bld.new_layer("fc")
    y = bld.linear(x, n_cls, "none", "fc", "he")
    return bld.finish(y, n_slices=3, cuts_after=None, k_by_layer={rd_layer: k_rd})


def resnet50(batch=8, hw=224, blocks=(3, 4, 6, 3), widths=(64, 128, 256, 512), n_cls=1000,
             k_rd=4, seed=1002):
    """ResNet-50-shaped CNN (v1.5: stride on the 3x3), bf16, BN folded into the convs."""
    bld = _Builder("resnet50", BF16, batch, seed, cfg=2)
    x = bld.tensor((batch, 3, hw, hw), F32)
    bld.new_layer("stem")
    x = bld.conv(x, widths[0], 7, 2, 3, "relu", "stem.conv", bn_fold=True)
    x = bld.maxpool(x, 3, 2, 1, "stem.pool")
    k_by_layer, cuts = {}, []
    cin = widths[0]
    for si, (nb, wmid) in enumerate(zip(blocks, widths)):
        wout = wmid * 4
        for bi in range(nb):
            stride = 2 if (bi == 0 and si > 0) else 1
            nm = f"s{si + 1}b{bi + 1}"
            bld.new_layer(nm)
            a = bld.conv(x, wmid, 1, 1, 0, "relu", nm + ".a", bn_fold=True, branch=1, pos=1)
            b = bld.conv(a, wmid, 3, stride, 1, "relu", nm + ".b", bn_fold=True, branch=1, pos=2, rd=True)
            if bi == 0:
                sc = bld.conv(x, wout, 1, stride, 0, "none", nm + ".sc", bn_fold=True, branch=2, pos=1)
            else:
                sc = x
            x = bld.conv(b, wout, 1, 1, 0, "relu", nm + ".c", res=sc, bn_fold=True, branch=1, pos=3)
            k_by_layer[bld.layer] = k_rd
            cin = wout
        if si < len(blocks) - 1:
            cuts.append(bld.layer)
    bld.new_layer("head")
    x = bld.avgpool(x, "head.pool")
    y = bld.linear(x, n_cls, "none", "head.fc", "he")
    return bld.finish(y, n_slices=len(cuts) + 1, cuts_after=cuts, k_by_layer=k_by_layer)


VGG16_CFG = (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M")


def vgg16(batch=16, hw=224, arch=VGG16_CFG, fc=(4096, 4096), n_cls=1000, k_rd=8, seed=1003,
          cut_after_pools=(3, 5)):
    """VGG-16-shaped CNN, bf16; fc6 is the RD GEMM."""
    bld = _Builder("vgg16", BF16, batch, seed, cfg=3)
    x = bld.tensor((batch, 3, hw, hw), F32)
    cuts, blk, ci, npool = [], 1, 1, 0
    for v in arch:
        if v == "M":
            npool += 1
            bld.new_layer(f"pool{npool}")
            x = bld.maxpool(x, 2, 2, 0, f"pool{npool}")
            if npool in cut_after_pools:
                cuts.append(bld.layer)
            blk, ci = blk + 1, 1
        else:
            nm = f"conv{blk}_{ci}"
            bld.new_layer(nm)
            x = bld.conv(x, v, 3, 1, 1, "relu", nm)
            ci += 1
    k_by_layer = {}
    for i, f in enumerate(fc):
        nm = f"fc{6 + i}"
        bld.new_layer(nm)
        x = bld.linear(x, f, "relu", nm, "he", rd=(i == 0))
        if i == 0:
            k_by_layer[bld.layer] = k_rd
    bld.new_layer(f"fc{6 + len(fc)}")
    y = bld.linear(x, n_cls, "none", f"fc{6 + len(fc)}", "he")
    return bld.finish(y, n_slices=len(cuts) + 1, cuts_after=cuts, k_by_layer=k_by_layer)


def bert_base(batch=32, seq=128, layers=12, hidden=768, heads=12, ffn=3072, vocab=30522,
              max_pos=512, k_rd=4, slice_every=3, seed=1004):
    """BERT-base-shaped post-LN encoder, bf16; both FFN GEMMs are RD ops."""
    bld = _Builder("bert_base", BF16, batch, seed, cfg=4)
    ids = bld.tensor((batch, seq), I32)
    bld.new_layer("embed")
    x = bld.embed_bert(ids, vocab, max_pos, 2, hidden, "embed", 1e-12)
    k_by_layer, cuts = {}, []
    for li in range(layers):
        nm = f"L{li + 1}"
        bld.new_layer(nm)
        qkv = bld.linear(x, 3 * hidden, "none", nm + ".qkv", "bert")
        att = bld.attention(qkv, heads, nm + ".attn")
        a = bld.linear(att, hidden, "none", nm + ".proj", "bert", res=x)
        a = bld.layernorm(a, nm + ".ln1", 1e-12)
        h = bld.linear(a, ffn, "gelu", nm + ".ffn1", "bert", rd=True)
        h = bld.linear(h, hidden, "none", nm + ".ffn2", "bert", res=a, rd=True)
        x = bld.layernorm(h, nm + ".ln2", 1e-12)
        k_by_layer[bld.layer] = k_rd
        if (li + 1) % slice_every == 0 and li + 1 < layers:
            cuts.append(bld.layer)
    return bld.finish(x, n_slices=len(cuts) + 1, cuts_after=cuts, k_by_layer=k_by_layer)


def lstm_lm(batch=64, seq=128, hidden=1024, emb=1024, vocab=32000, n_layers=2, k_rd=8, seed=1005):
    """Two-layer LSTM language model, bf16; the vocabulary projection is the RD GEMM."""
    bld = _Builder("lstm_lm", BF16, batch, seed, cfg=5)
    ids = bld.tensor((batch, seq), I32)
    bld.new_layer("embed")
    x = bld.embed(ids, vocab, emb, "embed", -0.05, 0.05)
    cuts = [bld.layer]
    for li in range(n_layers):
        bld.new_layer(f"lstm{li + 1}")
        x = bld.lstm(x, hidden, f"lstm{li + 1}", -0.05, 0.05)
    cuts.append(bld.layer)
    bld.new_layer("proj")
    y = bld.linear(x, vocab, "none", "proj", "lstm", rd=True)
    return bld.finish(y, n_slices=len(cuts) + 1, cuts_after=cuts, k_by_layer={bld.layer: k_rd})




def inception_mini(batch=2, hw=32, k_rd=2, seed=1006, dtype=BF16):
    """Small Inception-style CNN (the branching family of the paper's CNN benchmarks): a
    stem conv and max pool, three four-branch nodes whose branch outputs are concatenated
    in place (some at channel offsets that are not a whole 16-byte chunk), a second pool,
    global average pool and a classifier.  Each node's 3x3 branch conv is the RD op."""
    bld = _Builder("inception_mini", dtype, batch, seed, cfg=6)
    x = bld.tensor((batch, 3, hw, hw), F32)
    bld.new_layer("stem")
    x = bld.conv(x, 32, 3, 2, 1, "relu", "stem.conv", bn_fold=True)
    bld.new_layer("pool1")
    x = bld.maxpool(x, 3, 2, 1, "pool1")
    k_by_layer = {}
    for nm, ch in (("inc3a", (16, 16, 24, 8, 12, 12)), ("inc3b", (24, 24, 32, 8, 20, 20)),
                   ("pool2", None), ("inc4a", (32, 32, 48, 8, 16, 16))):
        bld.new_layer(nm)
        if ch is None:
            x = bld.maxpool(x, 3, 2, 1, nm)
            continue
        x = bld.inception(x, *ch, nm, rd=True)
        k_by_layer[bld.layer] = k_rd
    bld.new_layer("head")
    x = bld.avgpool(x, "gap")
    y = bld.linear(x, 10, "none", "fc", "he")
    return bld.finish(y, n_slices=3, k_by_layer=k_by_layer)




def skipnet_mini(batch=2, hw=16, k_rd=2, seed=1007, dtype=BF16):
    """Small CNN with skip edges across planning nodes (U-Net / DenseNet style): node 3
    adds the stem's output as a residual and node 4 concatenates node 1's output, so
    the cuts after nodes 0-3 carry one, two, three and two tensors."""
    bld = _Builder("skipnet_mini", dtype, batch, seed, cfg=7)
    x = bld.tensor((batch, 3, hw, hw), F32)
    bld.new_layer("stem")
    x0 = bld.conv(x, 16, 3, 1, 1, "relu", "stem", bn_fold=True)
    bld.new_layer("c1")
    x1 = bld.conv(x0, 16, 3, 1, 1, "relu", "c1", bn_fold=True)
    bld.new_layer("c2")
    x2 = bld.conv(x1, 16, 3, 1, 1, "relu", "c2", bn_fold=True, rd=True)
    rd_layer = bld.layer
    bld.new_layer("c3")
    x3 = bld.conv(x2, 16, 3, 1, 1, "relu", "c3", res=x0, bn_fold=True)
    bld.new_layer("cat")
    n, _, h, w = bld.shape(x3)
    cat = bld.tensor((n, 32, h, w))
    bld.conv(x3, 16, 1, 1, 0, "relu", "cat.a", bn_fold=True, branch=1, pos=1, into=(cat, 0))
    bld.conv(x1, 16, 1, 1, 0, "relu", "cat.b", bn_fold=True, branch=2, pos=1, into=(cat, 16))
    bld.new_layer("head")
    y = bld.linear(bld.avgpool(cat, "gap"), 10, "none", "fc", "he")
    return bld.finish(y, n_slices=3, k_by_layer={rd_layer: k_rd})


BUILDERS = {1: tiny_vgg, 2: resnet50, 3: vgg16, 4: bert_base, 5: lstm_lm, 6: inception_mini, 7: skipnet_mini}
NAMES = {1: "tiny_vgg", 2: "resnet50", 3: "vgg16", 4: "bert_base", 5: "lstm_lm", 6: "inception_mini",
         7: "skipnet_mini"}


def build(cfg: int, **kw) -> Model:
    """Full-size configuration ``cfg`` (1..5), or a shrunken variant via keyword arguments."""
    kw.setdefault("seed", 1000 + cfg)
    return BUILDERS[cfg](**kw)


def make_input(model: Model, seed: int | None = None) -> np.ndarray:
    """Seeded model input: images ~ N(0, 1) float32 NCHW, or uniform token ids int32 [B, S]."""
    seed = 2000 + model.cfg if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    t = model.tensors[model.input_tid]
    if t["dtype"] == I32:
        vocab = model.ops[0]["vocab"]
        return rng.integers(0, vocab, size=t["shape"], dtype=np.int64).astype(np.int32)
    return rng.standard_normal(t["shape"]).astype(np.float32)


def boundary_channels(model: Model, layer: int) -> int:
    """Channel (images) or feature (sequences) count of the tensor leaving ``layer``."""
    t = model.tensors[model.layer_output_tid(layer)]
    return t["shape"][1] if len(t["shape"]) == 4 else t["shape"][-1]


def tensor_channels(model: Model, tid: int) -> int:
    """Channel (images) or feature (sequences) count of tensor ``tid``."""
    s = model.tensors[tid]["shape"]
    return s[1] if len(s) == 4 else s[-1]


def make_codec_weights(model: Model, cut_layers, ratio: int = 8, seed: int | None = None, tensors=None):
    """Autoencoder weights for each boundary: W_e ~ N(0, 1/C) [C_e][C], W_d ~ N(0, 1/C_e) [C][C_e], biases 0.

    One set per cut (for the tensor leaving that node), or, when ``tensors`` lists
    the boundary tensor ids (several per cut where skip edges cross it), one per
    tensor in that order.  ``ratio`` may be an int or a list (one per boundary).
    Returns a list of dicts with keys c, c_code, w_enc, b_enc, w_dec, b_dec
    (float32, model-dtype values).
    """
    seed = 3000 + model.cfg if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    chans = ([tensor_channels(model, t) for t in tensors] if tensors is not None
             else [boundary_channels(model, layer) for layer in cut_layers])
    ratios = ratio if isinstance(ratio, (list, tuple)) else [ratio] * len(chans)
    out = []
    for c, r in zip(chans, ratios):
        if c % r:
            raise ValueError(f"channels {c} not divisible by ratio {r}")
        ce = c // r
        arrs = [rng.standard_normal((ce, c)) * math.sqrt(1.0 / c), np.zeros(ce),
                rng.standard_normal((c, ce)) * math.sqrt(1.0 / ce), np.zeros(c)]
        arrs = [np.asarray(a, dtype=np.float64).astype(np.float32) for a in arrs]
        if model.dtype == BF16:
            arrs = [to_bf16_values(a) for a in arrs]
        out.append(dict(c=c, c_code=ce, w_enc=arrs[0], b_enc=arrs[1], w_dec=arrs[2], b_dec=arrs[3]))
    return out


def random_codec_weights(c: int, c_code: int, dtype: str, seed: int):
    """Codec weights with non-zero biases, for kernel-level tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    arrs = [rng.standard_normal((c_code, c)) / math.sqrt(c), rng.standard_normal(c_code) * 0.5,
            rng.standard_normal((c, c_code)) / math.sqrt(c_code), rng.standard_normal(c) * 0.5]
    arrs = [np.asarray(a).astype(np.float32) for a in arrs]
    if dtype == BF16:
        arrs = [to_bf16_values(a) for a in arrs]
    return dict(c=c, c_code=c_code, w_enc=arrs[0], b_enc=arrs[1], w_dec=arrs[2], b_dec=arrs[3])


def random_tensor(shape, dtype: str, seed: int, scale: float = 1.0) -> np.ndarray:
    """Seeded N(0, scale^2) tensor holding ``dtype`` values (float32 array)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    a = (rng.standard_normal(shape) * scale).astype(np.float32)
    return to_bf16_values(a) if dtype == BF16 else a
