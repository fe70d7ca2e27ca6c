"""Pins for the oracle's operator profile (Sec. III-B, Eq. 1-4), every op kind.

The pins are numbers fixed outside the oracle, never its own formulas typed
again:

* the algorithmic FLOP per batch of the five workloads, from the standard
  multiply-accumulate counts of the architectures (ResNet-50 v1.5: 4 089 184 256
  MAC per 224x224 image; VGG-16: 15 470 264 320; BERT-base: 11 173 625 856 per
  128-token sequence; the 2-layer LSTM LM: 6 341 787 648 per 128-token sequence;
  the tiny VGG: 9 889 792 per 32x32 image), each re-derived below from the
  layer table as a cross-check of the constant;
* the published parameter counts of the standard architectures (ResNet-50
  25 557 032 with its batch-norm scales and shifts, here folded into one bias
  per conv channel; VGG-16 138 357 544; BERT-base without its pooler
  108 891 648), which the operator profile's parameter bytes must add up to;
* the sizes of the boundary tensors at the prescribed cuts;
* byte and FLOP counts of single operators at small shapes, evaluated by hand
  (the arithmetic is in the comments).

A dropped term (a bias, the second LSTM bias, the residual input), a wrong
element size (int32 ids, the f32 model input) or a transposed dimension moves at
least one of these numbers.
"""
import pytest

import synth
from oracle import plan as P

# ---------------------------------------------------------------------------
# whole workloads
# ---------------------------------------------------------------------------

FLOP_PER_BATCH = {1: 19_779_584, 2: 65_426_948_096, 3: 495_048_458_240, 4: 715_112_054_784,
                  5: 811_748_818_944}
BATCH = {1: 1, 2: 8, 3: 16, 4: 32, 5: 64}


def resnet50_mac_per_image():
    """ResNet-50 v1.5 (stride on the 3x3 conv of each stage's first block)."""
    mac = 112 * 112 * 64 * 3 * 49                       # 7x7/2 stem
    hw, cin = 56, 64                                    # after the 3x3/2 max pool
    for blocks, width, stride in ((3, 64, 1), (4, 128, 2), (6, 256, 2), (3, 512, 2)):
        for b in range(blocks):
            s = stride if b == 0 else 1
            ho = hw // s
            mac += hw * hw * cin * width                # 1x1 reduce
            mac += ho * ho * width * width * 9          # 3x3 (stride s)
            mac += ho * ho * width * 4 * width          # 1x1 expand
            if b == 0:
                mac += ho * ho * cin * 4 * width        # projection shortcut
            hw, cin = ho, 4 * width
    return mac + 2048 * 1000


def vgg16_mac_per_image():
    mac, hw, cin = 0, 224, 3
    for cout, n in ((64, 2), (128, 2), (256, 3), (512, 3), (512, 3)):
        for _ in range(n):
            mac += hw * hw * cin * cout * 9
            cin = cout
        hw //= 2
    return mac + 25088 * 4096 + 4096 * 4096 + 4096 * 1000


def bert_base_mac_per_sequence(s=128, f=768, ffn=3072, layers=12):
    per_layer = s * f * 3 * f + 2 * s * s * f + s * f * f + 2 * s * f * ffn   # QKV, QK^T and PV, O, FFN
    return layers * per_layer


def lstm_lm_mac_per_sequence(t=128, e=1024, h=1024, v=32000):
    layer1 = t * 4 * h * (e + h)
    layer2 = t * 4 * h * (h + h)
    return layer1 + layer2 + t * h * v


def tiny_vgg_mac():
    return (32 * 32 * 9 * (3 * 16 + 16 * 16) + 16 * 16 * 9 * (16 * 32 + 32 * 32)
            + 8 * 8 * 9 * (32 * 64 + 64 * 64) + 1024 * 10)


def test_flop_constants_match_the_layer_tables():
    assert tiny_vgg_mac() == 9_889_792
    assert resnet50_mac_per_image() == 4_089_184_256
    assert vgg16_mac_per_image() == 15_470_264_320
    assert bert_base_mac_per_sequence() == 11_173_625_856
    assert lstm_lm_mac_per_sequence() == 6_341_787_648
    per = {1: tiny_vgg_mac(), 2: resnet50_mac_per_image(), 3: vgg16_mac_per_image(),
           4: bert_base_mac_per_sequence(), 5: lstm_lm_mac_per_sequence()}
    for cfg, mac in per.items():
        assert 2 * mac * BATCH[cfg] == FLOP_PER_BATCH[cfg]


_FULL = {}


def full(cfg):
    if cfg not in _FULL:
        _FULL[cfg] = synth.build(cfg)
    return _FULL[cfg]


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_summed_op_flop_equals_workload_flop(cfg):
    m = full(cfg)
    assert sum(P.op_profile(m, op)[2] for op in m.ops) == FLOP_PER_BATCH[cfg]


def test_lstm_lm_flop_split():
    """Input projections 137.4, recurrence 137.4 and vocabulary projection 536.9 GFLOP per batch:
    the two LSTM ops carry the first two, the projection the third."""
    m = full(5)
    by_kind = {}
    for op in m.ops:
        by_kind[op["kind"]] = by_kind.get(op["kind"], 0) + P.op_profile(m, op)[2]
    # per layer 2 FLOP x (64 x 128 positions) x 4096 gate rows x 1024; two layers (E = H = 1024)
    in_proj = 2 * (2 * 64 * 128 * 4096 * 1024)           # x_t -> 4H gates
    recur = 2 * (2 * 64 * 128 * 4096 * 1024)             # h_{t-1} -> 4H gates
    assert in_proj == recur == 137_438_953_472
    assert by_kind["lstm"] == in_proj + recur
    assert by_kind["linear"] == 536_870_912_000 == 2 * 64 * 128 * 1024 * 32000
    assert by_kind.get("embed", 0) == 0


PUBLISHED_PARAMS = {
    # tiny VGG: six 3x3 convs with biases and a 1024 -> 10 classifier (counted by hand:
    # 448 + 2320 + 4640 + 9248 + 18496 + 36928 + 10250)
    1: 82_330,
    # ResNet-50: 25 557 032 published, with 2 x 26 560 batch-norm parameters; folding them
    # into the convs leaves one bias per channel: 25 557 032 - 26 560
    2: 25_530_472,
    3: 138_357_544,      # VGG-16 with 1000 classes
    4: 108_891_648,      # BERT-base (30 522-token vocabulary, 512 positions, 2 types), no pooler
    # LSTM LM: 32 000 x 1024 embedding; two layers of 4H x (E + H) weights and two 4H biases;
    # 1024 -> 32 000 projection with bias: 32 768 000 + 2 x 8 396 800 + 32 800 000
    5: 82_361_600,
}


def _act_bytes(m, op):
    """Bytes of the op's input and output tensors as stored (a concatenation writer counts its
    own channels only; no workload here has one)."""
    es = {"bf16": 2, "f32": 4, "i32": 4}
    n = 0
    for t in list(op["inputs"]) + [op["out"]]:
        size = 1
        for s in m.tensors[t]["shape"]:
            size *= s
        n += size * es[m.tensors[t]["dtype"]]
    return n


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_op_memory_counts_every_parameter_once(cfg):
    m = full(cfg)
    es = 2 if m.dtype == "bf16" else 4
    param_bytes = sum(P.op_profile(m, op)[0] - _act_bytes(m, op) for op in m.ops)
    assert param_bytes == PUBLISHED_PARAMS[cfg] * es


BOUNDARY_BYTES = {
    2: [8 * 56 * 56 * 256 * 2, 8 * 28 * 28 * 512 * 2, 8 * 14 * 14 * 1024 * 2],   # 12.85 / 6.42 / 3.21 MB
    3: [16 * 256 * 28 * 28 * 2, 16 * 512 * 7 * 7 * 2],                        # after pool3, pool5
    4: [32 * 128 * 768 * 2] * 3,
    5: [64 * 128 * 1024 * 2] * 2,
}


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_boundary_sizes_at_the_prescribed_cuts(cfg):
    m = full(cfg)
    cuts = [j for j, a in enumerate(m.slicing["allowed_cut"]) if a]
    prof = P.layer_profiles(m)
    assert [prof[j].out_bytes for j in cuts] == [float(b) for b in BOUNDARY_BYTES[cfg]]
    assert BOUNDARY_BYTES[2] == [12_845_056, 6_422_528, 3_211_264]
    assert BOUNDARY_BYTES[5] == [16_777_216] * 2


# ---------------------------------------------------------------------------
# single operators, counted by hand
# ---------------------------------------------------------------------------

def _one_op(dtype, in_shape, in_dtype, build):
    b = synth._Builder("one", dtype, in_shape[0], 3)
    x = b.tensor(in_shape, in_dtype)
    b.new_layer("L0")
    y = build(b, x)
    m = b.finish(y, 1)
    return m, m.ops[-1]


def _check(m, op, mem, flop):
    got_mem, got_t, got_flop = P.op_profile(m, op)
    assert got_mem == mem
    assert got_flop == flop
    peak = 2.5e15 if m.dtype == "bf16" else 157.3e12
    assert got_t == max(flop / peak, mem / 8e12)


def test_linear_with_residual():
    # x (2,5,64) bf16 -> 48 features, residual (2,5,48):
    # weight 48*64 + bias 48 = 3120 -> 6240 B; x 640 + residual 480 -> 2240 B; y 480 -> 960 B
    def build(b, x):
        r = b.linear(x, 48, "none", "r", "rand")
        return b.linear(x, 48, "relu", "lin", "rand", res=r)
    m, op = _one_op("bf16", (2, 5, 64), "bf16", build)
    _check(m, op, 9440.0, 2 * 10 * 48 * 64)


def test_linear_on_a_flattened_image():
    # x (2,4,3,3) bf16 flattened to K = 36 -> 10: weight 360 + bias 10 -> 740 B; x 72 -> 144 B;
    # y (2,10) -> 40 B; FLOP 2 * 2 * 10 * 36 = 1440
    m, op = _one_op("bf16", (2, 4, 3, 3), "bf16", lambda b, x: b.linear(x, 10, "none", "fc", "he"))
    _check(m, op, 924.0, 1440)


def test_linear_f32():
    # x (1,3,4) f32 -> 5: weight 20 + bias 5 -> 100 B; x 12 -> 48 B; y 15 -> 60 B; FLOP 120
    m, op = _one_op("f32", (1, 3, 4), "f32", lambda b, x: b.linear(x, 5, "none", "fc", "he"))
    _check(m, op, 208.0, 120)


def test_layernorm_with_residual():
    # x (3,7,32) + residual: gamma, beta 64 -> 128 B; two inputs 2 * 672 -> 2688 B; y -> 1344 B
    def build(b, x):
        r = b.linear(x, 32, "none", "r", "rand")
        return b.layernorm(x, "ln", 1e-12, res=r)
    m, op = _one_op("bf16", (3, 7, 32), "bf16", build)
    _check(m, op, 4160.0, 0)


def test_attention():
    # qkv (2,16,384), 2 heads of 64: no parameters; in 12288 -> 24576 B; out (2,16,128) -> 8192 B;
    # FLOP: QK^T and PV, 2 * (2 * 16 * 16 * 128) multiply-adds = 262144
    m, op = _one_op("bf16", (2, 16, 384), "bf16", lambda b, x: b.attention(x, 2, "att"))
    _check(m, op, 32768.0, 262144)


def test_embed_bert():
    # ids (2,8) int32 -> 64 B; tables (50 + 12 + 2) * 16 + gamma, beta 32 = 1056 -> 2112 B;
    # out (2,8,16) -> 512 B
    m, op = _one_op("bf16", (2, 8), "i32", lambda b, x: b.embed_bert(x, 50, 12, 2, 16, "emb", 1e-12))
    _check(m, op, 2688.0, 0)


def test_embed():
    # ids (3,4) int32 -> 48 B; table 20 x 8 -> 320 B; out (3,4,8) -> 192 B
    m, op = _one_op("bf16", (3, 4), "i32", lambda b, x: b.embed(x, 20, 8, "emb", -1.0, 1.0))
    _check(m, op, 560.0, 0)


def test_lstm():
    # x (2,3,8), H = 16: W_ih 64x8 = 512, W_hh 64x16 = 1024, b_ih 64, b_hh 64 -> 1664 -> 3328 B;
    # x 48 -> 96 B; h sequence (2,3,16) -> 192 B; FLOP 2 * (2*3) * 64 * (8 + 16) = 18432
    m, op = _one_op("bf16", (2, 3, 8), "bf16", lambda b, x: b.lstm(x, 16, "lstm", -0.1, 0.1))
    _check(m, op, 3616.0, 18432)


def test_pools():
    # max pool 2x2/2 of (1,8,6,6): in 288 -> 576 B, out (1,8,3,3) 72 -> 144 B
    m, op = _one_op("bf16", (1, 8, 6, 6), "bf16", lambda b, x: b.maxpool(x, 2, 2, 0, "p"))
    _check(m, op, 720.0, 0)
    # global average of (2,8,4,4): in 256 -> 512 B, out (2,8) -> 32 B
    m, op = _one_op("bf16", (2, 8, 4, 4), "bf16", lambda b, x: b.avgpool(x, "a"))
    _check(m, op, 544.0, 0)


def test_conv_reading_the_f32_model_input():
    # the model input stays float32 in a bf16 model: (1,3,8,8) -> 768 B; 3x3 conv to 4 channels,
    # pad 1: weight 4*3*9 + bias 4 = 112 -> 224 B; out (1,4,8,8) bf16 -> 512 B;
    # FLOP 2 * 256 * 27 = 13824
    m, op = _one_op("bf16", (1, 3, 8, 8), "f32", lambda b, x: b.conv(x, 4, 3, 1, 1, "relu", "c"))
    _check(m, op, 1504.0, 13824)
