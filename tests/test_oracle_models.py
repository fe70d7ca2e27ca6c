"""Pins for the oracle's model forward (CPU only).

A second evaluator built from torch library routines (conv2d, max_pool2d,
layer_norm, scaled_dot_product_attention, nn.LSTM) in float64, rounding each
op output to the storage type with torch's own casts, must agree with the
oracle on shrunken versions of all five workloads.  This pins the oracle's
op dispatch (which weight goes where, residual inputs, flatten order,
rounding points) against independent library code.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth


def _round(t, dtype):
    if dtype == "none":
        return t
    if dtype == "bf16":
        return t.to(torch.bfloat16).double()
    if dtype == "f32":
        return t.float().double()
    return t


def torch_forward(m, x, rnd=None):
    """The model evaluated with torch library routines in float64; every stored tensor rounded
    to ``rnd`` (None: the model dtype; 'none': no rounding, the LSTM cell state included)."""
    W = {k: torch.from_numpy(v.astype(np.float64)) for k, v in m.weights.items()}
    dt = m.dtype if rnd is None else rnd
    if m.tensors[m.input_tid]["dtype"] == "i32":
        env = {m.input_tid: torch.from_numpy(x.astype(np.int64))}
    else:
        env = {m.input_tid: _round(torch.from_numpy(x.astype(np.float64)), dt)}
    parts = {}
    for op in m.ops:
        ins = [env[t] for t in op["inputs"]]
        k = op["kind"]
        if k == "conv":
            v = F.conv2d(ins[0], W[op["w"]], W[op["b"]], op["stride"], op["pad"])
            if len(ins) > 1:
                v = v + ins[1]
            v = F.relu(v) if op["act"] == "relu" else v
            y = _round(v, dt)
        elif k == "maxpool":
            y = F.max_pool2d(ins[0], op["k"], op["stride"], op["pad"])
        elif k == "avgpool":
            y = _round(ins[0].mean(dim=(2, 3)), dt)
        elif k == "linear":
            a = ins[0].flatten(1) if ins[0].dim() == 4 else ins[0]
            v = F.linear(a, W[op["w"]], W[op["b"]])
            if len(ins) > 1:
                v = v + ins[1]
            if op["act"] == "relu":
                v = F.relu(v)
            elif op["act"] == "gelu":
                v = F.gelu(v, approximate="none")
            y = _round(v, dt)
        elif k == "layernorm":
            v = ins[0] + (ins[1] if len(ins) > 1 else 0)
            y = _round(F.layer_norm(v, v.shape[-1:], W[op["g"]], W[op["beta"]], op["eps"]), dt)
        elif k == "attention":
            b, s, f3 = ins[0].shape
            h = op["heads"]
            d = f3 // 3 // h
            t = ins[0].view(b, s, 3, h, d).permute(2, 0, 3, 1, 4)
            o = F.scaled_dot_product_attention(t[0], t[1], t[2], scale=op["scale"])
            y = _round(o.permute(0, 2, 1, 3).reshape(b, s, h * d), dt)
        elif k == "embed_bert":
            ids = ins[0]
            v = W[op["w_tok"]][ids] + W[op["w_pos"]][: ids.shape[1]][None] + W[op["w_type"]][0]
            y = _round(F.layer_norm(v, v.shape[-1:], W[op["g"]], W[op["beta"]], op["eps"]), dt)
        elif k == "embed":
            y = W[op["table"]][ins[0]]
        elif k == "lstm":
            xx = ins[0]
            b, t, _ = xx.shape
            hd = op["hidden"]
            h = torch.zeros(b, hd, dtype=torch.float64)
            c = torch.zeros(b, hd, dtype=torch.float64)
            outs = []
            for s in range(t):
                g = F.linear(xx[:, s], W[op["w_ih"]], W[op["b_ih"]]) + F.linear(h, W[op["w_hh"]], W[op["b_hh"]])
                i, f, gg, o = g.split(hd, dim=1)
                c = _round(torch.sigmoid(f) * c + torch.sigmoid(i) * torch.tanh(gg), "none" if dt == "none" else "f32")
                h = _round(torch.sigmoid(o) * torch.tanh(c), dt)
                outs.append(h)
            y = torch.stack(outs, 1)
        else:
            raise ValueError(k)
        if "out_off" in op:                 # branch of a parallel node: channel concatenation
            parts.setdefault(op["out"], []).append((op["out_off"], y))
            y = torch.cat([p for _, p in sorted(parts[op["out"]], key=lambda q: q[0])], dim=1)
        env[op["out"]] = y
    return env[m.output_tid].numpy()


SMALL = {
    1: dict(hw=16),
    2: dict(batch=2, hw=32, blocks=(1, 2, 1, 1), widths=(8, 16, 16, 32), n_cls=10),
    3: dict(batch=2, hw=32, arch=(8, "M", 16, "M", 16, 16, "M", 32, "M", 32, "M"), fc=(64, 48), n_cls=10,
            cut_after_pools=(2, 4)),
    4: dict(batch=2, seq=16, layers=2, hidden=64, heads=2, ffn=128, vocab=100, max_pos=32, slice_every=1),
    5: dict(batch=2, seq=6, hidden=32, emb=24, vocab=50),
    6: dict(batch=2, hw=16),
    7: dict(batch=2, hw=8),
}


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6, 7])
def test_oracle_model_matches_torch_library_forward(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    y = oracle.forward(m, x)
    ref = torch_forward(m, x)
    # both round at the same points; double-accumulation order differences can flip a
    # bf16 rounding, so compare with a bf16-ulp-scale tolerance relative to the tensor max
    scale = np.abs(ref).max()
    tol = 1e-12 if m.dtype == "f32" else 2e-2
    assert np.abs(y - ref).max() <= tol * scale


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6, 7])
def test_oracle_model_matches_torch_library_forward_unrounded(cfg):
    """Without storage rounding both evaluators compute the same real-valued function in double,
    so they agree to double-precision summation-order noise: any op-dispatch mistake in the oracle
    (a weight in the wrong place, a missing residual, a wrong flatten order) shows up far above
    1e-12, which the bf16-rounded comparison above, held to bf16 noise, cannot resolve."""
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    y = oracle.forward(m, x, rnd="none")
    ref = torch_forward(m, x, rnd="none")
    assert np.abs(y - ref).max() <= 1e-12 * np.abs(ref).max()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_sample_rows_equal_full_batch(cfg):
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    full = oracle.forward(m, x)
    part = oracle.forward(m, x, sample=[m.batch - 1])
    np.testing.assert_array_equal(part[0], full[m.batch - 1])


def test_full_size_configs_shapes():
    for cfg, out in [(1, (1, 10)), (2, (8, 1000)), (4, (32, 128, 768)), (5, (64, 128, 32000))]:
        m = synth.build(cfg)
        assert m.tensors[m.output_tid]["shape"] == out
        assert len(m.layers) == {1: 10, 2: 18, 4: 13, 5: 4}[cfg]


def test_codec_hand_off_changes_only_through_codec():
    m = synth.build(2, **SMALL[2])
    x = synth.make_input(m)
    cuts = [1, 3]
    cw = synth.make_codec_weights(m, cuts, ratio=8)
    y, env, codes, bounds = oracle.forward(m, x, cuts=cuts, codecs=cw, keep=True)
    for li, c in zip(cuts, cw):
        code = codes[li]
        assert code.shape[1] == bounds[li].shape[1] // 8
        np.testing.assert_array_equal(code, oracle.ae_encode(bounds[li], c["w_enc"], c["b_enc"], "bf16"))
        np.testing.assert_array_equal(env[m.layer_output_tid(li)],
                                      oracle.ae_decode(code, c["w_dec"], c["b_dec"], "bf16"))
    assert math.isfinite(float(np.abs(y).max()))


def _planted(monkeypatch, name):
    """Plant one plausible mistake in the oracle's op dispatch (CPU only, undone after the test)."""
    real = oracle.run_op

    def wrong(model, op, env, w_rows=None, rnd=None):
        k = op["kind"]
        if name == "linear_residual_dropped" and k == "linear" and len(op["inputs"]) > 1:
            op = dict(op, inputs=op["inputs"][:1])
        elif name == "attention_scale_over_hidden" and k == "attention":
            op = dict(op, scale=op["scale"] / np.sqrt(op["heads"]))     # 1/sqrt(F) in place of 1/sqrt(d)
        elif name == "lstm_gates_swapped" and k == "lstm":
            W = dict(model.weights)
            h = op["hidden"]
            for key in ("w_ih", "w_hh", "b_ih", "b_hh"):
                a = W[op[key]]
                W[op[key]] = np.concatenate([a[h:2 * h], a[:h], a[2 * h:]])   # i <-> f
            model = type(model)(**{**model.__dict__, "weights": W})
        elif name == "conv_residual_dropped" and k == "conv" and len(op["inputs"]) > 1:
            op = dict(op, inputs=op["inputs"][:1])
        return real(model, op, env, w_rows, rnd)
    monkeypatch.setattr(oracle, "run_op", wrong)


@pytest.mark.parametrize("cfg,mistake", [(4, "linear_residual_dropped"), (4, "attention_scale_over_hidden"),
                                         (5, "lstm_gates_swapped"), (2, "conv_residual_dropped")])
def test_unrounded_pin_catches_planted_mistakes(monkeypatch, cfg, mistake):
    m = synth.build(cfg, **SMALL[cfg])
    x = synth.make_input(m)
    ref = torch_forward(m, x, rnd="none")
    _planted(monkeypatch, mistake)
    y = oracle.forward(m, x, rnd="none")
    assert np.abs(y - ref).max() > 1e-9 * np.abs(ref).max()
