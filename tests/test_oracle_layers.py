"""Pins for the oracle's layer math (CPU only).

Each oracle routine is checked against something other than itself: a
brute-force loop written independently here, a library routine (torch CPU in
float64, numpy, scipy), a closed form or a known rounding value.  Shapes are
chosen so that a transposed operand, a wrong stride or pad, a dropped bias or
a mis-ordered gate fails a check.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

RNG = np.random.default_rng(7)


def rnd(*shape, scale=1.0):
    return RNG.standard_normal(shape) * scale


# ---- rounding ---------------------------------------------------------------

def test_bf16_rounding_known_values():
    u = 2.0 ** -7                       # bf16 spacing at 1.0
    cases = {
        1.0 + u / 2: 1.0,               # tie -> even (mantissa 0)
        1.0 + 3 * u / 2: 1.0 + 2 * u,   # tie -> even (mantissa 2)
        1.0 + u / 2 + 2 ** -20: 1.0 + u,
        -(1.0 + 3 * u / 2): -(1.0 + 2 * u),
        3.4e38: math.inf,               # above the largest bf16 plus half a spacing -> inf
        3.0e38: 226 * 2.0 ** 120,       # 3e38 = 225.69 * 2^120 -> 226 * 2^120
        2.0 ** -133: 2.0 ** -133,       # smallest subnormal bf16
        2.0 ** -135: 0.0,               # below half of it -> 0
        0.0: 0.0,
    }
    for x, want in cases.items():
        assert oracle.round_to(np.array([x]), "bf16")[0] == want, x


def test_bf16_rounding_matches_torch():
    x = (RNG.standard_normal(200000) * np.exp(RNG.uniform(-30, 30, 200000))).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.round_to(x.astype(np.float64), "bf16")
    np.testing.assert_array_equal(got, want)


def test_f32_rounding_matches_numpy():
    x = RNG.standard_normal(100000) * 1e3
    np.testing.assert_array_equal(oracle.round_to(x, "f32"), x.astype(np.float32).astype(np.float64))


def test_synth_bf16_rounding_matches_torch():
    x = RNG.standard_normal(50000).astype(np.float32) * 77
    np.testing.assert_array_equal(synth.to_bf16_values(x),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


# ---- conv2d -----------------------------------------------------------------

def conv_brute(x, w, b, st, pad):
    n, c, h, wd = x.shape
    co, _, kh, kw = w.shape
    ho, wo = (h + 2 * pad - kh) // st + 1, (wd + 2 * pad - kw) // st + 1
    y = np.zeros((n, co, ho, wo))
    for a in range(n):
        for o in range(co):
            for i in range(ho):
                for j in range(wo):
                    s = b[o]
                    for ci in range(c):
                        for r in range(kh):
                            for q in range(kw):
                                hi, wi = i * st - pad + r, j * st - pad + q
                                if 0 <= hi < h and 0 <= wi < wd:
                                    s += w[o, ci, r, q] * x[a, ci, hi, wi]
                    y[a, o, i, j] = s
    return y


@pytest.mark.parametrize("k,st,pad", [(1, 1, 0), (3, 1, 1), (3, 2, 1), (7, 2, 3), (1, 2, 0), (2, 2, 0)])
def test_conv2d_brute_force(k, st, pad):
    x, w, b = rnd(2, 3, 9, 8), rnd(4, 3, k, k), rnd(4)
    np.testing.assert_allclose(oracle.conv2d(x, w, b, st, pad), conv_brute(x, w, b, st, pad), rtol=1e-13, atol=1e-13)


def test_conv2d_torch_relu_residual():
    x, w, b = rnd(2, 16, 14, 14), rnd(32, 16, 3, 3), rnd(32)
    res = rnd(2, 32, 7, 7)
    y = oracle.conv2d(x, w, b, 2, 1, act="relu", res=res)
    t = F.relu(F.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b), 2, 1) + torch.from_numpy(res))
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-12, atol=1e-12)


def test_conv2d_rounds_once_to_bf16():
    x, w, b = rnd(1, 8, 6, 6), rnd(8, 8, 3, 3), rnd(8)
    y = oracle.conv2d(x, w, b, 1, 1, rnd="bf16")
    y64 = oracle.conv2d(x, w, b, 1, 1)
    np.testing.assert_array_equal(y, torch.from_numpy(y64).to(torch.bfloat16).double().numpy())


# ---- pooling, linear, activations --------------------------------------------

@pytest.mark.parametrize("k,st,pad", [(2, 2, 0), (3, 2, 1)])
def test_maxpool_torch(k, st, pad):
    x = rnd(2, 5, 11, 12)
    np.testing.assert_array_equal(oracle.maxpool2d(x, k, st, pad),
                                  F.max_pool2d(torch.from_numpy(x), k, st, pad).numpy())


def test_maxpool_all_negative_padding_is_minus_inf():
    x = -np.abs(rnd(1, 1, 4, 4)) - 1.0
    y = oracle.maxpool2d(x, 3, 2, 1)
    assert y[0, 0, 0, 0] == x[0, 0, :2, :2].max()


def test_avgpool_mean():
    x = rnd(3, 7, 5, 6)
    np.testing.assert_allclose(oracle.avgpool_global(x), x.mean(axis=(2, 3)), rtol=1e-13)


@pytest.mark.parametrize("act", ["none", "relu", "gelu"])
def test_linear_numpy(act):
    x, w, b, res = rnd(5, 37), rnd(11, 37), rnd(11), rnd(5, 11)
    y = oracle.linear(x, w, b, act=act, res=res)
    v = x @ w.T + b + res
    if act == "relu":
        v = np.maximum(v, 0)
    elif act == "gelu":
        v = F.gelu(torch.from_numpy(v), approximate="none").numpy()
    np.testing.assert_allclose(y, v, rtol=1e-12, atol=1e-12)


def test_linear_flattens_nchw():
    x, w, b = rnd(2, 3, 4, 5), rnd(6, 60), rnd(6)
    np.testing.assert_allclose(oracle.linear(x, w, b), x.reshape(2, -1) @ w.T + b, rtol=1e-12)


def test_gelu_closed_form_points():
    # gelu(0) = 0, gelu(x) -> x for large x, gelu(-x) = -x + gelu(x)
    x = np.array([[0.0, 6.0, -6.0, 1.0, -1.0]])
    y = oracle.linear(x.T, np.ones((1, 1)), np.zeros(1), act="gelu")[:, 0]
    assert y[0] == 0.0
    assert abs(y[1] - 6.0) < 1e-8 and abs(y[2]) < 1e-8
    assert abs((y[3] - y[4]) - 1.0) < 1e-15
    assert abs(y[3] - 0.8413447460685429) < 1e-15   # Phi(1) = 0.841344746...


# ---- layer norm, attention, embeddings ----------------------------------------

def test_layernorm_torch():
    x, res, g, be = rnd(6, 48), rnd(6, 48), rnd(48), rnd(48)
    y = oracle.layernorm(x, g, be, 1e-12, res=res)
    t = F.layer_norm(torch.from_numpy(x + res), (48,), torch.from_numpy(g), torch.from_numpy(be), 1e-12)
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-11, atol=1e-11)


def test_layernorm_invariants():
    x = rnd(4, 32) * 5 + 3
    y = oracle.layernorm(x, np.ones(32), np.zeros(32), 0.0)
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-13)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1, atol=1e-12)


def test_attention_torch_sdpa():
    b, s, h, d = 2, 9, 3, 8
    qkv = rnd(b, s, 3 * h * d)
    y = oracle.attention(qkv, h, 1 / math.sqrt(d))
    t = torch.from_numpy(qkv).view(b, s, 3, h, d).permute(2, 0, 3, 1, 4)
    o = F.scaled_dot_product_attention(t[0], t[1], t[2])
    np.testing.assert_allclose(y, o.permute(0, 2, 1, 3).reshape(b, s, h * d).numpy(), rtol=1e-11, atol=1e-12)


def test_attention_uniform_keys_average_values():
    # identical keys -> uniform softmax -> output = mean of the values
    b, s, h, d = 1, 5, 2, 4
    qkv = rnd(b, s, 3 * h * d)
    qkv[:, :, h * d:2 * h * d] = qkv[:, :1, h * d:2 * h * d]
    y = oracle.attention(qkv, h, 0.5)
    np.testing.assert_allclose(y[0], np.broadcast_to(qkv[0, :, 2 * h * d:].mean(axis=0), (s, h * d)), rtol=1e-12)


def test_embed_bert():
    ids = RNG.integers(0, 50, size=(2, 7)).astype(np.int32)
    tok, pos, typ, g, be = rnd(50, 16), rnd(10, 16), rnd(2, 16), rnd(16), rnd(16)
    y = oracle.embed_bert(ids, tok, pos, typ, g, be, 1e-12)
    v = tok[ids] + pos[None, :7] + typ[0]
    t = F.layer_norm(torch.from_numpy(v), (16,), torch.from_numpy(g), torch.from_numpy(be), 1e-12)
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-11, atol=1e-11)


def test_embed_gather():
    ids = RNG.integers(0, 30, size=(3, 4)).astype(np.int32)
    tab = rnd(30, 5)
    np.testing.assert_array_equal(oracle.embed(ids, tab), tab[ids])


# ---- LSTM ---------------------------------------------------------------------

def test_lstm_torch():
    b, t, e, h = 2, 6, 5, 4
    x = rnd(b, t, e)
    w_ih, w_hh, b_ih, b_hh = rnd(4 * h, e, scale=0.5), rnd(4 * h, h, scale=0.5), rnd(4 * h), rnd(4 * h)
    y = oracle.lstm(x, w_ih, w_hh, b_ih, b_hh)
    m = torch.nn.LSTM(e, h, batch_first=True).double()
    with torch.no_grad():
        m.weight_ih_l0.copy_(torch.from_numpy(w_ih))
        m.weight_hh_l0.copy_(torch.from_numpy(w_hh))
        m.bias_ih_l0.copy_(torch.from_numpy(b_ih))
        m.bias_hh_l0.copy_(torch.from_numpy(b_hh))
        ref, _ = m(torch.from_numpy(x))
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_lstm_bf16_storage_points():
    # h_t rounded to bf16 every step (so the output is bf16-representable)
    b, t, e, h = 1, 4, 3, 2
    y = oracle.lstm(rnd(b, t, e), rnd(4 * h, e), rnd(4 * h, h), rnd(4 * h), rnd(4 * h), rnd="bf16")
    np.testing.assert_array_equal(y, oracle.round_to(y, "bf16"))


# ---- codec ----------------------------------------------------------------------

def test_ae_matches_numpy_and_is_linear():
    x = rnd(2, 16, 3, 5)
    we, be = rnd(2, 16), np.zeros(2)
    c = oracle.ae_encode(x, we, be)
    assert c.shape == (2, 2, 3, 5)                        # C_e = C / R with R = 8
    np.testing.assert_allclose(c, np.einsum("ec,nchw->nehw", we, x), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(oracle.ae_encode(3.0 * x, we, be), 3.0 * c, rtol=1e-12)
    wd, bd = rnd(16, 2), rnd(16)
    y = oracle.ae_decode(c, wd, bd)
    np.testing.assert_allclose(y, np.einsum("ce,nehw->nchw", wd, c) + bd[None, :, None, None], rtol=1e-12)


def test_ae_sequences_per_token():
    x = rnd(2, 3, 24)
    we, be = rnd(3, 24), rnd(3)
    np.testing.assert_allclose(oracle.ae_encode(x, we, be), x @ we.T + be, rtol=1e-12)


def test_ae_identity_weights_round_trip_nonzero():
    # identity encoder/decoder (R = 1) returns the input (zeros aside) -- sanity of the layout
    x = rnd(1, 4, 2, 2)
    eye = np.eye(4)
    y = oracle.ae_decode(oracle.ae_encode(x, eye, np.zeros(4)), eye, np.zeros(4))
    np.testing.assert_array_equal(y, x)


# ---- sub-slicing ----------------------------------------------------------------

def test_subslice_range_matches_array_split():
    for n in [1, 7, 16, 64, 100, 3072]:
        for k in range(1, min(n, 9) + 1):
            sizes = [len(a) for a in np.array_split(np.arange(n), k)]
            got = [oracle.subslice_range(n, k, j) for j in range(k)]
            assert [hi - lo for lo, hi in got] == sizes
            assert got[0][0] == 0 and got[-1][1] == n
            assert all(got[j][1] == got[j + 1][0] for j in range(k - 1))
    with pytest.raises(ValueError):
        oracle.subslice_range(4, 5, 0)


@pytest.mark.parametrize("kind", ["conv", "linear"])
def test_subsliced_op_equals_unsplit_bitwise(kind):
    m = synth.tiny_vgg(hw=16, chans=(8, 8, 16, 16, 24, 24))
    x = synth.make_input(m)
    env = {m.input_tid: oracle.round_to(x, m.dtype)}
    for op in m.ops:
        full = oracle.run_op(m, op, env)
        if op["kind"] == kind:
            for k in (2, 3, 5):
                np.testing.assert_array_equal(oracle.run_op_sliced(m, op, env, k), full)
        env[op["out"]] = full


def test_sliced_raw_equals_unsliced_bitwise():
    m = synth.resnet50(batch=1, hw=32, blocks=(1, 2, 1, 1), widths=(8, 16, 16, 32), n_cls=7)
    x = synth.make_input(m)
    k = [4 if o else 1 for o in [any(op["rd"] for op in m.ops if op["layer"] == li) for li in range(len(m.layers))]]
    y0 = oracle.forward(m, x)
    y1 = oracle.forward(m, x, k=k, cuts=[1, 3, 4])
    np.testing.assert_array_equal(y0, y1)
