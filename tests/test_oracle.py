"""Pins of the CPU oracle against facts that do not come from the oracle:
brute force on tiny inputs, closed forms, delta kernels, hand-computed
examples and independent library routines (torch CPU in float64, numpy).
Each test is chosen so that a plausible slip in the oracle (a dropped bias,
a swapped index, a wrong pad or stride, the residual added on the wrong
side of the activation, a transposed flatten) fails it."""

import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import model as om

RNG = np.random.default_rng(1234)


def brute_conv(x, w, b, s, p):
    """Seven nested loops straight from the definition, in Python floats."""
    n, c, h, wd = x.shape
    o, _, kh, kw = w.shape
    ho, wo = (h + 2 * p - kh) // s + 1, (wd + 2 * p - kw) // s + 1
    y = np.zeros((n, o, ho, wo))
    for nn, oo, pp, qq in itertools.product(range(n), range(o), range(ho),
                                            range(wo)):
        acc = float(b[oo]) if b is not None else 0.0
        for cc, i, j in itertools.product(range(c), range(kh), range(kw)):
            hi, wi = pp * s - p + i, qq * s - p + j
            if 0 <= hi < h and 0 <= wi < wd:
                acc += float(x[nn, cc, hi, wi]) * float(w[oo, cc, i, j])
        y[nn, oo, pp, qq] = acc
    return y


@pytest.mark.parametrize("shape", [
    # n, c, h, w, o, k, s, p
    (2, 3, 5, 5, 4, 3, 1, 1),
    (1, 2, 6, 7, 3, 3, 2, 1),
    (2, 3, 7, 7, 2, 5, 2, 2),
    (1, 4, 4, 4, 5, 1, 2, 0),
    (1, 1, 5, 5, 1, 3, 1, 0),
])
def test_conv_matches_brute_force(shape):
    n, c, h, w, o, k, s, p = shape
    x = RNG.standard_normal((n, c, h, w)).astype(np.float32)
    wt = RNG.standard_normal((o, c, k, k)).astype(np.float32)
    b = RNG.standard_normal(o).astype(np.float32)
    y = oracle.conv2d(x, wt, b, s, p)
    ref = brute_conv(x, wt, b, s, p)
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("shape", [
    (2, 16, 20, 20, 24, 3, 1, 1),
    (1, 3, 37, 37, 16, 7, 2, 3),
    (2, 32, 13, 13, 8, 1, 2, 0),
    (1, 8, 9, 11, 8, 3, 2, 1),
])
def test_conv_matches_torch_float64(shape):
    n, c, h, w, o, k, s, p = shape
    x = RNG.standard_normal((n, c, h, w)).astype(np.float32)
    wt = RNG.standard_normal((o, c, k, k)).astype(np.float32)
    b = RNG.standard_normal(o).astype(np.float32)
    y = oracle.conv2d(x, wt, b, s, p)
    ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(wt).double(),
                   torch.from_numpy(b).double(), stride=s, padding=p).numpy()
    # one rounding to float32 at the end of a double sum
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=1e-6)


def test_conv_centre_delta_is_identity():
    c = 5
    x = RNG.standard_normal((2, c, 6, 6)).astype(np.float32)
    w = np.zeros((c, c, 3, 3), np.float32)
    for i in range(c):
        w[i, i, 1, 1] = 1.0
    assert np.array_equal(oracle.conv2d(x, w, None, 1, 1), x)


def test_conv_stride2_delta_subsamples():
    x = RNG.standard_normal((1, 2, 7, 7)).astype(np.float32)
    w = np.zeros((2, 2, 3, 3), np.float32)
    w[0, 0, 1, 1] = w[1, 1, 1, 1] = 1.0
    y = oracle.conv2d(x, w, None, 2, 1)
    assert y.shape == (1, 2, 4, 4)
    assert np.array_equal(y, x[:, :, ::2, ::2])


def test_conv_shifted_delta_shifts_with_zero_border():
    x = RNG.standard_normal((1, 1, 5, 6)).astype(np.float32)
    w = np.zeros((1, 1, 3, 3), np.float32)
    w[0, 0, 0, 0] = 1.0            # tap (i, j) = (0, 0) reads x[p-1, q-1]
    y = oracle.conv2d(x, w, None, 1, 1)
    ref = np.zeros_like(x)
    ref[:, :, 1:, 1:] = x[:, :, :-1, :-1]
    assert np.array_equal(y, ref)


def test_conv_channel_permutation_delta():
    perm = [2, 0, 3, 1]
    x = RNG.standard_normal((1, 4, 3, 3)).astype(np.float32)
    w = np.zeros((4, 4, 1, 1), np.float32)
    for o, c in enumerate(perm):
        w[o, c, 0, 0] = 1.0
    assert np.array_equal(oracle.conv2d(x, w, None, 1, 0), x[:, perm])


def test_conv_bias_and_power_of_two_linearity():
    x = RNG.standard_normal((1, 3, 6, 6)).astype(np.float32)
    w = RNG.standard_normal((4, 3, 3, 3)).astype(np.float32)
    b = np.array([1.0, -2.0, 0.5, 0.0], np.float32)
    y0 = oracle.conv2d(x, w, None, 1, 1)
    assert np.array_equal(oracle.conv2d(x, 8 * w, None, 1, 1), 8 * y0)
    # a zero input leaves exactly the bias, border included
    yb = oracle.conv2d(np.zeros_like(x), w, b, 1, 1)
    assert np.array_equal(yb, np.broadcast_to(b[None, :, None, None],
                                              yb.shape))


def test_fc_matches_numpy_float64_and_flatten_order():
    x = RNG.standard_normal((3, 50)).astype(np.float32)
    w = RNG.standard_normal((7, 50)).astype(np.float32)
    b = RNG.standard_normal(7).astype(np.float32)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b
    np.testing.assert_allclose(oracle.fc(x, w, b), ref, rtol=2e-7, atol=1e-6)
    # one-hot at (c, h, w) of a C x 7 x 7 map, identity weights: the
    # activation lands at index c*49 + h*7 + w (NCHW flatten)
    layers = [dict(name="fc", op="fc", src0=-1, src1=-1, cin=4 * 49,
                   cout=4 * 49, kh=1, kw=1, stride=1, pad=0, act="none",
                   res=-1, res_mode="add_act", bias=False, bn=False,
                   out=True)]
    params = [{"w": np.eye(4 * 49, dtype=np.float32), "b": None, "bn": None}]
    f = np.zeros((1, 4, 7, 7), np.float32)
    f[0, 2, 3, 5] = 1.0
    y = om.run_model(layers, params, f)[0]
    assert y.shape == (1, 196) and np.argmax(y[0]) == 2 * 49 + 3 * 7 + 5


def test_batchnorm_matches_folded_conv():
    x = RNG.standard_normal((2, 3, 8, 8)).astype(np.float32)
    w = RNG.standard_normal((5, 3, 3, 3)).astype(np.float32)
    gamma = RNG.uniform(0.5, 1.5, 5).astype(np.float32)
    beta = RNG.standard_normal(5).astype(np.float32)
    mean = RNG.standard_normal(5).astype(np.float32)
    var = RNG.uniform(0.5, 2.0, 5).astype(np.float32)
    eps = 1e-5
    layers = [dict(name="c", op="conv", src0=-1, src1=-1, cin=3, cout=5,
                   kh=3, kw=3, stride=1, pad=1, act="none", res=-1,
                   res_mode="add_act", bias=False, bn=True, out=True)]
    p = [{"w": w, "b": None, "bn": (gamma, beta, mean, var, eps)}]
    y = om.run_model(layers, p, x)[0]
    # fold: W' = W * g / sqrt(v + eps), b' = beta - mean * g / sqrt(v + eps)
    sc = gamma.astype(np.float64) / np.sqrt(var.astype(np.float64) + eps)
    wf = w.astype(np.float64) * sc[:, None, None, None]
    bf = beta - mean * sc
    ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(wf),
                   torch.from_numpy(bf), padding=1).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-5, atol=1e-5)


def _one_conv(act, res_mode):
    inp = dict(name="id", op="conv", src0=-1, src1=-1, cin=1, cout=1, kh=1,
               kw=1, stride=1, pad=0, act="none", res=-1, res_mode="add_act",
               bias=False, bn=False, out=False)
    neg = dict(inp, name="neg", src0=0, res=0, act=act, res_mode=res_mode,
               out=True)
    one = {"w": np.ones((1, 1, 1, 1), np.float32), "b": None, "bn": None}
    minus3 = {"w": np.full((1, 1, 1, 1), -3.0, np.float32), "b": None,
              "bn": None}
    return [inp, neg], [one, minus3]


@pytest.mark.parametrize("act,mode,expect", [
    # z = -3 r, r = x: add->act gives act(-2r), act->add gives act(-3r) + r
    ("relu", "add_act", [0.0, 1.0]),      # r = [0.5, -0.5]
    ("relu", "act_add", [0.5, 1.0]),
    ("leaky", "add_act", [-0.1, 1.0]),
    ("leaky", "act_add", [0.35, 1.0]),
])
def test_residual_order_hand_computed(act, mode, expect):
    layers, params = _one_conv(act, mode)
    x = np.array([0.5, -0.5], np.float32).reshape(2, 1, 1, 1)
    y = om.run_model(layers, params, x)[0].reshape(-1)
    np.testing.assert_allclose(y, expect, rtol=1e-6, atol=1e-7)


def _pool_layer(op, k=1, s=1, p=0):
    return [dict(name="p", op=op, src0=-1, src1=-1, cin=2, cout=2, kh=k,
                 kw=k, stride=s, pad=p, act="none", res=-1,
                 res_mode="add_act", bias=False, bn=False, out=True)]


def test_maxpool_constant_ramp_and_neg_inf_padding():
    run = lambda x, k, s, p: om.run_model(_pool_layer("maxpool", k, s, p),
                                          [None], x)[0]
    c = np.full((1, 2, 6, 6), -3.5, np.float32)
    # padding is -inf, so a negative constant survives the border windows
    assert np.array_equal(run(c, 3, 2, 1), np.full((1, 2, 3, 3), -3.5))
    ramp = np.arange(36, dtype=np.float32).reshape(1, 1, 6, 6)
    ramp = np.concatenate([ramp, -ramp], axis=1)
    y = run(ramp, 3, 2, 1)
    # window of output (p, q) covers rows 2p-1..2p+1, cols 2q-1..2q+1
    assert y[0, 0, 0, 0] == 7 and y[0, 0, 2, 2] == 35 and y[0, 0, 1, 2] == 23
    assert y[0, 1, 0, 0] == 0 and y[0, 1, 2, 2] == -21
    y2 = run(ramp, 2, 2, 0)
    assert y2.shape == (1, 2, 3, 3) and y2[0, 0, 0, 0] == 7 \
        and y2[0, 0, 2, 2] == 35


def test_avgpool_constant_and_ramp():
    run = lambda x: om.run_model(_pool_layer("avgpool"), [None], x)[0]
    assert np.array_equal(run(np.full((2, 2, 7, 7), 1.25, np.float32)),
                          np.full((2, 2, 1, 1), 1.25, np.float32))
    ramp = np.arange(49, dtype=np.float32).reshape(1, 1, 7, 7)
    y = run(np.concatenate([ramp, 2 * ramp], axis=1))
    assert y[0, 0, 0, 0] == 24.0 and y[0, 1, 0, 0] == 48.0


def test_upsample_and_concat_one_hot():
    up = [dict(name="u", op="upsample", src0=-1, src1=-1, cin=1, cout=1,
               kh=1, kw=1, stride=1, pad=0, act="none", res=-1,
               res_mode="add_act", bias=False, bn=False, out=True)]
    x = np.zeros((1, 1, 3, 3), np.float32)
    x[0, 0, 1, 2] = 1.0
    y = om.run_model(up, [None], x)[0]
    assert y.shape == (1, 1, 6, 6)
    assert set(zip(*np.nonzero(y[0, 0]))) == {(2, 4), (2, 5), (3, 4), (3, 5)}
    cat = [dict(up[0], out=False),
           dict(up[0], name="c", op="concat", src0=0, src1=-1, out=True)]
    # concat of [upsampled, input]: needs equal spatial size, so concat the
    # upsample with itself through src1 = 0
    cat[1]["src1"] = 0
    z = om.run_model(cat, [None, None], x)[0]
    assert z.shape == (1, 2, 6, 6) and np.array_equal(z[:, :1], y) \
        and np.array_equal(z[:, 1:], y)


def test_leaky_slope_and_relu_values():
    layers = [dict(name="c", op="conv", src0=-1, src1=-1, cin=1, cout=1,
                   kh=1, kw=1, stride=1, pad=0, act="leaky", res=-1,
                   res_mode="add_act", bias=False, bn=False, out=True)]
    p = [{"w": np.ones((1, 1, 1, 1), np.float32), "b": None, "bn": None}]
    x = np.array([-2.0, 3.0], np.float32).reshape(2, 1, 1, 1)
    np.testing.assert_allclose(om.run_model(layers, p, x)[0].ravel(),
                               [-0.2, 3.0], rtol=1e-7)
    layers[0]["act"] = "relu"
    assert np.array_equal(om.run_model(layers, p, x)[0].ravel(), [0.0, 3.0])


def test_round_bf16_ties_to_even():
    v = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5],
                 np.float32)
    r = om.round_bf16(v)
    np.testing.assert_array_equal(r, [1.0, 1.0 + 2 ** -6, 1.0, -2.5])
