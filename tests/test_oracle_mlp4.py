"""Pins of the CPU oracle's 4-layer regression head (Section 4.2, Eq. 2).

y^ = w4 . phi(W3 phi(W2 phi(W1 h + b1) + b2) + b3) + b4 with phi = ReLU,
d -> 2048 -> 512 -> 64 -> 1 in the paper.  The pins are:
* numpy's float64 matrix products over the same widened bits;
* special cases: zero weights; a dead third layer;
* all-positive weights and inputs, where ReLU is the identity and the head
  collapses to one matrix product;
* positive homogeneity of the bias-free network;
* row selection;
* the error-scale output;
* the EMA closed form.
"""
import numpy as np
import pytest

from paper_2510_13668_amd import synth


def _np_chain(x, with_scale=False):
    f = synth.bf16_bits_to_f32 if x.hidden.dtype == np.uint16 else (lambda a: a)
    h = f(x.hidden).astype(np.float64)
    W1, W2, W3 = (f(w).astype(np.float64) for w in (x.w1, x.w2, x.w3))
    b = [np.zeros(W.shape[0]) if bb is None else bb.astype(np.float64)
         for W, bb in ((W1, x.b1), (W2, x.b2), (W3, x.b3))]
    a1 = np.maximum(h @ W1.T + b[0], 0.0)
    a2 = np.maximum(a1 @ W2.T + b[1], 0.0)
    a3 = np.maximum(a2 @ W3.T + b[2], 0.0)
    y = a3 @ x.w4.astype(np.float64) + x.b4
    if with_scale:
        return y, np.abs(a3 * x.w4.astype(np.float64)).sum(1) + abs(x.b4)
    return y


def _run(oracle_mod, x, dtype, **kw):
    return oracle_mod.predict_mlp4(x.hidden, x.w1, x.w2, x.w3, x.w4, dtype=dtype, b1=x.b1,
                                   b2=x.b2, b3=x.b3, b4=x.b4, **kw)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("bias", [False, True])
def test_against_numpy_products(oracle_mod, dtype, bias):
    x = synth.make_mlp4(9, (40, 24, 16, 8), dtype=dtype, seed=3, with_bias=bias)
    out = _run(oracle_mod, x, dtype)
    y, scale = _np_chain(x, with_scale=True)
    np.testing.assert_allclose(out["expected"], y, rtol=1e-12, atol=1e-9)
    np.testing.assert_allclose(out["scale"], scale, rtol=1e-12)


def test_zero_weights_and_dead_layer(oracle_mod):
    x = synth.make_mlp4(5, (16, 12, 8, 4), dtype=synth.F32, seed=1, with_bias=True)
    z = synth.Mlp4Inputs(x.hidden, x.w1 * 0, x.w2 * 0, x.w3 * 0, x.w4, None, None, None, 123.5)
    np.testing.assert_array_equal(_run(oracle_mod, z, synth.F32)["expected"], 123.5)
    # W3 = 0: a3 = relu(b3) whatever the input
    d = synth.Mlp4Inputs(x.hidden, x.w1, x.w2, x.w3 * 0, x.w4, x.b1, x.b2, x.b3, 7.0)
    expect = float(np.maximum(x.b3.astype(np.float64), 0) @ x.w4.astype(np.float64)) + 7.0
    np.testing.assert_allclose(_run(oracle_mod, d, synth.F32)["expected"], expect, rtol=1e-12)


def test_positive_network_is_one_linear_map(oracle_mod):
    """Non-negative inputs and weights: every ReLU passes its input, so
    y^ = w4 W3 W2 W1 h + b4 (a wrong layer order or a transposed operand
    breaks this)."""
    rng = np.random.default_rng(2)
    d, m1, m2, m3 = 20, 14, 10, 6
    x = synth.Mlp4Inputs(rng.random((4, d), dtype=np.float32), rng.random((m1, d), dtype=np.float32),
                         rng.random((m2, m1), dtype=np.float32), rng.random((m3, m2), dtype=np.float32),
                         rng.random(m3, dtype=np.float32), None, None, None, -3.0)
    M = (x.w4.astype(np.float64) @ x.w3.astype(np.float64) @ x.w2.astype(np.float64)
         @ x.w1.astype(np.float64))
    expect = x.hidden.astype(np.float64) @ M - 3.0
    np.testing.assert_allclose(_run(oracle_mod, x, synth.F32)["expected"], expect, rtol=1e-12)


def test_positive_homogeneity_without_biases(oracle_mod):
    """ReLU networks without biases scale with their input: y(2h) is exactly
    twice y(h) (doubling commutes with every rounding)."""
    x = synth.make_mlp4(6, (32, 16, 8, 4), dtype=synth.F32, seed=5)
    x = synth.Mlp4Inputs(x.hidden, x.w1, x.w2, x.w3, x.w4, None, None, None, 0.0)
    y1 = _run(oracle_mod, x, synth.F32)["expected"]
    x2 = synth.Mlp4Inputs(x.hidden * np.float32(2), x.w1, x.w2, x.w3, x.w4, None, None, None, 0.0)
    y2 = _run(oracle_mod, x2, synth.F32)["expected"]
    np.testing.assert_array_equal(y2, 2 * y1)
    assert (y1 != 0).sum() >= 4


def test_row_selection_and_integerisation(oracle_mod):
    x = synth.make_mlp4(12, (24, 16, 8, 4), dtype=synth.BF16, seed=7, with_bias=True,
                        y_mean=0.0, y_spread=60.0)
    full = _run(oracle_mod, x, synth.BF16, len_max=60)
    rows = np.array([11, 0, 5, 5], np.int64)
    part = _run(oracle_mod, x, synth.BF16, rows=rows, len_max=60)
    np.testing.assert_array_equal(part["expected"], full["expected"][rows])
    y = full["expected"]
    expect = np.clip(np.where(np.rint(y) >= 1, np.rint(y), 1), 1, 60)
    np.testing.assert_array_equal(full["rem_len"], expect.astype(np.int32))
    assert (full["rem_len"] == 1).any() and (full["rem_len"] == 60).any()


def test_ema_closed_form(oracle_mod):
    x = synth.make_mlp4(5, (24, 16, 8, 4), dtype=synth.F32, seed=9, steps=3)
    st = np.zeros(5, np.float64)
    ys = []
    for t in range(3):
        xt = synth.Mlp4Inputs(x.hidden[t], x.w1, x.w2, x.w3, x.w4, None, None, None, x.b4)
        ys.append(_run(oracle_mod, xt, synth.F32, ema_alpha=0.25, ema_init=(t == 0),
                       ema_state=st)["expected"])
    expect = 0.25 * ys[2] + 0.75 * (0.25 * ys[1] + 0.75 * ys[0])
    np.testing.assert_allclose(st, expect, rtol=1e-13)
