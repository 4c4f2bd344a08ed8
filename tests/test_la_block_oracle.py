"""The fp64 layer-block oracle (oracle/la_block.py) against facts that hold
independently of it (CPU only).

  * the causal convolution equals NumPy's full convolution with the reversed
    kernel, truncated (a library routine), restarts at every sequence, and
    moves inputs by K - 1 tokens with a one-hot first tap;
  * one token from zero gives the state beta k v^T and the output
    scale beta v (k . q) of the block's own q, k, v (the recurrence receives
    the right columns), with alpha = beta = 1/2 when the gate inputs vanish
    (softplus(0) = ln 2, sigmoid(0) = 1/2);
  * gate parameters away from zero (A_log = (ln 2, ln 3), dt_bias = (1, -1/2),
    zero gate inputs) give g = -exp(A_log) softplus(dt_bias) in closed form
    per head, and two tokens carry that gate into the state as Eq. 1 says;
  * q and k come out with unit norm; g <= 0 and 0 < beta < 1;
  * the gated RMS norm removes any positive scale of o (o is linear in V
    from the zero state), with a worked case of exact decimals;
  * the output is linear in W_out, and vanishes when the z rows of W_in do
    (silu(0) = 0);
  * which weights reach which result: the state ignores the q and z rows,
    w_norm and W_out; beta ignores the a rows and g the b rows; the
    state-only run gives the same state;
  * replaying a tail behind K - 1 zero tokens changes nothing (zero hiddens
    give zero keys and values, so the state stays zero and the convolution
    sees zeros either way): the reading that the conv history restarts with
    the replay.
Each planted mistake below breaks at least one of these.
"""
import numpy as np
import pytest

from oracle import la_block as lb

HK, HV, DK, DV, D, K = 1, 2, 4, 3, 6, 4


def _weights(rng, scale_v=1.0):
    cq, cv = HK * DK, HV * DV
    w_in = rng.standard_normal((2 * cq + 2 * cv + 2 * HV, D)) / np.sqrt(D)
    w_in[2 * cq:2 * cq + cv] *= scale_v
    return dict(w_in=w_in, conv_w=rng.standard_normal((2 * cq + cv, K)) * 0.5,
                a_log=rng.uniform(-1.0, 0.5, HV), dt_bias=rng.uniform(-1.0, 1.0, HV),
                w_norm=rng.uniform(0.5, 1.5, DV), w_out=rng.standard_normal((D, HV * DV)) / np.sqrt(HV * DV))


def _run(x, w, cu, fn=None, **kw):
    fn = fn or lb.la_block
    return fn(x, w["w_in"], w["conv_w"], w["a_log"], w["dt_bias"], w["w_norm"], w["w_out"], cu,
              HK, HV, DK, DV, scale=0.5, **kw)


# ---------------------------------------------------------------- pins (take the block function)

def pin_conv_is_numpy_convolution(conv):
    rng = np.random.default_rng(1)
    cu = np.array([0, 7, 7, 12])
    u = rng.standard_normal((12, 5))
    w = rng.standard_normal((5, K))
    got = conv(u, w, cu)
    for n in range(3):
        a, b = cu[n], cu[n + 1]
        if a == b:
            continue
        for ch in range(5):
            want = np.convolve(u[a:b, ch], w[ch, ::-1])[:b - a]
            np.testing.assert_allclose(got[a:b, ch], want, rtol=1e-12, atol=1e-12)
    onehot = np.zeros((5, K))
    onehot[:, 0] = 1.0
    got = conv(u, onehot, np.array([0, 12]))
    np.testing.assert_allclose(got[K - 1:], u[:12 - (K - 1)], rtol=0, atol=0)
    assert np.all(got[:K - 1] == 0.0)


def pin_single_token(block):
    rng = np.random.default_rng(2)
    w = _weights(rng)
    cq, cv = HK * DK, HV * DV
    w["w_in"][2 * cq + cv:2 * cq + cv + 2 * HV] = 0.0   # a = b = 0
    w["a_log"][:] = 0.0
    w["dt_bias"][:] = 0.0                          # g = -softplus(0) = -ln 2, beta = 1/2
    x = rng.standard_normal((1, D))
    state, out, p = block(x, w["w_in"], w["conv_w"], w["a_log"], w["dt_bias"], w["w_norm"], w["w_out"],
                          np.array([0, 1]), HK, HV, DK, DV, scale=0.5)
    np.testing.assert_allclose(p["g"], -np.log(2.0), rtol=1e-14)
    np.testing.assert_allclose(p["beta"], 0.5, rtol=1e-14)
    for h in range(HV):
        kk, qq, vv = p["k"][0, h * HK // HV], p["q"][0, h * HK // HV], p["v"][0, h]
        np.testing.assert_allclose(state[0, h], 0.5 * np.outer(kk, vv), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(p["o"][0, h], 0.5 * 0.5 * vv * (kk @ qq), rtol=1e-12, atol=1e-15)


def pin_gate_closed_form(block):
    """Gate parameters away from zero: with the a and b rows of W_in zeroed,
    a = b = 0, so beta = 1/2 and g[h] = -exp(A_log[h]) softplus(dt_bias[h])
    exactly.  A_log = (ln 2, ln 3) and dt_bias = (1, -1/2) give
    g = (-2 ln(1 + e), -3 ln(1 + e^{-1/2})).  Two tokens carry the gate into
    the state: M2 = alpha2 (M1 - beta2 k2 (k2^T M1)) + beta2 k2 v2^T with
    M1 = beta1 k1 v1^T, alpha2 = exp(g[h]) (Eq. 1, transposed layout)."""
    rng = np.random.default_rng(11)
    w = _weights(rng)
    cq, cv = HK * DK, HV * DV
    w["w_in"][2 * cq + cv:2 * cq + cv + 2 * HV] = 0.0
    w["a_log"] = np.array([np.log(2.0), np.log(3.0)])
    w["dt_bias"] = np.array([1.0, -0.5])
    want_g = np.array([-2.0 * np.log1p(np.e), -3.0 * np.log1p(np.exp(-0.5))])
    x = rng.standard_normal((2, D))
    state, _, p = _run(x, w, np.array([0, 2]), block)
    np.testing.assert_allclose(p["g"], np.broadcast_to(want_g, (2, HV)), rtol=1e-14)
    np.testing.assert_allclose(p["beta"], 0.5, rtol=1e-14)
    for h in range(HV):
        k1, k2 = p["k"][0, h * HK // HV], p["k"][1, h * HK // HV]
        v1, v2 = p["v"][0, h], p["v"][1, h]
        m1 = 0.5 * np.outer(k1, v1)
        m2 = np.exp(want_g[h]) * (m1 - 0.5 * np.outer(k2, k2 @ m1)) + 0.5 * np.outer(k2, v2)
        np.testing.assert_allclose(state[0, h], m2, rtol=1e-12, atol=1e-15)


def pin_norms_and_gate_ranges(block):
    rng = np.random.default_rng(3)
    w = _weights(rng)
    x = rng.standard_normal((9, D))
    _, _, p = _run(x, w, np.array([0, 4, 9]), block, l2_eps=1e-30)
    np.testing.assert_allclose(np.linalg.norm(p["q"], axis=-1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(p["k"], axis=-1), 1.0, rtol=1e-12)
    assert np.all(p["g"] <= 0.0) and np.all((p["beta"] > 0) & (p["beta"] < 1))


def pin_gated_norm(block):
    """The gated RMS norm removes any positive scale of o (checked through the
    block: o is linear in V from the zero state, so scaling V by 3 after the
    convolution scales o by 3 and leaves the block output alone), and a worked
    case: o = (1, -1, 1, -1) has rms 1, so with w_norm = 2 and z = ln 3
    (silu = 3/4 ln 3) the output is 1.5 ln 3 * o."""
    rng = np.random.default_rng(6)
    w = _weights(rng)
    x = rng.standard_normal((8, D))
    cu = np.array([0, 8])
    _, out, p = _run(x, w, cu, block, norm_eps=1e-30)
    from oracle import recurrence
    o3, _ = recurrence(p["k"], 3.0 * p["v"], p["g"], p["beta"], cu, q=p["q"], scale=0.5)
    np.testing.assert_allclose(o3, 3.0 * p["o"], rtol=1e-12, atol=1e-14)
    y3 = lb.gated_rmsnorm(o3, p["z"].reshape(8, HV, DV), w["w_norm"], 1e-30)
    np.testing.assert_allclose(y3, p["y"], rtol=1e-12, atol=1e-15)
    o = np.array([[1.0, -1.0, 1.0, -1.0]])
    y = lb.gated_rmsnorm(o, np.full((1, 4), np.log(3.0)), np.full(4, 2.0), 0.0)
    np.testing.assert_allclose(y, 1.5 * np.log(3.0) * o, rtol=1e-15)


def pin_out_is_linear_in_w_out(block):
    rng = np.random.default_rng(7)
    w = _weights(rng)
    x = rng.standard_normal((7, D))
    cu = np.array([0, 7])
    _, out1, _ = _run(x, w, cu, block)
    w2 = dict(w, w_out=2.5 * w["w_out"])
    _, out2, _ = _run(x, w2, cu, block)
    np.testing.assert_allclose(out2, 2.5 * out1, rtol=1e-12, atol=1e-14)
    w3 = dict(w, w_out=np.zeros_like(w["w_out"]))
    _, out3, _ = _run(x, w3, cu, block)
    assert np.all(out3 == 0.0)


def pin_zero_prefix_changes_nothing(block):
    rng = np.random.default_rng(8)
    w = _weights(rng)
    x = rng.standard_normal((11, D))
    s1, o1, _ = _run(x, w, np.array([0, 11]), block)
    xz = np.concatenate([np.zeros((K - 1, D)), x])
    s2, o2, _ = _run(xz, w, np.array([0, 11 + K - 1]), block)
    np.testing.assert_allclose(s2, s1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(o2[K - 1:], o1, rtol=1e-12, atol=1e-15)


def pin_zero_gate_silences_output(block):
    """Zero rows of W_in for z give z = 0, silu(0) = 0, so y = 0 and out = 0
    exactly, whatever the state does; zero rows for v give v = 0 and a zero
    state."""
    rng = np.random.default_rng(9)
    w = _weights(rng)
    cq, cv = HK * DK, HV * DV
    w["w_in"][2 * cq + cv + 2 * HV:] = 0.0
    x = rng.standard_normal((6, D))
    s, out, _ = _run(x, w, np.array([0, 6]), block)
    assert np.all(out == 0.0) and np.any(s != 0.0)
    w = _weights(rng)
    w["w_in"][2 * cq:2 * cq + cv] = 0.0
    s, out, _ = _run(x, w, np.array([0, 6]), block)
    assert np.all(s == 0.0)


def pin_what_depends_on_what(block):
    """Which weights reach which result: the state does not see the q or z
    rows of W_in, w_norm or W_out; beta does not see the a rows, g not the b
    rows; and the state-only run (outputs=False) gives the same state."""
    rng = np.random.default_rng(10)
    w = _weights(rng)
    cq, cv = HK * DK, HV * DV
    x = rng.standard_normal((10, D))
    cu = np.array([0, 3, 10])
    s0, _, p0 = _run(x, w, cu, block)
    rows = dict(q=slice(0, cq), a=slice(2 * cq + cv, 2 * cq + cv + HV),
                b=slice(2 * cq + cv + HV, 2 * cq + cv + 2 * HV), z=slice(2 * cq + cv + 2 * HV, None))
    for name in ("q", "z"):
        w1 = dict(w, w_in=w["w_in"].copy())
        w1["w_in"][rows[name]] = rng.standard_normal(w1["w_in"][rows[name]].shape)
        s1, _, _ = _run(x, w1, cu, block)
        assert np.array_equal(s1, s0), name
    w1 = dict(w, w_norm=2.0 * w["w_norm"], w_out=-w["w_out"])
    s1, _, _ = _run(x, w1, cu, block)
    assert np.array_equal(s1, s0)
    for name, kept in (("a", "beta"), ("b", "g")):
        w1 = dict(w, w_in=w["w_in"].copy())
        w1["w_in"][rows[name]] += 1.0
        _, _, p1 = _run(x, w1, cu, block)
        assert np.array_equal(p1[kept], p0[kept]), name
        other = "g" if kept == "beta" else "beta"
        assert not np.allclose(p1[other], p0[other]), name
    s2, out2, _ = _run(x, w, cu, block, outputs=False)
    assert out2 is None
    np.testing.assert_allclose(s2, s0, rtol=1e-13, atol=1e-15)


BLOCK_PINS = [pin_what_depends_on_what, pin_single_token, pin_gate_closed_form, pin_norms_and_gate_ranges,
              pin_gated_norm,
              pin_out_is_linear_in_w_out, pin_zero_prefix_changes_nothing,
              pin_zero_gate_silences_output]


def test_conv_pin():
    pin_conv_is_numpy_convolution(lb.causal_conv)


@pytest.mark.parametrize("pin", BLOCK_PINS, ids=lambda p: p.__name__)
def test_block_pin(pin):
    pin(lb.la_block)


def test_activation_identities():
    np.testing.assert_allclose(lb.softplus(0.0), np.log(2.0), rtol=1e-15)
    np.testing.assert_allclose(lb.softplus(800.0), 800.0, rtol=1e-15)
    np.testing.assert_allclose(lb.sigmoid(0.0), 0.5, rtol=0)


# ---------------------------------------------------------------- planted mistakes

def _mutant_conv_unreversed(u, w, cu):
    return lb.causal_conv(u, w[:, ::-1], cu)


def _mutant_conv_no_restart(u, w, cu):
    return lb.causal_conv(u, w, np.array([0, u.shape[0]]))


def _block_with(**over):
    def block(x, w_in, conv_w, a_log, dt_bias, w_norm, w_out, cu, hk, hv, dk, dv, scale, norm_eps=1e-6,
              l2_eps=1e-6, outputs=True):
        saved = {k: getattr(lb, k) for k in over}
        try:
            for k, v in over.items():
                setattr(lb, k, v)
            return lb.la_block(x, w_in, conv_w, a_log, dt_bias, w_norm, w_out, cu, hk, hv, dk, dv, scale,
                               norm_eps, l2_eps, outputs)
        finally:
            for k, v in saved.items():
                setattr(lb, k, v)
    return block


_conv = lb.causal_conv


def _shifted_conv(u, w, cu):   # off by one token
    c = _conv(u, w, cu)
    out = np.zeros_like(c)
    out[1:] = c[:-1]
    return out


def _rows_read_as(order):
    """The block reading W_in's row blocks in another order (a slicing mistake)."""
    def block(x, w_in, *args, **kw):
        cq, cv = HK * DK, HV * DV
        spans = dict(q=(0, cq), k=(cq, 2 * cq), v=(2 * cq, 2 * cq + cv), a=(2 * cq + cv, 2 * cq + cv + HV),
                     b=(2 * cq + cv + HV, 2 * cq + cv + 2 * HV), z=(2 * cq + cv + 2 * HV, 2 * cq + 2 * cv + 2 * HV))
        # sizes follow the true order; contents come from `order`'s reading of the rows
        flat = np.concatenate([w_in[slice(*spans[n])] for n in order])
        return lb.la_block(x, flat, *args, **kw)
    return block


MUTANTS = {
    "conv taps not reversed": ("conv", _mutant_conv_unreversed),
    "conv history across sequences": ("conv", _mutant_conv_no_restart),
    "conv off by one token": ("block", _block_with(causal_conv=_shifted_conv)),
    "gate sign": ("block", _block_with(softplus=lambda x: -np.logaddexp(0.0, x))),
    "beta without sigmoid": ("block", _block_with(sigmoid=lambda x: np.clip(x, 1e-3, 0.999))),
    "silu as identity": ("block", _block_with(silu=lambda x: x)),
    "norm without the rms": ("block", _block_with(gated_rmsnorm=lambda o, z, w, e: o * w * lb.silu(z))),
    "l2 norm missing": ("block", _block_with(l2norm=lambda x, e: x)),
    "gate without exp(A_log)": ("block", _block_with(
        gates=lambda a, b, al, dt: (-lb.softplus(a + np.asarray(dt)[None, :]), lb.sigmoid(b)))),
    "gate with A_log not exponentiated": ("block", _block_with(
        gates=lambda a, b, al, dt: (-np.asarray(al)[None, :] * lb.softplus(a + np.asarray(dt)[None, :]),
                                    lb.sigmoid(b)))),
    "gate with a - dt_bias": ("block", _block_with(
        gates=lambda a, b, al, dt: (-np.exp(np.asarray(al))[None, :] * lb.softplus(a - np.asarray(dt)[None, :]),
                                    lb.sigmoid(b)))),
    "gate with exp(-A_log)": ("block", _block_with(
        gates=lambda a, b, al, dt: (-np.exp(-np.asarray(al))[None, :] * lb.softplus(a + np.asarray(dt)[None, :]),
                                    lb.sigmoid(b)))),
    "gate parameters of the wrong head": ("block", _block_with(
        gates=lambda a, b, al, dt, _g=lb.gates: _g(a, b, np.asarray(al)[::-1], np.asarray(dt)[::-1]))),
    "a and b swapped": ("block", _rows_read_as("qkvbaz")),
    "q and k swapped": ("block", _rows_read_as("kqvabz")),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_catch_planted_mistake(name):
    kind, fn = MUTANTS[name]
    caught = False
    if kind == "conv":
        try:
            pin_conv_is_numpy_convolution(fn)
        except AssertionError:
            caught = True
    else:
        for pin in BLOCK_PINS:
            try:
                pin(fn)
            except AssertionError:
                caught = True
                break
    assert caught, f"no pin caught: {name}"
