"""Which MFMA passes the bf16 scan may drop (CPU only).

The scan multiplies fp32 operands split into bf16 hi + lo parts.  Using the
model of exactly those roundings (tests/precision_model.py), checked against
the fp64 oracle: the passes the kernels use for bf16 inputs (hi(T) alone in
T R, every other product with both parts) keep the state within 1e-3 relative
of the exact recurrence across gate scales 0 to 0.5 with beta up to 1, and the
outputs within their bar; dropping hi(M0)'s partner in K M0, or the lo part
of Delta in K^T Delta, does not (each passes 1e-3 in some case), which is why
those passes stay.  Folding the row weights beta and e^{G_last - G} into T
before taking hi(T) also does (its diagonal is no longer exact in bf16).
The rounding model itself is anchored by the GPU test
that compares the kernels' measured error with the model's prediction.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from tests import precision_model as pm

SHAPE = synth.Shape(hk=2, hv=4, dk=128, dv=128, dtype="bf16")


def _head(r, gate_scale, beta_scale, h=1, seed=0):
    t = synth.tokens(400 + seed, 0, 0, 0, r, SHAPE, gate_scale=gate_scale)
    t = dataclasses.replace(t, beta=(t.beta * beta_scale).astype(np.float32))
    ex = synth.pack([t]).exact()
    kh = h // 2
    return ex["k"][:, kh], ex["v"][:, h], ex["g"][:, h], ex["beta"][:, h], ex["q"][:, kh]


def _errors(r, gate_scale, beta_scale, passes, outputs=False):
    k, v, g, b, q = _head(r, gate_scale, beta_scale)
    cu = np.array([0, r])
    w_o, w = oracle.recurrence(k[:, None], v[:, None], g[:, None], b[:, None], cu,
                               q=q[:, None] if outputs else None)
    o, m = pm.run(k, v, g, b, q=q if outputs else None, passes=passes)
    e_state = np.linalg.norm(m - w[0, 0]) / np.linalg.norm(w[0, 0])
    e_out = np.linalg.norm(o - w_o[:, 0]) / np.linalg.norm(w_o[:, 0]) if outputs else 0.0
    return e_state, e_out


def test_split_identity():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(10000).astype(np.float32)
    hi, lo = pm.split(x)
    assert np.all(np.abs(x - hi - lo) <= 2.0 ** -16 * np.abs(x))
    assert np.array_equal(hi, pm.split(hi)[0]) and np.all(pm.split(hi)[1] == 0)


def test_all_passes_track_the_oracle():
    # the three-pass form only leaves fp32-level rounding
    e_state, e_out = _errors(640, 0.1, 1.0, pm.ALL_PASSES, outputs=True)
    assert e_state < 2e-5
    assert e_out < 3e-3          # dominated by rounding the outputs to bf16


@pytest.mark.parametrize("gate_scale,beta_scale", [(0.0, 1.0), (0.002, 1.0), (0.02, 1.0), (0.1, 1.0),
                                                   (0.5, 1.0), (0.002, 0.1)])
def test_kernel_passes_stay_within_1e3(gate_scale, beta_scale):
    e_state, e_out = _errors(1600, gate_scale, beta_scale, pm.KERNEL, outputs=True)
    print(f"[passes] gate {gate_scale} beta x{beta_scale}: state {e_state:.2e} out {e_out:.2e}")
    assert e_state <= 1e-3
    assert e_out <= 3e-3


@pytest.mark.parametrize("name,passes", [("K M0 with hi(M0) alone", pm.Passes(tr="2a", km="1")),
                                         ("K^T Delta with hi(Delta) alone", pm.Passes(tr="2a", ktd="1")),
                                         ("row weights folded into hi(T)", pm.Passes(tr="2a", fold=True))])
def test_dropping_another_pass_exceeds_1e3(name, passes):
    e_state, _ = _errors(3277, 0.0, 1.0, passes)
    assert e_state > 1e-3, name


def test_unknown_pass_mode_is_rejected():
    k, v, g, b, _ = _head(64, 0.1, 1.0)
    with pytest.raises(ValueError):
        pm.run(k, v, g, b, passes=pm.Passes(tr="2t"))
