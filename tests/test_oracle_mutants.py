"""Planted mistakes in a copy of the oracle's recurrence must each break a pin.

This shows the pins of ``tests/pins.py`` are strong enough: a dropped term, a
wrong sign, a transposed operand, a wrong index or a wrong gate form anywhere
in the recurrence fails at least one of them.  The mistakes are planted in
pure-Python copies on the CPU; the real oracle is untouched.
"""
import numpy as np
import pytest

from tests import pins


def _unit_with(bug):
    def unit(k, v, g, beta, q, M0, scale):
        L, dk = k.shape
        dv = v.shape[1]
        M = np.zeros((dk, dv)) if (M0 is None or bug == "ignores_state_in") else np.array(M0)
        o = None if q is None else np.zeros((L, dv))
        steps = L - 1 if (bug == "drops_last_token" and L > 0) else L
        for t in range(steps):
            a = 1.0 + g[t] if bug == "linear_gate" else np.exp(g[t])
            b = beta[t]
            if bug == "transposed_recall":
                p = M @ k[t]
            else:
                p = k[t] @ M
            if bug == "recall_without_gate":
                w = b * (v[t] - p)
            elif bug == "recall_sign":
                w = b * (v[t] + a * p)
            elif bug == "beta_on_value_only":
                w = b * v[t] - a * p
            elif bug == "beta_squared":
                w = b * b * (v[t] - a * p)
            else:
                w = b * (v[t] - a * p)
            prev = M
            if bug == "no_decay":
                M = M + np.outer(k[t], w)
            elif bug == "rank1_transposed":
                M = a * M + np.outer(w, k[t])
            elif bug == "gate_after_write":
                M = a * (M + np.outer(k[t], w))
            else:
                M = a * M + np.outer(k[t], w)
            if q is not None:
                src = prev if bug == "output_before_update" else M
                vec = k[t] if bug == "output_reads_key" else q[t]
                sc = 1.0 if bug == "no_scale" else scale
                o[t] = sc * (vec @ src)
        return o, M
    return unit


UNIT_BUGS = [
    "recall_without_gate", "recall_sign", "beta_on_value_only", "beta_squared",
    "transposed_recall", "no_decay", "rank1_transposed", "gate_after_write",
    "output_before_update", "output_reads_key", "no_scale", "linear_gate",
    "ignores_state_in", "drops_last_token",
]


def _gqa_modulo():
    """Grouped heads mapped by h % Hk instead of h // (Hv / Hk)."""
    unit = _unit_with(None)

    def fn(k, v, g, beta, cu_seqlens, q=None, state_in=None, scale=1.0):
        k = np.asarray(k)
        v = np.asarray(v)
        T, hk, dk = k.shape
        hv, dv = v.shape[1:]
        cu = np.asarray(cu_seqlens)
        n = cu.size - 1
        o = None if q is None else np.zeros((T, hv, dv))
        st = np.zeros((n, hv, dk, dv))
        for s in range(n):
            a, b = int(cu[s]), int(cu[s + 1])
            for h in range(hv):
                kh = h % hk
                M0 = None if state_in is None else np.asarray(state_in)[s, h]
                oh, M = unit(k[a:b, kh], v[a:b, h], np.asarray(g)[a:b, h],
                             np.asarray(beta)[a:b, h],
                             None if q is None else np.asarray(q)[a:b, kh], M0, scale)
                st[s, h] = M
                if q is not None:
                    o[a:b, h] = oh
        return o, st
    return fn


def _carries_across_sequences():
    """Forgets to restart the state at each sequence boundary."""
    unit = _unit_with(None)

    def fn(k, v, g, beta, cu_seqlens, q=None, state_in=None, scale=1.0):
        k = np.asarray(k)
        v = np.asarray(v)
        T, hk, dk = k.shape
        hv, dv = v.shape[1:]
        cu = np.asarray(cu_seqlens)
        n = cu.size - 1
        o = None if q is None else np.zeros((T, hv, dv))
        st = np.zeros((n, hv, dk, dv))
        for h in range(hv):
            kh = h // (hv // hk)
            M = None if state_in is None else np.asarray(state_in)[0, h]
            for s in range(n):
                a, b = int(cu[s]), int(cu[s + 1])
                oh, M = unit(k[a:b, kh], v[a:b, h], np.asarray(g)[a:b, h],
                             np.asarray(beta)[a:b, h],
                             None if q is None else np.asarray(q)[a:b, kh], M, scale)
                st[s, h] = M
                if q is not None:
                    o[a:b, h] = oh
        return o, st
    return fn


MUTANTS = {b: pins.packed_from_unit(_unit_with(b)) for b in UNIT_BUGS}
MUTANTS["gqa_modulo"] = _gqa_modulo()
MUTANTS["carries_across_sequences"] = _carries_across_sequences()


def test_unmutated_copy_passes_every_pin():
    fn = pins.packed_from_unit(_unit_with(None))
    for pin in pins.ALL_PINS:
        pin(fn)


@pytest.mark.parametrize("name", list(MUTANTS))
def test_mutant_breaks_a_pin(name):
    fn = MUTANTS[name]
    broken = []
    for pin in pins.ALL_PINS:
        try:
            pin(fn)
        except (AssertionError, ValueError):
            broken.append(pin.__name__)
    assert broken, f"planted mistake '{name}' passed every pin"
