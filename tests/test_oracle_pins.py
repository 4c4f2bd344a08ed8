"""The oracle against facts fixed by the paper and by mathematics (CPU only).

Runs every pin of ``tests/pins.py`` on
  * the compiled fp64 oracle (``oracle.recurrence``), the value the GPU is
    compared with, and
  * the NumPy chunked (UT/WY) form at two chunk sizes and the explicit
    matrix form of Eq. 1, so the algorithm the kernels implement is pinned by
    the same facts.
"""
import numpy as np
import pytest

import oracle
from oracle import reference as ref
from tests import pins


def _chunked(C):
    def unit(k, v, g, beta, q, M0, scale):
        o, S = ref.chunked(k, v, g, beta, C, q=q,
                           S0=None if M0 is None else np.asarray(M0).T, scale=scale)
        return o, S.T
    return pins.packed_from_unit(unit)


def _matrix_form(k, v, g, beta, q, M0, scale):
    o, S = ref.step_matrix_form(k, v, g, beta, q=q,
                                S0=None if M0 is None else np.asarray(M0).T, scale=scale)
    return o, S.T


IMPLS = {
    "oracle": oracle.recurrence,
    "chunked4": _chunked(4),
    "chunked16": _chunked(16),
    "matrix_form": pins.packed_from_unit(_matrix_form),
}


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin, impl):
    pin(IMPLS[impl])


def test_oracle_threads_do_not_change_bits():
    rng = np.random.default_rng(5)
    hk, hv, dk, dv = 2, 4, 16, 8
    lens = [33, 0, 70, 5]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    k = rng.standard_normal((T, hk, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    q = rng.standard_normal((T, hk, dk))
    v = rng.standard_normal((T, hv, dv))
    g = -rng.uniform(0, 0.3, (T, hv))
    b = rng.uniform(0, 1, (T, hv))
    o1, s1 = oracle.recurrence(k, v, g, b, cu, q=q, nthreads=1)
    o4, s4 = oracle.recurrence(k, v, g, b, cu, q=q, nthreads=4)
    assert np.array_equal(o1, o4) and np.array_equal(s1, s4)


def test_oracle_rejects_bad_arguments():
    k = np.zeros((4, 1, 2))
    v = np.zeros((4, 3, 2))          # 3 value heads, 1 key head: fine
    g = np.zeros((4, 3))
    with pytest.raises(ValueError):
        oracle.recurrence(k, v, g, g, [0, 5])          # offsets past T
    with pytest.raises(ValueError):
        oracle.recurrence(k, v, g, g, [0, 3, 2, 4])    # decreasing
    with pytest.raises(ValueError):
        oracle.recurrence(k, np.zeros((4, 3, 2)), g, g, [1, 4])
    v2 = np.zeros((4, 3, 2))
    k2 = np.zeros((4, 2, 2))         # Hv % Hk != 0
    with pytest.raises(ValueError):
        oracle.recurrence(k2, v2, g, g, [0, 4])


def test_replay_len_is_the_papers_ceiling():
    # k = ceil(r m), Section 3; exact rational arithmetic.
    assert oracle.replay_len(8192, "0.1") == 820
    assert oracle.replay_len(8192, "0.05") == 410
    assert oracle.replay_len(32768, "0.05") == 1639
    assert oracle.replay_len(32768, "0.1") == 3277
    assert oracle.replay_len(2048, "0.1") == 205
    assert oracle.replay_len(100, "0.1") == 10
    assert oracle.replay_len(0, "0.1") == 0
    assert oracle.replay_len(7, 1) == 7
    with pytest.raises(TypeError):
        oracle.replay_len(8192, 0.1)
    for m in range(1, 300):
        for num in (1, 5, 7, 10, 33):
            r = oracle.replay_len(m, f"{num}/100")
            assert (r - 1) * 100 < num * m <= r * 100
