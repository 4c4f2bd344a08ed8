"""Oracle for the Gated DeltaNet tail-replay hot path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls anything here, and nothing
here imports the product package.

Contents
--------
``recurrence``   the fp64 token-by-token GDN recurrence (paper Section 2,
                 Eq. 1), compiled C with OpenMP over independent
                 (sequence, value head) units.  With ``state_in=None`` over a
                 tail of the matched prefix it is Independent Tail-Replay
                 (paper Section 3, Eq. 2): the replay starts from a zero state.
``replay_len``   the replay budget k = ceil(r * m) (paper Section 3), exact
                 integer arithmetic.
``reference``    NumPy forms used to pin the recurrence: the explicit product
                 formula, the transition product, and the chunked (UT/WY)
                 rewrite that the GPU kernels implement.

Layouts (all float64, C-contiguous):
    q, k      [T, Hk, d_k]        packed varlen tokens, token-major
    v         [T, Hv, d_v]
    g, beta   [T, Hv]             g = log alpha (alpha = exp(g))
    state     [N, Hv, d_k, d_v]   M = S^T of the paper's S in R^{d_v x d_k}
    o         [T, Hv, d_v]        o_t = scale * S_t q_t (after the update)
Value head h reads key/query head h // (Hv // Hk).
"""
from __future__ import annotations

import ctypes
import os
from fractions import Fraction

import numpy as np

from . import build as _build

__all__ = ["recurrence", "replay_len", "max_threads", "library_path"]

_LIB = None


def library_path() -> str:
    return _build.LIB_PATH


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB_PATH):
            _build.build()
        lib = ctypes.CDLL(_build.LIB_PATH)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.gdn_oracle_recurrence.argtypes = [
            i32, i32, i32, i32, i32, P, P, P, P, P, P, P, ctypes.c_double, P, P, i32]
        lib.gdn_oracle_recurrence.restype = ctypes.c_int
        lib.gdn_oracle_max_threads.argtypes = []
        lib.gdn_oracle_max_threads.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def max_threads() -> int:
    """Threads the oracle uses when ``nthreads`` is not given."""
    return int(_lib().gdn_oracle_max_threads())


def _f64(x, name, shape=None):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {a.shape}")
    return a


def recurrence(k, v, g, beta, cu_seqlens, q=None, state_in=None, scale=1.0,
               nthreads=None):
    """Gated delta rule, token by token in fp64 (paper Section 2, Eq. 1).

    Returns ``(o, state)``: ``o`` is ``[T, Hv, d_v]`` when ``q`` is given,
    else ``None``; ``state`` is the state after each sequence's last token,
    ``[N, Hv, d_k, d_v]``.  ``state_in=None`` starts every sequence from the
    zero state, which over a tail is Independent Tail-Replay (Section 3,
    Eq. 2).
    """
    k = _f64(k, "k")
    if k.ndim != 3:
        raise ValueError("k must be [T, Hk, d_k]")
    T, hk, dk = k.shape
    v = _f64(v, "v")
    if v.ndim != 3 or v.shape[0] != T:
        raise ValueError("v must be [T, Hv, d_v]")
    hv, dv = v.shape[1], v.shape[2]
    g = _f64(g, "g", (T, hv))
    beta = _f64(beta, "beta", (T, hv))
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64))
    if cu.ndim != 1 or cu.size < 1 or cu[0] != 0 or cu[-1] != T or np.any(np.diff(cu) < 0):
        raise ValueError("cu_seqlens must be non-decreasing, start at 0 and end at T")
    n = cu.size - 1
    if q is not None:
        q = _f64(q, "q", (T, hk, dk))
    if state_in is not None:
        state_in = _f64(state_in, "state_in", (n, hv, dk, dv))
    o = np.zeros((T, hv, dv), np.float64) if q is not None else None
    state = np.zeros((n, hv, dk, dv), np.float64)

    def ptr(a):
        return None if a is None else a.ctypes.data_as(ctypes.c_void_p)

    nt = 0 if nthreads is None else int(nthreads)
    rc = _lib().gdn_oracle_recurrence(
        n, hk, hv, dk, dv, ptr(cu), ptr(q), ptr(k), ptr(v), ptr(g), ptr(beta),
        ptr(state_in), float(scale), ptr(o), ptr(state), nt)
    if rc != 0:
        raise ValueError(f"gdn_oracle_recurrence rejected its arguments (code {rc})")
    return o, state


def replay_len(m: int, ratio) -> int:
    """Replay budget k = ceil(r * m) of the paper (Section 3), exactly.

    ``ratio`` may be a ``Fraction``, an int, or a decimal string such as
    ``"0.05"``; floats are refused because 0.1 * 8192 rounds up in binary.
    """
    if isinstance(ratio, float):
        raise TypeError("pass the ratio as a Fraction or decimal string, not a float")
    r = Fraction(ratio)
    if m < 0 or r < 0:
        raise ValueError("m and r must be non-negative")
    num = r.numerator * m
    return -(-num // r.denominator)
