"""A model of the HIP kernels' operand rounding, for choosing MFMA passes.

Test-side only (it models the HIP path's arithmetic; it is not part of the
oracle and shares nothing with it).  It evaluates the chunked (UT/WY) form of
the gated delta rule (paper Section 2, Eq. 1, rewritten per 64-token chunk)
in fp64, except that every operand the kernels feed to a bf16 MFMA is rounded
the way the kernels round it: bf16 inputs exactly, fp32 operands (the state
M0, R, Delta and its weighted form, T and P) split into x = hi + lo with
hi = bf16(x) and lo = bf16(x - hi) (both round to nearest even) and
multiplied in the passes a variant names:
    km   K M0        "2": K hi(M0) + K lo(M0)       "1": K hi(M0)
    tr   T R         "3": hi hi + hi lo + lo hi      "2a": hi(T) (hi + lo)(R)
                     "2b": (hi + lo)(T) hi(R)        "1": hi(T) hi(R)
    ktd  K^T Dw      "2": K^T (hi + lo)(Dw)         "1": K^T hi(Dw)
    qm   Q M0        "2": Q (hi + lo)(M0)           "1": Q hi(M0)
    pd   P Delta     "3", "2a", "2b", "1" as for T R (P in the place of T)
With ``fold`` (tail replay, no outputs) the row weights would go into T
before it is split: T~ = diag(e^{G_last - G}) T diag(beta), R~ = V - diag(e^G)
K M0 and Dw = T~ R~ directly; the kernels do not do this, since hi(T~) loses
the exact unit diagonal that hi(T) keeps.  Results are rounded to fp32 where
the kernels hold fp32 (R, Delta, M1) and outputs to the storage dtype
(``out_bf16``).  The model covers bf16 inputs (K and Q exact operands).  The
kernels' choice for bf16 inputs is ``KERNEL``: km=2, tr=2a, ktd=2, qm=2, pd=3
(``ALL_PASSES`` is the three-pass form they used before).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

import synth

C = 64


@dataclass(frozen=True)
class Passes:
    km: str = "2"
    tr: str = "3"
    ktd: str = "2"
    qm: str = "2"
    pd: str = "3"
    fold: bool = False


ALL_PASSES = Passes()
KERNEL = Passes(tr="2a")


def _f32(x):
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)


def _bf16(x32):
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.asarray(x32, np.float32))).astype(np.float64)


def split(x):
    """fp32 value -> (hi, lo) bf16 parts, as float64."""
    x32 = np.asarray(x, np.float64).astype(np.float32)
    hi = _bf16(x32)
    lo = _bf16((x32.astype(np.float64) - hi).astype(np.float32))
    return hi, lo


def _mm_exact_split(a, b_split, mode):
    """a (exact bf16) times b (split): "2" both parts, "1" hi only."""
    bh, bl = b_split
    return a @ bh + (a @ bl if mode == "2" else 0.0)


def _mm_split_split(a_split, b_split, mode):
    ah, al = a_split
    bh, bl = b_split
    out = ah @ bh
    if mode not in ("3", "2a", "2b", "1"):
        raise ValueError(f"unknown pass mode {mode!r}")
    if mode in ("3", "2a"):
        out = out + ah @ bl
    if mode in ("3", "2b"):
        out = out + al @ bh
    return out


def run(k, v, g, beta, q=None, m0=None, scale=1.0, passes: Passes = KERNEL, out_bf16=True):
    """One (sequence, value head): k, q [T, d_k], v [T, d_v] (exact stored
    values), g, beta [T].  Returns (outputs [T, d_v] or None, final state
    M [d_k, d_v])."""
    for mode in (passes.km, passes.ktd, passes.qm):
        if mode not in ("2", "1"):
            raise ValueError(f"unknown pass mode {mode!r}")
    k, v, g, beta = (np.asarray(x, np.float64) for x in (k, v, g, beta))
    T, dk = k.shape
    dv = v.shape[1]
    M = np.zeros((dk, dv)) if m0 is None else _f32(m0)
    outs = np.zeros((T, dv)) if q is not None else None
    tri_strict = np.tril(np.ones((C, C)), -1)
    tri_incl = np.tril(np.ones((C, C)))
    for c0 in range(0, T, C):
        n = min(C, T - c0)
        K = np.zeros((C, dk))
        V = np.zeros((C, dv))
        gg = np.zeros(C)
        bb = np.zeros(C)
        K[:n], V[:n], gg[:n], bb[:n] = k[c0:c0 + n], v[c0:c0 + n], g[c0:c0 + n], beta[c0:c0 + n]
        G = np.cumsum(gg)
        L = np.exp(np.minimum(G[:, None] - G[None, :], 0.0))
        A = bb[:, None] * (K @ K.T) * L * tri_strict
        Tm = _f32(np.linalg.inv(np.eye(C) + A))
        ms = split(M)
        KM = _mm_exact_split(K, ms, passes.km)
        w = np.exp(G[-1] - G)
        if passes.fold and q is None:
            Tw = _f32(w[:, None] * Tm * bb[None, :])
            R = _f32(V - np.exp(G)[:, None] * KM)
            Dw = _f32(_mm_split_split(split(Tw), split(R), passes.tr))
            M = _f32(np.exp(G[-1]) * M + _mm_exact_split(K.T, split(Dw), passes.ktd))
            continue
        R = _f32(bb[:, None] * V - (bb * np.exp(G))[:, None] * KM)
        D = _f32(_mm_split_split(split(Tm), split(R), passes.tr))
        if q is not None:
            Q = np.zeros((C, dk))
            Q[:n] = np.asarray(q, np.float64)[c0:c0 + n]
            P = _f32(scale * (Q @ K.T) * L * tri_incl)
            QM = _mm_exact_split(Q, ms, passes.qm)
            O = _f32(scale * np.exp(G)[:, None] * QM + _mm_split_split(split(P), split(D), passes.pd))
            outs[c0:c0 + n] = _bf16(O[:n]) if out_bf16 else O[:n]
        Dw = w[:, None] * D
        M = _f32(np.exp(G[-1]) * M + _mm_exact_split(K.T, split(Dw), passes.ktd))
    return outs, M
