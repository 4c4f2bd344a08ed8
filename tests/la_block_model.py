"""The layer block's fp64 oracle with the HIP path's storage roundings.

Test-side only (a model of where the GPU path stores bf16; it is not part of
the oracle).  It composes the oracle's own steps (``oracle.la_block``) and
rounds to bf16, round to nearest even, exactly where the block stores bf16:
the in-projection P, the recurrence inputs q, k, v and its output o when the
intermediates are bf16, and always the gated norm's output y (the
out-projection's operand) and the block output.  Everything else is fp64, so
the GPU path and this model differ by fp32 arithmetic alone (and the rare
element whose bf16 rounding flips with it): the states can be held to the
recurrence's own bar and every sequence's outputs, one-token sequences
included, to the output bar.
"""
from __future__ import annotations

import numpy as np

import synth
from oracle import la_block as lb
from oracle import recurrence


def bf16(x):
    x32 = np.asarray(x, np.float64).astype(np.float32)
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x32)).astype(np.float64)


def la_block_rounded(x, w_in, conv_w, a_log, dt_bias, w_norm, w_out, cu_seqlens, hk, hv, dk, dv, scale,
                     act, outputs=True, norm_eps=1e-6, l2_eps=1e-6):
    """``(state, out)`` as ``oracle.la_block`` computes them, with the block's
    bf16 stores; ``act`` is the intermediates' type, "bf16" or "f32"."""
    rnd = bf16 if act == "bf16" else (lambda t: t)
    x = np.asarray(x, np.float64)
    T = x.shape[0]
    cq, cv = hk * dk, hv * dv
    P = rnd(x @ np.asarray(w_in, np.float64).T)
    u = P[:, :2 * cq + cv]
    a = P[:, 2 * cq + cv:2 * cq + cv + hv]
    b = P[:, 2 * cq + cv + hv:2 * cq + cv + 2 * hv]
    z = P[:, 2 * cq + cv + 2 * hv:]
    c = lb.silu(lb.causal_conv(u, conv_w, cu_seqlens))
    q = rnd(lb.l2norm(c[:, :cq].reshape(T, hk, dk), l2_eps))
    k = rnd(lb.l2norm(c[:, cq:2 * cq].reshape(T, hk, dk), l2_eps))
    v = rnd(c[:, 2 * cq:].reshape(T, hv, dv))
    g, beta = lb.gates(a, b, a_log, dt_bias)
    o, state = recurrence(k, v, g, beta, cu_seqlens, q=q if outputs else None, scale=scale)
    if not outputs:
        return state, None
    y = bf16(lb.gated_rmsnorm(rnd(o), z.reshape(T, hv, dv), w_norm, norm_eps))
    out = bf16(y.reshape(T, cv) @ np.asarray(w_out, np.float64).T)
    return state, out
