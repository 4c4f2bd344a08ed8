"""Seeded synthetic weights and hiddens for one linear-attention layer block.

Serves the oracle side and the HIP side alike and holds none of the block's
arithmetic: it draws random numbers in the ranges such layers are initialised
with, rounds the two projection matrices and the hiddens to bfloat16, and packs
hidden rows by sequence.

Recipe (float64 draws, then the storage dtype):
  * W_in  [2 Hk d_k + 2 Hv d_v + 2 Hv, D] ~ N(0, 1/D), bf16;
  * conv_w [2 Hk d_k + Hv d_v, 4] ~ U(-1/2, 1/2) (a depthwise 4-tap
    convolution's default uniform bound 1/sqrt(4)), fp32;
  * A_log [Hv] = log U(1, 16), fp32;
  * dt_bias [Hv] = softplus^-1(dt), dt = exp U(log 1e-3, log 1e-1), fp32
    (so softplus(a + dt_bias) starts near dt for a near 0);
  * norm_w [d_v] ~ U(1/2, 3/2), fp32;
  * W_out [D, Hv d_v] ~ N(0, 1/(Hv d_v)), bf16;
  * hiddens x [L, D] ~ N(0, 1), bf16, drawn per block of 64 token positions
    from ``SeedSequence([workload, layer, seq, block, 1])`` so any tail of any
    prefix is reproducible without drawing the head.
Weights come from ``SeedSequence([workload, layer, 2])``.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence

import numpy as np

from . import BLOCK, bf16_bits_to_f32, f32_to_bf16_bits

__all__ = ["LayerDims", "layer_weights", "hiddens", "pack_hiddens", "exact_weights"]

CONV_TAPS = 4


@dataclass(frozen=True)
class LayerDims:
    hidden: int
    hk: int
    hv: int
    dk: int
    dv: int

    @property
    def cq(self) -> int:
        return self.hk * self.dk

    @property
    def cv(self) -> int:
        return self.hv * self.dv

    @property
    def in_rows(self) -> int:
        return 2 * self.cq + 2 * self.cv + 2 * self.hv


def layer_weights(workload: int, layer: int, dims: LayerDims) -> dict:
    """Storage arrays: w_in, w_out as uint16 bf16 bits; the rest float32."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([workload, layer, 2])))
    d = dims
    w_in = rng.standard_normal((d.in_rows, d.hidden)) / np.sqrt(d.hidden)
    conv_w = rng.uniform(-0.5, 0.5, (2 * d.cq + d.cv, CONV_TAPS))
    a_log = np.log(rng.uniform(1.0, 16.0, d.hv))
    dt = np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), d.hv))
    dt_bias = dt + np.log(-np.expm1(-dt))
    norm_w = rng.uniform(0.5, 1.5, d.dv)
    w_out = rng.standard_normal((d.hidden, d.cv)) / np.sqrt(d.cv)
    return dict(w_in=f32_to_bf16_bits(w_in.astype(np.float32)),
                conv_w=conv_w.astype(np.float32), a_log=a_log.astype(np.float32),
                dt_bias=dt_bias.astype(np.float32), norm_w=norm_w.astype(np.float32),
                w_out=f32_to_bf16_bits(w_out.astype(np.float32)))


def exact_weights(w: dict) -> dict:
    """float64 copies of exactly the stored weight values."""
    out = {}
    for name, a in w.items():
        out[name] = (bf16_bits_to_f32(a) if a.dtype == np.uint16 else a).astype(np.float64)
    return out


def hiddens(workload: int, layer: int, seq: int, start: int, stop: int, hidden: int) -> np.ndarray:
    """bf16 bits [stop - start, hidden] of token positions [start, stop)."""
    if not 0 <= start <= stop:
        raise ValueError("need 0 <= start <= stop")
    parts = []
    for b in range(start // BLOCK, -(-stop // BLOCK)):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([workload, layer, seq, b, 1])))
        x = rng.standard_normal((BLOCK, hidden))
        lo = max(start - b * BLOCK, 0)
        hi = min(stop - b * BLOCK, BLOCK)
        parts.append(x[lo:hi])
    x = np.concatenate(parts, axis=0) if parts else np.zeros((0, hidden))
    return f32_to_bf16_bits(x.astype(np.float32))


def pack_hiddens(rows: Sequence[np.ndarray], hidden: int):
    """Concatenates per-sequence hidden rows; returns (x [T, D] bf16 bits, cu_seqlens int32)."""
    lens = [r.shape[0] for r in rows]
    cu = np.zeros(len(rows) + 1, np.int64)
    cu[1:] = np.cumsum(lens)
    x = np.concatenate(rows, axis=0) if rows else np.zeros((0, hidden), np.uint16)
    return np.ascontiguousarray(x, dtype=np.uint16), cu.astype(np.int32)
