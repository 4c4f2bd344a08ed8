"""Seeded synthetic inputs for the GDN tail-replay path.

This module serves both the oracle side and the HIP side of every test and of
the benchmark.  It holds none of the method's arithmetic: it only draws random
numbers, shapes them into the distributions of the paper's workloads, rounds
them to the storage dtype and packs sequences.

Recipe (one token block = 64 consecutive token positions of one sequence):
  * the block's values come from
    ``Generator(PCG64(SeedSequence([workload, layer, seq, block])))`` so any
    tail of any prefix is reproducible without drawing the head;
  * draw order per block: q[64,Hk,d_k], k[64,Hk,d_k], v[64,Hv,d_v],
    z_beta[64,Hv], z_g[64,Hv], all standard normal float64;
  * q and k are L2-normalised per (token, head); beta = sigmoid(z_beta);
    g = -softplus(z_g) * gate_scale (so alpha = exp(g) lies in (0, 1]);
  * everything is cast to float32; q, k, v are then rounded to bfloat16
    (round to nearest, ties to even) when the workload stores bf16.
The exact float64 value of every stored number is available through
``Packed.exact()`` so the oracle sees the same bits the GPU receives.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
from scipy.special import expit

BLOCK = 64

__all__ = ["BLOCK", "Shape", "Tokens", "Packed", "tokens", "pack",
           "f32_to_bf16_bits", "bf16_bits_to_f32"]


@dataclass(frozen=True)
class Shape:
    """Head layout of one GDN layer."""
    hk: int          # query/key heads
    hv: int          # value heads (g, beta, state, output)
    dk: int
    dv: int
    dtype: str       # storage dtype of q, k, v, o: "bf16" or "f32"

    def __post_init__(self):
        if self.hv % self.hk:
            raise ValueError("hv must be a multiple of hk")
        if self.dtype not in ("bf16", "f32"):
            raise ValueError("dtype must be 'bf16' or 'f32'")


def f32_to_bf16_bits(x) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    Inputs here are finite, so no NaN handling is needed.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Tokens:
    """Token positions [start, stop) of one sequence, storage dtypes.

    q, k: [L, Hk, d_k]; v: [L, Hv, d_v] -- uint16 bf16 bits or float32;
    g, beta: [L, Hv] float32.
    """
    shape: Shape
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray

    @property
    def length(self) -> int:
        return int(self.k.shape[0])


@dataclass
class Packed:
    """Several sequences packed token-major with ``cu_seqlens`` offsets."""
    shape: Shape
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray
    cu_seqlens: np.ndarray   # int32 [N+1]

    @property
    def num_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def num_seqs(self) -> int:
        return int(self.cu_seqlens.size - 1)

    def _to_f64(self, a):
        if self.shape.dtype == "bf16":
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)

    def exact(self) -> dict:
        """float64 copies of exactly the stored values."""
        return dict(q=self._to_f64(self.q), k=self._to_f64(self.k),
                    v=self._to_f64(self.v), g=self.g.astype(np.float64),
                    beta=self.beta.astype(np.float64),
                    cu_seqlens=self.cu_seqlens.astype(np.int64))


def _block_draw(workload: int, layer: int, seq: int, block: int, shape: Shape):
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([workload, layer, seq, block])))
    q = rng.standard_normal((BLOCK, shape.hk, shape.dk))
    k = rng.standard_normal((BLOCK, shape.hk, shape.dk))
    v = rng.standard_normal((BLOCK, shape.hv, shape.dv))
    zb = rng.standard_normal((BLOCK, shape.hv))
    zg = rng.standard_normal((BLOCK, shape.hv))
    return q, k, v, zb, zg


def tokens(workload: int, layer: int, seq: int, start: int, stop: int,
           shape: Shape, gate_scale: float = 0.1) -> Tokens:
    """Token positions [start, stop) of sequence ``seq`` of ``layer``."""
    if not 0 <= start <= stop:
        raise ValueError("need 0 <= start <= stop")
    parts = []
    for b in range(start // BLOCK, -(-stop // BLOCK)):
        q, k, v, zb, zg = _block_draw(workload, layer, seq, b, shape)
        lo = max(start - b * BLOCK, 0)
        hi = min(stop - b * BLOCK, BLOCK)
        parts.append((q[lo:hi], k[lo:hi], v[lo:hi], zb[lo:hi], zg[lo:hi]))
    if parts:
        q, k, v, zb, zg = (np.concatenate(x, axis=0) for x in zip(*parts))
    else:
        q = np.zeros((0, shape.hk, shape.dk))
        k = np.zeros((0, shape.hk, shape.dk))
        v = np.zeros((0, shape.hv, shape.dv))
        zb = np.zeros((0, shape.hv))
        zg = np.zeros((0, shape.hv))
    q = q / np.linalg.norm(q, axis=-1, keepdims=True)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    beta = expit(zb)
    g = -np.logaddexp(0.0, zg) * gate_scale
    q32, k32, v32 = (x.astype(np.float32) for x in (q, k, v))
    if shape.dtype == "bf16":
        q32, k32, v32 = (f32_to_bf16_bits(x) for x in (q32, k32, v32))
    return Tokens(shape, q32, k32, v32, g.astype(np.float32), beta.astype(np.float32))


def pack(seqs: Sequence[Tokens], shape: Optional[Shape] = None) -> Packed:
    """Concatenates sequences token-major; ``cu_seqlens`` marks the boundaries."""
    if shape is None:
        if not seqs:
            raise ValueError("pack() of no sequences needs a shape")
        shape = seqs[0].shape
    for s in seqs:
        if s.shape != shape:
            raise ValueError("all sequences must share one shape")
    lens = [s.length for s in seqs]
    cu = np.zeros(len(seqs) + 1, np.int64)
    cu[1:] = np.cumsum(lens)
    if cu[-1] >= 2 ** 31:
        raise ValueError("too many tokens for int32 offsets")
    sd = np.uint16 if shape.dtype == "bf16" else np.float32

    def cat(name, tail_shape, dt):
        arrs = [getattr(s, name) for s in seqs]
        if not arrs:
            return np.zeros((0,) + tail_shape, dt)
        return np.ascontiguousarray(np.concatenate(arrs, axis=0))

    return Packed(shape,
                  cat("q", (shape.hk, shape.dk), sd),
                  cat("k", (shape.hk, shape.dk), sd),
                  cat("v", (shape.hv, shape.dv), sd),
                  cat("g", (shape.hv,), np.float32),
                  cat("beta", (shape.hv,), np.float32),
                  cu.astype(np.int32))
