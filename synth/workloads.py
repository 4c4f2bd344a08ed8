"""The benchmark workloads as seeded cache hits (shapes and sizes only).

A cache hit covers the first ``m`` tokens of a sequence; the replay tail is the
last ``r`` of them, positions [m - r, m), and the new suffix is [m, m + s)
(paper Section 3).  Token values come from ``synth.tokens`` keyed by
(workload id, layer, sequence, block).

  workload 0  one layer, 1 sequence, Hk = Hv = 4, d = 64, float32;
              m = 2048, r = 205, s = 256, gate scale 0.1
  workload 1  one layer with hybrid-LLM head shapes: Hk = 16, Hv = 32,
              d = 128, bf16 q/k/v; m = 8192, r in {410, 819}, s = 512
  workload 2  36 independent layers (shapes of workload 1), m = 32768,
              r = 3277, s = 1024
  workload 3  16 concurrent hits on one layer (shapes of workload 1):
              m uniform on {8192, 16384, 32768}, replay ratio uniform on the
              grid {0.0500, 0.0501, ..., 0.1000}, s uniform on [128, 2048]
  workload 4  one layer (shapes of workload 1), m = 32768: full prefix versus
              tails r in {256, 1024, 1638, 3277}, gate scales {0.02, 0.1, 0.5}
The replay length of workload 3 is derived from (m, ratio) by the caller with
the paper's ceiling rule; this module only draws the ratio.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from fractions import Fraction
from typing import List, Sequence, Tuple

import numpy as np

from . import Shape, Tokens, tokens

SMALL = Shape(hk=4, hv=4, dk=64, dv=64, dtype="f32")
HYBRID = Shape(hk=16, hv=32, dk=128, dv=128, dtype="bf16")
CHUNK = 64


@dataclass(frozen=True)
class Hit:
    workload: int
    layer: int
    seq: int
    m: int          # matched prefix length
    r: int          # replay tail length
    s: int          # new suffix length
    gate_scale: float = 0.1

    def tail(self, shape: Shape) -> Tokens:
        return tokens(self.workload, self.layer, self.seq, self.m - self.r,
                      self.m, shape, self.gate_scale)

    def suffix(self, shape: Shape) -> Tokens:
        return tokens(self.workload, self.layer, self.seq, self.m,
                      self.m + self.s, shape, self.gate_scale)

    def prefix(self, shape: Shape) -> Tokens:
        return tokens(self.workload, self.layer, self.seq, 0, self.m, shape,
                      self.gate_scale)

    def span(self, shape: Shape, start: int, stop: int) -> Tokens:
        return tokens(self.workload, self.layer, self.seq, start, stop, shape,
                      self.gate_scale)


def workload0() -> Tuple[Shape, List[Hit]]:
    return SMALL, [Hit(0, 0, 0, 2048, 205, 256)]


def workload1(r: int = 819) -> Tuple[Shape, List[Hit]]:
    if r not in (410, 819):
        raise ValueError("workload 1 replays 410 or 819 tokens")
    return HYBRID, [Hit(1, 0, 0, 8192, r, 512)]


def workload2(layers: int = 36) -> Tuple[Shape, List[Hit]]:
    return HYBRID, [Hit(2, l, 0, 32768, 3277, 1024) for l in range(layers)]


def workload3_draw(n: int = 16) -> List[Tuple[int, Fraction, int]]:
    """(m, replay ratio, suffix length) for each of the ``n`` hits."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([3])))
    m = rng.choice(np.array([8192, 16384, 32768]), size=n)
    ratio = rng.integers(500, 1001, size=n)
    s = rng.integers(128, 2049, size=n)
    return [(int(m[i]), Fraction(int(ratio[i]), 10000), int(s[i])) for i in range(n)]


def workload3(replay_lengths: List[int]) -> Tuple[Shape, List[Hit]]:
    """Hits of workload 3 given the replay length of each (same order as the draw)."""
    draw = workload3_draw(len(replay_lengths))
    return HYBRID, [Hit(3, 0, i, m, r, s) for i, ((m, _, s), r) in
                    enumerate(zip(draw, replay_lengths))]


WORKLOAD4_TAILS = (256, 1024, 1638, 3277)
WORKLOAD4_GATE_SCALES = (0.02, 0.1, 0.5)


def workload4(r: int, gate_scale: float) -> Tuple[Shape, Hit]:
    return HYBRID, Hit(4, 0, 0, 32768, r, 0, gate_scale)


def draw_hits(hits: Sequence[Hit], shape: Shape, parts: Sequence[str] = ("tail", "suffix"),
              threads: int = 0) -> List[Tuple[Tokens, ...]]:
    """The named parts ("tail", "suffix", "prefix") of every hit, drawn on a
    pool of threads (NumPy's generators and array kernels release the GIL).
    The values are those of calling the parts one by one."""
    if threads <= 0:
        try:
            threads = len(os.sched_getaffinity(0))
        except AttributeError:
            threads = os.cpu_count() or 1
        threads = min(16, threads)

    def one(h):
        return tuple(getattr(h, p)(shape) for p in parts)

    if threads == 1 or len(hits) <= 1:
        return [one(h) for h in hits]
    with ThreadPoolExecutor(threads) as ex:
        return list(ex.map(one, hits))
