"""Helpers shared by the GPU tests: host arrays -> device tensors, error metrics."""
from __future__ import annotations

import numpy as np
import torch

import oracle

STATE_TOL = 2e-3     # max relative Frobenius error per (sequence, head) state
OUTPUT_TOL = 5e-3    # max relative Frobenius error per (sequence, head) output block


def device_inputs(p, device="cuda:0"):
    """synth.Packed -> dict of device tensors in the storage dtypes."""
    def qkv(a):
        if p.shape.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
        return torch.from_numpy(a).to(device)
    return dict(q=qkv(p.q), k=qkv(p.k), v=qkv(p.v),
                g=torch.from_numpy(p.g).to(device), beta=torch.from_numpy(p.beta).to(device),
                cu=torch.from_numpy(p.cu_seqlens).to(device),
                cu_host=torch.from_numpy(p.cu_seqlens.copy()))


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def oracle_run(p, state_in=None, outputs=False, scale=1.0):
    ex = p.exact()
    return oracle.recurrence(ex["k"], ex["v"], ex["g"], ex["beta"], ex["cu_seqlens"],
                             q=ex["q"] if outputs else None, state_in=state_in, scale=scale)


def state_err(got, want):
    """max over (seq, head) of ||got - want||_F / ||want||_F (absolute if want == 0)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape
    worst = 0.0
    for idx in np.ndindex(*want.shape[:2]):
        den = np.linalg.norm(want[idx])
        num = np.linalg.norm(got[idx] - want[idx])
        worst = max(worst, num / den if den > 0 else num)
    return worst


def output_err(got, want, cu):
    """max over (seq, head) of the relative Frobenius error of the [len, d_v] block."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape
    worst = 0.0
    for n in range(len(cu) - 1):
        a, b = int(cu[n]), int(cu[n + 1])
        if a == b:
            continue
        for h in range(want.shape[1]):
            den = np.linalg.norm(want[a:b, h])
            num = np.linalg.norm(got[a:b, h] - want[a:b, h])
            worst = max(worst, num / den if den > 0 else num)
    return worst
