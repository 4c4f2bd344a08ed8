"""One Gated DeltaNet layer block in fp64 -- TEST INFRASTRUCTURE.

The replay of a whole linear-attention layer (paper Section 3: a group's
linear-attention layers turn the cached full-attention output hiddens of the
tail into k, v, alpha, beta at each replay step, and for the group's last layer
only the linear-attention block runs).  The paper does not print the block; it
is written out here as the usual Gated DeltaNet layer, every step in plain
NumPy on one packed batch of sequences, with the recurrence itself from the
compiled oracle (``oracle.recurrence``, Eq. 1 and Eq. 2):

1. in-projection   P = X W_in^T, columns [q | k | v | a | b | z]
                   (Hk d_k, Hk d_k, Hv d_v, Hv, Hv, Hv d_v);
2. short causal depthwise convolution over the q, k, v channels, K taps,
                   c[t] = sum_j w[:, j] u[t - (K - 1) + j], with u = 0 before
                   each sequence's first token (the conv history restarts with
                   the replay, as the state does), then SiLU;
3. q and k L2-normalised per (token, head): x / sqrt(sum x^2 + eps);
4. beta = sigmoid(b), g = log alpha = -exp(A_log[h]) softplus(a + dt_bias[h]);
5. the recurrence from the zero state, o_t = scale S_t q_t;
6. gated RMS norm per (token, head): y = o / sqrt(mean(o^2) + eps) * w_norm
                   * silu(z);
7. out-projection  out = Y W_out^T.

Layouts (float64; the two projections as linear layers store them,
[out_features, in_features]): X [T, D]; W_in [2 Hk d_k + 2 Hv d_v + 2 Hv, D];
conv_w [2 Hk d_k + Hv d_v, K]; A_log, dt_bias [Hv]; w_norm [d_v];
W_out [D, Hv d_v]; state [N, Hv, d_k, d_v] (M = S^T); out [T, D].
The column order puts everything the state needs (k, v, a, b) in one
contiguous block, so a state-only replay projects onto rows cq .. of W_in
alone.
"""
from __future__ import annotations

import numpy as np

from . import recurrence

__all__ = ["causal_conv", "silu", "softplus", "sigmoid", "l2norm", "gates", "gated_rmsnorm", "la_block"]


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def silu(x):
    return x * sigmoid(x)


def softplus(x):
    # log(1 + e^x) without overflow for large x
    return np.logaddexp(0.0, x)


def causal_conv(u, w, cu_seqlens):
    """Depthwise causal convolution of u [T, C] with w [C, K] per sequence:
    c[t, ch] = sum_{j<K} w[ch, j] u[t - (K - 1) + j, ch], zero before each
    sequence's first token."""
    u = np.asarray(u, np.float64)
    w = np.asarray(w, np.float64)
    T, C = u.shape
    K = w.shape[1]
    out = np.zeros_like(u)
    for n in range(len(cu_seqlens) - 1):
        a, b = int(cu_seqlens[n]), int(cu_seqlens[n + 1])
        for t in range(a, b):
            for j in range(K):
                src = t - (K - 1) + j
                if src >= a:
                    out[t] += w[:, j] * u[src]
    return out


def l2norm(x, eps):
    """x / sqrt(sum x^2 + eps) over the last axis."""
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def gates(a, b, a_log, dt_bias):
    """beta = sigmoid(b), g = log alpha = -exp(A_log) softplus(a + dt_bias), per value head."""
    beta = sigmoid(b)
    g = -np.exp(np.asarray(a_log, np.float64))[None, :] * softplus(a + np.asarray(dt_bias, np.float64)[None, :])
    return g, beta


def gated_rmsnorm(o, z, w_norm, eps):
    """o / sqrt(mean(o^2) + eps) * w_norm * silu(z) over the last axis."""
    return o / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps) * np.asarray(w_norm, np.float64) * silu(z)


def la_block(x, w_in, conv_w, a_log, dt_bias, w_norm, w_out, cu_seqlens, hk, hv, dk, dv,
             scale, norm_eps=1e-6, l2_eps=1e-6, outputs=True):
    """Returns ``(state, out, parts)``: the state after each sequence's last
    token, the block output [T, D] (None when ``outputs`` is False: the
    recurrence then runs without queries and steps 6-7 are skipped) and the
    intermediate tensors by name."""
    x = np.asarray(x, np.float64)
    T = x.shape[0]
    cq, cv = hk * dk, hv * dv
    P = x @ np.asarray(w_in, np.float64).T
    u = P[:, :2 * cq + cv]
    a = P[:, 2 * cq + cv:2 * cq + cv + hv]
    b = P[:, 2 * cq + cv + hv:2 * cq + cv + 2 * hv]
    z = P[:, 2 * cq + cv + 2 * hv:]
    c = silu(causal_conv(u, conv_w, cu_seqlens))
    q = c[:, :cq].reshape(T, hk, dk)
    k = c[:, cq:2 * cq].reshape(T, hk, dk)
    v = c[:, 2 * cq:].reshape(T, hv, dv)
    q = l2norm(q, l2_eps)
    k = l2norm(k, l2_eps)
    g, beta = gates(a, b, a_log, dt_bias)
    o, state = recurrence(k, v, g, beta, cu_seqlens, q=q if outputs else None, scale=scale)
    parts = dict(q=q, k=k, v=v, z=z, g=g, beta=beta, o=o)
    if not outputs:
        return state, None, parts
    y = gated_rmsnorm(o, z.reshape(T, hv, dv), w_norm, norm_eps)
    parts["y"] = y
    out = y.reshape(T, cv) @ np.asarray(w_out, np.float64).T
    return state, out, parts
