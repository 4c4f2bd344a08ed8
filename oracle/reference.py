"""NumPy forms of the GDN recurrence used to pin the oracle -- TEST INFRASTRUCTURE.

Every function works on ONE (sequence, value head) unit in float64:
    k [L, d_k], v [L, d_v], g [L], beta [L], q [L, d_k] or None,
    S0 [d_v, d_k] or None (zero), in the paper's orientation S in R^{d_v x d_k}.

``transition``      T_i = alpha_i (I - beta_i k_i k_i^T)        (Section 2, Eq. 1)
``step_matrix_form`` S_i = S_{i-1} T_i + beta_i v_i k_i^T, with T_i built as an
                    explicit matrix (Eq. 1 with the transition on the key side,
                    the only orientation that is dimensionally valid when
                    d_k != d_v)
``product_formula`` the recurrence unrolled:
                    S_L = S0 prod_{j=1..L} T_j + sum_i beta_i v_i k_i^T prod_{j>i} T_j
``chunked``         the chunked (UT/WY) rewrite the GPU kernels compute: per
                    chunk of C tokens with in-chunk cumulative log-gates G,
                    A = strict_tril(diag(beta) K K^T * exp(G_i - G_j)),
                    T = (I + A)^-1, U = T diag(beta) V, W = T diag(beta e^G) K,
                    Delta = U - W M0, M <- e^{G_C} M0 + K^T diag(e^{G_C - G}) Delta,
                    O = scale (diag(e^G) Q M0 + (Q K^T * L) Delta), M = S^T.
                    It is an exact algebraic rewrite of Eq. 1, so it must equal
                    the recurrence up to rounding for any chunk size.
"""
from __future__ import annotations

import numpy as np
from scipy.linalg import solve_triangular

__all__ = ["transition", "transition_product", "step_matrix_form",
           "product_formula", "chunked"]


def transition(k_i, g_i, beta_i):
    """T_i = alpha_i (I - beta_i k_i k_i^T), alpha_i = exp(g_i)  (Eq. 1)."""
    k_i = np.asarray(k_i, np.float64)
    d = k_i.shape[0]
    return np.exp(g_i) * (np.eye(d) - beta_i * np.outer(k_i, k_i))


def transition_product(k, g, beta):
    """Ordered right product T_1 T_2 ... T_L (identity for L = 0)."""
    k = np.asarray(k, np.float64)
    P = np.eye(k.shape[1])
    for i in range(k.shape[0]):
        P = P @ transition(k[i], g[i], beta[i])
    return P


def step_matrix_form(k, v, g, beta, q=None, S0=None, scale=1.0):
    """Eq. 1 applied token by token with explicit d_k x d_k transition matrices.

    Returns ``(o [L, d_v] or None, S [d_v, d_k])``.
    """
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    L, dk = k.shape
    dv = v.shape[1]
    S = np.zeros((dv, dk)) if S0 is None else np.array(S0, np.float64)
    o = None if q is None else np.zeros((L, dv))
    for i in range(L):
        S = S @ transition(k[i], g[i], beta[i]) + beta[i] * np.outer(v[i], k[i])
        if q is not None:
            o[i] = scale * (S @ np.asarray(q[i], np.float64))
    return o, S


def product_formula(k, v, g, beta, S0=None):
    """Closed form of the unrolled recurrence (brute force, O(L^2 d^3))."""
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    L, dk = k.shape
    dv = v.shape[1]
    S = np.zeros((dv, dk))
    if S0 is not None:
        S = S + np.asarray(S0, np.float64) @ transition_product(k, g, beta)
    for i in range(L):
        tail = transition_product(k[i + 1:], g[i + 1:], beta[i + 1:])
        S = S + beta[i] * np.outer(v[i], k[i]) @ tail
    return S


def chunked(k, v, g, beta, C, q=None, S0=None, scale=1.0):
    """Chunked UT/WY form of Eq. 1 in float64.  Returns ``(o or None, S)``.

    Works in the transposed layout M = S^T (d_k x d_v) like the GPU path.
    Decay factors are only ever formed as exp(G_i - G_j) with i >= j, or as
    exp(G_i) with G_i <= 0, so nothing overflows.
    """
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    g = np.asarray(g, np.float64)
    beta = np.asarray(beta, np.float64)
    L, dk = k.shape
    dv = v.shape[1]
    M = np.zeros((dk, dv)) if S0 is None else np.array(S0, np.float64).T.copy()
    o = None if q is None else np.zeros((L, dv))
    for s in range(0, L, C):
        e = min(s + C, L)
        n = e - s
        K = k[s:e]
        V = v[s:e]
        b = beta[s:e]
        G = np.cumsum(g[s:e])
        lower = np.tril(np.ones((n, n), bool))
        diff = np.where(lower, G[:, None] - G[None, :], -np.inf)
        decay = np.exp(diff)                       # L_ij = e^{G_i - G_j}, j <= i
        A = np.tril(b[:, None] * (K @ K.T) * decay, -1)
        Tm = solve_triangular(np.eye(n) + A, np.eye(n), lower=True,
                              unit_diagonal=True)
        U = Tm @ (b[:, None] * V)
        W = Tm @ ((b * np.exp(G))[:, None] * K)
        D = U - W @ M
        if q is not None:
            Q = np.asarray(q[s:e], np.float64)
            P = (Q @ K.T) * decay
            o[s:e] = scale * (np.exp(G)[:, None] * (Q @ M) + P @ D)
        M = np.exp(G[-1]) * M + K.T @ (np.exp(G[-1] - G)[:, None] * D)
    return o, M.T.copy()
