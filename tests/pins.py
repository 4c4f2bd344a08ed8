"""Pins for the GDN recurrence oracle: facts fixed by the paper or by mathematics.

Each ``pin_*`` takes an implementation ``fn`` with the interface of
``oracle.recurrence``::

    fn(k, v, g, beta, cu_seqlens, q=None, state_in=None, scale=1.0) -> (o, state)

(k [T,Hk,dk], v [T,Hv,dv], g/beta [T,Hv], state [N,Hv,dk,dv] = S^T) and raises
``AssertionError`` when the implementation violates the fact.  The same pins
are run against the oracle (all must hold) and against planted mistakes (each
must break at least one), so together they cover every term of Eq. 1.

Sources of each fact:
  * closed forms of Eq. 1 (paper Section 2) for one and two tokens and for
    one token from a nonzero state (a decode step), a worked
    two-token example with hand-derived decimals, the textbook delta rule
    (alpha = beta = 1), pure decay (beta = 0) and the identity step;
  * Eq. 2 (Section 3): replaying the whole prefix from zero is full prefill;
    the tail error equals S_head times the product of the tail transitions
    and is bounded by ||S_head||_F prod(alpha) when beta ||k||^2 <= 2;
  * the unrolled product formula (brute force), linearity/affinity, grouped
    heads, varlen independence, state hand-off, the per-step norm bound;
  * the chunked (UT/WY) rewrite, an independent algorithm for the same value.
"""
from __future__ import annotations

import numpy as np

from oracle import reference as ref

RTOL = 1e-12


def _rng(seed):
    return np.random.default_rng(seed)


def _unit(rng, *shape):
    x = rng.standard_normal(shape)
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _close(a, b, tol=RTOL, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} != {b.shape}"
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol * scale, f"{what}: max abs err {err:.3e} (scale {scale:.3e})"


def one(fn, k, v, g, beta, q=None, S0=None, scale=1.0):
    """One sequence, one head.  k [L,dk], v [L,dv]; S0 in S orientation [dv,dk].

    Returns (o [L,dv] or None, S [dv,dk]) in the paper's orientation.
    """
    k = np.asarray(k, np.float64)
    L = k.shape[0]
    o, st = fn(k[:, None, :], np.asarray(v, np.float64)[:, None, :],
               np.asarray(g, np.float64)[:, None],
               np.asarray(beta, np.float64)[:, None], np.array([0, L]),
               q=None if q is None else np.asarray(q, np.float64)[:, None, :],
               state_in=None if S0 is None else np.asarray(S0, np.float64).T[None, None],
               scale=scale)
    return (None if o is None else o[:, 0, :]), st[0, 0].T


def _random_unit(rng, L, dk, dv, gate=(-1.0, 0.0)):
    k = _unit(rng, L, dk)
    v = rng.standard_normal((L, dv))
    q = rng.standard_normal((L, dk))
    g = rng.uniform(gate[0], gate[1], L)
    beta = rng.uniform(0.05, 1.0, L)
    return k, v, q, g, beta


# ---------------------------------------------------------------- closed forms

def pin_single_token(fn):
    """From zero, one token gives S = beta v k^T and o = scale beta v (k . q)."""
    rng = _rng(11)
    dk, dv = 3, 5
    k = _unit(rng, 1, dk)
    v = rng.standard_normal((1, dv))
    q = rng.standard_normal((1, dk))
    o, S = one(fn, k, v, [np.log(0.6)], [0.7], q=q, scale=1.3)
    _close(S, 0.7 * np.outer(v[0], k[0]), what="single-token state")
    _close(o[0], 1.3 * 0.7 * v[0] * float(k[0] @ q[0]), what="single-token output")


def pin_worked_example(fn):
    """Eq. 1 worked by hand for d_k = d_v = 2 (exact decimals).

    k1 = (1, 0), v1 = (2, 3), beta1 = 1/2, alpha1 = 1/2;
    k2 = (0.6, 0.8), v2 = (1, -1), beta2 = 1, alpha2 = 1/4.
    S1 = beta1 v1 k1^T = [[1, 0], [1.5, 0]].
    T2 = alpha2 (I - k2 k2^T) = [[0.16, -0.12], [-0.12, 0.09]],
    S1 T2 = [[0.16, -0.12], [0.24, -0.18]], beta2 v2 k2^T = [[0.6, 0.8], [-0.6, -0.8]],
    S2 = [[0.76, 0.68], [-0.36, -0.98]].
    With q1 = (1, 1), q2 = (1, 0): o1 = S1 q1 = (1, 1.5), o2 = S2 q2 = (0.76, -0.36).
    (Applying T on the value side instead would give S2 = [[0.58, 0.8], [-0.585, -0.8]].)
    """
    k = np.array([[1.0, 0.0], [0.6, 0.8]])
    v = np.array([[2.0, 3.0], [1.0, -1.0]])
    q = np.array([[1.0, 1.0], [1.0, 0.0]])
    g = np.log([0.5, 0.25])
    beta = np.array([0.5, 1.0])
    o, S = one(fn, k, v, g, beta, q=q)
    _close(S, [[0.76, 0.68], [-0.36, -0.98]], 1e-14, "worked example state")
    _close(o, [[1.0, 1.5], [0.76, -0.36]], 1e-14, "worked example outputs")


def pin_two_tokens(fn):
    """S2 = alpha2 beta1 v1 k1^T (I - beta2 k2 k2^T) + beta2 v2 k2^T from zero."""
    rng = _rng(12)
    dk, dv = 4, 3
    k = _unit(rng, 2, dk)
    v = rng.standard_normal((2, dv))
    g = np.array([-0.3, -0.7])
    beta = np.array([0.4, 0.9])
    _, S = one(fn, k, v, g, beta)
    a2 = np.exp(g[1])
    want = (a2 * beta[0] * np.outer(v[0], k[0]) @ (np.eye(dk) - beta[1] * np.outer(k[1], k[1]))
            + beta[1] * np.outer(v[1], k[1]))
    _close(S, want, what="two-token state")


def pin_decode_step(fn):
    """One token from a nonzero state (a decode step): S1 = alpha S0 (I - beta k k^T)
    + beta v k^T and o = scale S1 q, for several batched (sequence, head) pairs."""
    rng = _rng(19)
    dk, dv, n, hk, hv = 5, 3, 3, 1, 2
    k = _unit(rng, n, hk, dk)
    q = rng.standard_normal((n, hk, dk))
    v = rng.standard_normal((n, hv, dv))
    g = rng.uniform(-1.0, 0.0, (n, hv))
    beta = rng.uniform(0.05, 1.0, (n, hv))
    M0 = rng.standard_normal((n, hv, dk, dv))          # state = S^T
    o, M = fn(k, v, g, beta, np.arange(n + 1), q=q, state_in=M0, scale=0.7)
    for s in range(n):
        for h in range(hv):
            kk, qq = k[s, 0], q[s, 0]
            S0 = M0[s, h].T
            S1 = (np.exp(g[s, h]) * S0 @ (np.eye(dk) - beta[s, h] * np.outer(kk, kk))
                  + beta[s, h] * np.outer(v[s, h], kk))
            _close(M[s, h].T, S1, what="decode-step state")
            _close(o[s, h], 0.7 * S1 @ qq, what="decode-step output")


def pin_identity_step(fn):
    """alpha = 1, beta = 0 is the identity on any state; o_t = scale S0 q_t."""
    rng = _rng(13)
    dk, dv, L = 4, 6, 5
    k = _unit(rng, L, dk)
    v = rng.standard_normal((L, dv))
    q = rng.standard_normal((L, dk))
    S0 = rng.standard_normal((dv, dk))
    o, S = one(fn, k, v, np.zeros(L), np.zeros(L), q=q, S0=S0, scale=0.5)
    _close(S, S0, 0.0, "identity step state")
    _close(o, 0.5 * q @ S0.T, what="identity step outputs")
    _, Z = one(fn, k, v, np.zeros(L), np.zeros(L))
    assert np.all(Z == 0.0), "alpha=1, beta=0 must keep a zero state at zero"


def pin_delta_rule_textbook(fn):
    """alpha = beta = 1: orthonormal keys store their values; a repeated key overwrites."""
    rng = _rng(14)
    dk, dv = 4, 3
    order = [2, 0, 3, 1]
    k = np.eye(dk)[order]
    v = rng.standard_normal((dk, dv))
    _, S = one(fn, k, v, np.zeros(dk), np.ones(dk))
    _close(S, sum(np.outer(v[i], k[i]) for i in range(dk)), what="orthonormal keys")
    kk = _unit(rng, 1, dk)[0]
    v2 = rng.standard_normal((2, dv))
    _, S = one(fn, np.stack([kk, kk]), v2, np.zeros(2), np.ones(2))
    _close(S, np.outer(v2[1], kk), what="repeated key overwrites")


def pin_pure_decay(fn):
    """beta = 0: S_t = exp(sum_{j<=t} g_j) S0 and o_t = scale exp(G_t) S0 q_t."""
    rng = _rng(15)
    dk, dv, L = 3, 4, 6
    k = _unit(rng, L, dk)
    v = rng.standard_normal((L, dv))
    q = rng.standard_normal((L, dk))
    g = rng.uniform(-0.5, 0.0, L)
    S0 = rng.standard_normal((dv, dk))
    o, S = one(fn, k, v, g, np.zeros(L), q=q, S0=S0, scale=2.0)
    _close(S, np.exp(g.sum()) * S0, what="pure decay state")
    G = np.cumsum(g)
    _close(o, 2.0 * np.exp(G)[:, None] * (q @ S0.T), what="pure decay outputs")


# -------------------------------------------------------------- brute force

def pin_product_formula(fn):
    """The unrolled product formula equals the recurrence (tiny, many seeds)."""
    for seed in range(6):
        rng = _rng(100 + seed)
        dk, dv, L = 3, 4, 7
        k, v, _, g, beta = _random_unit(rng, L, dk, dv)
        S0 = rng.standard_normal((dv, dk)) if seed % 2 else None
        _, S = one(fn, k, v, g, beta, S0=S0)
        _close(S, ref.product_formula(k, v, g, beta, S0), what=f"product formula seed {seed}")


def pin_chunked_form(fn):
    """The chunked UT/WY rewrite equals the implementation for several chunk sizes."""
    rng = _rng(16)
    dk, dv, L = 8, 6, 150
    k, v, q, g, beta = _random_unit(rng, L, dk, dv, gate=(-0.3, 0.0))
    S0 = rng.standard_normal((dv, dk))
    o, S = one(fn, k, v, g, beta, q=q, S0=S0, scale=0.7)
    for C in (1, 4, 16, 64):
        oc, Sc = ref.chunked(k, v, g, beta, C, q=q, S0=S0, scale=0.7)
        _close(S, Sc, 1e-11, f"chunked C={C} state")
        _close(o, oc, 1e-11, f"chunked C={C} outputs")


# --------------------------------------------------------------- invariants

def pin_linearity(fn):
    """From zero the state is linear in V; in general it is affine in S0."""
    rng = _rng(17)
    dk, dv, L = 5, 3, 9
    k, v1, _, g, beta = _random_unit(rng, L, dk, dv)
    v2 = rng.standard_normal((L, dv))
    _, A = one(fn, k, v1, g, beta)
    _, B = one(fn, k, v2, g, beta)
    _, C = one(fn, k, 2.0 * v1 - 3.0 * v2, g, beta)
    _close(C, 2.0 * A - 3.0 * B, what="linear in V")
    X0 = rng.standard_normal((dv, dk))
    Y0 = rng.standard_normal((dv, dk))
    _, F0 = one(fn, k, v1, g, beta)
    _, FX = one(fn, k, v1, g, beta, S0=X0)
    _, FY = one(fn, k, v1, g, beta, S0=Y0)
    _, FXY = one(fn, k, v1, g, beta, S0=X0 + Y0)
    _close(FXY - F0, (FX - F0) + (FY - F0), 1e-11, "affine in S0")


def pin_grouped_heads(fn):
    """Value head h reads key/query head h // (Hv / Hk)."""
    rng = _rng(18)
    hk, hv, dk, dv, L = 2, 4, 4, 3, 6
    k = _unit(rng, L, hk, dk)
    q = rng.standard_normal((L, hk, dk))
    v = rng.standard_normal((L, hv, dv))
    g = rng.uniform(-0.5, 0.0, (L, hv))
    beta = rng.uniform(0.1, 1.0, (L, hv))
    o, st = fn(k, v, g, beta, np.array([0, L]), q=q)
    for h in range(hv):
        kh = h // (hv // hk)
        oh, Sh = one(fn, k[:, kh], v[:, h], g[:, h], beta[:, h], q=q[:, kh])
        _close(st[0, h], Sh.T, what=f"grouped head {h} state")
        _close(o[:, h], oh, what=f"grouped head {h} outputs")


def pin_varlen(fn):
    """Packed sequences are independent; an empty one keeps its initial state."""
    rng = _rng(19)
    hk, hv, dk, dv = 1, 2, 3, 4
    lens = [5, 0, 7]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    k = _unit(rng, T, hk, dk)
    q = rng.standard_normal((T, hk, dk))
    v = rng.standard_normal((T, hv, dv))
    g = rng.uniform(-0.5, 0.0, (T, hv))
    beta = rng.uniform(0.1, 1.0, (T, hv))
    s0 = rng.standard_normal((len(lens), hv, dk, dv))
    o, st = fn(k, v, g, beta, cu, q=q, state_in=s0)
    for n in range(len(lens)):
        a, b = int(cu[n]), int(cu[n + 1])
        on, sn = fn(k[a:b], v[a:b], g[a:b], beta[a:b], np.array([0, b - a]),
                    q=q[a:b], state_in=s0[n:n + 1])
        _close(st[n], sn[0], 0.0, f"varlen seq {n} state")
        _close(o[a:b], on, 0.0, f"varlen seq {n} outputs")
    assert np.array_equal(st[1], s0[1]), "an empty sequence must return state_in"
    _, z = fn(k, v, g, beta, cu)
    assert np.all(z[1] == 0.0), "an empty sequence from zero must return zeros"


def pin_continuation(fn):
    """forward(x[:a]) then forward(x[a:], state) equals forward(x) for every a."""
    rng = _rng(20)
    dk, dv, L = 4, 5, 9
    k, v, q, g, beta = _random_unit(rng, L, dk, dv)
    o, S = one(fn, k, v, g, beta, q=q, scale=0.9)
    for a in range(L + 1):
        o1, S1 = one(fn, k[:a], v[:a], g[:a], beta[:a], q=q[:a], scale=0.9)
        o2, S2 = one(fn, k[a:], v[a:], g[a:], beta[a:], q=q[a:], S0=S1, scale=0.9)
        _close(S2, S, what=f"continuation at {a} state")
        _close(np.concatenate([o1, o2]), o, what=f"continuation at {a} outputs")


def pin_norm_bound(fn):
    """||S_t||_F <= alpha_t ||S_{t-1}||_F + beta_t ||v_t|| ||k_t|| (unit k, beta <= 1)."""
    rng = _rng(21)
    dk, dv, L = 4, 4, 12
    k, v, _, g, beta = _random_unit(rng, L, dk, dv)
    S = rng.standard_normal((dv, dk))
    for t in range(L):
        _, Sn = one(fn, k[t:t + 1], v[t:t + 1], g[t:t + 1], beta[t:t + 1], S0=S)
        bound = np.exp(g[t]) * np.linalg.norm(S) + beta[t] * np.linalg.norm(v[t])
        assert np.linalg.norm(Sn) <= bound * (1 + 1e-12), f"norm bound broken at {t}"
        S = Sn


def pin_tail_replay_full(fn):
    """Eq. 2 with k = m (replay the whole prefix from zero) is full prefill."""
    rng = _rng(22)
    dk, dv, m = 4, 3, 10
    k, v, _, g, beta = _random_unit(rng, m, dk, dv)
    _, full = one(fn, k, v, g, beta)
    _, tail = one(fn, k[m - m:], v[m - m:], g[m - m:], beta[m - m:])
    assert np.array_equal(full, tail)
    _close(full, ref.product_formula(k, v, g, beta), what="r = m state")


def pin_tail_error(fn):
    """Tail-Replay error (Eq. 2 vs Eq. 1): S_full - S_tail = S_head prod_tail T_i,
    bounded by ||S_head||_F prod_tail alpha_i for unit keys and beta in [0, 1]."""
    for seed in range(20):
        rng = _rng(200 + seed)
        d = int(rng.integers(2, 5))
        m = int(rng.integers(3, 13))
        k, v, _, g, beta = _random_unit(rng, m, d, d, gate=(-0.4, 0.0))
        for r in range(0, m + 1):
            h = m - r
            _, S_full = one(fn, k, v, g, beta)
            _, S_head = one(fn, k[:h], v[:h], g[:h], beta[:h])
            _, S_tail = one(fn, k[h:], v[h:], g[h:], beta[h:])
            diff = S_full - S_tail
            _, carried = one(fn, k[h:], np.zeros_like(v[h:]), g[h:], beta[h:], S0=S_head)
            _close(diff, carried, 1e-11, f"tail identity seed {seed} r={r}")
            _close(diff, S_head @ ref.transition_product(k[h:], g[h:], beta[h:]),
                   1e-11, f"tail product seed {seed} r={r}")
            bound = np.linalg.norm(S_head) * np.exp(g[h:].sum())
            assert np.linalg.norm(diff) <= bound * (1 + 1e-12) + 1e-15, \
                f"tail bound broken seed {seed} r={r}"


ALL_PINS = [
    pin_single_token, pin_worked_example, pin_two_tokens, pin_decode_step, pin_identity_step,
    pin_delta_rule_textbook, pin_pure_decay, pin_product_formula,
    pin_chunked_form, pin_linearity, pin_grouped_heads, pin_varlen,
    pin_continuation, pin_norm_bound, pin_tail_replay_full, pin_tail_error,
]


def packed_from_unit(unit_fn):
    """Lifts a one-(sequence, head) function ``unit_fn(k, v, g, beta, q, S0, scale)
    -> (o [L,dv] or None, M [dk,dv])`` to the packed interface of the oracle."""
    def fn(k, v, g, beta, cu_seqlens, q=None, state_in=None, scale=1.0):
        k = np.asarray(k, np.float64)
        v = np.asarray(v, np.float64)
        T, hk, dk = k.shape
        hv, dv = v.shape[1:]
        cu = np.asarray(cu_seqlens, np.int64)
        n = cu.size - 1
        o = None if q is None else np.zeros((T, hv, dv))
        st = np.zeros((n, hv, dk, dv))
        for s in range(n):
            a, b = int(cu[s]), int(cu[s + 1])
            for h in range(hv):
                kh = h // (hv // hk)
                M0 = None if state_in is None else np.asarray(state_in)[s, h]
                oh, M = unit_fn(k[a:b, kh], v[a:b, h], np.asarray(g)[a:b, h],
                                np.asarray(beta)[a:b, h],
                                None if q is None else np.asarray(q)[a:b, kh], M0, scale)
                st[s, h] = M
                if q is not None:
                    o[a:b, h] = oh
        return o, st
    return fn
