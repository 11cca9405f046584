"""Brute-force O(T^2) definitions of the estimators, for pinning the oracle on small inputs.

These do not use the alpha/beta recurrences at all: each one sums over future (or past) steps
of the current episode segment, as the estimator is defined in the work the paper cites for it.
They are written independently of ``oracle/`` and share nothing with it but the readings of
the boundary rules (Section 3.2): a step with both flags set counts as terminated; a
truncated step continues from the supplied value ``bv_t``; the last step of the window
continues from the row bootstrap ``B``.

Plain Python loops over Python floats (fp64); intended for T up to about 16.
"""
from __future__ import annotations

import math
from typing import List, Sequence

import numpy as np


def _f(a):
    return [float(x) for x in a]


def done_flags(term: Sequence[int], trunc: Sequence[int]) -> List[int]:
    return [1 if (a or b) else 0 for a, b in zip(term, trunc)]


def segment_end(d: Sequence[int], t: int) -> int:
    """e_t: the first step k >= t whose flag is set, or the last step of the window."""
    T = len(d)
    for k in range(t, T):
        if d[k]:
            return k
    return T - 1


def segment_start(d: Sequence[int], t: int, starts_at: bool = False) -> int:
    """s_t: the first step of t's episode segment. With the ends_at convention a flag at k-1
    starts a segment at k; with starts_at a flag at k starts a segment at k."""
    for k in range(t, -1, -1):
        if k == 0:
            return 0
        if starts_at and d[k]:
            return k
        if not starts_at and d[k - 1]:
            return k
    return 0


def continuation(term, trunc, bv, B, e: int, T: int) -> float:
    """Value of the state after the segment's last step e."""
    if term[e]:
        return 0.0
    if trunc[e]:
        return float(bv[e])
    assert e == T - 1
    return float(B)


def gae_sum(r, v, term, trunc, bv, B, gamma, lam):
    """A_t = sum_{k=t}^{e_t} (gamma lambda)^(k-t) delta_k (the sum form of GAE, Section 3.3.1)."""
    r, v, bv = _f(r), _f(v), _f(bv)
    T = len(r)
    d = done_flags(term, trunc)
    delta = []
    for k in range(T):
        if term[k]:
            nxt = 0.0
        elif trunc[k]:
            nxt = bv[k]
        elif k == T - 1:
            nxt = float(B)
        else:
            nxt = v[k + 1]
        delta.append(r[k] + gamma * nxt - v[k])
    A = []
    for t in range(T):
        e = segment_end(d, t)
        A.append(sum((gamma * lam) ** (k - t) * delta[k] for k in range(t, e + 1)))
    return A


def discounted_sum(r, term, trunc, bv, B, gamma):
    """G_t = sum_{k=t}^{e_t} gamma^(k-t) r_k + gamma^(e_t-t+1) * continuation(e_t)."""
    r, bv = _f(r), _f(bv)
    T = len(r)
    d = done_flags(term, trunc)
    G = []
    for t in range(T):
        e = segment_end(d, t)
        g = sum(gamma ** (k - t) * r[k] for k in range(t, e + 1))
        g += gamma ** (e - t + 1) * continuation(term, trunc, bv, B, e, T)
        G.append(g)
    return G


def lambda_return(r, v, term, trunc, bv, B, gamma, lam):
    """The truncated lambda-return (Sutton and Barto, cited for TD(lambda) in Section 3.3.4):
    with h = e_t - t + 1 steps left in the segment,
    G_t = (1 - lambda) sum_{n=1}^{h-1} lambda^(n-1) G_t^(n) + lambda^(h-1) G_t^(h),
    where G_t^(n) bootstraps from V(s_{t+n}) for n < h and G_t^(h) from the continuation."""
    r, v, bv = _f(r), _f(v), _f(bv)
    T = len(r)
    d = done_flags(term, trunc)
    out = []
    for t in range(T):
        e = segment_end(d, t)
        h = e - t + 1

        def n_step(n):
            g = sum(gamma ** k * r[t + k] for k in range(n))
            if n < h:
                g += gamma ** n * v[t + n]
            else:
                g += gamma ** n * continuation(term, trunc, bv, B, e, T)
            return g

        total = sum((1 - lam) * lam ** (n - 1) * n_step(n) for n in range(1, h))
        total += lam ** (h - 1) * n_step(h)
        out.append(total)
    return out


def vtrace_sum(r, v, log_rho, term, trunc, bv, B, gamma, rho_bar, c_bar):
    """IMPALA's sum form: Delta_s = sum_{k=s}^{e_s} gamma^(k-s) (prod_{i=s}^{k-1} c_i) dV_k with
    dV_k = rho_k (r_k + gamma V(s_{k+1}) - V_k); vs = V + Delta;
    pg_s = rho_s (r_s + gamma vs(s_{s+1}) - V_s)."""
    r, v, lr, bv = _f(r), _f(v), _f(log_rho), _f(bv)
    T = len(r)
    d = done_flags(term, trunc)
    rho = [min(rho_bar, math.exp(x)) for x in lr]
    c = [min(c_bar, math.exp(x)) for x in lr]

    def nxt(u, k):
        if term[k]:
            return 0.0
        if trunc[k]:
            return bv[k]
        if k == T - 1:
            return float(B)
        return u[k + 1]

    dV = [rho[k] * (r[k] + gamma * nxt(v, k) - v[k]) for k in range(T)]
    Delta = []
    for s in range(T):
        e = segment_end(d, s)
        acc = 0.0
        for k in range(s, e + 1):
            prod = 1.0
            for i in range(s, k):
                prod *= c[i]
            acc += gamma ** (k - s) * prod * dV[k]
        Delta.append(acc)
    vs = [Delta[k] + v[k] for k in range(T)]
    pg = [rho[k] * (r[k] + gamma * nxt(vs, k) - v[k]) for k in range(T)]
    return vs, pg


def retrace_sum(r, q, eq, log_rho, term, trunc, bv, B, gamma, lam, c_bar):
    """Munos et al.'s sum form: Delta_s = sum_{k=s}^{e_s} gamma^(k-s) (prod_{i=s+1}^{k} c_i) delta_k,
    c_i = lambda min(c_bar, rho_i), delta_k = r_k + gamma E_pi Q(s_{k+1}) - Q(s_k, a_k)."""
    r, q, eq, lr, bv = _f(r), _f(q), _f(eq), _f(log_rho), _f(bv)
    T = len(r)
    d = done_flags(term, trunc)
    c = [lam * min(c_bar, math.exp(x)) for x in lr]

    def nxt(k):
        if term[k]:
            return 0.0
        if trunc[k]:
            return bv[k]
        if k == T - 1:
            return float(B)
        return eq[k + 1]

    td = [r[k] + gamma * nxt(k) - q[k] for k in range(T)]
    Delta = []
    for s in range(T):
        e = segment_end(d, s)
        acc = 0.0
        for k in range(s, e + 1):
            prod = 1.0
            for i in range(s + 1, k + 1):
                prod *= c[i]
            acc += gamma ** (k - s) * prod * td[k]
        Delta.append(acc)
    return Delta, [q[k] + Delta[k] for k in range(T)]


def elig_sum(x, term, trunc, gamma, lam):
    """z_t = sum_{k=s_t}^{t} (gamma lambda)^(t-k) x_k."""
    x = _f(x)
    d = done_flags(term, trunc)
    return [sum((gamma * lam) ** (t - k) * x[k] for k in range(segment_start(d, t), t + 1))
            for t in range(len(x))]


def prefix_sum(x, term, trunc, starts_at=False):
    """C_t = sum_{k=s_t}^{t} x_k."""
    x = _f(x)
    d = done_flags(term, trunc)
    return [sum(x[k] for k in range(segment_start(d, t, starts_at), t + 1))
            for t in range(len(x))]



def retrace_full_sum(r, q3, pi3, actions, mu, term, trunc, bv, B, gamma, lam, c_bar):
    """Munos et al.'s sum form with the per-step terms taken from the [T, A] tensors:
    E_pi Q(s_t) = sum_a pi(a|s_t) Q(s_t, a), Q(s_t, a_t), c_t = lambda min(c_bar, pi(a_t)/mu_t);
    an action outside [0, A) selects nothing."""
    T = len(r)
    A = len(q3[0]) if T else 0
    eq, qt, lr_c = [], [], []
    for t in range(T):
        eq.append(sum(float(pi3[t][k]) * float(q3[t][k]) for k in range(A)))
        a = int(actions[t])
        ok = 0 <= a < A
        qt.append(float(q3[t][a]) if ok else 0.0)
        p = float(pi3[t][a]) if ok else 0.0
        lr_c.append(lam * min(c_bar, p / float(mu[t])))
    r, bv = _f(r), _f(bv)
    d = done_flags(term, trunc)

    def nxt(k):
        if term[k]:
            return 0.0
        if trunc[k]:
            return bv[k]
        if k == T - 1:
            return float(B)
        return eq[k + 1]

    td = [r[k] + gamma * nxt(k) - qt[k] for k in range(T)]
    Delta = []
    for s in range(T):
        e = segment_end(d, s)
        acc = 0.0
        for k in range(s, e + 1):
            prod = 1.0
            for i in range(s + 1, k + 1):
                prod *= lr_c[i]
            acc += gamma ** (k - s) * prod * td[k]
        Delta.append(acc)
    return Delta, [qt[k] + Delta[k] for k in range(T)]
