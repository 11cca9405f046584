"""Pins for the fp64 oracle: it is checked against things other than itself.

* the combine of Eq. 2 (associativity, identity, annihilator) and the Appendix A trace;
* brute-force sum definitions of every estimator (tests/brute.py), exhaustively over all flag
  patterns for short rows and on random patterns up to T = 16;
* closed forms (geometric series), special cases (lambda = 0 / 1, on-policy V-Trace and
  Retrace) and identities that follow from the definitions (TD(lambda) returns equal GAE
  advantages plus values);
* the boundary rules of Section 3.2 and the severing argument of Section 5.2.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import brute
import oracle
from oracle import scan_algebra

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

G, L = 0.99, 0.95  # stored exactly as the oracle sees them (float32-rounded)
g32, l32 = oracle.param(G), oracle.param(L)


def rtol_close(a, b, rel=1e-12):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    scale = 1.0 + np.max(np.abs(b)) if b.size else 1.0
    assert np.max(np.abs(a - b), initial=0.0) <= rel * scale, (np.max(np.abs(a - b)), scale)


def all_flag_patterns(T):
    """Every (term, trunc) assignment over T steps: 4**T rows (none / term / trunc / both)."""
    codes = np.array(list(itertools.product(range(4), repeat=T)), dtype=np.uint8).reshape(-1, T)
    return (codes & 1).astype(np.uint8), ((codes >> 1) & 1).astype(np.uint8)


def random_inputs(N, T, seed, dyadic=False):
    rng = np.random.default_rng(seed)
    if dyadic:
        f = lambda: (rng.integers(-16, 17, size=(N, T)) / 8.0)
    else:
        f = lambda: rng.standard_normal((N, T))
    return dict(r=f(), v=f(), bv=f(), lr=0.5 * rng.standard_normal((N, T)), q=f(), eq=f(),
                boot=rng.standard_normal(N))


# ---------------------------------------------------------------- combine (Eq. 2)

def test_combine_associative_exhaustive_on_dyadics():
    """Proposition 1, exhaustively on all triples of pairs with entries in {k/4 : |k| <= 4}:
    fp64 products and sums of these are exact, so both groupings agree bitwise."""
    vals = np.arange(-4, 5) / 4.0
    grid = np.array(list(itertools.product(vals, repeat=6)))
    aC, bC, aB, bB, aA, bA = grid.T
    # [(C (+) B)] (+) A
    l_a, l_b = aC + bC * aB, bB * bC
    left = (l_a + l_b * aA, bA * l_b)
    # C (+) [(B (+) A)]
    r_a, r_b = aB + bB * aA, bA * bB
    right = (aC + bC * r_a, r_b * bC)
    assert np.array_equal(left[0], right[0]) and np.array_equal(left[1], right[1])
    # and the module's own combine agrees on a sample of them
    for row in grid[::997]:
        C, B, A = (row[0], row[1]), (row[2], row[3]), (row[4], row[5])
        assert scan_algebra.combine(scan_algebra.combine(C, B), A) == \
            scan_algebra.combine(C, scan_algebra.combine(B, A))


def test_combine_associative_random_reals():
    rng = np.random.default_rng(1)
    for _ in range(2000):
        C, B, A = [tuple(rng.standard_normal(2)) for _ in range(3)]
        x = scan_algebra.combine(scan_algebra.combine(C, B), A)
        y = scan_algebra.combine(C, scan_algebra.combine(B, A))
        assert abs(x[0] - y[0]) <= 1e-14 * (1 + abs(x[0]))
        assert abs(x[1] - y[1]) <= 1e-14 * (1 + abs(x[1]))


def test_combine_identity_and_annihilator():
    """(0, 1) is the identity; (alpha, 0) (+) X = (alpha, 0) severs the carry (Section 5.2)."""
    rng = np.random.default_rng(2)
    for _ in range(200):
        X = tuple(rng.standard_normal(2))
        assert scan_algebra.combine(scan_algebra.IDENTITY, X) == X
        assert scan_algebra.combine(X, scan_algebra.IDENTITY) == X
        a = float(rng.standard_normal())
        assert scan_algebra.combine((a, 0.0), X) == (a, 0.0)


def test_combine_orientation_is_earlier_first():
    """Eq. 2 composes the earlier step on the left: (a0, b0) (+) (a1, b1) gives
    A_0 = a0 + b0 * A_1 for a zero carry; the reversed orientation does not."""
    e, l = (1.0, 0.5), (4.0, 0.25)
    assert scan_algebra.combine(e, l)[0] == 1.0 + 0.5 * 4.0
    assert scan_algebra.combine(l, e)[0] != 1.0 + 0.5 * 4.0


# ---------------------------------------------------------------- Appendix A

def test_appendix_a_trace_matches_golden():
    with open(os.path.join(GOLDEN, "appendix_a_trace.json")) as f:
        gold = json.load(f)
    alpha, beta = gold["alpha"], gold["beta"]
    hist = scan_algebra.hillis_steele_backward(alpha, beta)
    assert len(hist) == 3  # initial + log2(4) passes
    p1, p2 = hist[1], hist[2]
    # positions are 0-based here: paper position k is index k-1
    assert p1[0] == tuple(gold["pass1"]["T_1..1"])
    assert p1[1] == tuple(gold["pass1"]["T_1..2"])
    assert p1[2] == tuple(gold["pass1"]["T_2..3"])
    assert p1[3] == tuple(gold["pass1"]["T_3..4"])
    assert p2[2] == tuple(gold["pass2"]["T_1..3"])
    assert p2[3] == tuple(gold["pass2"]["T_1..4"])
    # the sequential oracle reproduces the same A_t exactly
    A = oracle.affine_scan(np.array([alpha]), np.array([beta]), reverse=True)[0]
    assert list(A) == gold["A"]
    assert scan_algebra.scan_backward_by_combine(alpha, beta) == gold["A"]


@pytest.mark.parametrize("T", [1, 2, 3, 4, 5, 7, 8, 16, 31, 33])
def test_tree_scan_equals_sequential_oracle_exactly(T):
    """On dyadic inputs small enough that every partial result is exact, the log-depth scan
    by combine and the oracle's sequential recurrence agree bitwise, carry included."""
    rng = np.random.default_rng(T)
    # five rows in one call: each row is its own recurrence with its own carry
    a = rng.integers(-8, 9, size=(5, T)) / 4.0
    b = rng.integers(0, 3, size=(5, T)) / 2.0  # 0, 0.5, 1: products stay dyadic
    carry = rng.integers(-8, 9, size=5) / 4.0
    seq = oracle.affine_scan(a, b, carry, reverse=True)
    fwd = oracle.affine_scan(a, b, carry, reverse=False)
    for n in range(5):
        tree = scan_algebra.scan_backward_by_combine(list(a[n]), list(b[n]), float(carry[n]))
        assert list(seq[n]) == tree
        # forward mirror: reverse the arrays
        tree_f = scan_algebra.scan_backward_by_combine(list(a[n][::-1]), list(b[n][::-1]),
                                                       float(carry[n]))[::-1]
        assert list(fwd[n]) == tree_f


# ---------------------------------------------------------------- brute force, exhaustive

@pytest.mark.parametrize("T", [1, 2, 3, 4, 5, 6])
def test_brute_force_exhaustive_flags(T):
    term, trunc = all_flag_patterns(T)
    N = term.shape[0]
    x = random_inputs(N, T, seed=100 + T)
    r, v, bv, lr, q, eq, boot = x["r"], x["v"], x["bv"], x["lr"], x["q"], x["eq"], x["boot"]

    adv, ret = oracle.gae(r, v, term, trunc, bv, boot, gamma=G, lam=L)
    bf = np.array([brute.gae_sum(r[n], v[n], term[n], trunc[n], bv[n], boot[n], g32, l32)
                   for n in range(N)])
    rtol_close(adv, bf)
    rtol_close(ret, bf + v)

    td = oracle.td_lambda(r, v, term, trunc, bv, boot, gamma=G, lam=L)
    bf = np.array([brute.lambda_return(r[n], v[n], term[n], trunc[n], bv[n], boot[n], g32, l32)
                   for n in range(N)])
    rtol_close(td, bf)

    dr = oracle.discounted(r, term, trunc, bv, boot, gamma=G)
    bf = np.array([brute.discounted_sum(r[n], term[n], trunc[n], bv[n], boot[n], g32)
                   for n in range(N)])
    rtol_close(dr, bf)

    rho_bar, c_bar = 1.2, 0.9
    vs, pg = oracle.vtrace(r, v, lr, term, trunc, bv, boot, gamma=G, rho_bar=rho_bar, c_bar=c_bar)
    res = [brute.vtrace_sum(r[n], v[n], lr[n], term[n], trunc[n], bv[n], boot[n], g32,
                            oracle.param(rho_bar), oracle.param(c_bar)) for n in range(N)]
    rtol_close(vs, np.array([a for a, _ in res]))
    rtol_close(pg, np.array([b for _, b in res]))

    dl, qr = oracle.retrace(r, q, eq, lr, term, trunc, bv, boot, gamma=G, lam=L, c_bar=c_bar)
    res = [brute.retrace_sum(r[n], q[n], eq[n], lr[n], term[n], trunc[n], bv[n], boot[n], g32,
                             l32, oracle.param(c_bar)) for n in range(N)]
    rtol_close(dl, np.array([a for a, _ in res]))
    rtol_close(qr, np.array([b for _, b in res]))

    z = oracle.elig_trace(r, term, trunc, gamma=G, lam=L)
    rtol_close(z, np.array([brute.elig_sum(r[n], term[n], trunc[n], g32, l32) for n in range(N)]))

    for starts_at in (False, True):
        c = oracle.episodic_prefix(r, term, trunc,
                                   boundary="starts_at" if starts_at else "ends_at")
        rtol_close(c, np.array([brute.prefix_sum(r[n], term[n], trunc[n], starts_at)
                                for n in range(N)]))


@pytest.mark.parametrize("T", [7, 9, 12, 16])
def test_brute_force_random_flags(T):
    N = 200
    rng = np.random.default_rng(7 * T)
    term = (rng.random((N, T)) < 0.15).astype(np.uint8)
    trunc = (rng.random((N, T)) < 0.15).astype(np.uint8)
    x = random_inputs(N, T, seed=200 + T)
    r, v, bv, lr, q, eq, boot = x["r"], x["v"], x["bv"], x["lr"], x["q"], x["eq"], x["boot"]
    adv, _ = oracle.gae(r, v, term, trunc, bv, boot, gamma=G, lam=L)
    rtol_close(adv, [brute.gae_sum(r[n], v[n], term[n], trunc[n], bv[n], boot[n], g32, l32)
                     for n in range(N)])
    td = oracle.td_lambda(r, v, term, trunc, bv, boot, gamma=G, lam=L)
    rtol_close(td, [brute.lambda_return(r[n], v[n], term[n], trunc[n], bv[n], boot[n], g32, l32)
                    for n in range(N)])
    vs, pg = oracle.vtrace(r, v, lr, term, trunc, bv, boot, gamma=G)
    res = [brute.vtrace_sum(r[n], v[n], lr[n], term[n], trunc[n], bv[n], boot[n], g32, 1.0, 1.0)
           for n in range(N)]
    rtol_close(vs, [a for a, _ in res])
    rtol_close(pg, [b for _, b in res])
    dl, _ = oracle.retrace(r, q, eq, lr, term, trunc, bv, boot, gamma=G, lam=L)
    rtol_close(dl, [brute.retrace_sum(r[n], q[n], eq[n], lr[n], term[n], trunc[n], bv[n],
                                      boot[n], g32, l32, 1.0)[0] for n in range(N)])
    z = oracle.elig_trace(r, term, trunc, gamma=G, lam=L)
    rtol_close(z, [brute.elig_sum(r[n], term[n], trunc[n], g32, l32) for n in range(N)])


def test_brute_force_without_optional_inputs():
    """NULL flags / NULL bootstrap behave as all-clear / zero."""
    N, T = 50, 11
    x = random_inputs(N, T, seed=5)
    zeros8 = np.zeros((N, T), np.uint8)
    a1, _ = oracle.gae(x["r"], x["v"], gamma=G, lam=L)
    a2, _ = oracle.gae(x["r"], x["v"], zeros8, zeros8, x["bv"], np.zeros(N), gamma=G, lam=L)
    assert np.array_equal(a1, a2)
    d1 = oracle.discounted(x["r"], gamma=G)
    d2 = oracle.discounted(x["r"], zeros8, None, None, np.zeros(N), gamma=G)
    assert np.array_equal(d1, d2)


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("T", [1, 5, 64, 300])
def test_gae_closed_form_geometric(T):
    """r = c, V = 0, B = 0, no flags: A_t = c (1 - (gl)^(T-t)) / (1 - gl)."""
    c = 0.7
    r = np.full((1, T), c)
    v = np.zeros((1, T))
    adv, ret = oracle.gae(r, v, gamma=G, lam=L)
    gl = g32 * l32
    k = T - np.arange(T)
    rtol_close(adv[0], c * (1 - gl ** k) / (1 - gl))
    assert np.array_equal(ret, adv)


@pytest.mark.parametrize("T", [1, 7, 128])
def test_discounted_closed_form(T):
    c = -1.25
    r = np.full((1, T), c)
    k = T - np.arange(T)
    rtol_close(oracle.discounted(r, gamma=G)[0], c * (1 - g32 ** k) / (1 - g32))
    # gamma = 1: c * (T - t), exact in fp64
    assert np.array_equal(oracle.discounted(r, gamma=1.0)[0], c * k)


@pytest.mark.parametrize("T", [1, 9, 100])
def test_elig_closed_form(T):
    x = np.ones((1, T))
    gl = g32 * l32
    t = np.arange(T)
    rtol_close(oracle.elig_trace(x, gamma=G, lam=L)[0], (1 - gl ** (t + 1)) / (1 - gl))


def test_prefix_counts_exact():
    T = 1000
    x = np.ones((1, T))
    assert np.array_equal(oracle.episodic_prefix(x)[0], np.arange(T) + 1.0)
    for m in (1, 3, 17):
        term = np.zeros((1, T), np.uint8)
        term[0, m - 1::m] = 1
        assert np.array_equal(oracle.episodic_prefix(x, term)[0], (np.arange(T) % m) + 1.0)
        # starts_at: a flag at t starts a new segment at t
        starts = np.zeros((1, T), np.uint8)
        starts[0, ::m] = 1
        assert np.array_equal(oracle.episodic_prefix(x, None, starts, boundary="starts_at")[0],
                              (np.arange(T) % m) + 1.0)


# ---------------------------------------------------------------- special cases / identities

def _flags(N, T, seed, p=0.1):
    rng = np.random.default_rng(seed)
    return ((rng.random((N, T)) < p).astype(np.uint8), (rng.random((N, T)) < p).astype(np.uint8))


def test_gae_lambda_zero_is_one_step_td():
    """Section 3.3.1: lambda = 0 gives A_t = delta_t."""
    N, T = 40, 33
    x = random_inputs(N, T, 11)
    term, trunc = _flags(N, T, 11)
    adv, _ = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=0.0)
    nxt = np.concatenate([x["v"][:, 1:], x["boot"][:, None]], axis=1)
    nxt = np.where(trunc == 1, x["bv"], nxt)
    nxt = np.where(term == 1, 0.0, nxt)
    rtol_close(adv, x["r"] + g32 * nxt - x["v"], rel=1e-15)


def test_gae_lambda_one_is_monte_carlo_minus_baseline():
    """Section 3.3.1: lambda = 1 gives the discounted return minus V."""
    N, T = 40, 33
    x = random_inputs(N, T, 12)
    term, trunc = _flags(N, T, 12)
    adv, _ = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=1.0)
    dr = oracle.discounted(x["r"], term, trunc, x["bv"], x["boot"], gamma=G)
    rtol_close(adv, dr - x["v"])


def test_td_lambda_equals_gae_returns():
    """TD(lambda) returns equal GAE advantages plus values for the same inputs, boundary cases
    included (Table 1: both share beta = gamma lambda (1 - d); the window identity of
    Section 3.3.4 matches GAE's window bootstrap)."""
    N, T = 60, 40
    x = random_inputs(N, T, 13)
    term, trunc = _flags(N, T, 13)
    _, ret = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    td = oracle.td_lambda(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    rtol_close(td, ret)


def test_td_lambda_one_is_discounted():
    N, T = 30, 25
    x = random_inputs(N, T, 14)
    term, trunc = _flags(N, T, 14)
    td = oracle.td_lambda(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=1.0)
    dr = oracle.discounted(x["r"], term, trunc, x["bv"], x["boot"], gamma=G)
    rtol_close(td, dr, rel=1e-15)


def test_td_lambda_window_edge():
    """Section 3.3.4: at the last step of a continuing episode G_{T-1} = r + gamma V(s_T)."""
    N, T = 20, 6
    x = random_inputs(N, T, 15)
    td = oracle.td_lambda(x["r"], x["v"], None, None, None, x["boot"], gamma=G, lam=L)
    rtol_close(td[:, -1], x["r"][:, -1] + g32 * x["boot"], rel=1e-15)


def test_vtrace_on_policy_is_gae_lambda_one():
    """On-policy (log rho = 0, rho_bar = c_bar = 1): rho = c = 1, so the V-Trace correction is
    the lambda = 1 GAE advantage and vs the lambda = 1 GAE return."""
    N, T = 30, 50
    x = random_inputs(N, T, 16)
    term, trunc = _flags(N, T, 16)
    zero = np.zeros((N, T))
    vs, pg = oracle.vtrace(x["r"], x["v"], zero, term, trunc, x["bv"], x["boot"], gamma=G)
    adv, ret = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=1.0)
    rtol_close(vs, ret)
    rtol_close(vs - x["v"], adv)


def test_vtrace_rho_clip():
    """Large ratios are clipped at rho_bar (value target) and c_bar (trace)."""
    N, T = 10, 12
    x = random_inputs(N, T, 17)
    big = np.full((N, T), 3.0)  # exp(3) ~ 20
    vs_a, pg_a = oracle.vtrace(x["r"], x["v"], big, gamma=G, rho_bar=1.0, c_bar=1.0)
    vs_b, pg_b = oracle.vtrace(x["r"], x["v"], np.zeros((N, T)), gamma=G, rho_bar=1.0, c_bar=1.0)
    assert np.array_equal(vs_a, vs_b) and np.array_equal(pg_a, pg_b)
    # unclipped: rho = exp(lr) exactly
    vs_c, pg_c = oracle.vtrace(x["r"], x["v"], big, gamma=G, rho_bar=math.inf, c_bar=math.inf)
    assert not np.allclose(vs_c, vs_b)


def test_retrace_reduces_to_gae():
    """log rho = 0, c_bar = 1, Q = E_pi Q = V: c = lambda and delta is GAE's TD error, so the
    Retrace correction equals the GAE advantage with the same lambda (c_T = 0 matches A_T = 0)."""
    N, T = 30, 45
    x = random_inputs(N, T, 18)
    term, trunc = _flags(N, T, 18)
    zero = np.zeros((N, T))
    dl, qr = oracle.retrace(x["r"], x["v"], x["v"], zero, term, trunc, x["bv"], x["boot"],
                            gamma=G, lam=L)
    adv, ret = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    rtol_close(dl, adv)
    rtol_close(qr, ret)


def test_retrace_lambda_zero_is_td_error():
    N, T = 20, 30
    x = random_inputs(N, T, 19)
    term, trunc = _flags(N, T, 19)
    dl, _ = oracle.retrace(x["r"], x["q"], x["eq"], x["lr"], term, trunc, x["bv"], x["boot"],
                           gamma=G, lam=0.0)
    nxt = np.concatenate([x["eq"][:, 1:], x["boot"][:, None]], axis=1)
    nxt = np.where(trunc == 1, x["bv"], nxt)
    nxt = np.where(term == 1, 0.0, nxt)
    rtol_close(dl, x["r"] + g32 * nxt - x["q"], rel=1e-15)


def test_elig_unit_decay_is_prefix():
    N, T = 20, 64
    x = random_inputs(N, T, 20)
    term, trunc = _flags(N, T, 20)
    z = oracle.elig_trace(x["r"], term, trunc, gamma=1.0, lam=1.0)
    c = oracle.episodic_prefix(x["r"], term, trunc)
    assert np.array_equal(z, c)


def test_prefix_starts_at_is_shifted_ends_at():
    """starts_at with flags d equals ends_at with the flags moved one step earlier."""
    N, T = 30, 40
    x = random_inputs(N, T, 21)
    term, _ = _flags(N, T, 21, p=0.2)
    s = oracle.episodic_prefix(x["r"], term, boundary="starts_at")
    shifted = np.zeros_like(term)
    shifted[:, :-1] = term[:, 1:]
    e = oracle.episodic_prefix(x["r"], shifted, boundary="ends_at")
    assert np.array_equal(s, e)


# ---------------------------------------------------------------- boundaries (Sections 3.2, 5.2)

BACKWARD = ["gae", "td_lambda", "discounted", "vtrace", "retrace"]


def _run_backward(name, x, term, trunc):
    if name == "gae":
        return oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    if name == "td_lambda":
        return (oracle.td_lambda(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L),)
    if name == "discounted":
        return (oracle.discounted(x["r"], term, trunc, x["bv"], x["boot"], gamma=G),)
    if name == "vtrace":
        return oracle.vtrace(x["r"], x["v"], x["lr"], term, trunc, x["bv"], x["boot"], gamma=G)
    return oracle.retrace(x["r"], x["q"], x["eq"], x["lr"], term, trunc, x["bv"], x["boot"],
                          gamma=G, lam=L)


@pytest.mark.parametrize("name", BACKWARD)
@pytest.mark.parametrize("kind", ["term", "trunc"])
def test_severing_backward(name, kind):
    """With a flag at t, outputs at steps <= t do not change, bitwise, when anything after t
    (or the row bootstrap) changes."""
    N, T, t = 8, 20, 9
    x = random_inputs(N, T, 30)
    term = np.zeros((N, T), np.uint8)
    trunc = np.zeros((N, T), np.uint8)
    (term if kind == "term" else trunc)[:, t] = 1
    base = _run_backward(name, x, term, trunc)
    y = {k: v.copy() for k, v in x.items()}
    rng = np.random.default_rng(31)
    for k in ("r", "v", "bv", "lr", "q", "eq"):
        y[k][:, t + 1:] = rng.standard_normal((N, T - t - 1))
    y["boot"] = rng.standard_normal(N)
    pert = _run_backward(name, y, term, trunc)
    for a, b in zip(base, pert):
        assert np.array_equal(a[:, :t + 1], b[:, :t + 1])
        assert not np.array_equal(a[:, t + 1:], b[:, t + 1:])


@pytest.mark.parametrize("boundary", ["ends_at", "starts_at"])
def test_severing_forward(boundary):
    N, T, t = 8, 20, 9
    x = random_inputs(N, T, 32)
    term = np.zeros((N, T), np.uint8)
    term[:, t] = 1
    first_free = t + 1 if boundary == "ends_at" else t
    y = x["r"].copy()
    y[:, :first_free] = np.random.default_rng(33).standard_normal((N, first_free))
    runs = [lambda a: oracle.episodic_prefix(a, term, boundary=boundary)]
    if boundary == "ends_at":
        runs.append(lambda a: oracle.elig_trace(a, term, gamma=G, lam=L))
    for run in runs:
        a, b = run(x["r"]), run(y)
        assert np.array_equal(a[:, first_free:], b[:, first_free:])
        assert not np.array_equal(a[:, :first_free], b[:, :first_free])


def test_terminated_and_truncated_step_values():
    """Section 3.2: at a terminated step GAE A = r - V, TD/discounted G = r, V-Trace
    Delta = rho (r - V), Retrace Delta = r - Q; at a truncated step GAE A = r + gamma bv - V
    and TD/discounted G = r + gamma bv, with nothing carried from later steps."""
    N, T, t = 6, 15, 7
    x = random_inputs(N, T, 34)
    rho = np.minimum(1.0, np.exp(x["lr"]))
    for kind in ("term", "trunc"):
        term = np.zeros((N, T), np.uint8)
        trunc = np.zeros((N, T), np.uint8)
        (term if kind == "term" else trunc)[:, t] = 1
        cont = 0.0 if kind == "term" else g32 * x["bv"][:, t]
        r, v = x["r"][:, t], x["v"][:, t]
        adv, _ = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
        assert np.allclose(adv[:, t], r + cont - v, rtol=0, atol=1e-15)
        td = oracle.td_lambda(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
        assert np.allclose(td[:, t], r + cont, rtol=0, atol=1e-15)
        dr = oracle.discounted(x["r"], term, trunc, x["bv"], x["boot"], gamma=G)
        assert np.allclose(dr[:, t], r + cont, rtol=0, atol=1e-15)
        vs, _ = oracle.vtrace(x["r"], x["v"], x["lr"], term, trunc, x["bv"], x["boot"], gamma=G)
        assert np.allclose(vs[:, t] - v, rho[:, t] * (r + cont - v), rtol=0, atol=1e-14)
        dl, _ = oracle.retrace(x["r"], x["q"], x["eq"], x["lr"], term, trunc, x["bv"],
                               x["boot"], gamma=G, lam=L)
        assert np.allclose(dl[:, t], r + cont - x["q"][:, t], rtol=0, atol=1e-15)


def test_truncated_last_step_not_double_counted():
    """Section 3.2: a truncated last step bootstraps from bv once; the row bootstrap is unused."""
    N, T = 6, 9
    x = random_inputs(N, T, 35)
    trunc = np.zeros((N, T), np.uint8)
    trunc[:, -1] = 1
    for boot in (x["boot"], 100 * x["boot"]):
        td = oracle.td_lambda(x["r"], x["v"], None, trunc, x["bv"], boot, gamma=G, lam=L)
        assert np.allclose(td[:, -1], x["r"][:, -1] + g32 * x["bv"][:, -1], rtol=0, atol=1e-15)
        adv, _ = oracle.gae(x["r"], x["v"], None, trunc, x["bv"], boot, gamma=G, lam=L)
        assert np.allclose(adv[:, -1], x["r"][:, -1] + g32 * x["bv"][:, -1] - x["v"][:, -1],
                           rtol=0, atol=1e-15)


def test_bf16_widening_is_exact():
    import workloads
    ro = workloads.make_rollout(4, 8, seed=3, dtype="bf16")
    w = oracle.widen(ro["r"])
    assert w.dtype == np.float64
    back = workloads.bf16_bits_from_f32(w.astype(np.float32))
    assert np.array_equal(back, ro["r"])


# ---------------------------------------------------------------- full-form Retrace (Section 7.3)

@pytest.mark.parametrize("A", [1, 3, 4, 7])
def test_retrace_full_brute_force(A):
    """Full-form Retrace against the Munos sum with the per-step terms computed from the
    [T, A] tensors in the test, including out-of-range actions and every flag pattern mix."""
    import workloads
    N, T = 120, 11
    ro = workloads.make_retrace_full(N, T, A, seed=40 + A, p_term=0.15, p_trunc=0.15)
    act = ro["actions"].copy()
    act[::7, ::3] = A + 2      # out of range: selects nothing
    act[1::9, 1::4] = -1
    act[2::11, 2::5] = A       # the first index past the last action
    c_bar = 0.8
    dl, qr = oracle.retrace_full(ro["r"], ro["q3"], ro["pi3"], act, ro["mu"], ro["term"],
                                 ro["trunc"], ro["bv"], ro["boot"], gamma=G, lam=L, c_bar=c_bar)
    res = [brute.retrace_full_sum(ro["r"][n], ro["q3"][n], ro["pi3"][n], act[n], ro["mu"][n],
                                  ro["term"][n], ro["trunc"][n], ro["bv"][n], ro["boot"][n],
                                  g32, l32, oracle.param(c_bar)) for n in range(N)]
    rtol_close(dl, [a for a, _ in res])
    rtol_close(qr, [b for _, b in res])


def test_retrace_full_single_action_is_gae():
    """A = 1 with pi = mu = 1: E_pi Q = Q, rho = 1, c = lambda, so the correction is the GAE
    advantage with V = Q (Section 3.3.3 with Table 1's GAE row)."""
    N, T = 40, 30
    x = random_inputs(N, T, 41)
    term, trunc = _flags(N, T, 41)
    q3 = x["q"][:, :, None]
    ones = np.ones((N, T))
    dl, _ = oracle.retrace_full(x["r"], q3, ones[:, :, None], np.zeros((N, T), np.int32), ones,
                                term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    adv, _ = oracle.gae(x["r"], x["q"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    rtol_close(dl, adv)


# ---------------------------------------------------------------- vector eligibility traces (Section 3.3.5)

@pytest.mark.parametrize("F", [1, 3, 8])
def test_elig_trace_vec_brute_force(F):
    """Every feature of z_t against the past-weighted sum over the episode segment, with the
    step's flags shared by all features."""
    N, T = 60, 13
    rng = np.random.default_rng(90 + F)
    term = (rng.random((N, T)) < 0.15).astype(np.uint8)
    trunc = (rng.random((N, T)) < 0.15).astype(np.uint8)
    x = rng.standard_normal((N, T, F))
    z = oracle.elig_trace_vec(x, term, trunc, gamma=G, lam=L)
    ref = np.array([[brute.elig_sum(x[n, :, f], term[n], trunc[n], g32, l32) for f in range(F)]
                    for n in range(N)])  # [N, F, T]
    rtol_close(z, ref.transpose(0, 2, 1))


def test_elig_trace_vec_exhaustive_flags():
    """All 4**5 flag patterns of a 5-step row, two features."""
    T = 5
    term, trunc = all_flag_patterns(T)
    N = term.shape[0]
    rng = np.random.default_rng(3)
    x = rng.standard_normal((N, T, 2))
    z = oracle.elig_trace_vec(x, term, trunc, gamma=G, lam=L)
    for f in range(2):
        rtol_close(z[:, :, f], [brute.elig_sum(x[n, :, f], term[n], trunc[n], g32, l32)
                                for n in range(N)])


def test_elig_trace_vec_one_feature_is_scalar_trace():
    """F = 1 is the scalar eligibility trace, bit for bit (same fp64 steps)."""
    N, T = 30, 40
    term, trunc = _flags(N, T, 11)
    x = np.random.default_rng(12).standard_normal((N, T))
    zv = oracle.elig_trace_vec(x[:, :, None], term, trunc, gamma=G, lam=L)[:, :, 0]
    assert np.array_equal(zv, oracle.elig_trace(x, term, trunc, gamma=G, lam=L))


def test_elig_trace_vec_feature_permutation_and_linearity():
    """Features are independent scans with a shared coefficient: permuting features permutes
    the traces bit for bit, and the map x -> z is linear."""
    N, T, F = 20, 50, 6
    term, trunc = _flags(N, T, 13)
    rng = np.random.default_rng(14)
    x1, x2 = rng.standard_normal((N, T, F)), rng.standard_normal((N, T, F))
    perm = rng.permutation(F)
    z1 = oracle.elig_trace_vec(x1, term, trunc, gamma=G, lam=L)
    assert np.array_equal(oracle.elig_trace_vec(x1[:, :, perm], term, trunc, gamma=G, lam=L),
                          z1[:, :, perm])
    z2 = oracle.elig_trace_vec(x2, term, trunc, gamma=G, lam=L)
    z12 = oracle.elig_trace_vec(2.0 * x1 - x2, term, trunc, gamma=G, lam=L)
    rtol_close(z12, 2.0 * z1 - z2)


def test_elig_trace_vec_closed_form():
    """x = 1 in every feature, no flags: (1 - (gamma lambda)^(t+1)) / (1 - gamma lambda)."""
    T, F = 200, 4
    z = oracle.elig_trace_vec(np.ones((1, T, F)), gamma=G, lam=L)
    gl = g32 * l32
    ref = (1 - gl ** (np.arange(T) + 1)) / (1 - gl)
    for f in range(F):
        rtol_close(z[0, :, f], ref)


# ---------------------------------------------------------------- time-major [T, N] layout

def test_time_major_oracle_brute_force():
    """Each environment's column of the time-major arrays against the sum forms."""
    T, N = 14, 40
    rng = np.random.default_rng(21)
    term = (rng.random((T, N)) < 0.15).astype(np.uint8)
    trunc = (rng.random((T, N)) < 0.15).astype(np.uint8)
    r, v, bv, lr = (rng.standard_normal((T, N)) for _ in range(4))
    q, eq = rng.standard_normal((T, N)), rng.standard_normal((T, N))
    boot = rng.standard_normal(N)
    col = lambda a, n: a[:, n]
    adv, ret = oracle.time_major(oracle.gae, r, v, term, trunc, bv, boot, gamma=G, lam=L)
    assert adv.shape == (T, N)
    rtol_close(adv, np.array([brute.gae_sum(col(r, n), col(v, n), col(term, n), col(trunc, n),
                                            col(bv, n), boot[n], g32, l32) for n in range(N)]).T)
    rtol_close(ret, adv + v)
    vs, pg = oracle.time_major(oracle.vtrace, r, v, lr, term, trunc, bv, boot, gamma=G)
    res = [brute.vtrace_sum(col(r, n), col(v, n), col(lr, n), col(term, n), col(trunc, n),
                            col(bv, n), boot[n], g32, 1.0, 1.0) for n in range(N)]
    rtol_close(vs, np.array([a for a, _ in res]).T)
    rtol_close(pg, np.array([b for _, b in res]).T)
    dl, _ = oracle.time_major(oracle.retrace, r, q, eq, lr, term, trunc, bv, boot, gamma=G, lam=L)
    rtol_close(dl, np.array([brute.retrace_sum(col(r, n), col(q, n), col(eq, n), col(lr, n),
                                               col(term, n), col(trunc, n), col(bv, n), boot[n],
                                               g32, l32, 1.0)[0] for n in range(N)]).T)
    td = oracle.time_major(oracle.td_lambda, r, v, term, trunc, bv, boot, gamma=G, lam=L)
    rtol_close(td, np.array([brute.lambda_return(col(r, n), col(v, n), col(term, n),
                                                 col(trunc, n), col(bv, n), boot[n], g32, l32)
                             for n in range(N)]).T)
    dr = oracle.time_major(oracle.discounted, r, term, trunc, bv, boot, gamma=G)
    rtol_close(dr, np.array([brute.discounted_sum(col(r, n), col(term, n), col(trunc, n),
                                                  col(bv, n), boot[n], g32) for n in range(N)]).T)
    z = oracle.time_major(oracle.elig_trace, r, term, trunc, gamma=G, lam=L)
    rtol_close(z, np.array([brute.elig_sum(col(r, n), col(term, n), col(trunc, n), g32, l32)
                            for n in range(N)]).T)
    for starts in (False, True):
        c = oracle.time_major(oracle.episodic_prefix, r, term, trunc,
                              boundary="starts_at" if starts else "ends_at")
        rtol_close(c, np.array([brute.prefix_sum(col(r, n), col(term, n), col(trunc, n), starts)
                                for n in range(N)]).T)


# ---------------------------------------------------------------- observation-skip masking (Section 9.3)

def _compacted_masked_gae(r, v, mask, term, trunc, bv, B):
    """Masked GAE of one row from its definition by compaction: the unmasked steps form the
    sequence, a flag anywhere between an unmasked step and the next one (the first one found
    from the step itself) is that step's flag, with the continuation of the truncated step;
    the GAE sum form runs on that sequence; a masked step takes the advantage of the first
    step at or after it that is unmasked, or 0 if a flagged step or the window end comes
    first."""
    T = len(r)
    U = [t for t in range(T) if mask[t]]
    tc, rc, bc = [], [], []
    for i, u in enumerate(U):
        end = U[i + 1] if i + 1 < len(U) else T
        te = tr = 0
        b = 0.0
        for s in range(u, end):
            if term[s] or trunc[s]:
                te = 1 if term[s] else 0
                tr = 0 if term[s] else 1
                b = bv[s]
                break
        tc.append(te); rc.append(tr); bc.append(b)
    Ac = brute.gae_sum([r[u] for u in U], [v[u] for u in U], tc, rc, bc, B, g32, l32) if U else []
    pos = {u: i for i, u in enumerate(U)}
    A = []
    for t in range(T):
        if mask[t]:
            A.append(Ac[pos[t]])
            continue
        val = 0.0
        for s in range(t, T):
            if mask[s]:
                val = Ac[pos[s]]
                break
            if term[s] or trunc[s]:
                break
        A.append(val)
    return A


@pytest.mark.parametrize("p_mask", [0.2, 0.6, 0.9])
def test_gae_masked_against_compaction(p_mask):
    N, T = 150, 17
    rng = np.random.default_rng(int(100 * p_mask))
    x = random_inputs(N, T, seed=int(1000 * p_mask))
    term = (rng.random((N, T)) < 0.12).astype(np.uint8)
    trunc = (rng.random((N, T)) < 0.12).astype(np.uint8)
    mask = (rng.random((N, T)) >= p_mask).astype(np.uint8)
    mask[0] = 0  # a row with no unmasked step
    mask[1] = 1  # a row with every step unmasked
    adv, ret = oracle.gae_masked(x["r"], x["v"], mask, term, trunc, x["bv"], x["boot"], gamma=G,
                                 lam=L)
    ref = [_compacted_masked_gae(x["r"][n], x["v"][n], mask[n], term[n], trunc[n], x["bv"][n],
                                 x["boot"][n]) for n in range(N)]
    rtol_close(adv, ref)
    rtol_close(ret, np.asarray(ref) + x["v"])
    assert np.all(adv[0] == 0.0)


def test_gae_masked_exhaustive_small():
    """Every mask pattern of a 5-step row under every flag pattern of its steps."""
    T = 5
    term, trunc = all_flag_patterns(T)
    rng = np.random.default_rng(31)
    for mbits in range(2 ** T):
        mrow = np.array([(mbits >> k) & 1 for k in range(T)], np.uint8)
        N = term.shape[0]
        mask = np.tile(mrow, (N, 1))
        r, v, bv = (rng.standard_normal((N, T)) for _ in range(3))
        boot = rng.standard_normal(N)
        adv, _ = oracle.gae_masked(r, v, mask, term, trunc, bv, boot, gamma=G, lam=L)
        rtol_close(adv, [_compacted_masked_gae(r[n], v[n], mrow, term[n], trunc[n], bv[n], boot[n])
                         for n in range(N)])


def test_gae_masked_all_unmasked_is_gae():
    N, T = 40, 60
    x = random_inputs(N, T, 33)
    term, trunc = _flags(N, T, 33)
    ones = np.ones((N, T), np.uint8)
    a1, r1 = oracle.gae_masked(x["r"], x["v"], ones, term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    a0, r0 = oracle.gae_masked(x["r"], x["v"], None, term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    a2, r2 = oracle.gae(x["r"], x["v"], term, trunc, x["bv"], x["boot"], gamma=G, lam=L)
    assert np.array_equal(a1, a0) and np.array_equal(r1, r0)
    rtol_close(a1, a2)
    rtol_close(r1, r2)


def test_normalize_advantages_exact_moments():
    """Mean and unbiased variance of the steps that take part, from exactly rounded sums."""
    import math
    rng = np.random.default_rng(41)
    adv = 3.0 + 2.0 * rng.standard_normal((30, 50))
    mask = (rng.random((30, 50)) < 0.7).astype(np.uint8)
    eps = 1e-8
    out = oracle.normalize_advantages(adv, mask, eps=eps)
    sel = [float(a) for a, m in zip(adv.reshape(-1), mask.reshape(-1)) if m]
    n = len(sel)
    mean = math.fsum(sel) / n
    var = math.fsum((a - mean) ** 2 for a in sel) / (n - 1)
    rtol_close(out, (adv - mean) / math.sqrt(var + oracle.param(eps)))
    z = out[mask != 0]
    assert abs(math.fsum(z.tolist())) < 1e-9
    rtol_close(math.fsum(((z - z.mean()) ** 2).tolist()) / (n - 1), var / (var + oracle.param(eps)))
    # one step taking part: variance 0
    one = np.zeros_like(mask); one[3, 4] = 1
    out1 = oracle.normalize_advantages(adv, one, eps=eps)
    rtol_close(out1, (adv - adv[3, 4]) / math.sqrt(oracle.param(eps)))


# ---------------------------------------------------------------- memory discipline

def test_oracle_writes_only_its_outputs():
    """Every oracle routine writes exactly its [N, T] outputs: called through the C ABI with
    output buffers that carry 32 sentinel doubles before and after, the sentinels survive and
    every output element is written."""
    import ctypes
    lib = oracle._load()
    N, T, A, F, G = 3, 9, 4, 2, 32
    rng = np.random.default_rng(5)
    D, U8, I32 = ctypes.c_double, ctypes.c_uint8, ctypes.c_int32
    keep = []

    def data(*shape):
        x = np.ascontiguousarray(rng.normal(size=shape))
        keep.append(x)
        return x.ctypes.data_as(ctypes.POINTER(D))

    def flags(p):
        f = np.ascontiguousarray((rng.random((N, T)) < p).astype(np.uint8))
        keep.append(f)
        return f.ctypes.data_as(ctypes.POINTER(U8))

    def out(n):
        buf = np.full(n + 2 * G, 12345.0)
        buf[G:G + n] = np.nan
        keep.append(buf)
        return buf, buf[G:].ctypes.data_as(ctypes.POINTER(D))

    def check(bufs, n):
        for buf in bufs:
            assert np.all(buf[:G] == 12345.0) and np.all(buf[G + n:] == 12345.0)
            assert np.all(np.isfinite(buf[G:G + n]))

    g, lam = 0.99, 0.95
    nt = N * T
    o1, p1 = out(nt); o2, p2 = out(nt)
    lib.oracle_gae(data(N, T), data(N, T), flags(0.2), flags(0.2), data(N, T), data(N), p1, p2, N, T, g, lam)
    check((o1, o2), nt)
    o1, p1 = out(nt)
    lib.oracle_td_lambda(data(N, T), data(N, T), flags(0.2), flags(0.2), data(N, T), data(N), p1, N, T, g, lam)
    check((o1,), nt)
    o1, p1 = out(nt)
    lib.oracle_discounted(data(N, T), flags(0.2), flags(0.2), data(N, T), data(N), p1, N, T, g)
    check((o1,), nt)
    o1, p1 = out(nt); o2, p2 = out(nt)
    lib.oracle_vtrace(data(N, T), data(N, T), data(N, T), flags(0.2), flags(0.2), data(N, T), data(N),
                      p1, p2, N, T, g, 1.0, 1.0)
    check((o1, o2), nt)
    o1, p1 = out(nt); o2, p2 = out(nt)
    lib.oracle_retrace(data(N, T), data(N, T), data(N, T), data(N, T), flags(0.2), flags(0.2), data(N, T),
                       data(N), p1, p2, N, T, g, lam, 1.0)
    check((o1, o2), nt)
    acts = np.ascontiguousarray(rng.integers(-1, A + 1, size=(N, T)).astype(np.int32))
    mu = np.ascontiguousarray(rng.uniform(0.1, 1.0, size=(N, T)))
    keep += [acts, mu]
    o1, p1 = out(nt); o2, p2 = out(nt)
    lib.oracle_retrace_full(data(N, T), data(N, T, A), data(N, T, A), acts.ctypes.data_as(ctypes.POINTER(I32)),
                            mu.ctypes.data_as(ctypes.POINTER(D)), flags(0.2), flags(0.2), data(N, T), data(N),
                            p1, p2, N, T, A, g, lam, 1.0)
    check((o1, o2), nt)
    o1, p1 = out(nt)
    lib.oracle_elig_trace(data(N, T), flags(0.2), flags(0.2), p1, N, T, g, lam)
    check((o1,), nt)
    o1, p1 = out(nt * F)
    lib.oracle_elig_trace_vec(data(N, T, F), flags(0.2), flags(0.2), p1, N, T, F, g, lam)
    check((o1,), nt * F)
    o1, p1 = out(nt); o2, p2 = out(nt)
    lib.oracle_gae_masked(data(N, T), data(N, T), flags(0.6), flags(0.2), flags(0.2), data(N, T), data(N),
                          p1, p2, N, T, g, lam)
    check((o1, o2), nt)
    for starts_at in (0, 1):
        o1, p1 = out(nt)
        lib.oracle_episodic_prefix(data(N, T), flags(0.2), flags(0.2), p1, N, T, starts_at)
        check((o1,), nt)
    for reverse in (0, 1):
        o1, p1 = out(nt)
        lib.oracle_affine_scan(data(N, T), data(N, T), data(N), p1, N, T, reverse)
        check((o1,), nt)
