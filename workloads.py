"""Seeded synthetic rollout generators shared by the tests, the bench and the smoke check.

This module only draws random inputs; it contains none of the estimators' arithmetic.
Every array it returns is a plain numpy array on the host:

* floating inputs are float32 arrays, or for ``dtype="bf16"`` uint16 arrays holding bfloat16
  bit patterns (the float32 draw rounded to nearest-even, which is how a bf16 rollout buffer
  would be produced);
* flags are uint8 arrays of 0/1 (``term`` and ``trunc``; both may be set at one step);
* ``boot`` is float32/bf16 of shape ``[N]``; everything else is ``[N, T]`` row-major.

The paper evaluates on synthetic rollouts in three regimes (few environments with short
rollouts; thousands of environments; long RLHF-style rows, Sections 1, 7.1 and 9.1) without
stating the value distributions, so the distributions below are a stated choice:
rewards, values, Q-values, truncation continuations and bootstraps ~ N(0, 1); behaviour and
target log-probabilities ~ N(0, 0.5) whose difference is log-rho; flags ~ Bernoulli.

Draw order is fixed (rewards, values, bootstrap[N], bv, log-pi, log-mu, q_taken, expected_q,
term, trunc) so that any one array can be regenerated from the seed alone.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "Rollout",
    "make_rollout",
    "make_rlhf_rollout",
    "make_affine",
    "make_retrace_full",
    "make_rollout_time_major",
    "make_multiturn",
    "make_vector_trace",
    "bf16_bits_from_f32",
    "f32_from_bf16_bits",
    "CONFIGS",
]


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even) and return the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    return ((u + rounding) >> 16).astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 exactly."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Rollout(dict):
    """A dict of input arrays plus the shape and dtype they were generated with."""

    def __init__(self, N: int, T: int, dtype: str, **arrays):
        super().__init__(**arrays)
        self.N, self.T, self.dtype = N, T, dtype


def _finish(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return bf16_bits_from_f32(x) if dtype == "bf16" else x


def make_rollout(N: int, T: int, seed: int = 0, *, dtype: str = "f32",
                 p_term: float = 0.02, p_trunc: float = 0.01,
                 logp_sigma: float = 0.5) -> Rollout:
    """Rollout buffer of ``N`` environment rows by ``T`` steps.

    ``p_trunc=0`` still returns an all-zero ``trunc`` array; callers decide whether to pass it.
    """
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    shape = (N, T)
    rewards = rng.standard_normal(shape, dtype=np.float32)
    values = rng.standard_normal(shape, dtype=np.float32)
    boot = rng.standard_normal((N,), dtype=np.float32)
    bv = rng.standard_normal(shape, dtype=np.float32)
    logp_pi = (logp_sigma * rng.standard_normal(shape)).astype(np.float32)
    logp_mu = (logp_sigma * rng.standard_normal(shape)).astype(np.float32)
    q_taken = rng.standard_normal(shape, dtype=np.float32)
    expected_q = rng.standard_normal(shape, dtype=np.float32)
    term = (rng.random(shape) < p_term).astype(np.uint8)
    trunc = (rng.random(shape) < p_trunc).astype(np.uint8)
    log_rho = (logp_pi - logp_mu).astype(np.float32)
    return Rollout(
        N, T, dtype,
        r=_finish(rewards, dtype), v=_finish(values, dtype), boot=_finish(boot, dtype),
        bv=_finish(bv, dtype), log_rho=_finish(log_rho, dtype),
        q=_finish(q_taken, dtype), eq=_finish(expected_q, dtype),
        x=_finish(rewards, dtype),
        term=np.ascontiguousarray(term), trunc=np.ascontiguousarray(trunc),
    )


def make_rlhf_rollout(N: int, T: int, seed: int = 0, *, dtype: str = "f32",
                      kl_sigma: float = 0.01) -> Rollout:
    """Long-row RLHF-style rollout: a per-token KL penalty ~ N(0, kl_sigma) on every step plus
    a sequence-level score ~ N(0, 1) on the final step; values ~ N(0, 1); each row terminates
    at its last step only; no truncation."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    kl = (kl_sigma * rng.standard_normal((N, T))).astype(np.float32)
    score = rng.standard_normal((N,), dtype=np.float32)
    values = rng.standard_normal((N, T), dtype=np.float32)
    rewards = kl.copy()
    rewards[:, T - 1] += score
    term = np.zeros((N, T), dtype=np.uint8)
    if T > 0:
        term[:, T - 1] = 1
    trunc = np.zeros((N, T), dtype=np.uint8)
    zeros = np.zeros((N, T), dtype=np.float32)
    return Rollout(
        N, T, dtype,
        r=_finish(rewards, dtype), v=_finish(values, dtype),
        boot=_finish(np.zeros((N,), np.float32), dtype), bv=_finish(zeros, dtype),
        log_rho=_finish(zeros, dtype), q=_finish(values, dtype), eq=_finish(values, dtype),
        x=_finish(rewards, dtype), term=term, trunc=trunc,
    )


def make_affine(N: int, T: int, seed: int = 0, *, dtype: str = "f32",
                p_zero: float = 0.02) -> Rollout:
    """Coefficients for the bare recurrence: alpha ~ N(0, 1), beta ~ U(0, 1) with a fraction
    p_zero of exact zeros (episode cuts), one carry per row ~ N(0, 1)."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    alpha = rng.standard_normal((N, T), dtype=np.float32)
    beta = rng.random((N, T), dtype=np.float32)
    beta[rng.random((N, T)) < p_zero] = 0.0
    carry = rng.standard_normal((N,), dtype=np.float32)
    return Rollout(N, T, dtype, alpha=_finish(alpha, dtype), beta=_finish(beta, dtype),
                   carry=_finish(carry, dtype))


def _softmax(z: np.ndarray) -> np.ndarray:
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def make_retrace_full(N: int, T: int, A: int, seed: int = 0, *, dtype: str = "f32",
                      p_term: float = 0.02, p_trunc: float = 0.01,
                      logit_sigma: float = 1.0) -> Rollout:
    """Rollout for Retrace in its full form: Q(s_t, .) ~ N(0, 1) over A actions, target and
    behaviour policies as softmaxes of independent N(0, logit_sigma) logits, actions drawn from
    the behaviour policy, mu = the behaviour probability of the drawn action (all [N, T] or
    [N, T, A]); rewards, truncation continuations (E_pi Q of the true successor) and
    bootstraps ~ N(0, 1); Bernoulli flags. Actions are int32."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    rewards = rng.standard_normal((N, T), dtype=np.float32)
    q = rng.standard_normal((N, T, A), dtype=np.float32)
    pi = _softmax(logit_sigma * rng.standard_normal((N, T, A))).astype(np.float32)
    mu_all = _softmax(logit_sigma * rng.standard_normal((N, T, A)))
    u = rng.random((N, T, 1))
    actions = np.minimum((np.cumsum(mu_all, axis=-1) < u).sum(axis=-1), A - 1).astype(np.int32)
    mu = np.take_along_axis(mu_all, actions[..., None].astype(np.int64), axis=-1)[..., 0]
    boot = rng.standard_normal((N,), dtype=np.float32)
    bv = rng.standard_normal((N, T), dtype=np.float32)
    term = (rng.random((N, T)) < p_term).astype(np.uint8)
    trunc = (rng.random((N, T)) < p_trunc).astype(np.uint8)
    ro = Rollout(N, T, dtype, r=_finish(rewards, dtype), q3=_finish(q, dtype),
                 pi3=_finish(pi, dtype), mu=_finish(mu.astype(np.float32), dtype),
                 actions=np.ascontiguousarray(actions), bv=_finish(bv, dtype),
                 boot=_finish(boot, dtype), term=term, trunc=trunc)
    ro.A = A
    return ro


def make_rollout_time_major(T: int, N: int, seed: int = 0, **kw) -> Rollout:
    """The rollout of ``make_rollout(N, T, seed, **kw)`` stored time-major: every [N, T] array
    becomes its [T, N] transpose (step t of environment n at [t, n]); ``boot`` stays [N]."""
    ro = make_rollout(N, T, seed, **kw)
    out = Rollout(N, T, ro.dtype)
    for k, v in ro.items():
        out[k] = np.ascontiguousarray(v.T) if v.ndim == 2 else v
    return out


def make_multiturn(N: int, T: int, seed: int = 0, *, dtype: str = "f32", mean_action: float = 48.0,
                   mean_obs: float = 96.0, kl_sigma: float = 0.01) -> Rollout:
    """Multi-turn / tool-use rows for masked GAE: each row alternates runs of observation
    tokens (mask 0; the row starts with one, the prompt) and action tokens (mask 1) with
    geometric run lengths of the given means; a per-token KL penalty ~ N(0, kl_sigma) on action
    tokens plus a score ~ N(0, 1) on the row's last action token; values ~ N(0, 1); the row
    terminates at its last step; no truncation; zero bootstrap."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    mask = np.zeros((N, T), dtype=np.uint8)
    for n in range(N):
        t, act = 0, False
        while t < T:
            run = int(rng.geometric(1.0 / (mean_action if act else mean_obs)))
            mask[n, t:t + run] = 1 if act else 0
            t += run
            act = not act
    kl = (kl_sigma * rng.standard_normal((N, T))).astype(np.float32) * mask
    score = rng.standard_normal((N,), dtype=np.float32)
    rewards = kl.copy()
    for n in range(N):
        idx = np.nonzero(mask[n])[0]
        if idx.size:
            rewards[n, idx[-1]] += score[n]
    values = rng.standard_normal((N, T), dtype=np.float32)
    term = np.zeros((N, T), dtype=np.uint8)
    if T > 0:
        term[:, T - 1] = 1
    zeros = np.zeros((N, T), dtype=np.float32)
    return Rollout(N, T, dtype, r=_finish(rewards, dtype), v=_finish(values, dtype),
                   bv=_finish(zeros, dtype), boot=_finish(np.zeros((N,), np.float32), dtype),
                   term=term, trunc=np.zeros((N, T), dtype=np.uint8), mask=mask)


def make_vector_trace(N: int, T: int, F: int, seed: int = 0, *, dtype: str = "f32",
                      p_term: float = 0.02, p_trunc: float = 0.01) -> Rollout:
    """Inputs of eligibility traces over F-vectors (linear function approximation): feature
    vectors x [N, T, F] ~ N(0, 1) and Bernoulli flags [N, T]."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(f"dtype must be 'f32' or 'bf16', got {dtype!r}")
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, T, F), dtype=np.float32)
    term = (rng.random((N, T)) < p_term).astype(np.uint8)
    trunc = (rng.random((N, T)) < p_trunc).astype(np.uint8)
    ro = Rollout(N, T, dtype, x=_finish(x, dtype), term=term, trunc=trunc)
    ro.F = F
    return ro


# The five synthetic workloads (shapes, dtypes, flag rates and parameters).
CONFIGS = {
    "gae_8x128": dict(N=8, T=128, dtype="f32", p_term=0.01, p_trunc=0.0,
                      gamma=0.99, lam=0.95, trunc=False, estimators=("gae",)),
    "all7_4096x32": dict(N=4096, T=32, dtype="f32", p_term=0.02, p_trunc=0.01,
                         gamma=0.99, lam=0.95, trunc=True,
                         estimators=("gae", "vtrace", "retrace", "td_lambda", "discounted",
                                     "elig_trace", "episodic_prefix")),
    "gae_vtrace_4096x256": dict(N=4096, T=256, dtype="f32", p_term=0.02, p_trunc=0.01,
                                gamma=0.99, lam=0.95, trunc=True,
                                estimators=("gae", "vtrace")),
    "rlhf_64x4096": dict(N=64, T=4096, dtype="f32", gamma=1.0, lam=0.95, trunc=False,
                         rlhf=True, estimators=("gae", "td_lambda")),
    "sweep_bf16": dict(N=(16384, 65536), T=(64, 512, 2048), dtype="bf16", p_term=0.005,
                       p_trunc=0.005, gamma=0.99, lam=0.95, trunc=True,
                       estimators=("gae", "vtrace", "retrace", "td_lambda", "discounted",
                                   "elig_trace", "episodic_prefix")),
}
