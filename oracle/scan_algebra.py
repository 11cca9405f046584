"""The combine operator of Eq. 2 and the Hillis-Steele scan of Appendix A, in plain Python.

TEST INFRASTRUCTURE ONLY (part of the oracle): these pin the algebra that the GPU scan relies
on. They are deliberately naive, operate on Python floats (fp64), and are only meant for the
small cases in the tests.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

Pair = Tuple[float, float]

IDENTITY: Pair = (0.0, 1.0)


def combine(earlier: Pair, later: Pair) -> Pair:
    """Eq. 2: (alpha_B, beta_B) (+) (alpha_A, beta_A) = (alpha_B + beta_B alpha_A, beta_A beta_B),
    where B is the chronologically earlier step (Section 2.2)."""
    a_b, b_b = earlier
    a_a, b_a = later
    return (a_b + b_b * a_a, b_a * b_b)


def hillis_steele_backward(alpha: Sequence[float], beta: Sequence[float]) -> List[List[Pair]]:
    """Appendix A: load the steps in reverse time order (position 1 = last step), then in pass
    k every position combines its current tuple with the one 2**(k-1) positions to its left,
    all reads happening before any write. Returns the list of tuples after each pass, indexed
    by position (position 0 here is the paper's position 1, i.e. the last step).

    The final pass leaves at position i the tuple covering time steps T-1-i .. T-1, whose alpha
    is A_{T-1-i} for a zero carry."""
    T = len(alpha)
    assert len(beta) == T
    cur: List[Pair] = [(float(alpha[T - 1 - i]), float(beta[T - 1 - i])) for i in range(T)]
    history = [list(cur)]
    stride = 1
    while stride < T:
        nxt = list(cur)
        for i in range(stride, T):
            # cur[i] covers chronologically earlier steps than cur[i - stride]
            nxt[i] = combine(cur[i], cur[i - stride])
        cur = nxt
        history.append(list(cur))
        stride *= 2
    return history


def scan_backward_by_combine(alpha: Sequence[float], beta: Sequence[float],
                             carry: float = 0.0) -> List[float]:
    """A_t for all t from the last Hillis-Steele pass, with the carry A_T applied afterwards as
    scan_alpha + scan_beta * carry (Section 4.1, step 4)."""
    T = len(alpha)
    if T == 0:
        return []
    final = hillis_steele_backward(alpha, beta)[-1]
    out = [0.0] * T
    for i, (a, b) in enumerate(final):
        out[T - 1 - i] = a + b * carry
    return out
