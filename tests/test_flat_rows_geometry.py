"""CPU emulation of flat_rows_kernel's lane geometry (csrc/rlcs_kernels.h; plan in
csrc/rlcs_dispatch.h), restated from the kernel. For dense rows of T steps, K < T <= 1024*K
(float32, K = 4) or 64*K (bfloat16, K = 8), not a power of two of at most 64*K steps, N*T a
multiple of K: workgroup g of W waves owns rows [g*R, g*R + R), R the most whole rows in W*64*K
steps that is a multiple of K / gcd(T, K) (W = 4, or 16 for float32 rows of which no such R fits
four waves: rows of more than 1024 steps, or more than 256 not a multiple of K), the range
[lo, hi) = [g*R*T, min(g*R + R, N)*T); lane l of wave w holds the K steps
at offset q = (64*w + g(l))*K (g(l) = 63 - l backward, l forward), live when lo + q < hi; its row
is g*R + floor(q * magic / 2^s), magic = ceil(2^s / T) with s = 22 for four waves and 26 for
sixteen, and its step q - T*floor(q / T). Checked: the multiply-shift division is exact and its
32-bit product does not overflow for every (K, T, q) the kernel sees; sixteen waves are taken
only where four hold no aligned range; every range starts and ends on a vector boundary and the
live lanes cover every step exactly once; a lane holds at most one row edge, where the kernel's
edge computation puts it, and the per-row value it reads is that edge step's row's; the
neighbour a live lane takes (lane l-1 through the wave shift, or lane 0's read at p0 + K
backward / p0 - 1 forward) is the adjacent step whenever the lane's carry-source edge step is
not a row edge, and lane 0's read address lies inside the range then; and the bf16 whole-line
stores of each wave ([lo + 512*w, ...) up to hi) cover exactly the live lanes' outputs. Nothing
here runs on a GPU."""
import pytest

WAVE = 64


def shift(W):
    return 26 if W > 4 else 22


def magic(T, W=4):
    return ((1 << shift(W)) + T - 1) // T


def flat_max(K):
    return 16 * WAVE * K if K == 4 else WAVE * K


def plan(T, K):
    """(W, R) as the dispatcher picks them: R the most whole rows that fit W*64*K steps, a
    multiple of K / gcd(T, K) so that the range starts and ends on vector boundaries; four waves,
    or sixteen for float32 rows of which no such R fits four; (4, 0): not taken."""
    from math import gcd
    step = K // gcd(T, K)
    R = 4 * WAVE * K // T // step * step
    W = 4
    if R == 0 and K == 4:
        R, W = 16 * WAVE * K // T // step * step, 16
    if R > 0 and (W * WAVE * K - 1) * magic(T, W) >= 1 << 32:
        R = 0
    return W, R


def rows_per_group(T, K):
    return plan(T, K)[1]


def is_flat(T, K, N=None):
    return (K < T <= flat_max(K) and not ((T & (T - 1)) == 0 and T <= WAVE * K)
            and rows_per_group(T, K) > 0 and (N is None or (N * T) % K == 0))


def flat_shapes(K):
    return [T for T in range(K + 1, flat_max(K) + 1) if is_flat(T, K)]


@pytest.mark.parametrize("K", [4, 8])
def test_multiply_shift_division_is_exact(K):
    for T in flat_shapes(K):
        W = plan(T, K)[0]
        m = magic(T, W)
        for q in range(0, W * WAVE * K):
            assert (q * m) >> shift(W) == q // T, (K, T, q)
        assert (W * WAVE * K - 1) * m < 2 ** 32  # no overflow of the 32-bit product


def test_sixteen_waves_only_where_four_hold_no_aligned_range():
    for T in flat_shapes(4):
        W, R = plan(T, 4)
        if W == 16:
            assert T > 256 and 4 * WAVE * 4 // T // (4 // __import__("math").gcd(T, 4)) == 0
    assert plan(1001, 4) == (16, 4) and plan(499, 4) == (16, 8) and plan(1023, 4) == (16, 4)
    assert plan(255, 4) == (4, 4) and plan(250, 4)[0] == 4


def lanes(N, T, K, backward):
    W, R = plan(T, K)
    for wg in range(-(-N // R)):
        row0 = wg * R
        lo, hi = row0 * T, min(row0 + R, N) * T
        for wave in range(W):
            for lane in range(WAVE):
                g = WAVE - 1 - lane if backward else lane
                q = (wave * WAVE + g) * K
                p0 = lo + q
                live = p0 < hi
                r_in = (q * magic(T, W)) >> shift(W)
                yield dict(wg=wg, wave=wave, lane=lane, g=g, lo=lo, hi=hi, p0=p0, live=live,
                           row=row0 + r_in, t=q - r_in * T)


@pytest.mark.parametrize("K", [4, 8])
@pytest.mark.parametrize("backward", [False, True])
@pytest.mark.parametrize("N,T", [(8, 1001), (12, 499), (8, 1023), (4, 1001), (16, 259), (6, 514),
                                 (5, 2000), (3, 3000), (2, 4096), (7, 1100), (4, 1500), (9, 2048),
                                 (1, 12), (7, 20), (5, 24), (33, 40), (100, 96), (13, 136),
                                 (9, 192), (64, 200), (3, 240), (17, 252), (11, 264), (4, 504),
                                 (50, 100), (5, 300), (7, 500), (6, 512), (3, 1000), (5, 1020),
                                 (4, 1024), (8, 255), (16, 255), (12, 129), (8, 100), (16, 101),
                                 (8, 251), (4, 1001), (8, 33), (32, 9)])
def test_flat_lanes_cover_rows_and_neighbours(N, T, K, backward):
    if not is_flat(T, K, N):
        pytest.skip("not a flat-rows shape for this K")
    W = plan(T, K)[0]
    L = list(lanes(N, T, K, backward))
    seen = set()
    where = {}
    for x in L:
        if not x["live"]:
            continue
        assert x["lo"] % K == 0 and x["hi"] % K == 0  # whole, aligned vectors
        p0 = x["p0"]
        assert p0 == x["row"] * T + x["t"] and 0 <= x["t"] < T
        for k in range(K):  # each step once
            assert p0 + k not in seen
            seen.add(p0 + k)
        where[(x["wg"], x["wave"], x["lane"])] = x
    assert seen == set(range(N * T))
    for (wg, wave, lane), x in where.items():
        t = x["t"]
        # at most one row edge in the lane (T >= K); the lane's carry-source edge step is a row
        # edge exactly when the kernel's edge bit sits there
        edges = [k for k in range(K) if (t + k) % T == (T - 1 if backward else 0)]
        assert len(edges) <= 1
        if backward:
            ke = T - 1 - t if t + K >= T else -1
        else:
            ke = 0 if t == 0 else (T - t if t + K > T else -1)
        assert edges == ([ke] if ke >= 0 else [])
        if ke >= 0:  # the per-row value read for the edge belongs to the edge step's row
            row_e = x["row"] + 1 if (not backward and ke > 0) else x["row"]
            assert (x["p0"] + ke) // T == row_e
        if ke == (K - 1 if backward else 0):
            continue
        want = x["p0"] + K if backward else x["p0"] - K  # the adjacent group's first step
        if lane > 0:  # the wave shift: lane l-1 of the same wave
            y = where.get((wg, wave, lane - 1))
            assert y is not None and y["p0"] == want
        else:         # lane 0 reads the step from memory, inside the range
            pn = x["p0"] + K if backward else x["p0"] - 1
            assert x["lo"] <= pn < x["hi"]
    if K == 8:  # whole-line stores per wave cover exactly the live outputs
        for wg in {x["wg"] for x in L}:
            for wave in range(W):
                xs = [x for x in L if x["wg"] == wg and x["wave"] == wave]
                lo, hi = xs[0]["lo"], xs[0]["hi"]
                base = lo + wave * WAVE * K
                pieces = [base + 4 * i for i in range(2 * WAVE) if base + 4 * i < hi]
                covered = sorted(p for x in xs if x["live"] for p in (x["p0"], x["p0"] + 4))
                assert covered == pieces
