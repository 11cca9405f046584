"""CPU emulation of flat_rows_kernel's lane geometry (csrc/rlcs_kernels.h; plan in
csrc/rlcs_dispatch.h), restated from the kernel. For dense rows of T steps, T a multiple of K,
K < T <= 256*K (float32, K = 4) or 64*K (bfloat16, K = 8), and not a power of two of at most 64*K
steps: workgroup g owns rows [g*R, g*R + R), R = floor(256*K / T),
the range [lo, hi) = [g*R*T, min(g*R + R, N)*T); lane l of wave w holds the K steps at offset
q = (64*w + g(l))*K (g(l) = 63 - l backward, l forward), live when lo + q < hi; its row is
g*R + floor(q * magic / 2^22), magic = ceil(2^22 / T), and its step q - T*floor(q / T).
Checked: the multiply-shift division is exact for every (K, T, q) the kernel sees; the live lanes
cover every (row, step group) exactly once, each in one row; the neighbour a live lane takes (lane
l-1 through the wave shift, or lane 0's read at p0 + K backward / p0 - 1 forward) is the adjacent
step of the same row whenever the lane's edge step is not a row edge, and lane 0's read address
lies inside the range then; and the bf16 whole-line stores of each wave ([lo + 512*w, ...) up to
hi) cover exactly the live lanes' outputs. Nothing here runs on a GPU."""
import pytest

WAVE, W = 64, 4


def magic(T):
    return ((1 << 22) + T - 1) // T


def flat_max(K):
    return W * WAVE * K if K == 4 else WAVE * K


def is_flat(T, K):
    return T % K == 0 and K < T <= flat_max(K) and not ((T & (T - 1)) == 0 and T <= WAVE * K)


def flat_shapes(K):
    return [T for T in range(2 * K, flat_max(K) + 1, K) if is_flat(T, K)]


@pytest.mark.parametrize("K", [4, 8])
def test_multiply_shift_division_is_exact(K):
    for T in flat_shapes(K):
        m = magic(T)
        for q in range(0, W * WAVE * K):
            assert (q * m) >> 22 == q // T, (K, T, q)
        assert (W * WAVE * K - 1) * m < 2 ** 32  # no overflow of the 32-bit product


def lanes(N, T, K, backward):
    R = W * WAVE * K // T
    for wg in range(-(-N // R)):
        row0 = wg * R
        lo, hi = row0 * T, min(row0 + R, N) * T
        for wave in range(W):
            for lane in range(WAVE):
                g = WAVE - 1 - lane if backward else lane
                q = (wave * WAVE + g) * K
                p0 = lo + q
                live = p0 < hi
                r_in = (q * magic(T)) >> 22
                yield dict(wg=wg, wave=wave, lane=lane, g=g, lo=lo, hi=hi, p0=p0, live=live,
                           row=row0 + r_in, t=q - r_in * T)


@pytest.mark.parametrize("K", [4, 8])
@pytest.mark.parametrize("backward", [False, True])
@pytest.mark.parametrize("N,T", [(1, 12), (7, 20), (5, 24), (33, 40), (100, 96), (13, 136),
                                 (9, 192), (64, 200), (3, 240), (17, 252), (11, 264), (4, 504),
                                 (50, 100), (5, 300), (7, 500), (6, 512), (3, 1000), (5, 1020),
                                 (4, 1024)])
def test_flat_lanes_cover_rows_and_neighbours(N, T, K, backward):
    if not is_flat(T, K):
        pytest.skip("not a flat-rows shape for this K")
    L = list(lanes(N, T, K, backward))
    seen = set()
    where = {}
    for x in L:
        if not x["live"]:
            continue
        row, t = x["row"], x["t"]
        assert 0 <= row < N and t % K == 0 and t + K <= T
        assert x["p0"] == row * T + t
        assert (row, t) not in seen
        seen.add((row, t))
        where[(x["wg"], x["wave"], x["lane"])] = x
    assert seen == {(n, t) for n in range(N) for t in range(0, T, K)}
    for (wg, wave, lane), x in where.items():
        row, t = x["row"], x["t"]
        at_edge = (t + K == T) if backward else (t == 0)
        if at_edge:
            continue
        want = (row, t + K) if backward else (row, t - K)
        if lane > 0:  # the wave shift: lane l-1 of the same wave
            y = where.get((wg, wave, lane - 1))
            assert y is not None and (y["row"], y["t"]) == want
        else:         # lane 0 reads the step from memory
            pn = x["p0"] + K if backward else x["p0"] - 1
            assert x["lo"] <= pn < x["hi"]
            assert pn == (want[0] * T + want[1] if backward else want[0] * T + want[1] + K - 1)
    if K == 8:  # whole-line stores per wave cover exactly the live outputs
        for wg in {x["wg"] for x in L}:
            for wave in range(W):
                xs = [x for x in L if x["wg"] == wg and x["wave"] == wave]
                lo, hi = xs[0]["lo"], xs[0]["hi"]
                base = lo + wave * WAVE * K
                pieces = [base + 4 * i for i in range(2 * WAVE) if base + 4 * i < hi]
                covered = sorted(p for x in xs if x["live"] for p in (x["p0"], x["p0"] + 4))
                assert covered == pieces
