"""CPU emulation of vec_rows_kernel (csrc/rlcs_vec.h; host choice in vec_rows_launch), restated
from the kernel: eligibility traces of F-vectors, F = L * V with V = 4 float32 (8 bfloat16)
features per lane and L a power of two up to 64, S = 64 / L step groups per wave, 4 consecutive
steps per lane, W the fewest waves (a power of two) that hold a row, and R = W * 4S / T whole
rows per workgroup scanned as one range. Checked: the host's choice (wave count, LDS bound,
rows per workgroup, fewest workgroups); every feature of every step of a range is loaded once
(in one 16-byte piece of its wave's staged span for steps under 128 bytes, where each lane then
takes its own steps' features from the staged pieces) and no access leaves the range; the
output slot pieces stay inside the wave's slot and the whole-line stores of the waves write
every output of the range once and nothing past it; the flag word of a lane never crosses the
range's end; and the kernel's order of composition (lane steps, a scan over lanes L apart, the
map of the earlier step groups, the earlier waves through LDS), with a row start wherever a
step's place in its row is 0, reproduces the recurrence z_t = beta_t z_{t-1} + x_t of every row
in float64, the last workgroup's partial range included. Nothing here runs on a GPU."""
import numpy as np
import pytest

WAVE, KS, MAX_LDS, MIN_GROUPS = 64, 4, 160 * 1024, 256


def lds_bytes(W, F, V):
    return W * WAVE * KS * V * 4 + W * F * 4 + W * 4


def plan(T, F, V, N=1 << 20):
    """(L, S, W, R) as vec_rows_launch picks them, or None when the row kernel is not taken."""
    if F % V:
        return None
    L = F // V
    if L > WAVE or L & (L - 1):
        return None
    S = WAVE // L
    W = 1
    while W < 16 and W * S * KS < T:
        W *= 2
    if W * S * KS < T or lds_bytes(W, F, V) > MAX_LDS:
        return None
    R = W * S * KS // T
    if -(-N // R) < MIN_GROUPS:
        return None
    return L, S, W, R


SHAPES = [(4096, 4, 4), (2048, 4, 4), (1999, 4, 4), (1024, 16, 4), (777, 16, 4), (2048, 8, 8),
          (1000, 16, 8), (64, 256, 4), (65, 8, 4), (1, 8, 4), (3, 16, 4), (511, 16, 4),
          (512, 16, 4), (65, 16, 4), (32, 16, 4), (255, 32, 4), (33, 64, 4), (5, 64, 4),
          (64, 128, 4), (31, 256, 4), (32, 256, 4), (100, 16, 4), (256, 16, 4), (1024, 8, 8),
          (257, 16, 8), (63, 64, 8), (16, 512, 8), (5, 512, 8), (2, 512, 8), (7, 8, 8)]


@pytest.mark.parametrize("T,F,V", SHAPES)
def test_plan_takes_the_shape_within_lds(T, F, V):
    p = plan(T, F, V)
    assert p is not None, (T, F, V)
    L, S, W, R = p
    assert W * S * KS >= T and (W == 1 or (W // 2) * S * KS < T)
    assert R >= 1 and R * T <= W * S * KS < (R + 1) * T
    assert lds_bytes(W, F, V) <= MAX_LDS and W * WAVE <= 1024


def test_plan_declines():
    assert plan(256, 12, 4) is None        # L = 3, not a power of two
    assert plan(256, 6, 4) is None         # F not a multiple of V
    assert plan(256, 16, 4, N=255) is None  # too few workgroups
    assert plan(32, 16, 4, N=510) is None  # two rows a workgroup: 256 workgroups need 511 rows
    assert plan(32, 16, 4, N=511) is not None
    assert plan(1025, 16, 4) is None       # needs 32 waves
    assert plan(4096, 4, 4) is not None and plan(4097, 4, 4) is None
    assert plan(65, 256, 4) is None        # L = 64: 4 steps per wave, 16 waves too many
    assert plan(256, 1024, 8) is None      # L = 128


def ranges(N, T, R):
    """(workgroup, first row, steps) of every workgroup."""
    for g in range(-(-N // R)):
        row0 = g * R
        yield g, row0, (min(row0 + R, N) - row0) * T


def lanes(S, L, W):
    for wave in range(W):
        for lane in range(WAVE):
            fg, sg = lane % L, lane // L
            yield wave, lane, fg, sg, (wave * S + sg) * KS


def rows_for(T, F, V):
    """Row counts that give a few full workgroups and a partial last one."""
    L, S, W, R = plan(T, F, V)
    return [3 * R + max(1, R // 2), R]


@pytest.mark.parametrize("T,F,V", SHAPES)
def test_loads_cover_each_range_once(T, F, V):
    """Steps under 128 bytes (L < 8): each wave loads 16-byte pieces i * 64 + lane (i < 4) of its
    span up to the range's end into its slot; a lane then takes piece (sg * 4 + k) * L + fg for
    its step k, which must have been loaded and hold the features [V fg, V fg + V) of step
    t0 + k. Longer steps: each lane loads its own steps' vectors, inside the range."""
    L, S, W, R = plan(T, F, V)
    for N in rows_for(T, F, V):
        for g, row0, E in ranges(N, T, R):
            seen = np.zeros((E, F), dtype=np.int64)
            loaded = {}
            if L < 8:
                for wave in range(W):
                    wbase = wave * S * KS * F
                    for i in range(KS):
                        for lane in range(WAVE):
                            p = wbase + (i * WAVE + lane) * V  # element offset in the range
                            if p < E * F:
                                assert p + V <= E * F and p % V == 0
                                loaded[(wave, i * WAVE + lane)] = p
                                t, f = divmod(p, F)
                                seen[t, f:f + V] += 1
            for wave, lane, fg, sg, t0 in lanes(S, L, W):
                nv = max(0, min(KS, E - t0))
                for k in range(nv):
                    if L < 8:
                        piece = (sg * KS + k) * L + fg
                        assert piece < KS * WAVE  # inside the input half of the slot
                        assert loaded[(wave, piece)] == (t0 + k) * F + fg * V
                    else:
                        p = (t0 + k) * F + fg * V
                        assert p + V <= E * F
                        seen[t0 + k, fg * V:(fg + 1) * V] += 1
                if nv and T % 4 == 0:  # flag word of steps t0 .. t0 + 3 (row0 * T is aligned)
                    assert t0 % 4 == 0 and t0 + 3 < E
            assert np.all(seen == 1)


@pytest.mark.parametrize("T,F,V", SHAPES)
def test_slot_pieces_and_stores(T, F, V):
    L, S, W, R = plan(T, F, V)
    pieces = WAVE * KS * V // 4
    for N in rows_for(T, F, V):
        for g, row0, E in ranges(N, T, R):
            written = np.zeros(E * F, dtype=np.int64)
            for wave in range(W):
                slot = np.full(pieces, -1)
                for lane in range(WAVE):
                    fg, sg = lane % L, lane // L
                    for k in range(KS):
                        piece = ((sg * KS + k) * F + fg * V) // 4
                        for i in range(V // 4):
                            assert 0 <= piece + i < pieces
                            assert slot[piece + i] == -1
                            slot[piece + i] = 1
                assert np.all(slot == 1)  # the lanes fill the slot exactly
                wbase = wave * S * KS * F
                for i in range(pieces // WAVE):
                    span = []
                    for lane in range(WAVE):
                        p = wbase + 4 * (i * WAVE + lane)
                        if p < E * F:
                            written[p:p + 4] += 1
                            span.append(p)
                    if len(span) == WAVE:  # a whole instruction: 1 KB of consecutive outputs
                        assert span == list(range(span[0], span[0] + 4 * WAVE, 4))
            assert np.all(written == 1)


def emulate_range(x, done, T, decay, F, V):
    """The kernel's arithmetic for one workgroup's range in float64: x [E, F] (the range's steps),
    done [E] (episode ends), T the row length (a row starts where the step's place is 0)."""
    E = x.shape[0]
    L, S, W, R = plan(T, F, V)
    nlanes = W * WAVE
    off = np.zeros((nlanes, V))
    fac = np.ones(nlanes)
    be_all = np.ones((nlanes, KS))
    xv_all = np.zeros((nlanes, KS, V))
    for wave, lane, fg, sg, t0 in lanes(S, L, W):
        i = wave * WAVE + lane
        nv = max(0, min(KS, E - t0))
        r = t0 % T
        for k in range(nv):
            xv_all[i, k] = x[t0 + k, fg * V:(fg + 1) * V]
            cut = r == 0 or done[t0 + k - 1]
            be_all[i, k] = 0.0 if cut else decay
            r = 0 if r + 1 == T else r + 1
        o, f = xv_all[i, 0].copy(), be_all[i, 0]
        for k in range(1, KS):
            o = be_all[i, k] * o + xv_all[i, k]
            f *= be_all[i, k]
        off[i], fac[i] = o, f
    # scan over lanes L apart within each wave (Hillis-Steele, as the shuffles do)
    eo = np.zeros((nlanes, V))
    ef = np.ones(nlanes)
    for wave in range(W):
        base = wave * WAVE
        d = 1
        while d < S:
            po, pf = off[base:base + WAVE].copy(), fac[base:base + WAVE].copy()
            for lane in range(WAVE):
                if lane // L >= d:
                    i = base + lane
                    off[i] = fac[i] * po[lane - d * L] + off[i]
                    fac[i] = fac[i] * pf[lane - d * L]
            d *= 2
        for lane in range(L, WAVE):
            eo[base + lane], ef[base + lane] = off[base + lane - L], fac[base + lane - L]
    s_off = np.zeros((W, F))
    s_fac = np.ones(W)
    for wave in range(W):
        for fg in range(L):
            s_off[wave, fg * V:(fg + 1) * V] = off[wave * WAVE + (S - 1) * L + fg]
        s_fac[wave] = fac[wave * WAVE + (S - 1) * L]
    z = np.zeros((E, F))
    for wave, lane, fg, sg, t0 in lanes(S, L, W):
        i = wave * WAVE + lane
        X = np.zeros(V)
        for j in range(wave):
            X = s_fac[j] * X + s_off[j, fg * V:(fg + 1) * V]
        X = ef[i] * X + eo[i]
        for k in range(KS):
            X = be_all[i, k] * X + xv_all[i, k]
            if t0 + k < E:
                z[t0 + k, fg * V:(fg + 1) * V] = X
    return z


def direct(x, done, decay):
    """Rows [n, T, F], done [n, T]: the recurrence row by row."""
    z = np.zeros_like(x)
    for n in range(x.shape[0]):
        prev = np.zeros(x.shape[2])
        for t in range(x.shape[1]):
            beta = 0.0 if t == 0 or done[n, t - 1] else decay
            prev = beta * prev + x[n, t]
            z[n, t] = prev
    return z


@pytest.mark.parametrize("T,F,V", [(2048, 4, 4), (1999, 4, 4), (65, 8, 4), (1, 8, 4), (3, 16, 4),
                                   (511, 16, 4), (65, 16, 4), (32, 16, 4), (255, 32, 4),
                                   (33, 64, 4), (5, 64, 4), (31, 256, 4), (257, 16, 8),
                                   (63, 64, 8), (5, 512, 8), (2, 512, 8), (7, 8, 8)])
def test_composition_order_reproduces_the_recurrence(T, F, V):
    L, S, W, R = plan(T, F, V)
    rng = np.random.default_rng(T * 1000 + F)
    N = 2 * R + max(1, R // 2)  # two full workgroups and a partial one
    x = rng.standard_normal((N, T, F))
    for done, decay in ((rng.random((N, T)) < 0.05, 0.99 * 0.95), (np.zeros((N, T), bool), 1.0)):
        want = direct(x, done, decay)
        for g, row0, E in ranges(N, T, R):
            rows = E // T
            z = emulate_range(x[row0:row0 + rows].reshape(E, F), done[row0:row0 + rows].reshape(E),
                              T, decay, F, V)
            np.testing.assert_allclose(z.reshape(rows, T, F), want[row0:row0 + rows],
                                       rtol=1e-9, atol=1e-9)
