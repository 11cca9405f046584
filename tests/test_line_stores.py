"""CPU emulation of the whole-line store of eight outputs per lane (store8_lines in
csrc/rlcs_device.h), restated here from the kernel: a wave whose lane l holds the eight outputs of
group g(l) of its 512 consecutive outputs [base, base + 512) writes them into a 2 KB slot as two
16-byte pieces (2g and 2g + 1), then lane l stores pieces l and 64 + l at base + 4l and
base + 256 + 4l, skipping pieces at or past `limit`. The memory this leaves must equal what the
lanes' own two stores each would leave (lanes whose group lies past `limit` storing nothing), for
forward lanes (g = l), backward lanes (g = 63 - l) and the masked kernels' backward layout, with
the limit anywhere on a group boundary (a partial last wave); and every store instruction must
cover whole 128-byte lines of a 16-byte aligned base. Nothing here runs on a GPU."""
import numpy as np
import pytest

WAVE, K = 64, 8


def per_lane(mem, base, limit, groups, vals):
    """Each lane's two 16-byte stores of its own eight outputs (the form replaced)."""
    for lane in range(WAVE):
        p0 = base + K * groups[lane]
        if p0 < limit:
            mem[p0:p0 + K] = vals[lane]


def line_stores(mem, base, limit, groups, vals):
    """store8_lines: the slot exchange, then pieces l and 64 + l per lane. Returns the byte
    ranges each of the two store instructions wrote."""
    slot = np.full((2 * WAVE, 4), np.nan)
    for lane in range(WAVE):
        g = groups[lane]
        slot[2 * g] = vals[lane][:4]
        slot[2 * g + 1] = vals[lane][4:]
    spans = []
    for j in range(2):
        wrote = []
        for lane in range(WAVE):
            p = base + 4 * lane + 4 * WAVE * j
            if p < limit:
                mem[p:p + 4] = slot[WAVE * j + lane]
                wrote.append((4 * p, 4 * p + 16))
        spans.append(wrote)
    return spans


@pytest.mark.parametrize("layout", ["forward", "backward"])
@pytest.mark.parametrize("live_groups", [64, 63, 33, 32, 31, 1, 0])
def test_line_stores_equal_per_lane_stores(layout, live_groups):
    rng = np.random.default_rng(live_groups * 2 + (layout == "backward"))
    groups = list(range(WAVE)) if layout == "forward" else [WAVE - 1 - l for l in range(WAVE)]
    base = 512 * 3  # a wave's span starts on a multiple of 512 outputs (2 KB)
    limit = base + K * live_groups  # N*T: a multiple of K, possibly inside the wave's span
    vals = [rng.standard_normal(K) for _ in range(WAVE)]
    a = np.full(base + 1024, -7.0)
    b = a.copy()
    per_lane(a, base, limit, groups, vals)
    spans = line_stores(b, base, limit, groups, vals)
    assert np.array_equal(a, b)
    assert np.all(b[limit:] == -7.0)  # nothing at or past the limit
    # a full wave: each store instruction covers 1 KB of whole, 128-byte aligned lines
    if live_groups == WAVE:
        for wrote in spans:
            lo, hi = min(w[0] for w in wrote), max(w[1] for w in wrote)
            assert hi - lo == 1024 and lo % 128 == 0
            assert sorted(wrote) == [(lo + 16 * i, lo + 16 * i + 16) for i in range(WAVE)]


def test_piece_limit_matches_group_liveness():
    """With `limit` a multiple of K, a piece is stored exactly when the group holding it is live:
    piece q covers outputs [4q, 4q + 4) of group q // 2."""
    base = 0
    for limit in range(0, 513, K):
        for q in range(2 * WAVE):
            assert (base + 4 * q < limit) == (base + K * (q // 2) < limit)
