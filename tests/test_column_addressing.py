"""CPU address emulation of the column kernels (time-major [T, N] layouts and F-vector
eligibility traces): the index arithmetic of every lane of every workgroup of cols_rows_kernel,
cols_tiles_kernel, cols_narrow_kernel and cols_narrow_tiles_kernel, restated here from the
kernels, over the shapes the GPU column tests run (ragged T, padded row strides, partly filled
column blocks, both dtypes), asserting that every data, flag, continuation, output, per-column
value, draw-slot and workspace-record access lies inside its array. A lane past the last column
or a step past T still issues its loads (from a clamped column and step), so those are checked
too. Nothing here runs on a GPU.

Geometry (as the column kernels take it): column j = b * C + c holds step t at
b * bstride + c + t * st; its flags at the same element (time-major) or at b * fbstride + t
(vector traces); its per-column value (bootstrap) at j."""
import numpy as np
import pytest

I = np.int32  # every index of these shapes fits in 31 bits
WAVE = 64
WS_SLOTS = 1024
COL_K, COL_W, COL_SPLIT_W = 8, 4, 8       # 64-column blocks: steps per lane, waves
LOOK_AHEAD, LIFT_AFTER = 4, 3             # look-back batch and the single-tile steps before doubling


class Geom:
    def __init__(self, J, C, st, bstride, fst, fbstride, fcol, data_extent, flag_extent):
        self.J, self.C, self.st, self.bstride = J, C, st, bstride
        self.fst, self.fbstride, self.fcol = fst, fbstride, fcol
        self.data_extent, self.flag_extent = data_extent, flag_extent


def time_major(T, N, ld=None):
    """[T, ld] buffers viewed as [N, T] (stride_n = 1, stride_t = ld): the minimal extent of a
    tensor whose last element is (N - 1) + (T - 1) * ld."""
    ld = N if ld is None else ld
    ext = (N - 1) + (T - 1) * ld + 1
    assert ext < 2 ** 31
    return Geom(N, 1, ld, 1, 0, 0, True, ext, ext)


def vector_trace(N, T, F):
    """[N, T, F] data with [N, T] flags: J = N * F columns of C = F per batch row."""
    return Geom(N * F, F, F, T * F, 1, T, False, N * T * F, N * T)


def paired_block(b, blocks):
    dealt = blocks // 16 * 16
    return np.where(b >= dealt, b, b // 16 * 16 + (b % 8) * 2 + (b // 8) % 2)


def narrow_group(b, groups):
    dealt = groups // 64 * 64
    return np.where(b >= dealt, b, b // 64 * 64 + (b % 8) * 8 + (b // 8) % 8)


def col_place(g, j):
    """ColLane: base and flag base of column j (column 0 for lanes past the last column)."""
    active = j < g.J
    jj = np.where(active, j, 0)
    b, c = jj // g.C, jj % g.C
    base = b * g.bstride + c
    fbase = base if g.fcol else b * g.fbstride
    fstep = g.st if g.fcol else g.fst
    return active, jj, base, fbase, fstep


def check_chunk(g, T, K, backward, j, t0, label):
    """ColChunk::issue / complete / finish for lanes owning column j (array) and the K steps
    from t0 (array of the same shape)."""
    active, jj, base, fbase, fstep = col_place(g, j)
    k = np.arange(K, dtype=I)
    t = t0[..., None] + k                    # the lane's steps
    tc = np.minimum(t, T - 1)                # clamped loads
    data = base[..., None] + tc * g.st
    flag = fbase[..., None] + tc * fstep
    assert data.min() >= 0 and data.max() < g.data_extent, (label, "data")
    assert flag.min() >= 0 and flag.max() < g.flag_extent, (label, "flag")
    valid = active[..., None] & (t < T)
    if valid.any():
        out = (base[..., None] + t * g.st)[valid]   # outputs and continuation values
        assert out.min() >= 0 and out.max() < g.data_extent, (label, "out")
    if backward:
        nbr = base + np.minimum(t0 + K, T - 1) * g.st
        assert nbr.min() >= 0 and nbr.max() < g.data_extent, (label, "neighbour")
        assert jj.max() < g.J, (label, "row value")
    else:
        tp = np.minimum(np.maximum(t0 - 1, 0), T - 1)
        prev = fbase + tp * fstep
        assert prev.min() >= 0 and prev.max() < g.flag_extent, (label, "previous flag")


def level_offset(P, l):
    return sum(P >> k for k in range(l))


def ctz(y):
    return (y & -y).bit_length() - 1


def record_indices(P, ticket, lift):
    """Tile-record slots (in units of J) that the tile of `ticket` writes and reads: its own
    map, the block aggregates it closes (reading their lower halves), and its look-back."""
    out = []
    if ticket < P - 1:
        out.append(ticket)
        if lift:
            off_prev, l = 0, 1
            while ((ticket + 1) & ((1 << l) - 1)) == 0:
                q = ((ticket + 1) >> l) - 1
                out.append(off_prev + 2 * q)
                off = off_prev + (P >> (l - 1))
                out.append(off + q)
                off_prev, l = off, l + 1
    if ticket > 0:
        if not lift:
            out.extend(range(ticket))
        else:
            y, step = ticket, 0
            while y > 0:
                yy, n = y, 0
                for k in range(LOOK_AHEAD):
                    if yy > 0:
                        lim = max(step + k - LIFT_AFTER, 0)
                        l = min(ctz(yy), lim)
                        out.append(level_offset(P, l) + (yy >> l) - 1)
                        yy -= 1 << l
                        n = k + 1
                y, step = yy, step + n
    return out


def records_capacity(J, T):
    """Records the column workspace of a [J columns, T] call holds: one per column per 32
    steps (col_ws_need)."""
    return ((T + 31) // 32) * J


def check_records(g, T, P, nblocks, C, label):
    cap = records_capacity(g.J, T)
    assert nblocks <= WS_SLOTS, (label, "draw slots")
    top = 0
    for lift in (False, True):
        for ticket in range(P):
            idx = record_indices(P, ticket, lift)
            if idx:
                top = max(top, max(idx))
    # the largest record index of any column j < J: top * J + j
    assert (top + 1) * g.J <= cap, (label, "records", top, cap)


def emulate_rows(g, T, backward):
    blocks = (g.J + WAVE - 1) // WAVE
    P = (T + COL_K * COL_W - 1) // (COL_K * COL_W)
    b = np.arange(blocks, dtype=I)
    pb = paired_block(b, blocks)
    assert sorted(pb.tolist()) == list(range(blocks))
    lane, wave, chunk = np.arange(WAVE, dtype=I), np.arange(COL_W, dtype=I), np.arange(P, dtype=I)
    cidx = (P - 1 - chunk) if backward else chunk
    for b0 in range(0, blocks, 8):
        sel = pb[b0:b0 + 8]
        j = (sel[:, None, None, None] * WAVE + lane[None, None, :, None]) + 0 * wave[None, :, None, None] + 0 * chunk
        t0 = cidx[None, None, None, :] * (COL_K * COL_W) + wave[None, :, None, None] * COL_K + 0 * j
        check_chunk(g, T, COL_K, backward, j, t0, "cols_rows_kernel")


def emulate_tiles(g, T, backward):
    blocks = (g.J + WAVE - 1) // WAVE
    L = COL_K * COL_SPLIT_W
    P = (T + L - 1) // L
    grid = np.arange(blocks * P, dtype=I)
    blk = paired_block(grid % blocks, blocks) if blocks % 8 == 0 else grid % blocks
    # tickets: every (block, ticket) pair occurs once; the emulation covers them all
    blk_u = np.unique(blk)
    assert blk_u.tolist() == list(range(blocks))
    ticket = np.arange(P, dtype=I)
    p = (P - 1 - ticket) if backward else ticket
    lane, wave = np.arange(WAVE, dtype=I), np.arange(COL_SPLIT_W, dtype=I)
    for b0 in range(0, blocks, 8):
        sel = blk_u[b0:b0 + 8]
        j = sel[:, None, None, None] * WAVE + lane[None, None, :, None] + 0 * wave[None, :, None, None] + 0 * p
        t0 = p[None, None, None, :] * L + wave[None, :, None, None] * COL_K + 0 * j
        check_chunk(g, T, COL_K, backward, j, t0, "cols_tiles_kernel")
    check_records(g, T, P, blocks, WAVE, "cols_tiles_kernel")


def narrow_shape(esz):
    C = 64 // esz
    return C, WAVE // C, C // 4          # columns per group, lane groups per wave, steps per lane


def emulate_narrow(g, T, backward, esz):
    C, G, K = narrow_shape(esz)
    W = 4 if T <= G * 4 * K else (8 if T <= G * 8 * K else 16)
    L = G * W * K
    P = (T + L - 1) // L
    groups = (g.J + C - 1) // C
    ng = narrow_group(np.arange(groups, dtype=I), groups)
    assert sorted(ng.tolist()) == list(range(groups))
    lane, wave, chunk = np.arange(WAVE, dtype=I), np.arange(W, dtype=I), np.arange(P, dtype=I)
    col, grp = lane % C, lane // C
    span = wave[:, None] * G + grp[None, :]                       # [W, 64]
    cidx = (P - 1 - chunk) if backward else chunk
    for b0 in range(0, groups, 16):
        sel = ng[b0:b0 + 16]
        j = sel[:, None, None, None] * C + col[None, None, :, None] + 0 * span[None, :, :, None] + 0 * chunk
        t0 = cidx[None, None, None, :] * L + span[None, :, :, None] * K + 0 * j
        check_chunk(g, T, K, backward, j, t0, f"cols_narrow_kernel W={W}")


def emulate_narrow_tiles(g, T, backward, esz, TL):
    C, G, K = narrow_shape(esz)
    W = TL // (G * K)
    P = (T + TL - 1) // TL
    groups = (g.J + C - 1) // C
    lane, wave = np.arange(WAVE, dtype=I), np.arange(W, dtype=I)
    col, grp = lane % C, lane // C
    span = wave[:, None] * G + grp[None, :]
    if P % 8 == 0:  # static dealing: workgroup b -> (block, ticket), onto every pair once
        b = np.arange(groups * P, dtype=I)
        r = b // 8
        pairs = (r % groups) * P + ((b % 8) * (P // 8) + r // groups)
        assert np.array_equal(np.sort(pairs), np.arange(groups * P, dtype=I))
    ticket = np.arange(P, dtype=I)
    p = (P - 1 - ticket) if backward else ticket
    for b0 in range(0, groups, 16):
        blk = np.arange(b0, min(groups, b0 + 16), dtype=I)
        j = blk[:, None, None, None] * C + col[None, None, :, None] + 0 * span[None, :, :, None] + 0 * p
        t0 = p[None, None, None, :] * TL + span[None, :, :, None] * K + 0 * j
        check_chunk(g, T, K, backward, j, t0, f"cols_narrow_tiles_kernel TL={TL}")
    check_records(g, T, P, groups, C, f"cols_narrow_tiles_kernel TL={TL}")


TIME_MAJOR = [(1, 1, None), (7, 3, None), (33, 64, None), (256, 100, None), (1000, 65, None),
              (4097, 5, None), (300, 130, 160), (70, 40, 48), (256, 4096, None), (1, 17, None),
              (64, 1000, None), (65, 1000, 1030), (300, 1000, None), (64, 1600, 1700),
              (1100, 4100, None), (2000, 530, 600), (5000, 4096, None), (500, 70, None),
              (3000, 17, None), (16384, 70, None), (4096, 64, None), (2048, 128, 136),
              (65, 16, None), (129, 1, 3), (1000, 33, None), (8192, 48, 50), (20000, 32, None),
              (999, 200, None)]
VECTOR = [(1, 1, 1), (3, 7, 5), (64, 256, 16), (7, 1000, 33), (2, 4097, 3), (5, 40, 300),
          (1, 33, 64), (2, 8192, 40), (16, 300, 40)]


def _kernels(g, T, esz):
    for backward in (True, False):
        emulate_rows(g, T, backward)
        emulate_narrow(g, T, backward, esz)
        if (g.J + WAVE - 1) // WAVE <= WS_SLOTS:
            emulate_tiles(g, T, backward)
        C = 64 // esz
        if (g.J + C - 1) // C <= WS_SLOTS:
            for TL in (64, 128):
                emulate_narrow_tiles(g, T, backward, esz, TL)


@pytest.mark.parametrize("esz", [4, 2])
@pytest.mark.parametrize("T,N,ld", TIME_MAJOR)
def test_time_major_addresses_in_bounds(T, N, ld, esz):
    _kernels(time_major(T, N, ld), T, esz)


@pytest.mark.parametrize("N,T,F", VECTOR)
def test_vector_trace_addresses_in_bounds(N, T, F):
    _kernels(vector_trace(N, T, F), T, 4)


def test_emulation_catches_an_unclamped_flag_read():
    """The check fails on the access pattern the kernels once had: the previous step's flag
    read at max(t0 - 1, 0) without clamping into the column, from lanes wholly past its end."""
    g = time_major(100, 40)
    j = np.arange(64, dtype=I)[None, :]
    t0 = np.array([[96 + 8 * w] for w in range(4)]) + 0 * j   # waves past T = 100
    active, jj, base, fbase, fstep = col_place(g, j)
    prev = fbase + np.maximum(t0 - 1, 0) * fstep               # the unclamped form
    assert prev.max() >= g.flag_extent
    with pytest.raises(AssertionError):
        assert prev.max() < g.flag_extent
    check_chunk(g, 100, 8, False, j, t0, "clamped")            # the kernels' form passes
