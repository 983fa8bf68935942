"""CPU model of the row-ragged tile decode with split tail tiles (host logic; no GPU).

The down projection of a layer whose grid is a few rounds of the chip splits each tail tile (a group's last m-tile
holding at most half a tile of rows) into column windows, one per workgroup. This model restates, in Python, the
tile plan of the m-tile prefix kernel (body and tail prefixes of 256-row m-tiles), the decode of a workgroup index
into (group, m-tile, n-tile, window), the host's grid size, and the 16-wavefront tile's mapping of wavefront
columns and B-operand load instructions to the window. It checks on random groups that:
- every body tile and every window of every tail tile is computed by exactly one workgroup, and no workgroup
  decodes past them;
- the host's grid covers every XCD's share;
- the windows partition a tile's columns along whole wavefront columns and whole direct-load instructions, so
  each output column of a tail tile is computed and stored exactly once, inside the output;
- the decode takes fewer windows per tail tile when the windows of all tails would not fit the chip's CUs.
"""
import random

import pytest

BM = BN = 256
GROUP_M = 8
XCDS = 8
# the 16-wavefront 256 x 256 tile of the down projection: 4 x 4 wavefronts of 64 x 64, 64-deep K-tiles, one
# direct-load instruction covers 1024 / (64 * 2) = 8 K-contiguous B rows
WN, WTN = 4, 64
RPI = 8
NW = 16
IB = BN * 64 * 2 // 1024 // NW


def plan(rows_of):
    """body and tail prefixes over groups (a tail: a last m-tile with at most half of BM rows)."""
    body, tail = [0], [0]
    for rows in rows_of:
        rem = rows % BM
        is_tail = 1 if (rem > 0 and 2 * rem <= BM) else 0
        body.append(body[-1] + (rows + BM - 1) // BM - is_tail)
        tail.append(tail[-1] + is_tail)
    return body, tail


def windows_per_tail(tail, n_tiles, ts, cus):
    """the largest power of two up to ts whose windows of all tail tiles fit cus workgroups"""
    ptiles = tail[-1] * n_tiles
    while ts > 1 and ptiles * ts > cus:
        ts //= 2
    return ts


def decode(bid, body, tail, n_tiles, ts_max, cus=256):
    """(g, mt, nt, sub, nsub) of workgroup bid, or None (the workgroup has no tile): column window sub of nsub
    equal windows of the tile (a body tile is one window of the whole tile)."""
    G = len(body) - 1
    ts = windows_per_tail(tail, n_tiles, ts_max, cus)
    total = body[G] * n_tiles
    x, lb = bid % XCDS, bid // XCDS
    q, r = divmod(total, XCDS)
    cnt = q + (1 if x < r else 0)
    if lb < cnt:
        L = x * q + min(x, r) + lb
        g = sum(1 for i in range(1, G) if body[i] * n_tiles <= L)
        l = L - body[g] * n_tiles
        n_mt = body[g + 1] - body[g]
        mblk = l // (GROUP_M * n_tiles)
        rem = l - mblk * GROUP_M * n_tiles
        gsz = min(GROUP_M, n_mt - mblk * GROUP_M)
        return g, mblk * GROUP_M + rem % gsz, rem // gsz, 0, 1
    ptot = tail[G] * n_tiles * ts
    qt, rt = divmod(ptot, XCDS)
    lt = lb - cnt
    if lt >= qt + (1 if x < rt else 0):
        return None
    L = x * qt + min(x, rt) + lt
    tix = L // (n_tiles * ts)
    g = sum(1 for i in range(1, G) if tail[i] <= tix)
    rem = L - tix * n_tiles * ts
    return g, body[g + 1] - body[g], rem // ts, rem % ts, ts


def host_grid(T, k, Eloc, S, n_tiles, ts):
    """the launch's workgroups: the m-tile bound of the row-ragged kinds, the rounding of the XCD shares (16) and
    the windows' extra workgroups (each group has at most one tail m-tile)."""
    bound = ((T * k + Eloc * (BM - 1)) // BM + S * ((T + BM - 1) // BM)) * n_tiles
    return bound + 16 + (ts - 1) * (Eloc + S) * n_tiles


def window(sub, ts):
    lo = sub * (BN // ts)
    return lo, lo + BN // ts


def random_layer(rng):
    Eloc = rng.randint(1, 80)
    S = rng.choice([0, 0, 1, 2])
    k = rng.randint(1, min(4, Eloc))
    T = rng.randint(1, 3000)
    # routed rows: a skewed partition of T * k over the local experts, some empty
    w = [rng.random() ** 3 * (0 if rng.random() < 0.15 else 1) for _ in range(Eloc)]
    if sum(w) == 0:
        w[0] = 1.0
    raw = [int(T * k * x / sum(w)) for x in w]
    raw[0] += T * k - sum(raw)
    return T, k, Eloc, S, raw + [T] * S


@pytest.mark.parametrize("ts", [1, 2, 4])
def test_split_tails_cover_every_tile_once(ts):
    rng = random.Random(1000 + ts)
    for _ in range(150):
        T, k, Eloc, S, rows_of = random_layer(rng)
        n_tiles = rng.randint(1, 24)
        body, tail = plan(rows_of)
        grid = host_grid(T, k, Eloc, S, n_tiles, ts)
        cols = {}  # (g, mt, nt) -> columns computed, through the windows the decode hands out
        for bid in range(grid + 8 * XCDS):  # past the grid: nothing may be left over
            t = decode(bid, body, tail, n_tiles, ts)
            if t is None:
                continue
            assert bid < grid, ("a tile past the host's grid", bid, grid)
            g, mt, nt, sub, nsub = t
            cols.setdefault((g, mt, nt), []).extend(range(*window(sub, nsub)))
        want = set()
        for g, rows in enumerate(rows_of):
            nb = body[g + 1] - body[g]
            has_tail = tail[g + 1] - tail[g]
            for mt in range(nb + has_tail):
                for nt in range(n_tiles):
                    want.add((g, mt, nt))
            if has_tail:  # the tail m-tile holds the group's last rows, at most half a tile
                assert 0 < rows - nb * BM <= BM // 2
            else:
                assert nb * BM >= rows
        assert set(cols) == want
        for key, c in cols.items():
            assert sorted(c) == list(range(BN)), ("columns of a tile not computed exactly once", key)


@pytest.mark.parametrize("ts", [1, 2, 4])
def test_windows_split_wave_columns_and_b_loads(ts):
    for sub in range(ts):
        lo, hi = window(sub, ts)
        # the wavefront columns that compute and store: whole 64-column blocks inside the window
        waves = [wn for wn in range(WN) if lo <= wn * WTN < hi]
        assert all(wn * WTN + WTN <= hi for wn in waves)
        assert sorted(c for wn in waves for c in range(wn * WTN, wn * WTN + WTN)) == list(range(lo, hi))
        # the B load instructions issued: rows RPI * jj .. RPI * jj + 7, all inside the window or all outside
        rows = []
        for wave in range(NW):
            for j in range(IB):
                jj = wave + NW * j
                inside = lo <= RPI * jj < hi
                assert inside == (lo <= RPI * jj + RPI - 1 < hi)
                if inside:
                    rows += range(RPI * jj, RPI * jj + RPI)
        # every B row a computing wavefront reads is loaded, exactly once
        assert sorted(rows) == list(range(lo, hi))
    # the windows of a tile partition its columns
    cols = sorted(c for sub in range(ts) for c in range(*window(sub, ts)))
    assert cols == list(range(BN))


def test_split_tail_stores_stay_in_the_output():
    """Stores of a tail window: rows below the group's row count, columns inside d_model (n_extent)."""
    rng = random.Random(7)
    for _ in range(200):
        T, k, Eloc, S, rows_of = random_layer(rng)
        d = 256 * rng.randint(1, 16)
        n_tiles = d // BN
        ts = rng.choice([2, 4])
        body, tail = plan(rows_of)
        for bid in range(host_grid(T, k, Eloc, S, n_tiles, ts)):
            t = decode(bid, body, tail, n_tiles, ts)
            if t is None:
                continue
            g, mt, nt, sub, nsub = t
            if not (tail[g + 1] - tail[g]) or mt != body[g + 1] - body[g]:
                assert (sub, nsub) == (0, 1)  # a body tile: whole columns, rows all inside the group
                assert (mt + 1) * BM <= rows_of[g] or mt * BM < rows_of[g] <= (mt + 1) * BM
                continue
            assert nsub == windows_per_tail(tail, n_tiles, ts, 256)
            lo, hi = window(sub, nsub)
            m0, n0 = mt * BM, nt * BN
            for wn in range(WN):
                if not (lo <= wn * WTN < hi) or n0 + wn * WTN >= d:
                    continue
                assert n0 + wn * WTN + WTN <= d
            assert m0 < rows_of[g] <= m0 + BM


def test_windows_per_tail_fit_the_chip():
    """Fewer windows per tail tile when those of all tails would not fit the CUs; one when even those would not."""
    assert windows_per_tail([0, 1, 2, 3], 16, 4, 256) == 4      # 48 tail tiles: 192 windows
    assert windows_per_tail([0, 1, 2, 3, 4, 5], 16, 4, 256) == 2  # 80 tail tiles: 160 windows
    assert windows_per_tail([0] + list(range(1, 21)), 16, 4, 256) == 1  # 320 tail tiles
    assert windows_per_tail([0, 0, 0], 16, 4, 256) == 4          # no tails
    rng = random.Random(11)
    for _ in range(100):  # the coverage holds whatever the window count the decode picks
        T, k, Eloc, S, rows_of = random_layer(rng)
        n_tiles = rng.randint(1, 24)
        body, tail = plan(rows_of)
        cus = rng.choice([8, 32, 256])
        grid = host_grid(T, k, Eloc, S, n_tiles, 4)
        cols = {}
        for bid in range(grid + 64):
            t = decode(bid, body, tail, n_tiles, 4, cus)
            if t is None:
                continue
            assert bid < grid
            g, mt, nt, sub, nsub = t
            cols.setdefault((g, mt, nt), []).extend(range(*window(sub, nsub)))
        for key, c in cols.items():
            assert sorted(c) == list(range(BN)), key
        assert len(cols) == (body[-1] + tail[-1]) * n_tiles
