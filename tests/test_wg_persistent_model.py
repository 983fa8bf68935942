"""CPU model of the persistent weight-gradient loop of the pipelined GEMM tile (wg_persistent in
grouped_gemm_bf16.hip), checked before the kernel runs on a GPU:
  * the tile claims (one counter per XCD, tiles L = x, x + 8, ... of XCD x, other XCDs' counters once a share is
    exhausted) hand out every tile exactly once and let every workgroup leave, under random interleavings;
  * the tile decode of the weight-gradient kinds is a bijection from L onto (group, m-tile, n-tile);
  * every 16-byte epilogue store lies inside its output buffer, and the stores of all tiles cover each output
    element inside N exactly once;
  * the LDS regions: the next tile's operand loads (the ring) and the finished tile's staging areas (past the ring)
    are disjoint and fit 160 KB, so the two may overlap in time between the same pair of barriers.
The arithmetic below restates the kernel's index formulas; a change there must be made here too."""
import random

import numpy as np

# Cfg2<256, 256, 32, 4, 2, 2>
BM = BN = 256
ROWB = 64
PAD = max(BM, 32 * (BM * ROWB // 1024))
A_BYTES = BM * ROWB + PAD
B_BYTES = BN * ROWB + PAD
STAGE = A_BYTES + B_BYTES
LDS_MAIN = 4 * STAGE
WTM = WTN = 128
STG_ROWS, P16 = 16, WTN + 8
STG_WAVE = STG_ROWS * P16 * 2
GROUP_M = 8


def decode(L, G, m_tiles, n_tiles, order, interleave):
    """The weight-gradient branch of decode_tile: tile L -> (group, m-tile, n-tile)."""
    if interleave:
        rank, l = L % G, L // G
    else:
        rank, l = L // (m_tiles * n_tiles), L % (m_tiles * n_tiles)
    g = order[rank]
    mblk = l // (GROUP_M * n_tiles)
    rem = l - mblk * GROUP_M * n_tiles
    gsz = min(GROUP_M, m_tiles - mblk * GROUP_M)
    return g, mblk * GROUP_M + rem % gsz, rem // gsz


def tile_of(t, x, n_tiles):
    return 8 * t + x if 0 <= t < (n_tiles - x + 7) // 8 else -1


def simulate_claims(n_tiles, workers, seed):
    """Workgroups on XCDs (index mod 8) claiming in a random order; returns the tiles each processed."""
    rng = random.Random(seed)
    queues = [0] * 8
    done = {w: [] for w in range(workers)}
    pending = {}  # worker -> own-counter value claimed one tile ahead (not yet read)

    def steal(x):
        for i in range(1, 8):
            y = (x + i) % 8
            t = queues[y]
            queues[y] += 1
            L = tile_of(t, y, n_tiles)
            if L >= 0:
                return L
        return -1

    def first_claim(x):
        t = queues[x]
        queues[x] += 1
        L = tile_of(t, x, n_tiles)
        return L if L >= 0 else steal(x)

    active = {}
    for w in range(workers):
        L = first_claim(w % 8)
        if L >= 0:
            active[w] = L
            x = w % 8
            pending[w] = queues[x]
            queues[x] += 1
    steps = 0
    while active:
        steps += 1
        assert steps < 100 * (n_tiles + workers), "a workgroup never leaves"
        w = rng.choice(sorted(active))
        done[w].append(active[w])
        x = w % 8
        L = tile_of(pending[w], x, n_tiles)
        if L < 0:
            L = steal(x)
        if L < 0:
            del active[w]
        else:
            active[w] = L
            pending[w] = queues[x]
            queues[x] += 1
    return done


def epilogue_stores(kind, g, mt, nt, d, f, n_extent):
    """Byte offsets (buffer, offset) of every 16-byte store of one tile, all four waves."""
    out = []
    m0, n0 = mt * 256, nt * 256
    for wave in range(4):
        wm, wn = wave // 2, wave % 2
        if not (n0 + wn * WTN < n_extent):
            continue
        cprw = WTN // 8
        for part in range(8):
            for it in range(STG_ROWS * cprw // 64):
                for lane in range(64):
                    qq = lane + 64 * it
                    rr, cc = qq // cprw, (qq % cprw) * 8
                    m = m0 + wm * WTM + part * STG_ROWS + rr
                    col = n0 + wn * WTN + cc
                    # staging read inside this wave's area
                    off = (rr * P16 + cc) * 2
                    assert 0 <= off and off + 16 <= STG_WAVE
                    if kind == "wg_down":
                        out.append(("out", ((g * d + m) * f + col) * 2))
                    elif m < f:
                        out.append(("out", ((g * f + m) * d + col) * 2))
                    else:
                        out.append(("out2", ((g * f + (m - f)) * d + col) * 2))
    return out


def test_lds_regions():
    assert LDS_MAIN == 135168 and STG_WAVE == 4352
    assert LDS_MAIN + 4 * STG_WAVE <= 160 * 1024  # ring + staging areas
    # the direct loads' destinations stay inside their stage (padded K-major layout of both operands)
    worst = 0
    for stage in range(4):
        for l in range(8):
            for wave in range(4):
                jj = wave + 4 * (l & 3)
                base = stage * STAGE + (0 if l < 4 else A_BYTES) + jj * 1024 + 32 * jj
                lo, hi = base, base + 16 * 63 + 16
                region = (stage * STAGE, stage * STAGE + A_BYTES) if l < 4 else \
                    (stage * STAGE + A_BYTES, (stage + 1) * STAGE)
                assert region[0] <= lo and hi <= region[1]
                worst = max(worst, hi)
    assert worst <= LDS_MAIN  # the loads never reach the staging areas
    # staging writes: row li, columns 16 j + 4 q .. + 3 of a 16-row part, 8 bytes each
    for li in range(16):
        for j in range(8):
            for q in range(4):
                off = (li * P16 + 16 * j + 4 * q) * 2
                assert 0 <= off and off + 8 <= STG_WAVE


def test_decode_bijection():
    for G, m_tiles, n_tiles, interleave in [(8, 112, 16, 1), (8, 16, 56, 0), (3, 3, 2, 1), (5, 9, 3, 0), (66, 8, 6, 0)]:
        order = list(range(G))
        random.Random(G).shuffle(order)
        seen = set()
        for L in range(G * m_tiles * n_tiles):
            g, mt, nt = decode(L, G, m_tiles, n_tiles, order, interleave)
            assert 0 <= g < G and 0 <= mt < m_tiles and 0 <= nt < n_tiles
            seen.add((g, mt, nt))
        assert len(seen) == G * m_tiles * n_tiles


def test_claims_cover_every_tile_once():
    for n_tiles, workers in [(14336, 256), (7168, 256), (100, 256), (7, 16), (1, 8), (513, 24), (64, 3)]:
        for seed in range(3):
            done = simulate_claims(n_tiles, workers, seed)
            tiles = sorted(L for v in done.values() for L in v)
            assert tiles == list(range(n_tiles)), (n_tiles, workers, seed)


def test_epilogue_stores_in_bounds_and_cover_once():
    # small shapes of both kinds, including a last n-tile of 128 columns (N = 384)
    for kind, G, d, f in [("wg_down", 3, 512, 384), ("wg_gu", 2, 256, 384), ("wg_down", 2, 256, 256)]:
        if kind == "wg_down":
            M, N = d, f
            sizes = {"out": G * d * f * 2}
        else:
            M, N = 2 * f, d
            sizes = {"out": G * f * d * 2, "out2": G * f * d * 2}
        m_tiles, n_tiles = M // 256, (N + 255) // 256
        covered = {k: np.zeros(v // 16, np.int64) for k, v in sizes.items()}
        order = list(range(G))
        for L in range(G * m_tiles * n_tiles):
            g, mt, nt = decode(L, G, m_tiles, n_tiles, order, 0)
            for buf, off in epilogue_stores(kind, g, mt, nt, d, f, N):
                assert off % 16 == 0 and 0 <= off and off + 16 <= sizes[buf], (kind, L, buf, off)
                covered[buf][off // 16] += 1
        for buf, c in covered.items():
            assert (c == 1).all(), (kind, buf, int(c.min()), int(c.max()))


def ticket_split(tiles, cus=256, forced=False, pair=True):
    """The ticket-claimed tail of a launch (run_pair2 / run2): returns (static count, dynamic count, ticket-taking
    workgroups); tiles are tiles_b for a pair, the grid (a multiple of 8) for a single launch."""
    if pair:
        if forced:
            dyn = min(tiles, max(tiles // 64 * 8, 8))
        elif tiles >= 8 * cus:
            dyn = tiles // 64 * 8
        else:
            dyn = 0
    else:
        grid = tiles
        if forced:
            dyn = min(grid, max(grid // 64 * 8, 8))
        elif grid >= 8 * cus:
            dyn = grid // 64 * 8
        else:
            dyn = 0
    return tiles - dyn, dyn, (dyn + 256 if dyn > 0 else 0)


def test_ticket_tails_cover_every_tile_once():
    # static workgroups take indices [0, static); ticket t < dyn takes static + t; the rest take nothing
    for tiles in [1, 7, 8, 63, 64, 100, 2047, 2048, 7168, 14336, 7504]:
        for forced in (False, True):
            for pair in (False, True):
                n = tiles if pair else (tiles + 7) // 8 * 8
                static, dyn, wgs = ticket_split(n, forced=forced, pair=pair)
                assert 0 <= dyn <= n and static + dyn == n and (dyn == 0 or wgs >= dyn)
                rng = random.Random(tiles)
                tickets = list(range(wgs))
                rng.shuffle(tickets)  # any order of arrival
                done = list(range(static)) + [static + t for t in tickets if t < dyn]
                assert sorted(done) == list(range(n))
