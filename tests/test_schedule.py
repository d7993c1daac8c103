"""Pins of the oracle's tile schedule (Alg. 1, Prop. 1) -- CPU only."""
import os

import numpy as np
import pytest

from oracle.schedule import all_tiles, lowbit, tile_after_step

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(v) for v in line.split()])
    return rows


def test_lowbit_is_largest_power_of_two_divisor():
    for i in range(1, 5000):
        u = lowbit(i)
        assert u & (u - 1) == 0          # a power of two
        assert i % u == 0                # divides i
        assert (i // u) % 2 == 1         # and is the largest such
        assert u == i & -i               # two's-complement identity


def test_golden_schedule_L8_hand_derived():
    """The L = 8 tiles written out by hand from Alg. 1 (1-indexed)."""
    want = [tuple(int(v) for v in r) for r in _rows("schedule_L8_alg1.txt")]
    got = []
    for (i, U, s0, s1, d0, d1) in all_tiles(8):
        # 0-indexed half-open -> 1-indexed closed ranges of the paper
        got.append((i, U, s0 + 1, s1, d0 + 1, d1))
    assert got == want


@pytest.mark.parametrize("P", range(1, 18))
def test_prop1_tile_counts(P):
    """Prop. 1: 2^(P-1-q) tiles of side 2^q, q = 0..P-1; L-1 tiles in all."""
    L = 1 << P
    counts = {}
    n = 0
    for t in range(L):
        tile = tile_after_step(t, L)
        if tile is None:
            continue
        n += 1
        counts[tile[1]] = counts.get(tile[1], 0) + 1
        assert tile[5] == tile[4] + tile[1]          # never clipped when L = 2^P
    assert n == L - 1
    assert counts == {1 << q: 1 << (P - 1 - q) for q in range(P)}


def test_golden_tile_fractions():
    """Sec. 5.1 / App. D: 93.75 % of positions use U <= 8, 87.5 % use U <= 4.

    Exactly: L/2 positions use U = 1, L/4 use U = 2, ..., so the counts are
    15L/16 and 7L/8 out of L positions (the last position runs no tile)."""
    for L in [1 << 10, 1 << 14, 1 << 17]:
        sizes = np.array([tile[1] for tile in all_tiles(L)])
        for max_u, pct in _rows("tile_fractions.txt"):
            share = np.count_nonzero(sizes <= max_u) / L
            assert share == pytest.approx(pct / 100.0, abs=0.0)


def _coverage(L):
    cover = np.zeros((L, L), dtype=np.int64)     # cover[t, s]
    for s in range(L):
        cover[s, s] += 1                          # red cells
    for (i, U, s0, s1, d0, d1) in all_tiles(L):
        cover[d0:d1, s0:s1] += 1
    return cover


@pytest.mark.parametrize("L", list(range(1, 70)) + [128, 255, 256, 1000, 1024, 4096])
def test_every_pair_covered_exactly_once(L):
    """Every (s, t) with s <= t is accounted for exactly once; nothing above
    the diagonal (no contribution of a future input)."""
    cover = _coverage(L)
    lower = np.tril(np.ones((L, L), dtype=np.int64))
    assert np.array_equal(cover, lower)


@pytest.mark.parametrize("L", [7, 64, 1000, 1 << 13])
def test_tiles_read_only_unlocked_inputs(L):
    """A tile run after z_t is emitted reads only y_s with s <= t and writes
    only z at positions > t; source and destination are disjoint."""
    for t in range(L):
        tile = tile_after_step(t, L)
        if tile is None:
            assert t == L - 1
            continue
        i, U, s0, s1, d0, d1 = tile
        assert s1 - 1 <= t < d0
        assert s1 <= d0 and s0 >= 0 and d1 <= L


def test_closed_form_covering_tile_large_L():
    """For s < t the pair is covered by the tile i = t with its low k bits
    cleared, U = 2^k, k = floor(log2(s xor t)) -- checked on random pairs at
    L = 2^17 against the schedule itself."""
    L = 1 << 17
    by_i = {tile[0]: tile for tile in all_tiles(L)}
    rng = np.random.default_rng(7)
    for _ in range(20000):
        s, t = sorted(int(v) for v in rng.integers(0, L, size=2))
        if s == t:
            continue
        k = (s ^ t).bit_length() - 1
        i = t & ~((1 << k) - 1)
        i_, U, s0, s1, d0, d1 = by_i[i]
        assert U == 1 << k
        assert s0 <= s < s1 and d0 <= t < d1


@pytest.mark.parametrize("P", [4, 10, 17])
def test_total_tile_area(P):
    """The tiles partition the strictly-lower triangle: sum U^2 = L(L-1)/2."""
    L = 1 << P
    assert sum(t[1] * t[1] for t in all_tiles(L)) == L * (L - 1) // 2


def test_non_power_of_two_clips_destination():
    L = 12
    tiles = all_tiles(L)
    assert tiles[7] == (8, 8, 0, 8, 8, 12)        # i = 8, U = 8 clipped at L
    assert tile_after_step(L - 1, L) is None


@pytest.mark.parametrize("L", [3, 5, 8, 12, 100, 129, 256, 1000, 4500, 8192])
def test_half_state_premise(L):
    """App. C's premise, on the schedule: with T the largest power of two
    below L, no tile before the one of i = T writes at a position >= T, that
    tile reads exactly y[0, T) and writes z[T, L), and every later tile reads
    and writes only positions >= T; the red cell of step t touches position t
    alone.  So T rows per layer suffice when the tile of i = T writes its
    outputs over its own inputs, and position p >= T is kept at row p - T."""
    T = 1
    while 2 * T < L:
        T *= 2
    seen_swap = False
    for (i, U, s0, s1, d0, d1) in all_tiles(L):
        if i < T:
            assert d1 <= T
        elif i == T:
            assert (U, s0, s1, d0, d1) == (T, 0, T, T, L)
            assert d1 - d0 <= s1 - s0      # the outputs fit in the inputs' rows
            seen_swap = True
        else:
            assert s0 >= T and d0 >= T and d1 <= L
            assert d1 - T <= T             # rows p - T stay below T
    assert seen_swap


@pytest.mark.parametrize("L", [64, 100, 1024, 4096 + 17])
@pytest.mark.parametrize("W", [32])
def test_small_tiles_stay_inside_their_block(L, W):
    """The premise of running the positions of one aligned block of W
    positions in one launch with the block's rows held in registers: in
    every block [b, b + W), the tile of each step t except the block's last
    has U <= W/2 and reads y and writes z only inside the block, and the
    last step's tile (i = b + W) has U >= W; so a tile that reads or writes
    a row of the block is either a small one of the block or a tile of
    U >= W launched at a block boundary."""
    for (i, U, s0, s1, d0, d1) in all_tiles(L):
        t = i - 1
        b = t - t % W
        if i < b + W:
            assert U <= W // 2
            assert b <= s0 and s1 <= b + W and b <= d0 and d1 <= b + W
        else:
            assert i == b + W and U >= W and i % W == 0
            # a large tile's inputs are whole earlier blocks, its outputs start
            # at a block boundary
            assert s0 % W == 0 and d0 % W == 0
