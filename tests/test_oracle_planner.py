"""Pins for the oracle's window-assignment planner (CPU only).

Values printed in the paper:
* Sec. VII-D: at w = 128 (p = 4, alpha = 2) on the 2041 x 4320 field, the
  minimally padded window grid is 2 x 5, the fixed Topo(4, 4) pads it to a
  4 x 8 grid of 32 windows, and the padding overheads are 280.6 % (fixed)
  against 18.9 % (ragged);
* Sec. V-B: ten windows on four ranks under ragged Topo(4, 1) give two
  ranks three windows and two ranks two; Topo(2, 1, 2) gives every one of
  the four ranks five sub-tiles;
* Sec. V-A: the 9 x 5 window grid of the fixed-assignment figure (M = 45).
Closed forms and invariants: every window owned exactly once, range sizes
differing by at most one, stripes partitioning the rows, every token needed
by exactly one rank, and shift-only fragments of exactly sh rows from the
next rank when window ranges and stripes line up.
"""

import itertools

import pytest

from oracle import Geometry
from oracle import planner as pl


def test_eq3_padding_of_the_paper_example():
    H, W = 2041, 4320
    minimal = pl.padded_grid(H, W, p=4, alpha=2, w=128)
    assert minimal == (2048, 5120)
    # Transformer-stage window grid: H_hat / (p alpha w) x W_hat / (p alpha w)
    assert (minimal[0] // (4 * 2 * 128), minimal[1] // (4 * 2 * 128)) == (2, 5)
    fixed = pl.padded_grid(H, W, p=4, alpha=2, w=128, m=4, n=4)
    assert fixed == (4096, 8192)
    assert (fixed[0] // 1024) * (fixed[1] // 1024) == 32        # a 4 x 8 grid of 32 windows
    assert round(100 * pl.padding_overhead(H, W, *fixed), 1) == 280.6
    assert round(100 * pl.padding_overhead(H, W, *minimal), 1) == 18.9


def test_eq3_is_the_least_multiple():
    # H_hat is the least multiple of p alpha w m that is >= H (brute force).
    for H, W, p, a, w, m, n in [(2041, 4320, 4, 2, 8, 2, 4), (100, 37, 2, 1, 3, 5, 1), (7, 7, 1, 1, 7, 1, 1)]:
        Hh, Wh = pl.padded_grid(H, W, p, a, w, m, n)
        assert Hh == min(x for x in range(H, H + p * a * w * m + 1) if x % (p * a * w * m) == 0)
        assert Wh == min(x for x in range(W, W + p * a * w * n + 1) if x % (p * a * w * n) == 0)
    assert pl.padding_overhead(64, 64, 64, 64) == 0.0


def test_eq4_worked_examples():
    sizes = lambda M, P: [R - L for L, R in pl.window_ranges(M, P)]  # noqa: E731
    assert sizes(10, 4) == [2, 3, 2, 3]
    assert sorted(sizes(10, 4)) == [2, 2, 3, 3]          # two ranks three, two ranks two
    assert sizes(45, 4) == [11, 11, 11, 12]              # the 9 x 5 grid on 2 x 2 ranks
    assert pl.subtiles_per_rank(10, 4, 2) == [5, 5, 5, 5]
    assert pl.subtiles_per_rank(10, 4, 1) == sizes(10, 4)


@pytest.mark.parametrize("M,P", [(1, 1), (1, 4), (10, 4), (45, 4), (1088, 8), (253, 16), (7, 9)])
def test_eq4_partitions_row_major_order(M, P):
    rng = pl.window_ranges(M, P)
    assert rng[0][0] == 0 and rng[-1][1] == M
    for (a, b), (c, d) in zip(rng, rng[1:]):
        assert b == c and a <= b
    sizes = [b - a for a, b in rng]
    assert max(sizes) - min(sizes) <= 1
    assert sum(sizes) == M


def test_stripes_partition_rows():
    for H, P in [(128, 4), (85, 4), (256, 8), (5, 7)]:
        st = pl.stripes(H, P)
        assert st[0][0] == 0 and st[-1][1] == H
        assert all(b == c for (_, b), (c, _) in zip(st, st[1:]))
        assert all(pl.stripe_owner(H, P, u) == r for r, (a, b) in enumerate(st) for u in range(a, b))


GEOMS = [
    Geometry(1, 32, 40, 8, 1, 8, 8, 8, 4, 4, 1),
    Geometry(2, 21, 52, 4, 1, 4, 8, 16, 4, 8, 1),       # ragged height
    Geometry(1, 17, 23, 4, 1, 4, 5, 6, 2, 3, 3),        # ragged both ways
    Geometry(1, 24, 30, 4, 1, 4, 6, 5, 0, 0, 1),        # no shift (the DMP route alone)
]


@pytest.mark.parametrize("g", GEOMS)
@pytest.mark.parametrize("P", [1, 2, 4, 8])
def test_every_token_needed_by_exactly_one_rank(g, P):
    seen = {}
    total = 0
    for r in range(P):
        begin, end = pl.rank_slots(g, P, r)
        need = pl.needed_tokens(g, P, r)
        n = sum(len(s) for s in need.values())
        assert n == end - begin
        total += n
        for src, pts in need.items():
            for (u, v) in pts:
                assert (u, v) not in seen
                seen[(u, v)] = r
                a, b = pl.stripes(g.H, P)[src]
                assert a <= u < b
    assert total == g.H * g.W and len(seen) == g.H * g.W


@pytest.mark.parametrize("sh,sw", [(4, 8), (0, 8), (4, 0), (0, 0)])
def test_aligned_ranks_exchange_only_the_shifted_rows(sh, sw):
    # 128 x 1080 grid, 8 x 16 windows (16 x 68 windows): on 4 ranks every
    # rank owns four whole window rows, exactly the 32 rows of its stripe
    # before the shift, so the only tokens from elsewhere are the sh rows
    # below its stripe, all columns, from the next rank (cyclically).
    g = Geometry(1, 128, 1080, 8, 1, 8, 8, 16, sh, sw, 1)
    P = 4
    for r in range(P):
        need = pl.needed_tokens(g, P, r)
        remote = {s: pts for s, pts in need.items() if s != r}
        if sh == 0:
            assert remote == {}
            continue
        nxt = (r + 1) % P
        assert set(remote) == {nxt}
        lo = (32 * r + 32) % 128
        assert remote[nxt] == {(u, v) for u, v in itertools.product(range(lo, lo + sh), range(1080))}
