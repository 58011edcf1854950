"""Pins for the oracle's window geometry and token routes (CPU only).

The oracle's route is checked against things it does not share code with:
the unshifted window coordinates of Sec. IV-D Eq. (2), numpy's reshape /
transpose window partition and numpy.roll for shifts, an independent
sort-based construction on ragged grids, and closed-form window counts.
"""

import numpy as np
import pytest

import terra_synth as ts
from oracle import Geometry, route, unroute, token_table, window_extents
from oracle.geometry import window_slots

GEOMS = [
    Geometry(1, 16, 32, 4, 1, 4, 8, 8, 4, 4),        # config-1 grid
    Geometry(2, 7, 9, 6, 2, 3, 3, 4, 1, 2, 3),       # ragged both ways, both masks
    Geometry(1, 85, 36, 2, 1, 2, 12, 12, 6, 6),      # ragged latitude (85 = 7*12 + 1)
    Geometry(1, 16, 40, 2, 1, 2, 8, 16, 4, 8),       # ragged longitude (40 = 2*16 + 8)
    Geometry(1, 12, 12, 3, 1, 3, 12, 12, 0, 0),      # one window
    Geometry(3, 5, 5, 1, 1, 1, 1, 1, 0, 0),          # 1x1 windows
]


def _x(g, seed=0):
    return np.random.default_rng(seed).standard_normal((g.B, g.H, g.W, g.C))


@pytest.mark.parametrize("g", GEOMS)
def test_token_table_is_a_permutation(g):
    tab = token_table(g)
    src = tab["u"] * g.W + tab["v"]
    assert np.array_equal(np.sort(src), np.arange(g.H * g.W))


@pytest.mark.parametrize("g", [Geometry(1, 16, 32, 1, 1, 1, 8, 8, 0, 0),
                               Geometry(1, 10, 11, 1, 1, 1, 4, 3, 0, 0)])
def test_unshifted_coordinates_follow_eq2(g):
    # Eq. (2): window (u // w, v // w), in-window offset (u mod w, v mod w).
    tab = token_table(g)
    Mh, Mw, _, _ = window_extents(g.H, g.W, g.wh, g.ww)
    assert np.array_equal(tab["win"], (tab["u"] // g.wh) * Mw + tab["v"] // g.ww)
    assert np.array_equal(tab["a"], tab["u"] % g.wh)
    assert np.array_equal(tab["c"], tab["v"] % g.ww)


def _partition(x, wh, ww):
    """Library window partition of a divisible NHWC grid."""
    B, H, W, C = x.shape
    y = x.reshape(B, H // wh, wh, W // ww, ww, C).transpose(0, 1, 3, 2, 4, 5)
    return y.reshape(B, H * W, C)


def test_shift0_divisible_equals_reshape_partition():
    g = Geometry(2, 16, 24, 3, 1, 3, 8, 8, 0, 0)
    x = _x(g)
    assert np.array_equal(route(x, g), _partition(x, 8, 8))


@pytest.mark.parametrize("shift", [(4, 4), (1, 7), (0, 3), (5, 0)])
def test_shift_divisible_equals_roll_then_partition(shift):
    g = Geometry(2, 16, 24, 3, 1, 3, 8, 8, shift[0], shift[1])
    x = _x(g)
    rolled = np.roll(x, (-shift[0], -shift[1]), axis=(1, 2))
    assert np.array_equal(route(x, g), _partition(rolled, 8, 8))


@pytest.mark.parametrize("g", GEOMS)
def test_ragged_route_equals_sort_construction(g):
    # Independent construction: sort original tokens by (window row, window
    # column, in-window row, in-window column) of their rolled coordinates.
    u, v = np.meshgrid(np.arange(g.H), np.arange(g.W), indexing="ij")
    r = (u - g.sh) % g.H
    s = (v - g.sw) % g.W
    order = np.lexsort(((s % g.ww).ravel(), (r % g.wh).ravel(),
                        (s // g.ww).ravel(), (r // g.wh).ravel()))
    x = _x(g)
    expect = x.reshape(g.B, g.H * g.W, g.C)[:, order, :]
    assert np.array_equal(route(x, g), expect)


@pytest.mark.parametrize("g", GEOMS)
def test_unroute_is_exact_inverse(g):
    cfg = ts.small_config("t", "f32", g.B, g.H, g.W, g.heads, g.head_dim, g.wh, g.ww, g.sh, g.sw)
    for width in (4, 2):
        x = ts.token_pattern(cfg, width)
        y = route(x, g)
        assert y.dtype == x.dtype
        assert np.array_equal(unroute(y, g), x)
        assert np.array_equal(route(unroute(y, g), g), y)


@pytest.mark.parametrize("g", GEOMS)
def test_wrap_labels_mark_the_wrapped_rows(g):
    tab = token_table(g)
    lat_expect = (g.mask_flags & 1) and g.sh > 0
    assert np.array_equal(tab["lat"].astype(bool), bool(lat_expect) & (tab["u"] < g.sh))
    lon_expect = (g.mask_flags & 2) and g.sw > 0
    assert np.array_equal(tab["lon"].astype(bool), bool(lon_expect) & (tab["v"] < g.sw))


def test_window_counts_of_the_five_configs():
    # Closed forms: Mh = ceil(H/wh), Mw = ceil(W/ww); partial rows/cols.
    expect = {
        "c1_f32_16x32_w8": {64: 8},
        "c2_bf16_128x256_w8": {64: 512},
        "c3_bf16_85x180_w12": {144: 105, 12: 15},
        "c4_bf16_128x1080_w8x16": {128: 1072, 64: 16},
        "c5_bf16_256x540_w24": {576: 220, 384: 22, 288: 10, 192: 1},
    }
    for name, counts in expect.items():
        cfg = ts.CONFIGS[name]
        g = Geometry(**cfg.geom_kwargs())
        got = {}
        for _, _, n in window_slots(g):
            got[n] = got.get(n, 0) + 1
        assert got == counts, name
        assert sum(n * c for n, c in counts.items()) == cfg.H * cfg.W


def test_window_offsets_are_prefix_sums_with_closed_form():
    g = Geometry(1, 85, 180, 1, 1, 1, 12, 12, 6, 6)
    Mh, Mw, rows, cols = window_extents(g.H, g.W, g.wh, g.ww)
    for w, start, n in window_slots(g):
        i, j = divmod(w, Mw)
        # offset(i, j) = i*wh*W + rows_i * j * ww  (every earlier window row is full)
        assert start == i * g.wh * g.W + rows[i] * j * g.ww
        assert n == rows[i] * cols[j]
