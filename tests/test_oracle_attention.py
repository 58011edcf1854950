"""Pins for the oracle's windowed attention forward (CPU only).

The windowed oracle is checked against: torch's scaled_dot_product_attention
in fp64 (a whole-grid window), the semantics of the bias table (one-hot
tables move attention to one neighbour), the brute-force whole-grid mask on
tiny ragged shifted grids, numpy.roll for unmasked shifts, seam isolation and
the softmax bounds.
"""

import numpy as np
import pytest
import torch

from oracle import Geometry, route, unroute, attn_fwd, brute


def _inputs(g, seed=1, scale=1.0):
    rng = np.random.default_rng(seed)
    shp = (g.B, g.H, g.W, g.C)
    q, k, v = (rng.standard_normal(shp) * s for s in (scale, 1.0, 1.0))
    table = 0.3 * rng.standard_normal((2 * g.wh - 1, 2 * g.ww - 1, g.heads))
    return q, k, v, table


def _windowed(q, k, v, table, g):
    o, lse = attn_fwd(route(q, g), route(k, g), route(v, g), table, g)
    return o, lse


def test_whole_grid_window_equals_torch_sdpa():
    g = Geometry(2, 6, 5, 8, 2, 4, 6, 5, 0, 0)
    q, k, v, _ = _inputs(g)
    table = np.zeros((11, 9, 2))
    o, lse = _windowed(q, k, v, table, g)
    o = unroute(o, g)
    tq, tk, tv = (torch.from_numpy(x.reshape(2, 30, 2, 4).transpose(0, 2, 1, 3).copy())
                  for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
    ref = ref.permute(0, 2, 1, 3).reshape(2, 6, 5, 8).numpy()
    assert np.abs(o - ref).max() < 1e-12
    # log-sum-exp of the scaled logits
    s = torch.einsum("bhqe,bhke->bhqk", tq, tk) / 2.0
    lse_ref = torch.logsumexp(s, dim=-1).numpy()        # NHWC token order (unshifted)
    assert np.abs(lse - lse_ref).max() < 1e-12


@pytest.mark.parametrize("delta", [(1, 0), (0, 1), (-1, 0), (0, -2), (2, 3)])
def test_one_hot_bias_moves_attention_to_the_offset_neighbour(delta):
    # With a +60 entry at bin (query - key) = delta, every query whose key at
    # offset -delta exists inside its window attends (almost) only to it.
    g = Geometry(1, 8, 8, 4, 2, 2, 4, 4, 0, 0, 0)
    q, k, v, _ = _inputs(g, seed=3)
    table = np.zeros((7, 7, 2))
    table[delta[0] + 3, delta[1] + 3, 1] = 60.0      # head 1 only
    o, _ = _windowed(q, k, v, table, g)
    o = unroute(o, g)
    o_free, _ = _windowed(q, k, v, np.zeros_like(table), g)
    o_free = unroute(o_free, g)
    for u in range(8):
        for w in range(8):
            ku, kw = u - delta[0], w - delta[1]
            same = (0 <= ku < 8 and 0 <= kw < 8 and ku // 4 == u // 4 and kw // 4 == w // 4)
            if same:
                assert np.allclose(o[0, u, w, 2:], v[0, ku, kw, 2:], atol=1e-12)
            else:
                assert np.allclose(o[0, u, w, 2:], o_free[0, u, w, 2:], atol=1e-12)
    assert np.allclose(o[..., :2], o_free[..., :2], atol=1e-14)   # head 0 untouched


GEOMS = [
    Geometry(1, 16, 32, 64, 2, 32, 8, 8, 4, 4, 1),      # config-1 geometry
    Geometry(2, 7, 9, 6, 2, 3, 3, 4, 1, 2, 1),
    Geometry(2, 7, 9, 6, 2, 3, 3, 4, 1, 2, 3),          # both wraps masked
    Geometry(1, 13, 10, 4, 1, 4, 6, 4, 3, 1, 1),        # ragged both ways
    Geometry(1, 9, 20, 8, 2, 4, 4, 8, 2, 4, 0),         # no mask at all
    Geometry(1, 10, 12, 4, 2, 2, 5, 4, 0, 0, 1),        # shift 0
]


@pytest.mark.parametrize("g", GEOMS)
def test_windowed_equals_brute_force_global_mask(g):
    q, k, v, table = _inputs(g, seed=5)
    o, lse = _windowed(q, k, v, table, g)
    ob, lb = brute.fwd(q, k, v, table, g)
    assert np.abs(o - route(ob, g)).max() < 1e-12
    lb_w = route(lb.transpose(0, 2, 3, 1), g).transpose(0, 2, 1)
    assert np.abs(lse - lb_w).max() < 1e-12


@pytest.mark.parametrize("shift,flags,axes", [((0, 3), 1, (2,)), ((2, 3), 0, (1, 2)),
                                              ((3, 0), 0, (1,))])
def test_unmasked_shift_equals_attention_on_rolled_grid(shift, flags, axes):
    # Where a wrap is not masked the shift is a plain cyclic roll of the grid.
    g = Geometry(1, 12, 16, 4, 2, 2, 4, 8, shift[0], shift[1], flags)
    g0 = Geometry(1, 12, 16, 4, 2, 2, 4, 8, 0, 0, flags)
    q, k, v, table = _inputs(g, seed=7)
    o, _ = _windowed(q, k, v, table, g)
    sh = tuple(-shift[a - 1] for a in axes)
    r = [np.roll(x, sh, axis=axes) for x in (q, k, v)]
    o0, _ = _windowed(*r, table, g0)
    assert np.abs(unroute(o, g) - np.roll(unroute(o0, g0), tuple(-s for s in sh), axis=axes)).max() < 1e-12


def test_seam_tokens_never_see_the_other_side():
    g = Geometry(1, 8, 8, 2, 1, 2, 4, 4, 2, 0, 1)
    q, k, v, table = _inputs(g, seed=9)
    o, _ = _windowed(q, k, v, table, g)
    v2 = v.copy()
    v2[0, 6:8, :, :] += 100.0      # original rows 6-7 share windows with rows 0-1 after the roll
    o2, _ = _windowed(q, k, v2, table, g)
    d = np.abs(unroute(o2, g) - unroute(o, g)).max(axis=-1)[0]
    assert np.all(d[0:2] < 1e-12)       # wrapped rows 0-1 are isolated from rows 6-7
    assert np.all(d[6:8] > 1.0)         # rows 6-7 see themselves
    assert np.all(d[2:6] < 1e-12)       # other windows untouched


def test_softmax_bounds():
    g = Geometry(1, 13, 10, 4, 1, 4, 6, 4, 3, 1, 3)
    q, k, v, table = _inputs(g, seed=11, scale=4.0)
    o, lse = _windowed(q, k, v, table, g)
    vw = route(v, g)
    ob, _ = brute.fwd(q, k, v, table, g)
    allowed = brute.allowed_pairs(g)
    counts = allowed.sum(1)
    # LSE >= own logit; convex combination of allowed values
    assert np.all(np.isfinite(lse))
    vmax, vmin = [], []
    vflat = v.reshape(g.H * g.W, g.C)
    for t in range(g.H * g.W):
        vmax.append(vflat[allowed[t]].max(0))
        vmin.append(vflat[allowed[t]].min(0))
    obf = ob.reshape(g.H * g.W, g.C)
    assert np.all(obf <= np.array(vmax) + 1e-12) and np.all(obf >= np.array(vmin) - 1e-12)
    assert counts.min() >= 1
    del vw
