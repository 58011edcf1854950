"""Pins for the oracle's window-restricted helpers (CPU only).

``attn_fwd_windows`` and ``attn_bwd_windows`` judge every sampled full-size
result, so they are tied here to two things outside themselves:

* the brute-force whole-grid attention (``brute.fwd``), which never forms the
  window-major layout: the restricted forward must equal the slots of the
  chosen windows of the brute-force result routed into window-major order;
* the unrestricted ``attn_fwd`` / ``attn_bwd`` (pinned by the brute force,
  finite differences and torch autograd): the restricted results must equal
  the same windows of the full results exactly.

The geometry is ragged both ways, shifted and masked both ways, and the
window set holds the first, last, latitude-seam, longitude-seam,
partial-row, partial-column and interior windows.  A wrong window to slot
map (a transposed window index, an off-by-one in the first slot, a window
taken from the wrong image) fails one of the comparisons.
"""

import numpy as np
import pytest

from oracle import Geometry, route, attn_fwd, attn_bwd, attn_fwd_windows, attn_bwd_windows, brute
from oracle.geometry import window_slots, window_extents

GEOMS = [
    # ragged both ways (13 = 2*5+3 rows, 23 = 3*6+5 columns), both wraps masked, 2 images
    Geometry(2, 13, 23, 6, 2, 3, 5, 6, 2, 3, 3),
    # shift 0 on a ragged grid, latitude mask bit set (no label ever set)
    Geometry(1, 11, 14, 4, 1, 4, 4, 5, 0, 0, 1),
]


def _inputs(g, seed=4):
    rng = np.random.default_rng(seed)
    shp = (g.B, g.H, g.W, g.C)
    q, k, v, do = (rng.standard_normal(shp) for _ in range(4))
    table = 0.3 * rng.standard_normal((2 * g.wh - 1, 2 * g.ww - 1, g.heads))
    return q, k, v, do, table


def _pick(g):
    Mh, Mw, rows, cols = window_extents(g.H, g.W, g.wh, g.ww)
    last = Mh * Mw - 1
    pick = {0, Mw - 1, (Mh - 1) * Mw, last, Mw + 1, (Mh - 2) * Mw + Mw - 1}
    # the restricted helpers must not depend on the order or repetition of the request
    return sorted(pick), [last, 0, Mw + 1, Mw + 1]


@pytest.mark.parametrize("g", GEOMS)
def test_restricted_forward_equals_brute_force_windows(g):
    q, k, v, _, table = _inputs(g)
    sel, _ = _pick(g)
    got = attn_fwd_windows(route(q, g), route(k, g), route(v, g), table, g, sel)
    ob, lb = brute.fwd(q, k, v, table, g)
    ow = route(ob, g)                                            # (B, HW, C) window-major
    lw = route(lb.transpose(0, 2, 3, 1), g).transpose(0, 2, 1)   # (B, heads, HW)
    slots = {w: (s, n) for w, s, n in window_slots(g)}
    assert set(got) == set(sel)
    for w in sel:
        s, n = slots[w]
        assert got[w][0].shape == (g.B, n, g.C)
        assert np.abs(got[w][0] - ow[:, s:s + n]).max() < 1e-12
        assert np.abs(got[w][1] - lw[:, :, s:s + n]).max() < 1e-12


@pytest.mark.parametrize("g", GEOMS)
def test_restricted_results_equal_slices_of_full_results(g):
    q, k, v, do, table = _inputs(g, seed=6)
    qw, kw, vw, dow = (route(x, g) for x in (q, k, v, do))
    o, lse = attn_fwd(qw, kw, vw, table, g)
    dq, dk, dv, _ = attn_bwd(qw, kw, vw, dow, table, g)
    slots = {w: (s, n) for w, s, n in window_slots(g)}
    for sel in _pick(g):
        fw = attn_fwd_windows(qw, kw, vw, table, g, sel)
        bw = attn_bwd_windows(qw, kw, vw, dow, table, g, sel)
        assert set(fw) == set(sel) and set(bw) == set(sel)
        for w in set(sel):
            s, n = slots[w]
            assert np.array_equal(fw[w][0], o[:, s:s + n])
            assert np.array_equal(fw[w][1], lse[:, :, s:s + n])
            for got, full in zip(bw[w], (dq, dk, dv)):
                assert got.shape == (g.B, n, g.C)
                assert np.array_equal(got, full[:, s:s + n])


def test_restricted_backward_ignores_other_windows():
    # Changing every token outside the chosen windows leaves their gradients
    # unchanged (windows are independent), and changing a token inside one
    # of them changes it.
    g = GEOMS[0]
    q, k, v, do, table = _inputs(g, seed=8)
    qw, kw, vw, dow = (route(x, g) for x in (q, k, v, do))
    sel = [0, 7]
    slots = {w: (s, n) for w, s, n in window_slots(g)}
    inside = np.zeros(g.H * g.W, bool)
    for w in sel:
        s, n = slots[w]
        inside[s:s + n] = True
    ref = attn_bwd_windows(qw, kw, vw, dow, table, g, sel)
    k2 = kw.copy()
    k2[:, ~inside] += 5.0
    same = attn_bwd_windows(qw, k2, vw, dow, table, g, sel)
    for w in sel:
        for a, b in zip(ref[w], same[w]):
            assert np.array_equal(a, b)
    k3 = kw.copy()
    s, n = slots[7]
    k3[:, s] += 1.0
    moved = attn_bwd_windows(qw, k3, vw, dow, table, g, sel)
    assert np.array_equal(moved[0][0], ref[0][0])
    assert np.abs(moved[7][0] - ref[7][0]).max() > 1e-6
