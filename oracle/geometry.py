"""Window partition of the shifted Transformer-stage token grid (oracle side).

Test infrastructure only (see the package docstring).

Definitions followed
--------------------
* Sec. IV-D, Eq. (2): a token of the H x W grid is identified by its global
  coordinate (u, v); its attention window is (floor(u / w), floor(v / w)) and
  its in-window offset is (u mod w, v mod w).  The window is generalised here
  to a rectangle (wh, ww).
* Sec. IV-D (shift route): the shifted window changes each token's
  coordinate.  Reading used: the grid is rolled so that content moves toward
  the top-left, i.e. the rolled coordinate of original (u, v) is
  (r, s) = ((u - sh) mod H, (v - sw) mod W), and the partition of Eq. (2) is
  applied to (r, s).
* Ragged edges: the grid is NOT padded.  When wh does not divide H (or ww
  does not divide W) the last window row (column) of the rolled grid is
  partial: rows_i = min(wh, H - i*wh), cols_j = min(ww, W - j*ww).
* Sec. V-A, Eq. (4): windows are flattened in row-major order.  Tokens within
  a window are ordered row-major over the window's actual extent.
* Shifted-window mask labels: longitude is periodic (no label) unless bit 1 of
  ``mask_flags`` is set; the latitude wrap is labelled when bit 0 is set.  A
  token carries latitude label 1 iff it is one of the sh rows that wrapped
  around (r >= H - sh, equivalently u < sh); longitude label likewise with sw.
  Two tokens may attend to each other iff they lie in the same window and
  carry equal labels.

Everything here is computed by enumerating tokens one by one, so that it can
be read against the definitions directly.
"""

from dataclasses import dataclass
from functools import lru_cache

import numpy as np

MASK_LAT = 1  # bit 0: latitude wrap masked
MASK_LON = 2  # bit 1: longitude wrap masked


@dataclass(frozen=True)
class Geometry:
    B: int
    H: int
    W: int
    C: int
    heads: int
    head_dim: int
    wh: int
    ww: int
    sh: int
    sw: int
    mask_flags: int = MASK_LAT

    def check(self):
        assert self.C == self.heads * self.head_dim
        assert 1 <= self.wh <= self.H and 1 <= self.ww <= self.W
        assert 0 <= self.sh < self.wh and 0 <= self.sw < self.ww
        assert self.B >= 1

    @property
    def tokens(self):
        return self.H * self.W


def window_extents(H, W, wh, ww):
    """Window grid size and per-row / per-column extents of the rolled grid."""
    Mh = -(-H // wh)
    Mw = -(-W // ww)
    rows = [min(wh, H - i * wh) for i in range(Mh)]
    cols = [min(ww, W - j * ww) for j in range(Mw)]
    return Mh, Mw, rows, cols


@lru_cache(maxsize=32)
def _table(H, W, wh, ww, sh, sw, mask_flags):
    Mh, Mw, rows, cols = window_extents(H, W, wh, ww)
    n_tok = H * W
    u = np.empty(n_tok, np.int64)
    v = np.empty(n_tok, np.int64)
    win = np.empty(n_tok, np.int64)
    a_in = np.empty(n_tok, np.int64)
    c_in = np.empty(n_tok, np.int64)
    lat = np.zeros(n_tok, np.int64)
    lon = np.zeros(n_tok, np.int64)
    t = 0
    for i in range(Mh):
        for j in range(Mw):
            for a in range(rows[i]):
                for c in range(cols[j]):
                    r = i * wh + a          # rolled row
                    s = j * ww + c          # rolled column
                    u[t] = (r + sh) % H     # original row that lands here
                    v[t] = (s + sw) % W     # original column that lands here
                    win[t] = i * Mw + j
                    a_in[t] = a
                    c_in[t] = c
                    if (mask_flags & MASK_LAT) and sh > 0 and r >= H - sh:
                        lat[t] = 1
                    if (mask_flags & MASK_LON) and sw > 0 and s >= W - sw:
                        lon[t] = 1
                    t += 1
    assert t == n_tok
    out = dict(u=u, v=v, win=win, a=a_in, c=c_in, lat=lat, lon=lon)
    for arr in out.values():
        arr.setflags(write=False)
    return out


def token_table(g):
    """Per window-major slot of one image: the source coordinate (u, v), the
    window index (row-major), the in-window offset (a, c) and the two mask
    labels.  Arrays of length H*W, read-only."""
    return _table(g.H, g.W, g.wh, g.ww, g.sh, g.sw, g.mask_flags)


def window_slots(g):
    """List of (window index, first slot, token count) in window-major order."""
    Mh, Mw, rows, cols = window_extents(g.H, g.W, g.wh, g.ww)
    out = []
    start = 0
    for i in range(Mh):
        for j in range(Mw):
            n = rows[i] * cols[j]
            out.append((i * Mw + j, start, n))
            start += n
    return out


def window_classes(g):
    """Group windows that share token count, in-window offsets and labels
    (hence the same bias matrix and mask).  Returns a list of
    (starts, n, a, c, lat, lon) with ``starts`` the first slot of every window
    in the class (per image) and the rest the per-token arrays of one member."""
    tab = token_table(g)
    groups = {}
    for _, start, n in window_slots(g):
        sl = slice(start, start + n)
        key = (n, tab["a"][sl].tobytes(), tab["c"][sl].tobytes(),
               tab["lat"][sl].tobytes(), tab["lon"][sl].tobytes())
        if key not in groups:
            groups[key] = dict(starts=[], n=n, a=tab["a"][sl].copy(),
                               c=tab["c"][sl].copy(), lat=tab["lat"][sl].copy(),
                               lon=tab["lon"][sl].copy())
        groups[key]["starts"].append(start)
    out = []
    for grp in groups.values():
        grp["starts"] = np.asarray(grp["starts"], np.int64)
        out.append(grp)
    return out
