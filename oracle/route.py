"""Token route between the NHWC layout and the window-major layout (oracle side).

Test infrastructure only (see the package docstring).

Sec. IV-D: both layouts are indexed by the same global token coordinate; the
route gathers every token into its window-major slot and the inverse route
puts every slot back (the backward of one is the other).  On one device the
route is a pure permutation of token rows; channels travel unchanged.

Window-major layout of one image: windows in row-major order, tokens
row-major within each window's actual extent, channels innermost
(B x (H*W) x C).
"""

import numpy as np

from .geometry import token_table


def _src_index(g):
    tab = token_table(g)
    return tab["u"] * g.W + tab["v"]


def route(x, g):
    """x: (B, H, W, C) -> (B, H*W, C) window-major.  Bit copy."""
    B, H, W, C = x.shape
    assert (H, W) == (g.H, g.W)
    src = _src_index(g)
    return x.reshape(B, H * W, C)[:, src, :].copy()


def unroute(y, g):
    """y: (B, H*W, C) window-major -> (B, H, W, C).  Exact inverse of route."""
    B, T, C = y.shape
    assert T == g.H * g.W
    src = _src_index(g)
    x = np.empty_like(y)
    x[:, src, :] = y
    return x.reshape(B, g.H, g.W, C)
