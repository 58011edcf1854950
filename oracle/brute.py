"""Brute-force shifted-window attention over the whole grid (oracle side).

Test infrastructure only (see the package docstring).

Independent of the window-major machinery: every pair of tokens of an image
is tested directly from its ORIGINAL coordinates (u, v) in NHWC order:

* rolled coordinate (r, s) = ((u - sh) mod H, (v - sw) mod W)  (shift route,
  Sec. IV-D; content moves toward the top-left);
* window (floor(r / wh), floor(s / ww)) and in-window offset
  (r mod wh, s mod ww)  (Sec. IV-D, Eq. (2));
* wrap labels [r >= H - sh] and [s >= W - sw] when the corresponding mask
  bit is set;
* two tokens attend iff same window and same labels; the bias of a pair is
  the table entry at (query offset - key offset) + (wh - 1, ww - 1).

Intended for tiny grids: it forms the (H*W) x (H*W) score matrix per head.
Outputs stay in NHWC order (O: B x H x W x C, LSE: B x heads x H x W).
"""

import numpy as np

MASK_LAT = 1
MASK_LON = 2


def _pair_structure(g):
    H, W = g.H, g.W
    uu, vv = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    u = uu.reshape(-1)
    v = vv.reshape(-1)
    r = (u - g.sh) % H
    s = (v - g.sw) % W
    wi, wj = r // g.wh, s // g.ww
    a, c = r % g.wh, s % g.ww
    lat = ((g.mask_flags & MASK_LAT) != 0) & (g.sh > 0) & (r >= H - g.sh)
    lon = ((g.mask_flags & MASK_LON) != 0) & (g.sw > 0) & (s >= W - g.sw)
    allowed = ((wi[:, None] == wi[None, :]) & (wj[:, None] == wj[None, :])
               & (lat[:, None] == lat[None, :]) & (lon[:, None] == lon[None, :]))
    ia = a[:, None] - a[None, :] + g.wh - 1
    ic = c[:, None] - c[None, :] + g.ww - 1
    return allowed, ia, ic


def fwd(q, k, v, table, g):
    """q, k, v: (B, H, W, C).  Returns (O (B,H,W,C), LSE (B,heads,H,W)), fp64."""
    B = q.shape[0]
    T = g.H * g.W
    allowed, ia, ic = _pair_structure(g)
    tab = np.asarray(table, np.float64)
    o = np.zeros((B, T, g.C))
    lse = np.zeros((B, g.heads, T))
    for b in range(B):
        for h in range(g.heads):
            sl = slice(h * g.head_dim, (h + 1) * g.head_dim)
            qh = np.asarray(q[b], np.float64).reshape(T, g.C)[:, sl]
            kh = np.asarray(k[b], np.float64).reshape(T, g.C)[:, sl]
            vh = np.asarray(v[b], np.float64).reshape(T, g.C)[:, sl]
            s = qh @ kh.T / np.sqrt(g.head_dim) + tab[ia, ic, h]
            s[~allowed] = -np.inf
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            l = e.sum(axis=1, keepdims=True)
            o[b][:, sl] = (e / l) @ vh
            lse[b, h] = (m + np.log(l))[:, 0]
    return o.reshape(B, g.H, g.W, g.C), lse.reshape(B, g.heads, g.H, g.W)


def allowed_pairs(g):
    """The (H*W) x (H*W) boolean attend-matrix in NHWC token order."""
    return _pair_structure(g)[0]
