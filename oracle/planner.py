"""Window assignment across ranks and the per-rank token route (oracle side).

Test infrastructure only (see the package docstring).

Definitions followed
--------------------
* Sec. V-A, Eq. (3): the fixed (two-dimensional round-robin) assignment of
  an M_h x M_w window grid to an m x n WP mesh pads the input field H x W to
      H_hat = ceil(H / (p alpha w m)) p alpha w m,
      W_hat = ceil(W / (p alpha w n)) p alpha w n,
  with p the patch size, alpha the down-sampling stride and w the window.
  Padding overhead is H_hat W_hat / (H W) - 1 (extra grid points over the
  real ones).  m = n = 1 gives the minimal padding to whole windows.
* Sec. V-A, Eq. (4): the ragged assignment Topo(mn, 1) flattens the window
  grid row-major and gives WP rank r the window range [L_r, R_r) with
  L_r = floor(r M / mn), R_r = floor((r + 1) M / mn).
* Sec. V-B: with SP degree s (Topo(mn/s, 1, s)) every window is cut into s
  sub-tiles, one per SP rank, and the mn/s WP groups take window ranges by
  Eq. (4); a rank then processes as many sub-tiles as its WP group owns
  windows.
* Sec. IV-B: the I/O topology cuts the grid into contiguous height stripes,
  one per DMP rank.  Reading used for grids whose height is not a multiple
  of the rank count (no grid is padded here): rank r holds rows
  [floor(r H / P), floor((r + 1) H / P)), the same floor rule as Eq. (4).
* Sec. IV-D: a token's global coordinate (u, v) fixes both its DMP source
  rank (the stripe holding row u) and, through the window shift, the window
  (and so the WP rank) that needs it.  The route of rank r gathers the
  window-major slots of its window range; tokens whose row lies in another
  rank's stripe arrive from that rank (the shift route's boundary
  fragments).  Here every needed token is listed one by one.

The window grid is the one of ``geometry`` (ragged last row and column, no
padding), so M = ceil(H / wh) ceil(W / ww) windows per image.
"""

from .geometry import token_table, window_slots, window_extents


def padded_grid(H, W, p, alpha, w, m=1, n=1):
    """Eq. (3): padded input size (H_hat, W_hat) for an m x n WP mesh."""
    unit_h = p * alpha * w * m
    unit_w = p * alpha * w * n
    H_hat = -(-H // unit_h) * unit_h
    W_hat = -(-W // unit_w) * unit_w
    return H_hat, W_hat


def padding_overhead(H, W, H_hat, W_hat):
    """Padded grid points over real grid points, minus one (0.189 = 18.9 %)."""
    return (H_hat * W_hat) / (H * W) - 1.0


def window_ranges(M, ranks):
    """Eq. (4): [(L_r, R_r)] for r = 0 .. ranks-1."""
    return [((r * M) // ranks, ((r + 1) * M) // ranks) for r in range(ranks)]


def subtiles_per_rank(M, mn, s):
    """Sec. V-B, Topo(mn/s, 1, s): sub-tiles processed by each of the mn
    ranks, listed WP group by WP group (each SP rank of a group takes one
    sub-tile of every window the group owns)."""
    assert mn % s == 0
    out = []
    for L, R in window_ranges(M, mn // s):
        out.extend([R - L] * s)
    return out


def stripes(H, ranks):
    """DMP height stripes: [(row_begin, row_end)] per rank."""
    return [((r * H) // ranks, ((r + 1) * H) // ranks) for r in range(ranks)]


def stripe_owner(H, ranks, u):
    for r, (a, b) in enumerate(stripes(H, ranks)):
        if a <= u < b:
            return r
    raise ValueError("row %d outside the grid" % u)


def rank_slots(g, ranks, r):
    """First and one-past-last window-major slot (per image) of rank r's
    window range."""
    Mh, Mw, _, _ = window_extents(g.H, g.W, g.wh, g.ww)
    L, R = window_ranges(Mh * Mw, ranks)[r]
    slots = window_slots(g)
    begin = slots[L][1] if L < len(slots) else g.H * g.W
    end = slots[R][1] if R < len(slots) else g.H * g.W
    return begin, end


def needed_tokens(g, ranks, r):
    """Every token rank r's route needs, one by one: a dict mapping each
    source DMP rank to the set of grid coordinates (u, v) it supplies."""
    tab = token_table(g)
    begin, end = rank_slots(g, ranks, r)
    need = {}
    for t in range(begin, end):
        u, v = int(tab["u"][t]), int(tab["v"][t])
        need.setdefault(stripe_owner(g.H, ranks, u), set()).add((u, v))
    return need
