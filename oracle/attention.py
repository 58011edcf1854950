"""Windowed multi-head self-attention with relative-position bias (oracle side).

Test infrastructure only (see the package docstring).

The paper's Swin blocks run W-MSA / SW-MSA (Sec. IV-A, citing Swin) on the
window-major layout produced by the token routes (Sec. IV-D).  The paper does
not write the attention formula out; the plain definition used here is the
Swin one, per window and head h:

    S[q, k] = <Q_q, K_k>_h / sqrt(head_dim) + T[a_q - a_k + wh - 1, c_q - c_k + ww - 1, h]
    S[q, k] = -inf where q and k carry different shifted-window labels
    P = softmax_k(S),  O_q = sum_k P[q, k] V_k,  LSE_q = ln sum_k exp S[q, k]

with (a, c) the in-window offset, T the (2wh-1) x (2ww-1) x heads bias table,
and labels as in ``geometry``.  The backward, for an upstream gradient dO:

    dV = P^T dO,  dP = dO V^T,  D_q = sum_k P[q, k] dP[q, k]
    dS = P * (dP - D),  dQ = dS K / sqrt(hd),  dK = dS^T Q / sqrt(hd)
    dT[bin(q, k), h] = sum over batch, windows and allowed pairs of dS[q, k]

Everything is fp64.  Inputs in window-major layout (B, H*W, C), channel
c = h*head_dim + e; LSE is (B, heads, H*W) in window-major token order.
Windows that share extent and labels are stacked and handled with batched
matmuls; nothing else is blocked, fused or reordered.
"""

import numpy as np

from .geometry import window_classes, window_slots, token_table

_CHUNK_BYTES = 1 << 28  # cap on the (.., n, n) fp64 score arrays per batch


def _class_bias(cls, table, g):
    """Bias matrix (heads, n, n) and allowed-pair matrix (n, n) of a class."""
    a, c = cls["a"], cls["c"]
    ia = a[:, None] - a[None, :] + g.wh - 1        # query minus key
    ic = c[:, None] - c[None, :] + g.ww - 1
    bias = np.asarray(table, np.float64)[ia, ic, :].transpose(2, 0, 1)
    allowed = ((cls["lat"][:, None] == cls["lat"][None, :])
               & (cls["lon"][:, None] == cls["lon"][None, :]))
    return bias, allowed, ia, ic


def _gather(x, idx, g):
    """x (B, HW, C) -> (B, nw, heads, n, hd) for slots idx (nw, n)."""
    B = x.shape[0]
    nw, n = idx.shape
    t = np.asarray(x, np.float64)[:, idx.reshape(-1), :]
    return t.reshape(B, nw, n, g.heads, g.head_dim).transpose(0, 1, 3, 2, 4)


def _scatter(out, idx, val, g):
    """Inverse of _gather into out (B, HW, C)."""
    B, nw, _, n, _ = val.shape
    out[:, idx.reshape(-1), :] = val.transpose(0, 1, 3, 2, 4).reshape(B, nw * n, g.C)


def _forward_block(qw, kw, vw, bias, allowed, hd):
    s = qw @ kw.swapaxes(-1, -2) / np.sqrt(hd) + bias
    s = np.where(allowed, s, -np.inf)
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=-1, keepdims=True)
    p = e / l
    o = p @ vw
    lse = (m + np.log(l))[..., 0]
    return o, lse, p


def _chunks(starts, B, heads, n):
    per_window = max(1, B * heads * n * n * 8)
    step = max(1, _CHUNK_BYTES // per_window)
    for lo in range(0, len(starts), step):
        yield starts[lo:lo + step]


def _select(cls, windows):
    if windows is None:
        return cls["starts"]
    return np.asarray([s for s in cls["starts"] if s in windows], np.int64)


def attn_fwd(q, k, v, table, g, _windows=None):
    """Forward over every window.  Returns (O (B,HW,C), LSE (B,heads,HW))."""
    B = q.shape[0]
    o = np.zeros((B, g.tokens, g.C), np.float64)
    lse = np.zeros((B, g.heads, g.tokens), np.float64)
    for cls in window_classes(g):
        bias, allowed, _, _ = _class_bias(cls, table, g)
        n = cls["n"]
        starts = _select(cls, _windows)
        for st in _chunks(starts, B, g.heads, n):
            idx = st[:, None] + np.arange(n)[None, :]
            ob, lb, _ = _forward_block(_gather(q, idx, g), _gather(k, idx, g),
                                       _gather(v, idx, g), bias, allowed, g.head_dim)
            _scatter(o, idx, ob, g)
            # lb: (B, nw, heads, n) -> lse[b, h, slot]
            lse[:, :, idx.reshape(-1)] = lb.transpose(0, 2, 1, 3).reshape(B, g.heads, -1)
    return o, lse


def attn_bwd(q, k, v, dout, table, g, _windows=None):
    """Backward over every window.  Returns (dQ, dK, dV, dT); dT has the bias
    table's shape (2wh-1, 2ww-1, heads) and sums over batch and windows."""
    B = q.shape[0]
    hd = g.head_dim
    dq = np.zeros((B, g.tokens, g.C), np.float64)
    dk = np.zeros_like(dq)
    dv = np.zeros_like(dq)
    dtab = np.zeros((2 * g.wh - 1, 2 * g.ww - 1, g.heads), np.float64)
    for cls in window_classes(g):
        bias, allowed, ia, ic = _class_bias(cls, table, g)
        n = cls["n"]
        starts = _select(cls, _windows)
        for st in _chunks(starts, B, g.heads, n):
            idx = st[:, None] + np.arange(n)[None, :]
            qw, kw, vw = _gather(q, idx, g), _gather(k, idx, g), _gather(v, idx, g)
            dow = _gather(dout, idx, g)
            _, _, p = _forward_block(qw, kw, vw, bias, allowed, hd)
            dvw = p.swapaxes(-1, -2) @ dow
            dp = dow @ vw.swapaxes(-1, -2)
            D = (p * dp).sum(axis=-1, keepdims=True)
            ds = p * (dp - D)
            dqw = ds @ kw / np.sqrt(hd)
            dkw = ds.swapaxes(-1, -2) @ qw / np.sqrt(hd)
            _scatter(dq, idx, dqw, g)
            _scatter(dk, idx, dkw, g)
            _scatter(dv, idx, dvw, g)
            ds_sum = ds.sum(axis=(0, 1))                     # (heads, n, n)
            np.add.at(dtab, (ia, ic), ds_sum.transpose(1, 2, 0))
    return dq, dk, dv, dtab


def _window_starts(g, windows):
    slots = {w: (st, n) for w, st, n in window_slots(g)}
    return {w: slots[w] for w in windows}


def attn_fwd_windows(q, k, v, table, g, windows):
    """Forward restricted to the given window indices (row-major window id).
    Returns {window: (O (B,n,C), LSE (B,heads,n))}; used to check samples of
    full-size runs one window at a time."""
    sel = _window_starts(g, windows)
    starts = {st for st, _ in sel.values()}
    o, lse = attn_fwd(q, k, v, table, g, _windows=starts)
    return {w: (o[:, st:st + n], lse[:, :, st:st + n]) for w, (st, n) in sel.items()}


def attn_bwd_windows(q, k, v, dout, table, g, windows):
    """Backward restricted to the given windows: {window: (dQ, dK, dV)} each
    (B, n, C).  (The bias-table gradient needs every window.)"""
    sel = _window_starts(g, windows)
    starts = {st for st, _ in sel.values()}
    dq, dk, dv, _ = attn_bwd(q, k, v, dout, table, g, _windows=starts)
    return {w: (dq[:, st:st + n], dk[:, st:st + n], dv[:, st:st + n])
            for w, (st, n) in sel.items()}


def token_labels(g):
    """(lat, lon) labels per window-major slot, for tests."""
    tab = token_table(g)
    return tab["lat"], tab["lon"]
