"""Pins for the oracle's attention backward (CPU only).

The backward is checked against central finite differences of the oracle's
own forward (which the forward pins tie to the definition), against torch
autograd of scaled_dot_product_attention in fp64 on a whole-grid window, and
against closed-form invariants of softmax attention.
"""

import numpy as np
import pytest
import torch

from oracle import Geometry, route, attn_fwd, attn_bwd
from oracle.geometry import window_slots


def _inputs(g, seed=2):
    rng = np.random.default_rng(seed)
    shp = (g.B, g.H * g.W, g.C)
    q, k, v, do = (rng.standard_normal(shp) for _ in range(4))
    table = 0.3 * rng.standard_normal((2 * g.wh - 1, 2 * g.ww - 1, g.heads))
    return q, k, v, do, table


def _loss(q, k, v, table, do, g):
    o, _ = attn_fwd(q, k, v, table, g)
    return float((o * do).sum())


@pytest.mark.parametrize("g", [Geometry(1, 5, 7, 4, 2, 2, 3, 4, 1, 2, 3),
                               Geometry(2, 4, 6, 2, 1, 2, 3, 3, 2, 1, 1)])
def test_gradients_equal_central_differences(g):
    q, k, v, do, table = _inputs(g)
    dq, dk, dv, dt = attn_bwd(q, k, v, do, table, g)
    h = 1e-6
    for name, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv), ("t", table, dt)):
        fd = np.zeros_like(arr)
        flat = arr.reshape(-1)
        for i in range(flat.size):
            keep = flat[i]
            flat[i] = keep + h
            lp = _loss(q, k, v, table, do, g)
            flat[i] = keep - h
            lm = _loss(q, k, v, table, do, g)
            flat[i] = keep
            fd.reshape(-1)[i] = (lp - lm) / (2 * h)
        assert np.abs(fd - grad).max() < 1e-7, name


def test_whole_grid_window_gradients_equal_torch_autograd():
    g = Geometry(1, 4, 6, 8, 2, 4, 4, 6, 0, 0)
    q, k, v, do, _ = _inputs(g, seed=4)
    table = np.zeros((7, 11, 2))
    dq, dk, dv, _ = attn_bwd(q, k, v, do, table, g)
    t = [torch.tensor(x.reshape(1, 24, 2, 4).transpose(0, 2, 1, 3).copy(), requires_grad=True)
         for x in (q, k, v)]
    o = torch.nn.functional.scaled_dot_product_attention(*t)
    o.backward(torch.from_numpy(do.reshape(1, 24, 2, 4).transpose(0, 2, 1, 3).copy()))
    for mine, ref in zip((dq, dk, dv), t):
        r = ref.grad.permute(0, 2, 1, 3).reshape(1, 24, 8).numpy()
        assert np.abs(mine - r).max() < 1e-12


def test_closed_form_invariants():
    g = Geometry(2, 13, 10, 6, 3, 2, 6, 4, 3, 1, 3)
    q, k, v, do, table = _inputs(g, seed=6)
    dq, dk, dv, dt = attn_bwd(q, k, v, do, table, g)
    for _, st, n in window_slots(g):
        sl = slice(st, st + n)
        # adding one vector to every key leaves softmax unchanged -> sum dK = 0
        assert np.abs(dk[:, sl].sum(axis=1)).max() < 1e-10
        # rows of P sum to one and stay inside the window -> sum dV = sum dO
        assert np.abs(dv[:, sl].sum(axis=1) - do[:, sl].sum(axis=1)).max() < 1e-10
    # each row of dS sums to zero -> the bias gradient of every head sums to zero
    assert np.abs(dt.sum(axis=(0, 1))).max() < 1e-10


def test_bias_gradient_of_one_bin_is_the_sum_of_its_pairs():
    # Cross-check the scatter of dS into bins with a one-bin perturbation of
    # the table: d loss / d T[bin] by differences for three bins.
    g = Geometry(1, 6, 8, 4, 2, 2, 3, 4, 1, 2, 1)
    q, k, v, do, table = _inputs(g, seed=8)
    _, _, _, dt = attn_bwd(q, k, v, do, table, g)
    for b in [(2, 3, 0), (0, 0, 1), (4, 6, 1)]:
        h = 1e-6
        tp, tm = table.copy(), table.copy()
        tp[b] += h
        tm[b] -= h
        fd = (_loss(q, k, v, tp, do, g) - _loss(q, k, v, tm, do, g)) / (2 * h)
        assert abs(fd - dt[b]) < 1e-7
