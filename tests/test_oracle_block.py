"""Pins for the oracle's Swin block (CPU only).

* LayerNorm and its backward against torch.nn.functional.layer_norm and
  torch autograd in fp64; GELU against torch's exact GELU and math.erf, its
  derivative against central differences.
* The whole block, forward and backward, against a torch fp64 autograd
  composition built from torch's own LayerNorm, Linear and GELU and an
  attention written from the brute-force whole-grid pair structure (never the
  window-major machinery): softmax(Q K^T / sqrt(hd) + bias, -inf where the
  pair is excluded) V.  This covers shifted, ragged, masked grids, the
  ordering of the Q/K/V rows of W_qkv and both residual branches.
* Central finite differences of L = sum(dx2 * x2) for sampled entries of x,
  every weight, bias, gain and shift, and the bias table.
"""

import math

import numpy as np
import pytest
import torch

from oracle import Geometry, brute
from oracle import block as ob


def _params(C, seed):
    rng = np.random.default_rng(seed)
    p = {}
    for name, shp in ob.PARAM_SHAPES.items():
        dims = shp(C)
        z = rng.standard_normal(dims)
        p[name] = 1.0 + 0.1 * z if name.endswith("_g") else (z / math.sqrt(dims[1]) if name.startswith("w_")
                                                              else 0.1 * z)
    return p


def test_layernorm_and_backward_equal_torch():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((5, 7, 12)) * 3 + 1
    gam, bet, dy = rng.standard_normal(12), rng.standard_normal(12), rng.standard_normal((5, 7, 12))
    y, zhat, rstd = ob.layernorm(z, gam, bet)
    tz, tg, tb = (torch.tensor(a, requires_grad=True) for a in (z, gam, bet))
    ty = torch.nn.functional.layer_norm(tz, (12,), tg, tb, eps=ob.EPS)
    assert np.abs(y - ty.detach().numpy()).max() < 1e-12
    ty.backward(torch.tensor(dy))
    dz, dg, db = ob.layernorm_bwd(dy, zhat, rstd, gam)
    assert np.abs(dz - tz.grad.numpy()).max() < 1e-12
    assert np.abs(dg - tg.grad.numpy()).max() < 1e-12
    assert np.abs(db - tb.grad.numpy()).max() < 1e-12


def test_gelu_and_derivative():
    t = np.linspace(-6, 6, 241)
    ref = torch.nn.functional.gelu(torch.tensor(t), approximate="none").numpy()
    assert np.abs(ob.gelu(t) - ref).max() < 1e-14
    assert abs(ob.gelu(np.array([1.3]))[0] - 1.3 * 0.5 * (1 + math.erf(1.3 / math.sqrt(2)))) < 1e-15
    h = 1e-6
    fd = (ob.gelu(t + h) - ob.gelu(t - h)) / (2 * h)
    assert np.abs(ob.gelu_grad(t) - fd).max() < 1e-8


def _torch_block(x, p, table, g):
    """The block as a torch fp64 graph; attention from the brute-force pair
    structure in NHWC order."""
    allowed, ia, ic = brute._pair_structure(g)
    T, C, hd = g.H * g.W, g.C, g.head_dim
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    tt = torch.tensor(table, requires_grad=True)
    tx = torch.tensor(x, requires_grad=True)
    ln1 = torch.nn.functional.layer_norm(tx, (C,), tp["ln1_g"], tp["ln1_b"], eps=ob.EPS)
    qkv = torch.nn.functional.linear(ln1, tp["w_qkv"], tp["b_qkv"]).reshape(g.B, T, 3 * C)
    q, k, v = (qkv[..., i * C:(i + 1) * C].reshape(g.B, T, g.heads, hd).transpose(1, 2) for i in range(3))
    bias = tt[torch.tensor(ia), torch.tensor(ic), :].permute(2, 0, 1)             # (heads, T, T)
    mask = torch.where(torch.tensor(allowed), 0.0, -math.inf).to(torch.float64)
    s = q @ k.transpose(-1, -2) / math.sqrt(hd) + bias + mask
    o = (torch.softmax(s, dim=-1) @ v).transpose(1, 2).reshape(g.B, g.H, g.W, C)
    x1 = tx + torch.nn.functional.linear(o, tp["w_proj"], tp["b_proj"])
    ln2 = torch.nn.functional.layer_norm(x1, (C,), tp["ln2_g"], tp["ln2_b"], eps=ob.EPS)
    a = torch.nn.functional.gelu(torch.nn.functional.linear(ln2, tp["w_fc1"], tp["b_fc1"]))
    x2 = x1 + torch.nn.functional.linear(a, tp["w_fc2"], tp["b_fc2"])
    return tx, tp, tt, x1, x2


GEOMS = [
    Geometry(1, 8, 8, 8, 2, 4, 8, 8, 0, 0, 0),           # one window, no shift
    Geometry(2, 7, 9, 8, 2, 4, 3, 4, 1, 2, 1),           # ragged, shifted, latitude mask
    Geometry(1, 10, 12, 12, 3, 4, 4, 5, 2, 3, 3),        # both masks
]


@pytest.mark.parametrize("g", GEOMS)
def test_block_equals_torch_autograd_composition(g):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((g.B, g.H, g.W, g.C))
    dx2 = rng.standard_normal((g.B, g.H, g.W, g.C))
    table = 0.3 * rng.standard_normal((2 * g.wh - 1, 2 * g.ww - 1, g.heads))
    p = _params(g.C, 4)
    x2, cache = ob.block_fwd(x, p, table, g)
    tx, tp, tt, tx1, tx2 = _torch_block(x, p, table, g)
    assert np.abs(x2 - tx2.detach().numpy()).max() < 1e-11
    assert np.abs(cache["x1"] - tx1.detach().numpy()).max() < 1e-11
    tx2.backward(torch.tensor(dx2))
    grads = ob.block_bwd(dx2, p, table, g, cache)
    assert np.abs(grads["x"] - tx.grad.numpy()).max() < 1e-10
    assert np.abs(grads["table"] - tt.grad.numpy()).max() < 1e-10
    for name in p:
        assert np.abs(grads[name] - tp[name].grad.numpy()).max() < 1e-10, name


def test_block_gradients_equal_central_differences():
    g = Geometry(1, 6, 7, 8, 2, 4, 3, 4, 1, 2, 3)
    rng = np.random.default_rng(9)
    x = rng.standard_normal((g.B, g.H, g.W, g.C))
    dx2 = rng.standard_normal((g.B, g.H, g.W, g.C))
    table = 0.3 * rng.standard_normal((2 * g.wh - 1, 2 * g.ww - 1, g.heads))
    p = _params(g.C, 5)
    _, cache = ob.block_fwd(x, p, table, g)
    grads = ob.block_bwd(dx2, p, table, g, cache)

    def loss():
        return float((ob.block_fwd(x, p, table, g)[0] * dx2).sum())

    h = 1e-6
    pick = np.random.default_rng(10)
    for name, arr in [("x", x), ("table", table)] + list(p.items()):
        flat = arr.reshape(-1)
        for i in pick.choice(flat.size, size=min(6, flat.size), replace=False):
            keep = flat[i]
            flat[i] = keep + h
            lp = loss()
            flat[i] = keep - h
            lm = loss()
            flat[i] = keep
            fd = (lp - lm) / (2 * h)
            assert abs(grads[name].reshape(-1)[i] - fd) < 1e-6 * max(1.0, abs(fd)), (name, i)
