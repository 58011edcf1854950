"""One Swin Transformer block around the shifted-window attention (oracle side).

Test infrastructure only (see the package docstring).

The paper's Transformer stage is a stack of Swin blocks (Sec. IV-A, citing
Swin) whose linear layers TP shards (Sec. IV-C); Table III gives d, N_h and
w.  The paper does not write the block out; the plain definition used here is
the Swin one (pre-norm, two residual branches), on a B x H x W x C token grid
with C = d:

    x1 = x  + Proj( A( LN1(x) W_qkv^T + b_qkv ) )
    x2 = x1 + ( GELU( LN2(x1) W_1^T + b_1 ) ) W_2^T + b_2

* LN(z) = (z - mean(z)) / sqrt(var(z) + eps) * gamma + beta over the C
  channels of one token, var the biased variance, eps = 1e-5;
* W_qkv is 3C x C: rows [0, C) give Q, [C, 2C) K, [2C, 3C) V, each with
  channel c = h * head_dim + e as the attention expects;
* A is the windowed attention of ``attention`` (route, softmax attention with
  the bias table and the shifted-window mask, inverse route);
* Proj(o) = o W_p^T + b_p with W_p C x C;
* W_1 is 4C x C, W_2 is C x 4C (MLP ratio 4); GELU(t) = t Phi(t) with Phi
  the standard normal distribution function (the exact, erf form).

The backward is the chain rule written out step by step, from the upstream
gradient dx2 to dx and every parameter's gradient (dW summed over all
tokens).  Everything is fp64; activations are kept in NHWC order.
"""

from math import sqrt

import numpy as np
from scipy.special import erf

from .attention import attn_fwd, attn_bwd
from .route import route, unroute

EPS = 1e-5


def _phi(t):
    """Standard normal distribution function, elementwise (scipy's erf)."""
    return 0.5 * (1.0 + erf(t / sqrt(2.0)))


def _pdf(t):
    return np.exp(-0.5 * t * t) / sqrt(2.0 * np.pi)


def gelu(t):
    return t * _phi(t)


def gelu_grad(t):
    """d/dt [t Phi(t)] = Phi(t) + t phi(t)."""
    return _phi(t) + t * _pdf(t)


def layernorm(z, gamma, beta):
    """Returns (LN(z), normalised zhat, 1/sqrt(var + eps)) over the last axis."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + EPS)
    zhat = (z - mu) * rstd
    return zhat * gamma + beta, zhat, rstd


def layernorm_bwd(dy, zhat, rstd, gamma):
    """Gradients of LN with respect to z, gamma and beta, from dy = dL/dLN(z)."""
    C = zhat.shape[-1]
    g = dy * gamma                                         # dL/dzhat
    dz = rstd * (g - g.sum(axis=-1, keepdims=True) / C
                 - zhat * (g * zhat).sum(axis=-1, keepdims=True) / C)
    dgamma = (dy * zhat).reshape(-1, C).sum(axis=0)
    dbeta = dy.reshape(-1, C).sum(axis=0)
    return dz, dgamma, dbeta


def _lin(z, W, b):
    return z @ np.asarray(W, np.float64).T + b


def block_fwd(x, p, table, g):
    """x: (B, H, W, C).  p: dict of parameters, names and shapes as in
    PARAM_SHAPES.  Returns (x2, cache) with every intermediate."""
    x = np.asarray(x, np.float64)
    C = g.C
    ln1, zhat1, rstd1 = layernorm(x, p["ln1_g"], p["ln1_b"])
    qkv = _lin(ln1, p["w_qkv"], p["b_qkv"])
    q, k, v = qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:]
    qw, kw, vw = (route(t, g) for t in (q, k, v))
    ow, lse = attn_fwd(qw, kw, vw, table, g)
    o = unroute(ow, g)
    x1 = x + _lin(o, p["w_proj"], p["b_proj"])
    ln2, zhat2, rstd2 = layernorm(x1, p["ln2_g"], p["ln2_b"])
    h = _lin(ln2, p["w_fc1"], p["b_fc1"])
    a = gelu(h)
    x2 = x1 + _lin(a, p["w_fc2"], p["b_fc2"])
    cache = dict(x=x, ln1=ln1, zhat1=zhat1, rstd1=rstd1, q=q, k=k, v=v, o=o, lse=lse, x1=x1,
                 ln2=ln2, zhat2=zhat2, rstd2=rstd2, h=h, a=a)
    return x2, cache


def _wgrad(dy, z):
    """dW = dy^T z summed over all tokens; dy (..., N), z (..., K) -> (N, K)."""
    return dy.reshape(-1, dy.shape[-1]).T @ z.reshape(-1, z.shape[-1])


def block_bwd(dx2, p, table, g, cache):
    """Gradients of the block for upstream dx2 (B, H, W, C): a dict with dx
    and d<name> for every parameter (and dtable for the bias table)."""
    c = cache
    C = g.C
    dx2 = np.asarray(dx2, np.float64)
    grads = {}
    # x2 = x1 + a W2^T + b2
    grads["w_fc2"] = _wgrad(dx2, c["a"])
    grads["b_fc2"] = dx2.reshape(-1, C).sum(axis=0)
    da = dx2 @ np.asarray(p["w_fc2"], np.float64)
    dh = da * gelu_grad(c["h"])
    grads["w_fc1"] = _wgrad(dh, c["ln2"])
    grads["b_fc1"] = dh.reshape(-1, dh.shape[-1]).sum(axis=0)
    dln2 = dh @ np.asarray(p["w_fc1"], np.float64)
    dx1_ln, grads["ln2_g"], grads["ln2_b"] = layernorm_bwd(dln2, c["zhat2"], c["rstd2"], p["ln2_g"])
    dx1 = dx2 + dx1_ln
    # x1 = x + o Wp^T + bp
    grads["w_proj"] = _wgrad(dx1, c["o"])
    grads["b_proj"] = dx1.reshape(-1, C).sum(axis=0)
    do = dx1 @ np.asarray(p["w_proj"], np.float64)
    qw, kw, vw, dow = (route(t, g) for t in (c["q"], c["k"], c["v"], do))
    dqw, dkw, dvw, dtab = attn_bwd(qw, kw, vw, dow, table, g)
    dqkv = np.concatenate([unroute(t, g) for t in (dqw, dkw, dvw)], axis=-1)
    grads["table"] = dtab
    grads["w_qkv"] = _wgrad(dqkv, c["ln1"])
    grads["b_qkv"] = dqkv.reshape(-1, 3 * C).sum(axis=0)
    dln1 = dqkv @ np.asarray(p["w_qkv"], np.float64)
    dx_ln, grads["ln1_g"], grads["ln1_b"] = layernorm_bwd(dln1, c["zhat1"], c["rstd1"], p["ln1_g"])
    grads["x"] = dx1 + dx_ln
    return grads


PARAM_SHAPES = {
    "ln1_g": lambda C: (C,), "ln1_b": lambda C: (C,),
    "w_qkv": lambda C: (3 * C, C), "b_qkv": lambda C: (3 * C,),
    "w_proj": lambda C: (C, C), "b_proj": lambda C: (C,),
    "ln2_g": lambda C: (C,), "ln2_b": lambda C: (C,),
    "w_fc1": lambda C: (4 * C, C), "b_fc1": lambda C: (4 * C,),
    "w_fc2": lambda C: (C, 4 * C), "b_fc2": lambda C: (C,),
}
