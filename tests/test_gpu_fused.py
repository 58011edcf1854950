"""GPU parity of the fused route + attention entry points (NHWC in place).

terra_winattn_fwd_nhwc / terra_winattn_bwd_nhwc read Q, K, V, dO straight
from the NHWC grid and write O, dQ, dK, dV back to it.  They are checked
(1) against the fp64 oracle composed as unroute(attention(route(x))) on the
small configurations and edge cases, with the tolerances of the window-major
tests, and (2) bit for bit against the window-major entry points followed by
the inverse route, on every configuration (the arithmetic is the same, only
the addressing differs).
"""

import sys

import numpy as np
import pytest

import terra_synth as ts
from oracle import Geometry, route as o_route, unroute as o_unroute
from oracle import attn_fwd, attn_bwd
from oracle.geometry import token_table

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2608_15211_amd")

pytestmark = pytest.mark.gpu

SMALL = ["c1_f32_16x32_w8", "c2_bf16_128x256_w8", "c3_bf16_85x180_w12"]
EDGE = [
    ts.small_config("f1", "bf16", 2, 9, 17, 3, 32, 4, 4, 2, 3, 3),
    ts.small_config("f2", "bf16", 1, 21, 52, 3, 32, 8, 16, 4, 8, 1),
    ts.small_config("f3", "bf16", 2, 16, 40, 2, 32, 8, 8, 4, 4, 3),
    ts.small_config("f4", "bf16", 1, 30, 20, 2, 64, 15, 12, 7, 5, 1),
    ts.small_config("f5", "f32", 1, 8, 24, 1, 32, 8, 8, 0, 5, 1),
    # unshifted 8x16 / 16x8 windows on ragged heights (short last window row
    # without wrap labels), no mask at all, and both wraps masked
    ts.small_config("f6", "bf16", 1, 20, 32, 2, 32, 8, 16, 0, 0, 1),
    ts.small_config("f7", "bf16", 1, 36, 24, 2, 32, 16, 8, 0, 0, 1),
    ts.small_config("f8", "bf16", 1, 20, 40, 2, 32, 8, 16, 4, 8, 0),
    ts.small_config("f9", "bf16", 1, 24, 48, 2, 32, 8, 16, 4, 8, 3),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.lib()
    yield
    torch.cuda.synchronize()


def _tdtype(cfg):
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def _dev(x, cfg):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(_tdtype(cfg))


def _host(t):
    return t.float().cpu().numpy().astype(np.float64)


def _assert_close(name, got, ref, cfg):
    err = np.abs(got - ref).max()
    if cfg.dtype == "f32":
        assert err <= 1e-5, "%s max abs err %.3g > 1e-5" % (name, err)
    else:
        assert err <= 2e-2, "%s max abs err %.3g > 2e-2" % (name, err)
        nrm = np.linalg.norm(ref)
        if nrm > 1e-6:
            rel = np.linalg.norm(got - ref) / nrm
            assert rel <= 5e-3, "%s rel L2 err %.3g > 5e-3" % (name, rel)


def _lse_to_nhwc(lse_win, g):
    """(B, heads, H*W) window-major token order -> NHWC token order (oracle side)."""
    tab = token_table(g)
    src = tab["u"] * g.W + tab["v"]
    out = np.empty_like(lse_win)
    out[:, :, src] = lse_win
    return out


def _fused(cfg, x, table):
    o, lse = P.terra_winattn_fwd_nhwc(x["q"], x["k"], x["v"], table, cfg)
    dq, dk, dv, dt = P.terra_winattn_bwd_nhwc(x["q"], x["k"], x["v"], o, x["dout"], lse, table, cfg)
    torch.cuda.synchronize()
    return dict(o=o, lse=lse, dq=dq, dk=dk, dv=dv, dt=dt)


@pytest.mark.parametrize("cfg", [ts.CONFIGS[n] for n in SMALL] + EDGE,
                         ids=SMALL + [c.name for c in EDGE])
def test_fused_against_oracle(cfg):
    g = Geometry(**cfg.geom_kwargs())
    _say("fused vs oracle %s" % cfg.name)
    inp = ts.make_inputs(cfg, seed=2)
    x = {n: _dev(inp[n], cfg) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to("cuda")
    got = _fused(cfg, x, table)
    q, k, v, do = (o_route(inp[n], g) for n in ("q", "k", "v", "dout"))
    o, lse = attn_fwd(q, k, v, inp["table"], g)
    dq, dk, dv, dt = attn_bwd(q, k, v, do, inp["table"], g)
    _assert_close("O", _host(got["o"]), o_unroute(o, g), cfg)
    _assert_close("LSE", _host(got["lse"]), _lse_to_nhwc(lse, g), cfg)
    _assert_close("dQ", _host(got["dq"]), o_unroute(dq, g), cfg)
    _assert_close("dK", _host(got["dk"]), o_unroute(dk, g), cfg)
    _assert_close("dV", _host(got["dv"]), o_unroute(dv, g), cfg)
    _assert_close("dT", _host(got["dt"]), dt, cfg)


def _bits(t):
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


@pytest.mark.parametrize("name", ts.ORDER)
def test_fused_equals_route_then_attention_bit_for_bit(name):
    cfg = ts.CONFIGS[name]
    g = Geometry(**cfg.geom_kwargs())
    _say("fused vs window-major %s" % name)
    inp = ts.make_inputs(cfg, seed=4)
    x = {n: _dev(inp[n], cfg) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to("cuda")
    del inp
    got = _fused(cfg, x, table)
    w = {n: P.terra_window_route(x[n], cfg) for n in x}
    o, lse = P.terra_winattn_fwd(w["q"], w["k"], w["v"], table, cfg)
    dq, dk, dv, dt = P.terra_winattn_bwd(w["q"], w["k"], w["v"], o, w["dout"], lse, table, cfg)
    ref = {"o": P.terra_window_unroute(o, cfg), "dq": P.terra_window_unroute(dq, cfg),
           "dk": P.terra_window_unroute(dk, cfg), "dv": P.terra_window_unroute(dv, cfg)}
    torch.cuda.synchronize()
    for n in ("o", "dq", "dk", "dv"):
        assert np.array_equal(_bits(got[n]), _bits(ref[n])), n
    tab = token_table(g)
    src = torch.from_numpy((tab["u"] * g.W + tab["v"]).astype(np.int64)).to("cuda")
    lse_nhwc = torch.empty_like(lse)
    lse_nhwc[:, :, src] = lse
    assert np.array_equal(_bits(got["lse"]), _bits(lse_nhwc)), "lse"
    assert np.array_equal(_bits(got["dt"]), _bits(dt)), "dt"
