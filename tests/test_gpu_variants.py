"""GPU parity of the paper-shaped variants: fp16 storage (the paper trains in
FP16 mixed precision), head_dim 128 (d / N_h of all three paper models) and
32 x 32 windows (the large model's window).

Small grids are compared with the fp64 oracle everywhere, through both the
window-major and the fused (NHWC in place) entry points.  The two full-size
variants (the small and large models' Transformer-stage grid 256 x 540) are
compared on sampled windows plus the whole bias-table gradient from stored
oracle values.  Tolerances: fp32 max abs 1e-5; fp16 and bf16 max abs 2e-2 and
relative L2 5e-3.
"""

import os
import sys

import numpy as np
import pytest

import terra_synth as ts
from oracle import Geometry, route as o_route, unroute as o_unroute
from oracle import attn_fwd, attn_bwd, attn_fwd_windows, attn_bwd_windows
from oracle.geometry import window_slots, token_table

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2608_15211_amd")

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TDT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

SMALL = [
    ts.small_config("v1_f16_hd32", "f16", 1, 16, 32, 2, 32, 8, 8, 4, 4),
    ts.small_config("v2_bf16_hd128", "bf16", 1, 24, 40, 2, 128, 8, 8, 4, 4),
    ts.small_config("v3_f32_hd128", "f32", 1, 16, 24, 1, 128, 8, 8, 4, 4),
    ts.small_config("v4_f16_hd128_w32", "f16", 1, 40, 70, 2, 128, 32, 32, 16, 16),
    ts.small_config("v5_f16_hd64_masks", "f16", 2, 36, 44, 2, 64, 12, 20, 6, 10, 3),
]
LARGE = ["p1_f16_256x540_hd128_w8", "p2_f16_256x540_hd128_w32"]


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


def _dev(x, cfg):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(TDT[cfg.dtype])


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
    tab = token_table(g)
    out = np.empty_like(lse_win)
    out[:, :, tab["u"] * g.W + tab["v"]] = lse_win
    return out


@pytest.mark.parametrize("cfg", SMALL, ids=[c.name for c in SMALL])
def test_variant_against_oracle(cfg):
    g = Geometry(**cfg.geom_kwargs())
    _say("variant %s" % cfg.name)
    inp = ts.make_inputs(cfg, seed=6)
    x = {n: _dev(inp[n], cfg) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to("cuda")
    q, k, v, do = (o_route(inp[n], g) for n in ("q", "k", "v", "dout"))
    o, lse = attn_fwd(q, k, v, inp["table"], g)
    dq, dk, dv, dt = attn_bwd(q, k, v, do, inp["table"], g)
    # window-major entry points
    w = {n: P.terra_window_route(x[n], cfg) for n in x}
    go, glse = P.terra_winattn_fwd(w["q"], w["k"], w["v"], table, cfg)
    gq, gk, gv, gt = P.terra_winattn_bwd(w["q"], w["k"], w["v"], go, w["dout"], glse, table, cfg)
    torch.cuda.synchronize()
    for nm, a, b in (("O", go, o), ("LSE", glse, lse), ("dQ", gq, dq), ("dK", gk, dk), ("dV", gv, dv),
                     ("dT", gt, dt)):
        _assert_close(nm, _host(a), b, cfg)
    # fused entry points, keeping O's rounding residual where the shape uses it
    lo = torch.empty_like(x["q"]) if P.terra_winattn_uses_o_lo(cfg, cfg.dtype) else None
    fo, flse = P.terra_winattn_fwd_nhwc(x["q"], x["k"], x["v"], table, cfg, o_lo=lo)
    fq, fk, fv, ft = P.terra_winattn_bwd_nhwc(x["q"], x["k"], x["v"], fo, x["dout"], flse, table, cfg,
                                              o_lo=lo)
    torch.cuda.synchronize()
    for nm, a, b in (("fused O", fo, o_unroute(o, g)), ("fused LSE", flse, _lse_to_nhwc(lse, g)),
                     ("fused dQ", fq, o_unroute(dq, g)), ("fused dK", fk, o_unroute(dk, g)),
                     ("fused dV", fv, o_unroute(dv, g)), ("fused dT", ft, dt)):
        _assert_close(nm, _host(a), b, cfg)


def _sample_windows(g, seed=0):
    mh, mw = -(-g.H // g.wh), -(-g.W // g.ww)
    last = mh * mw - 1
    pick = {0, mw - 1, (mh - 1) * mw, last, mw + mw - 1}
    rng = np.random.default_rng(seed)
    pick.update(int(x) for x in rng.integers(0, last + 1, 3))
    return sorted(pick)


@pytest.mark.parametrize("name", LARGE)
def test_variant_full_size_sampled(name):
    cfg = ts.VARIANTS[name]
    g = Geometry(**cfg.geom_kwargs())
    _say("full-size variant %s" % name)
    inp = ts.make_inputs(cfg)
    x = {n: _dev(inp[n], cfg) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to("cuda")
    # the timed path: O's rounding residual kept where the shape uses it
    lo = torch.empty_like(x["q"]) if P.terra_winattn_uses_o_lo(cfg, cfg.dtype) else None
    fo, flse = P.terra_winattn_fwd_nhwc(x["q"], x["k"], x["v"], table, cfg, o_lo=lo)
    fq, fk, fv, ft = P.terra_winattn_bwd_nhwc(x["q"], x["k"], x["v"], fo, x["dout"], flse, table, cfg,
                                              o_lo=lo)
    # window-major views of the fused results (the route is a bit copy)
    got = {n: P.terra_window_route(t, cfg) for n, t in (("o", fo), ("dq", fq), ("dk", fk), ("dv", fv))}
    torch.cuda.synchronize()
    sel = _sample_windows(g)
    q, k, v, do = (o_route(inp[n], g) for n in ("q", "k", "v", "dout"))
    fw = attn_fwd_windows(q, k, v, inp["table"], g, sel)
    bw = attn_bwd_windows(q, k, v, do, inp["table"], g, sel)
    tab = token_table(g)
    src = tab["u"] * g.W + tab["v"]
    lse_h = _host(flse)
    slots = {w: (s, n) for w, s, n in window_slots(g)}
    for w in sel:
        s, n = slots[w]
        _assert_close("O[w%d]" % w, _host(got["o"][:, s:s + n]), fw[w][0], cfg)
        _assert_close("LSE[w%d]" % w, lse_h[:, :, src[s:s + n]], fw[w][1], cfg)
        _assert_close("dQ[w%d]" % w, _host(got["dq"][:, s:s + n]), bw[w][0], cfg)
        _assert_close("dK[w%d]" % w, _host(got["dk"][:, s:s + n]), bw[w][1], cfg)
        _assert_close("dV[w%d]" % w, _host(got["dv"][:, s:s + n]), bw[w][2], cfg)
    gold = np.load(os.path.join(GOLDEN, "dtable_%s.npy" % name))
    _assert_close("dT", _host(ft), gold, cfg)
    assert np.abs(_host(ft).sum(axis=(0, 1))).max() < 1e-2
