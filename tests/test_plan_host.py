"""Host-side checks of the native window-assignment planner (no GPU needed).

terra_plan_padded_grid (Eq. (3)), terra_plan_window_ranges (Eq. (4)) and
terra_plan_rank (window range, slots, stripe and received fragments of one
rank) are compared with the paper's printed figures and with the oracle
planner, which lists every token a rank needs one by one: the fragments of
each source rank must cover exactly the tokens the oracle assigns to that
source, with no overlap, laid out back to back in source-rank order.
"""

import os

import pytest

import terra_synth as ts
from oracle import Geometry
from oracle import planner as opl

P = pytest.importorskip("paper_2608_15211_amd")
pytestmark = pytest.mark.skipif(not os.path.exists(P.LIB_PATH), reason="libterra_swin.so not built")


def test_eq3_paper_figures():
    hh, ww, ov = P.terra_plan_padded_grid(2041, 4320, 4, 2, 128, 4, 4)
    assert (hh, ww) == (4096, 8192) and round(100 * ov, 1) == 280.6
    hh, ww, ov = P.terra_plan_padded_grid(2041, 4320, 4, 2, 128)
    assert (hh, ww) == (2048, 5120) and round(100 * ov, 1) == 18.9
    for args in [(2041, 4320, 4, 2, 8, 2, 4), (100, 37, 2, 1, 3, 5, 1), (7, 7, 1, 1, 7, 1, 1)]:
        hh, ww, ov = P.terra_plan_padded_grid(*args)
        assert (hh, ww) == opl.padded_grid(*args)
        assert ov == pytest.approx(opl.padding_overhead(args[0], args[1], hh, ww), abs=1e-12)


def test_eq4_paper_figures():
    b = P.terra_plan_window_ranges(10, 4)
    assert [y - x for x, y in zip(b, b[1:])] == [2, 3, 2, 3]
    b = P.terra_plan_window_ranges(45, 4)
    assert [y - x for x, y in zip(b, b[1:])] == [11, 11, 11, 12]
    for M, R in [(1, 1), (1, 4), (1088, 8), (253, 16), (7, 9), (10 ** 9, 96)]:
        b = P.terra_plan_window_ranges(M, R)
        assert b == [x for x, _ in opl.window_ranges(M, R)] + [M]


def _geoms():
    out = [ts.CONFIGS["c4_bf16_128x1080_w8x16"], ts.CONFIGS["c5_bf16_256x540_w24"],
           ts.CONFIGS["c3_bf16_85x180_w12"]]
    out += [ts.small_config("g1", "bf16", 2, 21, 52, 1, 32, 8, 16, 4, 8, 3),
            ts.small_config("g2", "bf16", 1, 17, 23, 1, 32, 5, 6, 2, 3, 1),
            ts.small_config("g3", "f32", 1, 24, 30, 1, 32, 6, 5, 0, 0, 1),
            ts.small_config("g4", "bf16", 1, 40, 64, 1, 32, 8, 8, 7, 7, 0)]
    return out


@pytest.mark.parametrize("cfg", _geoms(), ids=lambda c: c.name)
@pytest.mark.parametrize("ranks", [1, 2, 3, 4, 8, 16])
def test_rank_plan_matches_the_oracle(cfg, ranks):
    g = Geometry(**cfg.geom_kwargs())
    Mh, Mw = -(-g.H // g.wh), -(-g.W // g.ww)
    big = g.H * g.W > 60000
    for r in range(ranks):
        if big and r not in (0, 1, ranks - 1):
            continue
        plan, frags = P.terra_plan_rank(cfg, ranks, r)
        L, R = opl.window_ranges(Mh * Mw, ranks)[r]
        assert (plan["win_begin"], plan["win_end"]) == (L, R)
        assert (plan["slot_begin"], plan["slot_end"]) == opl.rank_slots(g, ranks, r)
        assert (plan["row_begin"], plan["row_end"]) == opl.stripes(g.H, ranks)[r]
        assert plan["nfrag"] == len(frags)
        need = opl.needed_tokens(g, ranks, r)
        got = {}
        off = 0
        last_src = -1
        for f in frags:
            assert f["src_rank"] != r and f["src_rank"] >= last_src
            last_src = f["src_rank"]
            assert f["offset"] == off
            a, b = opl.stripes(g.H, ranks)[f["src_rank"]]
            assert a <= f["u0"] < f["u1"] <= b and 0 <= f["v0"] < f["v1"] <= g.W
            pts = got.setdefault(f["src_rank"], set())
            for u in range(f["u0"], f["u1"]):
                for v in range(f["v0"], f["v1"]):
                    assert (u, v) not in pts
                    pts.add((u, v))
            off += (f["u1"] - f["u0"]) * (f["v1"] - f["v0"])
        assert plan["frag_tokens"] == off
        assert got == {s: pts for s, pts in need.items() if s != r}


def test_plan_errors():
    cfg = ts.CONFIGS["c2_bf16_128x256_w8"]
    for ranks, rank in [(0, 0), (4, 4), (4, -1)]:
        with pytest.raises(P.TerraError) as e:
            P.terra_plan_rank(cfg, ranks, rank)
        assert e.value.status == 1
    with pytest.raises(P.TerraError):
        P.terra_plan_window_ranges(10, 0)
    with pytest.raises(P.TerraError):
        P.terra_plan_padded_grid(0, 10, 1, 1, 1, 1, 1)
    # one-row stripes under 64-row windows: a rank's window gathers from 64
    # stripes, each sending two column runs - more fragments than the cap
    thin = ts.small_config("thin", "bf16", 1, 256, 540, 1, 32, 64, 4, 12, 2)
    with pytest.raises(P.TerraError) as e:
        P.terra_plan_rank(thin, 256, 63)
    assert e.value.status == 2
