"""GPU parity of the per-rank token route (ragged window assignment).

The grid is cut into DMP height stripes; every rank, run one after another
on the one GPU, packs the fragments it receives out of the other ranks'
stripes (terra_fragment_pack, standing in for the point-to-point exchange)
and routes its window range (terra_window_route_rank).  Each rank's
window-major tensor must equal, bit for bit, its slots of the oracle's route
of the whole grid (unique bit patterns per element, so any misplaced element
shows).  Then every rank scatters its tensor back (terra_window_unroute_rank)
and returns the fragments (terra_fragment_unpack) into stripes that started
as a filler: the stripes must come back exactly, which also shows that the
ranks' windows cover every token once.
"""

import sys

import numpy as np
import pytest

import terra_synth as ts
from oracle import Geometry, route as o_route
from oracle import planner as opl

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2608_15211_amd")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P.lib()
    yield
    torch.cuda.synchronize()


CASES = [
    ("c4_4way", ts.CONFIGS["c4_bf16_128x1080_w8x16"], 4),
    ("c4_8way", ts.CONFIGS["c4_bf16_128x1080_w8x16"], 8),
    ("c4_7way", ts.CONFIGS["c4_bf16_128x1080_w8x16"], 7),        # ranges split window rows
    ("c5_4way", ts.CONFIGS["c5_bf16_256x540_w24"], 4),
    ("c5_8way", ts.CONFIGS["c5_bf16_256x540_w24"], 8),
    ("ragged_both_masks_5way", ts.small_config("r1", "bf16", 2, 21, 52, 3, 32, 8, 16, 4, 8, 3), 5),
    ("f32_noshift_4way", ts.small_config("r2", "f32", 1, 24, 30, 2, 32, 6, 5, 0, 0, 1), 4),
    ("small_windows_16way", ts.small_config("r3", "bf16", 1, 40, 64, 1, 32, 8, 8, 7, 7, 0), 16),
    ("more_ranks_than_windows", ts.small_config("r4", "bf16", 1, 16, 16, 1, 32, 8, 8, 4, 4, 1), 6),
]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("label,cfg,ranks", CASES, ids=[c[0] for c in CASES])
def test_rank_route_bit_exact_and_inverse(label, cfg, ranks):
    g = Geometry(**cfg.geom_kwargs())
    _say("rank route %s" % label)
    width = 4 if cfg.dtype == "f32" else 2
    idt = torch.int32 if width == 4 else torch.int16
    tdt = torch.float32 if width == 4 else torch.bfloat16
    pat = ts.token_pattern(cfg, width)
    npdt = np.int32 if width == 4 else np.int16
    x = torch.from_numpy(pat.view(npdt)).to("cuda")
    expect = o_route(pat, g)                                 # (B, HW, C) whole grid
    st = opl.stripes(g.H, ranks)
    stripes = [x[:, a:b].contiguous().view(tdt) for a, b in st]
    back = [torch.full_like(s.view(idt), -1).view(tdt) for s in stripes]
    for r in range(ranks):
        plan, frags = P.terra_plan_rank(cfg, ranks, r)
        fbuf = None
        if plan["frag_tokens"] > 0:
            fbuf = torch.empty((cfg.B, plan["frag_tokens"], cfg.C), dtype=tdt, device="cuda")
            for src in sorted({f["src_rank"] for f in frags}):
                P.terra_fragment_pack(stripes[src], fbuf, cfg, ranks, r, src)
        y = P.terra_window_route_rank(stripes[r], fbuf, cfg, ranks, r)
        torch.cuda.synchronize()
        s0, s1 = plan["slot_begin"], plan["slot_end"]
        got = y.view(idt).cpu().numpy().view(pat.dtype)
        assert np.array_equal(got, expect[:, s0:s1]), "rank %d" % r
        # inverse: back into a filled stripe and a fresh fragment buffer,
        # whose fragments then return to their source stripes
        fback = None if fbuf is None else torch.full_like(fbuf.view(idt), -1).view(tdt)
        P.terra_window_unroute_rank(y, cfg, ranks, r, back[r], fback)
        for src in sorted({f["src_rank"] for f in frags}):
            P.terra_fragment_unpack(fback, back[src], cfg, ranks, r, src)
    torch.cuda.synchronize()
    for r in range(ranks):
        assert torch.equal(back[r].view(idt), stripes[r].view(idt)), "stripe %d" % r
