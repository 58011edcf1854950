"""GPU check of the allocation-free fused backward (terra_winattn_bwd_nhwc_noalloc).

It runs the same kernels as terra_winattn_bwd_nhwc with the workspace taken
from the library's per-GPU scratch array, so its results must equal that
entry point's bit for bit.  Two calls in a row: a large generic-path
geometry (24 x 24 windows, head_dim 64: per-token D and bias partials in the
scratch), then a smaller window-path one (8 x 16 windows), which reuses the
array with the first call's contents still in it.  A geometry whose
workspace exceeds the array is refused before any device work.
"""

import sys

import numpy as np
import pytest

import terra_synth as ts

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2608_15211_amd")

pytestmark = pytest.mark.gpu


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


def _both(cfg, with_lo=False):
    inp = ts.make_inputs(cfg, seed=7)
    x = {n: torch.from_numpy(inp[n]).to("cuda").to(torch.bfloat16) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to("cuda")
    lo = torch.empty_like(x["q"]) if with_lo else None
    o, lse = P.terra_winattn_fwd_nhwc(x["q"], x["k"], x["v"], table, cfg, o_lo=lo)
    ref = P.terra_winattn_bwd_nhwc(x["q"], x["k"], x["v"], o, x["dout"], lse, table, cfg, o_lo=lo)
    out = (torch.full_like(x["q"], 7.0), torch.full_like(x["q"], 7.0), torch.full_like(x["q"], 7.0),
           torch.full_like(table, 7.0))
    got = P.terra_winattn_bwd_nhwc_noalloc(x["q"], x["k"], x["v"], o, x["dout"], lse, table, cfg, out, o_lo=lo)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv", "dtable"), got, ref):
        ai = a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32)
        bi = b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)
        assert torch.equal(ai, bi), "%s differs from terra_winattn_bwd_nhwc" % name


def test_noalloc_equals_workspace_backward_twice():
    big = ts.small_config("na_big", "bf16", 1, 96, 120, 8, 64, 24, 24, 12, 12)
    small = ts.small_config("na_small", "bf16", 1, 24, 80, 4, 32, 8, 16, 4, 8)
    assert P.terra_winattn_bwd_workspace_bytes(big, "bf16") > P.terra_winattn_bwd_workspace_bytes(small, "bf16")
    assert P.terra_winattn_bwd_workspace_bytes(big, "bf16") <= P.TERRA_SCRATCH_BYTES
    _say("noalloc: generic-path geometry")
    _both(big)
    _say("noalloc: generic-path geometry, D from the forward's O and O_lo")
    _both(big, with_lo=True)
    _say("noalloc: smaller window-path geometry")
    _both(small)


def test_noalloc_refuses_a_workspace_above_the_array():
    cfg = ts.small_config("na_huge", "bf16", 4, 256, 540, 24, 64, 24, 24, 12, 12)
    assert P.terra_winattn_bwd_workspace_bytes(cfg, "bf16") > P.TERRA_SCRATCH_BYTES
    t = torch.empty(1, dtype=torch.bfloat16, device="cuda")
    f = torch.empty(1, dtype=torch.float32, device="cuda")
    L = P.lib()
    import ctypes
    gg = P.terra_geom.make(**cfg.geom_kwargs())
    vp = lambda x: ctypes.c_void_p(x.data_ptr())  # noqa: E731
    st = L.terra_winattn_bwd_nhwc_noalloc(ctypes.byref(gg), P.TERRA_BF16, vp(t), vp(t), vp(t), vp(t), None,
                                          vp(t), vp(f), vp(f), vp(t), vp(t), vp(t), vp(f), None)
    assert st == 2
    assert b"scratch" in L.terra_last_error()
