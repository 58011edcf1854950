"""Host-side checks of the C-ABI library (no GPU needed).

The library must load, export every function declared in include/*.h, and
reject bad arguments with the documented status codes before any device
work.  Window counts and layouts from the library are compared with closed
forms and with the oracle's enumeration.
"""

import ctypes
import glob
import os
import re

import pytest

import terra_synth as ts
from oracle import Geometry
from oracle.geometry import window_slots

P = pytest.importorskip("paper_2608_15211_amd")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _have_lib():
    return os.path.exists(P.LIB_PATH)


pytestmark = pytest.mark.skipif(not _have_lib(), reason="libterra_swin.so not built")


def _declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"\b(terra_[a-z0-9_]+)\s*\(", text):
            names.add(m.group(1))
    return sorted(names)


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert len(names) >= 11
    L = ctypes.CDLL(P.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_version():
    assert P.lib().terra_version() >= 100


@pytest.mark.parametrize("name", ts.ORDER)
def test_configs_validate(name):
    P.terra_validate_geometry(ts.CONFIGS[name])


BAD = [
    (dict(C=63), 1),                          # C != heads * head_dim
    (dict(wh=17), 1),                         # window taller than the grid
    (dict(ww=0), 1),
    (dict(sh=8), 1),                          # shift not below window
    (dict(sw=-1), 1),
    (dict(mask_flags=4), 1),
    (dict(B=0), 1),
    (dict(heads=1, head_dim=64, C=64, wh=16, ww=32), 0),
    (dict(heads=1, head_dim=128, C=128), 0),   # head_dim 128 (the paper's models)
    (dict(heads=4, head_dim=16, C=64), 2),    # head_dim outside {32, 64}
]


@pytest.mark.parametrize("change,status", BAD)
def test_bad_geometry_is_rejected(change, status):
    base = dict(B=1, H=16, W=32, C=64, heads=2, head_dim=32, wh=8, ww=8, sh=4, sw=4, mask_flags=1)
    base.update(change)
    g = P.terra_geom.make(**base)
    if status == 0:
        P.terra_validate_geometry(g)
        return
    with pytest.raises(P.TerraError) as e:
        P.terra_validate_geometry(g)
    assert e.value.status == status
    assert P.lib().terra_last_error().decode() != ""


def test_device_calls_reject_bad_arguments_before_launch():
    L = P.lib()
    g = P.terra_geom.make(1, 16, 32, 64, 2, 32, 8, 8, 4, 4, 1)
    fake = ctypes.c_void_p(0x1000)
    null = ctypes.c_void_p(0)
    s = ctypes.c_void_p(0)
    assert L.terra_window_route(ctypes.byref(g), 7, fake, fake, null, null, s) == 1   # bad dtype
    assert L.terra_winattn_fwd(ctypes.byref(g), 3, *([fake] * 7), s) == 1     # bad dtype
    assert L.terra_winattn_bwd_workspace_bytes(ctypes.byref(g), 2) > 0       # fp16
    assert L.terra_window_route(ctypes.byref(g), 1, null, fake, null, null, s) == 1   # NULL
    assert L.terra_window_route(ctypes.byref(g), 1, fake, fake, fake, fake, s) == 1   # in place
    assert L.terra_winattn_fwd(ctypes.byref(g), 1, fake, fake, null, fake, fake, fake, fake, s) == 1
    assert L.terra_winattn_fwd(None, 1, *([fake] * 7), s) == 1
    # o_lo is optional: a NULL there is not an error (the NULL q below is)
    assert L.terra_winattn_fwd(ctypes.byref(g), 1, null, fake, fake, fake, fake, null, fake, s) == 1
    need = L.terra_winattn_bwd_workspace_bytes(ctypes.byref(g), 1)
    assert need > 0
    args = [fake] * 12
    assert L.terra_winattn_bwd(ctypes.byref(g), 1, *args, fake, ctypes.c_size_t(need - 4), s) == 3
    assert L.terra_winattn_bwd(ctypes.byref(g), 1, *args, null, ctypes.c_size_t(need), s) == 3
    # the fused (NHWC) entry points share the checks
    assert L.terra_winattn_fwd_nhwc(ctypes.byref(g), 1, fake, fake, null, fake, fake, fake, fake, s) == 1
    assert L.terra_winattn_fwd_nhwc(ctypes.byref(g), 5, *([fake] * 7), s) == 1
    assert L.terra_winattn_bwd_nhwc(ctypes.byref(g), 1, *args, fake, ctypes.c_size_t(need - 4), s) == 3
    assert L.terra_winattn_bwd_nhwc(ctypes.byref(g), 1, null, *args[1:], fake, ctypes.c_size_t(need),
                                    s) == 1
    g2 = P.terra_geom.make(1, 16, 32, 48, 3, 16, 8, 8, 4, 4, 1)
    assert L.terra_winattn_fwd(ctypes.byref(g2), 1, *([fake] * 7), s) == 2
    assert L.terra_winattn_fwd_nhwc(ctypes.byref(g2), 1, *([fake] * 7), s) == 2
    assert L.terra_winattn_bwd_workspace_bytes(ctypes.byref(g2), 1) == 0
    for code in range(5):
        assert L.terra_status_string(code)


def test_o_lo_is_used_for_16_bit_windows_above_256_tokens():
    # 16-bit windows of more than 256 tokens keep O's rounding residual;
    # smaller windows keep the D sweep (and bf16 windows of at most 128
    # tokens take the window-resident kernels, which form D in registers);
    # float32 never keeps it
    L = P.lib()
    expect = {"c1_f32_16x32_w8": 0, "c2_bf16_128x256_w8": 0, "c3_bf16_85x180_w12": 0,
              "c4_bf16_128x1080_w8x16": 0, "c5_bf16_256x540_w24": 1,
              "p1_f16_256x540_hd128_w8": 0, "p2_f16_256x540_hd128_w32": 1}
    for name, want in expect.items():
        cfg = ts.ALL[name]
        code = {"f32": 0, "bf16": 1, "f16": 2}[cfg.dtype]
        assert L.terra_winattn_uses_o_lo(ctypes.byref(P._geom(cfg)), code) == want, name
        assert P.terra_winattn_uses_o_lo(cfg, code) == bool(want)
    g = P.terra_geom.make(1, 34, 32, 64, 2, 32, 17, 16, 8, 8, 1)     # 272-token windows
    assert L.terra_winattn_uses_o_lo(ctypes.byref(g), 1) == 1          # bfloat16
    assert L.terra_winattn_uses_o_lo(ctypes.byref(g), 2) == 1          # float16
    assert L.terra_winattn_uses_o_lo(ctypes.byref(g), 0) == 0          # float32
    g = P.terra_geom.make(1, 32, 32, 64, 2, 32, 16, 16, 8, 8, 1)     # 256-token windows
    assert L.terra_winattn_uses_o_lo(ctypes.byref(g), 2) == 0
    assert L.terra_winattn_uses_o_lo(ctypes.byref(g), 7) == -1         # bad dtype
    assert L.terra_winattn_uses_o_lo(None, 1) == -1


@pytest.mark.parametrize("name", ts.ORDER)
def test_window_layout_matches_oracle_enumeration(name):
    cfg = ts.CONFIGS[name]
    mh, mw = P.terra_window_count(cfg)
    assert mh == -(-cfg.H // cfg.wh) and mw == -(-cfg.W // cfg.ww)
    off, cnt = P.terra_window_layout(cfg)
    slots = window_slots(Geometry(**cfg.geom_kwargs()))
    assert [s for _, s, _ in slots] == off[:-1]
    assert [n for _, _, n in slots] == cnt
    assert off[-1] == cfg.H * cfg.W


def test_block_calls_reject_bad_arguments_before_launch():
    L = P.lib()
    fake = ctypes.c_void_p(0x1000)
    s = ctypes.c_void_p(0)
    ok = P.terra_geom.make(1, 24, 40, 768, 24, 32, 8, 16, 4, 8, 1)
    bad_c = P.terra_geom.make(1, 24, 40, 96, 3, 32, 8, 16, 4, 8, 1)        # C not a multiple of 128
    assert L.terra_block_bwd_workspace_bytes(ctypes.byref(bad_c), 1) == 0
    assert L.terra_block_bwd_workspace_bytes(ctypes.byref(ok), 0) == 0    # fp32: bf16 only
    assert L.terra_block_bwd_workspace_bytes(ctypes.byref(ok), 1) > 0
    z = ctypes.c_size_t(0)
    assert L.terra_block_fwd_workspace_bytes(ctypes.byref(ok), 1) > 0
    assert L.terra_block_fwd(ctypes.byref(bad_c), 1, fake, None, fake, fake, None, fake, z, s) == 2
    assert L.terra_block_fwd(ctypes.byref(ok), 2, fake, None, fake, fake, None, fake, z, s) == 2
    assert L.terra_block_fwd(ctypes.byref(ok), 1, fake, None, fake, fake, None, fake, z, s) == 1   # NULL structs
    p = P.terra_block_params()
    sv = P.terra_block_saved()
    assert L.terra_block_fwd(ctypes.byref(ok), 1, fake, ctypes.byref(p), fake, fake, ctypes.byref(sv), fake, z,
                             s) == 1
    gr = P.terra_block_grads()
    need = L.terra_block_bwd_workspace_bytes(ctypes.byref(ok), 1)
    for n in P.BLOCK_PARAM_NAMES:
        setattr(p, n, 0x1000)
        setattr(gr, n, 0x1000)
    for n in P.BLOCK_SAVED_NAMES:
        setattr(sv, n, 0x1000)
    assert L.terra_block_bwd(ctypes.byref(ok), 1, fake, fake, ctypes.byref(p), fake, ctypes.byref(sv), fake,
                             ctypes.byref(gr), fake, fake, ctypes.c_size_t(need - 1), s) == 3
    fneed = L.terra_block_fwd_workspace_bytes(ctypes.byref(ok), 1)
    assert L.terra_block_fwd(ctypes.byref(ok), 1, fake, ctypes.byref(p), fake, fake, ctypes.byref(sv), fake,
                             ctypes.c_size_t(fneed - 1), s) == 3
