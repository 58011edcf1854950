"""Python binding of libterra_swin.so, the gfx950 shifted-window attention
library (C ABI in include/terra_swin.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
the library.  Tensors are torch tensors used as device memory; the current
torch stream is passed as the HIP stream.  If the library has not been built
the functions raise; there is no fallback.

Entry points (same names as the C ABI):
    terra_validate_geometry, terra_window_count, terra_window_layout,
    terra_window_route, terra_window_unroute, terra_winattn_fwd,
    terra_winattn_bwd_workspace_bytes, terra_winattn_bwd,
    terra_winattn_fwd_nhwc, terra_winattn_bwd_nhwc (route fused in),
    terra_winattn_uses_o_lo (whether the forward's rounding residual of O
    serves the backward),
    terra_winattn_bwd_nhwc_noalloc (workspace from a library-held array),
    terra_plan_padded_grid, terra_plan_window_ranges, terra_plan_rank,
    terra_window_route_rank, terra_window_unroute_rank, terra_fragment_pack,
    terra_fragment_unpack (ragged window assignment and per-rank route),
    terra_block_fwd_workspace_bytes, terra_block_fwd,
    terra_block_bwd_workspace_bytes, terra_block_bwd (the
    Swin block around the attention: LayerNorm, projections, MLP)
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libterra_swin.so")

TERRA_F32 = 0
TERRA_BF16 = 1
TERRA_F16 = 2
TERRA_MASK_LAT = 1
TERRA_MASK_LON = 2
STATUS = {0: "TERRA_OK", 1: "TERRA_ERR_INVALID", 2: "TERRA_ERR_UNSUPPORTED",
          3: "TERRA_ERR_WORKSPACE", 4: "TERRA_ERR_HIP"}


class TerraError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s: %s" % (STATUS.get(status, status), message))
        self.status = status


class terra_geom(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "H", "W", "C", "heads", "head_dim", "wh", "ww", "sh", "sw", "mask_flags")]

    @classmethod
    def make(cls, B, H, W, C, heads, head_dim, wh, ww, sh, sw, mask_flags=TERRA_MASK_LAT):
        return cls(B, H, W, C, heads, head_dim, wh, ww, sh, sw, mask_flags)

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class terra_rank_plan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("win_begin", "win_end", "slot_begin", "slot_end", "row_begin", "row_end",
                 "nfrag", "frag_tokens")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class terra_fragment(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("src_rank", "u0", "u1", "v0", "v1", "offset")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


TERRA_MAX_FRAGMENTS = 64

BLOCK_PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_proj", "b_proj", "ln2_g", "ln2_b",
                     "w_fc1", "b_fc1", "w_fc2", "b_fc2")
BLOCK_SAVED_NAMES = ("mu1", "rstd1", "mu2", "rstd2", "q", "k", "v", "o", "lse", "x1", "h", "a")


class terra_block_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_PARAM_NAMES]


class terra_block_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_PARAM_NAMES]


class terra_block_saved(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_SAVED_NAMES]

_lib = None


def lib():
    """The loaded shared library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libterra_swin.so is not built (%s); run __graft_entry__.build() "
                           "or python paper_2608_15211_amd/build.py" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    G = ctypes.POINTER(terra_geom)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    L.terra_version.restype = i32
    L.terra_validate_geometry.argtypes = [G]
    L.terra_window_count.argtypes = [G, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]
    L.terra_window_layout.argtypes = [G, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]
    L.terra_window_route.argtypes = [G, i32, vp, vp, vp, vp, vp]
    L.terra_window_unroute.argtypes = [G, i32, vp, vp, vp]
    L.terra_winattn_fwd.argtypes = [G, i32] + [vp] * 8
    L.terra_winattn_fwd_nhwc.argtypes = [G, i32] + [vp] * 8
    L.terra_winattn_uses_o_lo.argtypes = [G, i32]
    L.terra_winattn_uses_o_lo.restype = i32
    L.terra_winattn_bwd_workspace_bytes.argtypes = [G, i32]
    L.terra_winattn_bwd_workspace_bytes.restype = sz
    L.terra_winattn_bwd.argtypes = [G, i32] + [vp] * 13 + [sz, vp]
    L.terra_winattn_bwd_nhwc.argtypes = [G, i32] + [vp] * 13 + [sz, vp]
    L.terra_winattn_bwd_nhwc_noalloc.argtypes = [G, i32] + [vp] * 13
    i64 = ctypes.c_int64
    L.terra_plan_padded_grid.argtypes = [i32] * 7 + [ctypes.POINTER(ctypes.c_int32)] * 2 + \
        [ctypes.POINTER(ctypes.c_double)]
    L.terra_plan_window_ranges.argtypes = [i64, i32, ctypes.POINTER(ctypes.c_int64)]
    L.terra_plan_rank.argtypes = [G, i32, i32, ctypes.POINTER(terra_rank_plan),
                                  ctypes.POINTER(terra_fragment)]
    L.terra_window_route_rank.argtypes = [G, i32, i32, i32, vp, vp, vp, vp]
    L.terra_window_unroute_rank.argtypes = [G, i32, i32, i32, vp, vp, vp, vp]
    L.terra_fragment_pack.argtypes = [G, i32, i32, i32, i32, vp, vp, vp]
    L.terra_fragment_unpack.argtypes = [G, i32, i32, i32, i32, vp, vp, vp]
    L.terra_block_fwd.argtypes = [G, i32, vp, ctypes.POINTER(terra_block_params), vp, vp,
                                  ctypes.POINTER(terra_block_saved), vp, sz, vp]
    L.terra_block_fwd_workspace_bytes.argtypes = [G, i32]
    L.terra_block_fwd_workspace_bytes.restype = sz
    L.terra_block_bwd_workspace_bytes.argtypes = [G, i32]
    L.terra_block_bwd_workspace_bytes.restype = sz
    L.terra_block_bwd.argtypes = [G, i32, vp, vp, ctypes.POINTER(terra_block_params), vp,
                                  ctypes.POINTER(terra_block_saved), vp, ctypes.POINTER(terra_block_grads),
                                  vp, vp, sz, vp]
    L.terra_status_string.argtypes = [i32]
    L.terra_status_string.restype = ctypes.c_char_p
    L.terra_last_error.restype = ctypes.c_char_p
    for name in ("terra_validate_geometry", "terra_window_count", "terra_window_layout",
                 "terra_window_route", "terra_window_unroute", "terra_winattn_fwd",
                 "terra_winattn_bwd", "terra_winattn_fwd_nhwc", "terra_winattn_bwd_nhwc",
                 "terra_winattn_bwd_nhwc_noalloc", "terra_winattn_uses_o_lo",
                 "terra_plan_padded_grid", "terra_plan_window_ranges", "terra_plan_rank",
                 "terra_window_route_rank", "terra_window_unroute_rank", "terra_fragment_pack",
                 "terra_fragment_unpack", "terra_block_fwd", "terra_block_bwd"):
        getattr(L, name).restype = i32
    _lib = L
    return L


def _check(status):
    if status != 0:
        raise TerraError(status, lib().terra_last_error().decode())


def _geom(g):
    if isinstance(g, terra_geom):
        return g
    if isinstance(g, dict):
        return terra_geom.make(**g)
    return terra_geom.make(**g.geom_kwargs())


# ---------------------------------------------------------------- host-only
def terra_validate_geometry(g):
    """Raises TerraError if the geometry is invalid or unsupported."""
    _check(lib().terra_validate_geometry(ctypes.byref(_geom(g))))


def terra_window_count(g):
    mh, mw = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().terra_window_count(ctypes.byref(_geom(g)), ctypes.byref(mh), ctypes.byref(mw)))
    return mh.value, mw.value


def terra_window_layout(g):
    """(offsets[Mh*Mw+1], counts[Mh*Mw]) of one image, as Python lists."""
    mh, mw = terra_window_count(g)
    off = (ctypes.c_int32 * (mh * mw + 1))()
    cnt = (ctypes.c_int32 * (mh * mw))()
    _check(lib().terra_window_layout(ctypes.byref(_geom(g)), off, cnt))
    return list(off), list(cnt)


def terra_winattn_bwd_workspace_bytes(g, dtype):
    return int(lib().terra_winattn_bwd_workspace_bytes(ctypes.byref(_geom(g)), _dtype_code(dtype)))


# ---------------------------------------------------------------- device calls
def _dtype_code(dtype):
    if isinstance(dtype, int):
        return dtype
    import torch
    if dtype in (torch.float32, "f32"):
        return TERRA_F32
    if dtype in (torch.bfloat16, "bf16"):
        return TERRA_BF16
    if dtype in (torch.float16, "f16"):
        return TERRA_F16
    raise TypeError("unsupported dtype %r" % (dtype,))


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, name, dtype=None, numel=None):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (name, t.numel(), numel))
    return ctypes.c_void_p(t.data_ptr())


def _sizes(gg):
    return gg.B * gg.H * gg.W * gg.C, gg.B * gg.heads * gg.H * gg.W, \
        (2 * gg.wh - 1) * (2 * gg.ww - 1) * gg.heads


def terra_window_route(x_nhwc, g, out=None, offsets=None, counts=None):
    """NHWC (B,H,W,C) -> window-major (B,H*W,C), same dtype.  offsets /
    counts: optional int32 device tensors of Mh*Mw+1 / Mh*Mw entries that
    receive the window layout of one image."""
    import torch
    gg = _geom(g)
    n, _, _ = _sizes(gg)
    if out is None:
        out = torch.empty((gg.B, gg.H * gg.W, gg.C), dtype=x_nhwc.dtype, device=x_nhwc.device)
    nw = (-(-gg.H // gg.wh)) * (-(-gg.W // gg.ww))
    d_off = ctypes.c_void_p(0) if offsets is None else _dev(offsets, "offsets", torch.int32, nw + 1)
    d_cnt = ctypes.c_void_p(0) if counts is None else _dev(counts, "counts", torch.int32, nw)
    _check(lib().terra_window_route(ctypes.byref(gg), _dtype_code(x_nhwc.dtype),
                                    _dev(x_nhwc, "x", None, n), _dev(out, "out", x_nhwc.dtype, n),
                                    d_off, d_cnt, _stream()))
    return out


def terra_window_unroute(y_win, g, out=None):
    """window-major (B,H*W,C) -> NHWC (B,H,W,C), same dtype."""
    import torch
    gg = _geom(g)
    n, _, _ = _sizes(gg)
    if out is None:
        out = torch.empty((gg.B, gg.H, gg.W, gg.C), dtype=y_win.dtype, device=y_win.device)
    _check(lib().terra_window_unroute(ctypes.byref(gg), _dtype_code(y_win.dtype),
                                      _dev(y_win, "y", None, n), _dev(out, "out", y_win.dtype, n),
                                      _stream()))
    return out


def _opt(t, name, dtype=None, numel=None):
    """Nullable device pointer: NULL for None, else as _dev."""
    return ctypes.c_void_p(None) if t is None else _dev(t, name, dtype, numel)


def _attn_fwd(fn, shape, q, k, v, table, g, out, lse, o_lo):
    import torch
    gg = _geom(g)
    n, nl, nt = _sizes(gg)
    dt = q.dtype
    if out is None:
        out = torch.empty(shape(gg), dtype=dt, device=q.device)
    if lse is None:
        lse = torch.empty((gg.B, gg.heads, gg.H * gg.W), dtype=torch.float32, device=q.device)
    _check(fn(ctypes.byref(gg), _dtype_code(dt), _dev(q, "q", dt, n), _dev(k, "k", dt, n),
              _dev(v, "v", dt, n), _dev(table, "table", torch.float32, nt), _dev(out, "o", dt, n),
              _opt(o_lo, "o_lo", dt, n), _dev(lse, "lse", torch.float32, nl), _stream()))
    return out, lse


def _attn_bwd(fn, q, k, v, o, dout, lse, table, g, out, workspace, o_lo):
    import torch
    gg = _geom(g)
    n, nl, nt = _sizes(gg)
    dt = q.dtype
    code = _dtype_code(dt)
    if out is None:
        out = (torch.empty_like(q), torch.empty_like(q), torch.empty_like(q),
               torch.empty(table.shape, dtype=torch.float32, device=q.device))
    dq, dk, dv, dtab = out
    need = terra_winattn_bwd_workspace_bytes(gg, code)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(fn(ctypes.byref(gg), code, _dev(q, "q", dt, n), _dev(k, "k", dt, n), _dev(v, "v", dt, n),
              _dev(o, "o", dt, n), _opt(o_lo, "o_lo", dt, n), _dev(dout, "dout", dt, n),
              _dev(lse, "lse", torch.float32, nl), _dev(table, "table", torch.float32, nt),
              _dev(dq, "dq", dt, n), _dev(dk, "dk", dt, n), _dev(dv, "dv", dt, n),
              _dev(dtab, "dtable", torch.float32, nt), _dev(workspace, "workspace"),
              ctypes.c_size_t(workspace.numel()), _stream()))
    return dq, dk, dv, dtab


def terra_winattn_fwd(q, k, v, table, g, out=None, lse=None, o_lo=None):
    """Window-major q, k, v (B,H*W,C) and float32 bias table
    (2wh-1,2ww-1,heads) -> (O (B,H*W,C), LSE float32 (B,heads,H*W)).
    o_lo: optional tensor like O for O's rounding residual (written only
    where terra_winattn_uses_o_lo is true)."""
    return _attn_fwd(lib().terra_winattn_fwd, lambda gg: (gg.B, gg.H * gg.W, gg.C),
                     q, k, v, table, g, out, lse, o_lo)


def terra_winattn_fwd_nhwc(q, k, v, table, g, out=None, lse=None, o_lo=None):
    """NHWC q, k, v (B,H,W,C), route fused in -> (O (B,H,W,C), LSE float32
    (B,heads,H*W) in NHWC token order); o_lo as for terra_winattn_fwd."""
    return _attn_fwd(lib().terra_winattn_fwd_nhwc, lambda gg: (gg.B, gg.H, gg.W, gg.C),
                     q, k, v, table, g, out, lse, o_lo)


def terra_winattn_uses_o_lo(g, dtype):
    """True when the forward writes o_lo and the backward reads it."""
    r = int(lib().terra_winattn_uses_o_lo(ctypes.byref(_geom(g)), _dtype_code(dtype)))
    if r < 0:
        _check(-r)
    return r == 1


def terra_winattn_bwd(q, k, v, o, dout, lse, table, g, out=None, workspace=None, o_lo=None):
    """Window-major tensors.  Returns (dQ, dK, dV, dTable).  `out` may hold
    preallocated (dq, dk, dv, dtable); `workspace` a uint8 device tensor;
    `o_lo` the forward's rounding residual of O, if it kept one."""
    return _attn_bwd(lib().terra_winattn_bwd, q, k, v, o, dout, lse, table, g, out, workspace, o_lo)


def terra_winattn_bwd_nhwc(q, k, v, o, dout, lse, table, g, out=None, workspace=None, o_lo=None):
    """As terra_winattn_bwd with NHWC tensors and NHWC-ordered LSE."""
    return _attn_bwd(lib().terra_winattn_bwd_nhwc, q, k, v, o, dout, lse, table, g, out, workspace, o_lo)


TERRA_SCRATCH_BYTES = 32 << 20


def terra_winattn_bwd_nhwc_noalloc(q, k, v, o, dout, lse, table, g, out, o_lo=None):
    """terra_winattn_bwd_nhwc with no workspace argument: the library's own
    per-GPU scratch array serves.  `out` = preallocated (dq, dk, dv, dtable)."""
    import torch
    gg = _geom(g)
    n, nl, nt = _sizes(gg)
    dt = q.dtype
    dq, dk, dv, dtab = out
    _check(lib().terra_winattn_bwd_nhwc_noalloc(
        ctypes.byref(gg), _dtype_code(dt), _dev(q, "q", dt, n), _dev(k, "k", dt, n), _dev(v, "v", dt, n),
        _dev(o, "o", dt, n), _opt(o_lo, "o_lo", dt, n), _dev(dout, "dout", dt, n),
        _dev(lse, "lse", torch.float32, nl), _dev(table, "table", torch.float32, nt),
        _dev(dq, "dq", dt, n), _dev(dk, "dk", dt, n), _dev(dv, "dv", dt, n),
        _dev(dtab, "dtable", torch.float32, nt), _stream()))
    return dq, dk, dv, dtab


# ---------------------------------------------------------------- ranks
def terra_plan_padded_grid(H, W, p, alpha, w, m=1, n=1):
    """Eq. (3): (H_hat, W_hat, overhead) of the fixed assignment on an m x n mesh."""
    hh, ww, ov = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
    _check(lib().terra_plan_padded_grid(H, W, p, alpha, w, m, n, ctypes.byref(hh), ctypes.byref(ww),
                                        ctypes.byref(ov)))
    return hh.value, ww.value, ov.value


def terra_plan_window_ranges(M, ranks):
    """Eq. (4): [L_0, L_1, ..., L_ranks = M]."""
    out = (ctypes.c_int64 * (ranks + 1))()
    _check(lib().terra_plan_window_ranges(M, ranks, out))
    return list(out)


def terra_plan_rank(g, ranks, rank):
    """(plan dict, [fragment dicts]) of one rank."""
    plan = terra_rank_plan()
    frags = (terra_fragment * TERRA_MAX_FRAGMENTS)()
    _check(lib().terra_plan_rank(ctypes.byref(_geom(g)), ranks, rank, ctypes.byref(plan), frags))
    return plan.as_dict(), [frags[i].as_dict() for i in range(plan.nfrag)]


def terra_window_route_rank(stripe, frag_buf, g, ranks, rank, out=None):
    """Rank `rank`'s window-major tensor (B, slot_end - slot_begin, C) from
    its stripe (B, rows, W, C) and fragment buffer (B, frag_tokens, C)."""
    import torch
    gg = _geom(g)
    plan, _ = terra_plan_rank(gg, ranks, rank)
    dt = stripe.dtype
    if stripe.numel() != gg.B * (plan["row_end"] - plan["row_begin"]) * gg.W * gg.C:
        raise ValueError("stripe has %d elements, expected B*rows*W*C" % stripe.numel())
    if frag_buf is not None and frag_buf.numel() != gg.B * plan["frag_tokens"] * gg.C:
        raise ValueError("fragment buffer has %d elements, expected B*frag_tokens*C" % frag_buf.numel())
    ntok = plan["slot_end"] - plan["slot_begin"]
    if out is None:
        out = torch.empty((gg.B, ntok, gg.C), dtype=dt, device=stripe.device)
    elif out.numel() != gg.B * ntok * gg.C:
        raise ValueError("out has %d elements, expected B*tokens*C" % out.numel())
    _check(lib().terra_window_route_rank(ctypes.byref(gg), _dtype_code(dt), ranks, rank,
                                         _dev(stripe, "stripe", dt), _opt(frag_buf, "frag_buf", dt),
                                         _dev(out, "out", dt), _stream()))
    return out


def terra_window_unroute_rank(y_win, g, ranks, rank, stripe, frag_buf):
    """Inverse of terra_window_route_rank: y_win back into stripe and frag_buf."""
    gg = _geom(g)
    plan, _ = terra_plan_rank(gg, ranks, rank)
    dt = y_win.dtype
    if y_win.numel() != gg.B * (plan["slot_end"] - plan["slot_begin"]) * gg.C:
        raise ValueError("y_win has %d elements, expected B*tokens*C" % y_win.numel())
    if stripe.numel() != gg.B * (plan["row_end"] - plan["row_begin"]) * gg.W * gg.C:
        raise ValueError("stripe has %d elements, expected B*rows*W*C" % stripe.numel())
    if frag_buf is not None and frag_buf.numel() != gg.B * plan["frag_tokens"] * gg.C:
        raise ValueError("fragment buffer has %d elements, expected B*frag_tokens*C" % frag_buf.numel())
    _check(lib().terra_window_unroute_rank(ctypes.byref(gg), _dtype_code(dt), ranks, rank,
                                           _dev(y_win, "y_win", dt), _dev(stripe, "stripe", dt),
                                           _opt(frag_buf, "frag_buf", dt), _stream()))


def _frag_sizes(gg, ranks, dst_rank, src_rank, stripe, frag_buf):
    plan, _ = terra_plan_rank(gg, ranks, dst_rank)
    rows = (src_rank + 1) * gg.H // ranks - src_rank * gg.H // ranks
    if stripe.numel() != gg.B * rows * gg.W * gg.C:
        raise ValueError("source stripe has %d elements, expected B*rows*W*C" % stripe.numel())
    if frag_buf.numel() != gg.B * plan["frag_tokens"] * gg.C:
        raise ValueError("fragment buffer has %d elements, expected B*frag_tokens*C" % frag_buf.numel())


def terra_fragment_pack(src_stripe, frag_buf, g, ranks, dst_rank, src_rank):
    """Copy the fragments dst_rank receives from src_rank into its buffer."""
    gg = _geom(g)
    _frag_sizes(gg, ranks, dst_rank, src_rank, src_stripe, frag_buf)
    dt = src_stripe.dtype
    _check(lib().terra_fragment_pack(ctypes.byref(gg), _dtype_code(dt), ranks, dst_rank, src_rank,
                                     _dev(src_stripe, "src_stripe", dt), _dev(frag_buf, "frag_buf", dt),
                                     _stream()))


def terra_fragment_unpack(frag_buf, src_stripe, g, ranks, dst_rank, src_rank):
    """Copy those fragments back into src_rank's stripe (the backward)."""
    gg = _geom(g)
    _frag_sizes(gg, ranks, dst_rank, src_rank, src_stripe, frag_buf)
    dt = src_stripe.dtype
    _check(lib().terra_fragment_unpack(ctypes.byref(gg), _dtype_code(dt), ranks, dst_rank, src_rank,
                                       _dev(frag_buf, "frag_buf", dt), _dev(src_stripe, "src_stripe", dt),
                                       _stream()))


# ---------------------------------------------------------------- Swin block
def _block_shapes(gg):
    T, C = gg.B * gg.H * gg.W, gg.C
    return {"ln1_g": (C,), "ln1_b": (C,), "w_qkv": (3 * C, C), "b_qkv": (3 * C,), "w_proj": (C, C),
            "b_proj": (C,), "ln2_g": (C,), "ln2_b": (C,), "w_fc1": (4 * C, C), "b_fc1": (4 * C,),
            "w_fc2": (C, 4 * C), "b_fc2": (C,)}, T


def _params_struct(params, gg):
    import torch
    shapes, _ = _block_shapes(gg)
    st = terra_block_params()
    for n in BLOCK_PARAM_NAMES:
        t = params[n]
        dt = torch.bfloat16 if n.startswith("w_") else torch.float32
        setattr(st, n, _dev(t, n, dt, int(np.prod(shapes[n]))).value)
    return st


def terra_block_saved_alloc(g, device="cuda"):
    """Buffers for the activations the block forward saves."""
    import torch
    gg = _geom(g)
    T, C = gg.B * gg.H * gg.W, gg.C
    nhwc = (gg.B, gg.H, gg.W, C)
    f32, b16 = torch.float32, torch.bfloat16
    return {"mu1": torch.empty(T, dtype=f32, device=device), "rstd1": torch.empty(T, dtype=f32, device=device),
            "mu2": torch.empty(T, dtype=f32, device=device), "rstd2": torch.empty(T, dtype=f32, device=device),
            "q": torch.empty(nhwc, dtype=b16, device=device), "k": torch.empty(nhwc, dtype=b16, device=device),
            "v": torch.empty(nhwc, dtype=b16, device=device), "o": torch.empty(nhwc, dtype=b16, device=device),
            "lse": torch.empty((gg.B, gg.heads, gg.H * gg.W), dtype=f32, device=device),
            "x1": torch.empty(nhwc, dtype=b16, device=device),
            "h": torch.empty((gg.B, gg.H, gg.W, 4 * C), dtype=b16, device=device),
            "a": torch.empty((gg.B, gg.H, gg.W, 4 * C), dtype=b16, device=device)}


def _saved_struct(saved, gg):
    import torch
    T, C = gg.B * gg.H * gg.W, gg.C
    sizes = {"mu1": T, "rstd1": T, "mu2": T, "rstd2": T, "q": T * C, "k": T * C, "v": T * C, "o": T * C,
             "lse": T * gg.heads, "x1": T * C, "h": 4 * T * C, "a": 4 * T * C}
    st = terra_block_saved()
    for n in BLOCK_SAVED_NAMES:
        dt = torch.float32 if n in ("mu1", "rstd1", "mu2", "rstd2", "lse") else torch.bfloat16
        setattr(st, n, _dev(saved[n], n, dt, sizes[n]).value)
    return st


def terra_block_fwd_workspace_bytes(g, dtype="bf16"):
    return int(lib().terra_block_fwd_workspace_bytes(ctypes.byref(_geom(g)), _dtype_code(dtype)))


def terra_block_fwd(x, params, table, g, saved=None, out=None, workspace=None):
    """One Swin block forward on NHWC bf16 x.  params: dict of device tensors
    (weights bf16, the rest float32).  Returns (x2, saved)."""
    import torch
    gg = _geom(g)
    T, C = gg.B * gg.H * gg.W, gg.C
    if saved is None:
        saved = terra_block_saved_alloc(gg, x.device)
    if out is None:
        out = torch.empty_like(x)
    need = terra_block_fwd_workspace_bytes(gg)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check(lib().terra_block_fwd(ctypes.byref(gg), TERRA_BF16, _dev(x, "x", torch.bfloat16, T * C),
                                 ctypes.byref(_params_struct(params, gg)),
                                 _dev(table, "table", torch.float32, _sizes(gg)[2]),
                                 _dev(out, "x2", torch.bfloat16, T * C),
                                 ctypes.byref(_saved_struct(saved, gg)), _dev(workspace, "workspace"),
                                 ctypes.c_size_t(workspace.numel()), _stream()))
    return out, saved


def terra_block_bwd_workspace_bytes(g, dtype="bf16"):
    return int(lib().terra_block_bwd_workspace_bytes(ctypes.byref(_geom(g)), _dtype_code(dtype)))


def terra_block_bwd(dx2, x, params, table, g, saved, out=None, workspace=None):
    """Backward of the block.  Returns (dx, grads dict, dtable)."""
    import torch
    gg = _geom(g)
    T, C = gg.B * gg.H * gg.W, gg.C
    shapes, _ = _block_shapes(gg)
    if out is None:
        out = (torch.empty_like(x), {n: torch.empty(shapes[n], dtype=torch.float32, device=x.device)
                                     for n in BLOCK_PARAM_NAMES},
               torch.empty(table.shape, dtype=torch.float32, device=x.device))
    dx, grads, dtab = out
    gst = terra_block_grads()
    for n in BLOCK_PARAM_NAMES:
        setattr(gst, n, _dev(grads[n], "d" + n, torch.float32, int(np.prod(shapes[n]))).value)
    need = terra_block_bwd_workspace_bytes(gg)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check(lib().terra_block_bwd(ctypes.byref(gg), TERRA_BF16, _dev(dx2, "dx2", torch.bfloat16, T * C),
                                 _dev(x, "x", torch.bfloat16, T * C), ctypes.byref(_params_struct(params, gg)),
                                 _dev(table, "table", torch.float32, _sizes(gg)[2]),
                                 ctypes.byref(_saved_struct(saved, gg)), _dev(dx, "dx", torch.bfloat16, T * C),
                                 ctypes.byref(gst), _dev(dtab, "dtable", torch.float32, _sizes(gg)[2]),
                                 _dev(workspace, "workspace"), ctypes.c_size_t(workspace.numel()), _stream()))
    return dx, grads, dtab
