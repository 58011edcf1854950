"""Seeded synthetic inputs for the shifted-window attention path.

This module only draws numbers and rounds them to the storage type; it holds
none of the method's arithmetic.  Both the tests/benchmark side that drives
the HIP library and the oracle side consume what it returns.

The paper trains on GLORYS fields (2041 x 4320 grid, 93 variables) that are
not available here; the grids below stand in for the Transformer-stage token
grids of that workload (Sec. IV-B / IV-D: patch size 4, optional stride-2
down-sampling), with Gaussian activations in place of learned ones.

Recipe (all configurations): ``numpy.random.default_rng(seed)`` (PCG64),
draw order Q, K, V, dOut, each B x H x W x C standard normal in float64,
cast to float32 and, for bf16 (fp16) configurations, rounded to bf16
(IEEE half) with round-to-nearest-even; then the relative-position bias
table 0.02 * N(0, 1) of shape (2wh-1, 2ww-1, heads), float32.
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Config:
    name: str
    dtype: str          # "f32", "bf16" or "f16"
    B: int
    H: int
    W: int
    heads: int
    head_dim: int
    wh: int
    ww: int
    sh: int
    sw: int
    mask_flags: int = 1  # bit0 latitude wrap masked, bit1 longitude wrap masked

    @property
    def C(self):
        return self.heads * self.head_dim

    def geom_kwargs(self):
        return dict(B=self.B, H=self.H, W=self.W, C=self.C, heads=self.heads,
                    head_dim=self.head_dim, wh=self.wh, ww=self.ww, sh=self.sh,
                    sw=self.sw, mask_flags=self.mask_flags)


CONFIGS = {
    # fp32, 16x32 grid, 2 heads x 32, window 8x8, shift (4,4)
    "c1_f32_16x32_w8": Config("c1_f32_16x32_w8", "f32", 1, 16, 32, 2, 32, 8, 8, 4, 4),
    # bf16, 128x256, 6 heads x 32, window 8x8, shift (4,4): divisible grid
    "c2_bf16_128x256_w8": Config("c2_bf16_128x256_w8", "bf16", 1, 128, 256, 6, 32, 8, 8, 4, 4),
    # bf16, B=2, 85x180 (85 not divisible by 12), 8 heads x 32, window 12x12, shift (6,6)
    "c3_bf16_85x180_w12": Config("c3_bf16_85x180_w12", "bf16", 2, 85, 180, 8, 32, 12, 12, 6, 6),
    # bf16, one latitude slab of the 1/12-degree grid at patch 4: 128x1080,
    # 24 heads x 32, window 8x16 (1080/16 ragged), shift (4,8)
    "c4_bf16_128x1080_w8x16": Config("c4_bf16_128x1080_w8x16", "bf16", 1, 128, 1080, 24, 32, 8, 16, 4, 8),
    # bf16, the whole globe at patch 4 + one stride-2 down-sampling: 256x540,
    # 24 heads x 64, window 24x24 (ragged both ways), shift (12,12)
    "c5_bf16_256x540_w24": Config("c5_bf16_256x540_w24", "bf16", 1, 256, 540, 24, 64, 24, 24, 12, 12),
}

ORDER = list(CONFIGS)

# Paper-shaped variants (Table III models; Sec. VII-A: FP16 mixed precision).
# Every model has head_dim d / N_h = 128; the Transformer-stage grid of the
# 2041 x 4320 globe at patch 4 and one stride-2 down-sampling is 256 x 540.
VARIANTS = {
    # small model (d = 1024, 8 heads, w = 8), fp16
    "p1_f16_256x540_hd128_w8": Config("p1_f16_256x540_hd128_w8", "f16", 1, 256, 540, 8, 128, 8, 8, 4, 4),
    # large model (d = 8192, 64 heads, w = 32), fp16: 8 of its heads, one
    # GPU's share under 8-way head sharding
    "p2_f16_256x540_hd128_w32": Config("p2_f16_256x540_hd128_w32", "f16", 1, 256, 540, 8, 128, 32, 32, 16, 16),
}
ALL = dict(CONFIGS, **VARIANTS)


def bf16_round(x):
    """Round float32 values to the nearest bf16 (ties to even).  Returns
    float32 values that are exactly representable in bf16."""
    x = np.ascontiguousarray(x, np.float32)
    assert np.isfinite(x).all(), "bf16_round takes finite values only"
    bits = x.view(np.uint32)
    # finite values have bits <= 0xFF7FFFFF, so the sum stays below 2^32
    r = (bits >> np.uint32(16)) & np.uint32(1)
    r += bits
    r += np.uint32(0x7FFF)
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(x.shape)


def bf16_bits(x):
    """uint16 bit patterns of float32 values that are exact bf16 numbers."""
    x = np.ascontiguousarray(x, np.float32)
    bits = x.view(np.uint32)
    assert np.all((bits & 0xFFFF) == 0), "value is not an exact bf16 number"
    return (bits >> 16).astype(np.uint16)


def bf16_from_bits(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def make_inputs(cfg, seed=0, q_scale=1.0):
    """Q, K, V, dOut as B x H x W x C float32 arrays (exact in the storage
    type of the configuration) and the bias table, drawn in the documented
    order."""
    rng = np.random.default_rng(seed)
    shape = (cfg.B, cfg.H, cfg.W, cfg.C)
    out = {}
    for name in ("q", "k", "v", "dout"):
        x = rng.standard_normal(shape).astype(np.float32)
        if name == "q" and q_scale != 1.0:
            x = (x * np.float32(q_scale)).astype(np.float32)
        if cfg.dtype == "bf16":
            x = bf16_round(x)
        elif cfg.dtype == "f16":
            x = x.astype(np.float16).astype(np.float32)
        out[name] = x
    tshape = (2 * cfg.wh - 1, 2 * cfg.ww - 1, cfg.heads)
    out["table"] = (0.02 * rng.standard_normal(tshape)).astype(np.float32)
    return out


def token_pattern(cfg, width_bytes):
    """Unique per-element bit patterns (B, H, W, C) for bit-exact route tests:
    uint32 (width 4) or uint16 (width 2) built from the flat element index."""
    n = cfg.B * cfg.H * cfg.W * cfg.C
    z = np.arange(n, dtype=np.uint64) + np.uint64(0x9E3779B97F4A7C15)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    if width_bytes == 4:
        return (z & np.uint64(0xFFFFFFFF)).astype(np.uint32).reshape(cfg.B, cfg.H, cfg.W, cfg.C)
    return (z & np.uint64(0xFFFF)).astype(np.uint16).reshape(cfg.B, cfg.H, cfg.W, cfg.C)


def small_config(name, dtype, B, H, W, heads, head_dim, wh, ww, sh, sw, mask_flags=1):
    return Config(name, dtype, B, H, W, heads, head_dim, wh, ww, sh, sw, mask_flags)


# ---------------------------------------------------------------- Swin block
# Parameter names and shapes of one block for embedding width C (MLP ratio 4).
BLOCK_PARAMS = [
    ("ln1_g", lambda C: (C,)), ("ln1_b", lambda C: (C,)),
    ("w_qkv", lambda C: (3 * C, C)), ("b_qkv", lambda C: (3 * C,)),
    ("w_proj", lambda C: (C, C)), ("b_proj", lambda C: (C,)),
    ("ln2_g", lambda C: (C,)), ("ln2_b", lambda C: (C,)),
    ("w_fc1", lambda C: (4 * C, C)), ("b_fc1", lambda C: (4 * C,)),
    ("w_fc2", lambda C: (C, 4 * C)), ("b_fc2", lambda C: (C,)),
]


def make_block_inputs(cfg, seed=0):
    """Input x and upstream gradient dx2 (B x H x W x C, N(0, 1)), the block
    parameters and the attention bias table, drawn in this order from
    numpy.random.default_rng(seed): x, dx2, then each parameter in
    BLOCK_PARAMS order -- LayerNorm gains 1 + 0.1 N(0, 1), LayerNorm shifts
    and biases 0.02 N(0, 1), weights N(0, 1) / sqrt(fan_in) -- then the table
    0.02 N(0, 1) of shape (2wh-1, 2ww-1, heads).  x, dx2 and the weights are
    rounded to the storage type (bf16 / fp16); gains, shifts and biases stay
    float32."""
    rng = np.random.default_rng(seed)
    C = cfg.C
    shape = (cfg.B, cfg.H, cfg.W, C)

    def store(a):
        a = a.astype(np.float32)
        if cfg.dtype == "bf16":
            return bf16_round(a)
        if cfg.dtype == "f16":
            return a.astype(np.float16).astype(np.float32)
        return a

    out = {"x": store(rng.standard_normal(shape)), "dx2": store(rng.standard_normal(shape))}
    params = {}
    for name, shp in BLOCK_PARAMS:
        dims = shp(C)
        z = rng.standard_normal(dims)
        if name.endswith("_g"):
            params[name] = (1.0 + 0.1 * z).astype(np.float32)
        elif name.startswith("w_"):
            params[name] = store(z / np.sqrt(dims[1]))
        else:
            params[name] = (0.02 * z).astype(np.float32)
    out["params"] = params
    out["table"] = (0.02 * rng.standard_normal((2 * cfg.wh - 1, 2 * cfg.ww - 1, cfg.heads))).astype(np.float32)
    return out
