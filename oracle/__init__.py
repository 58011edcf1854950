"""Plain fp64 CPU oracle for the shifted-window attention hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) imports, calls or links anything in this package; only
the tests, the smoke check and the CPU-baseline leg of the benchmark do.

What it computes (the readings of the paper are listed next to each function):

* ``geometry``  - the window partition of the shifted token grid (Sec. IV-D,
  Eq. (2); row-major window flattening of Sec. V-A), written out by
  enumeration of every token.
* ``route``     - the token route between the spatially contiguous NHWC
  layout and the window-major layout, and its inverse (Sec. IV-D).
* ``attention`` - windowed multi-head self-attention with relative-position
  bias and the shifted-window mask, forward (O and log-sum-exp) and backward
  (dQ, dK, dV and the bias-table gradient), one window class at a time in
  fp64 (W-MSA / SW-MSA of the Swin blocks, Sec. IV-A).
* ``brute``     - the same attention computed over the whole grid in NHWC
  order from a full token-pair mask; it never forms the window-major layout.
* ``block``     - one pre-norm Swin block around the attention (LayerNorm,
  QKV projection, attention, output projection, MLP with GELU, two residual
  branches; Sec. IV-A, IV-C, Table III), forward and backward.
* ``planner``   - padding of the fixed window assignment (Sec. V-A, Eq. (3)),
  the ragged window ranges of Eq. (4), the SP sub-tile counts of Sec. V-B,
  the DMP height stripes, and every token each rank's route needs, listed
  one by one with its source rank (Sec. IV-D).

Parity status: the paper prints no numeric value for the attention or the
routes, so parity *with the paper's numbers* is unpinned for every function
here.  Each function is instead pinned to mathematics and library routines
(see the tests whose names start with ``test_oracle_``).
"""

from .geometry import Geometry, window_extents, token_table, window_classes
from .route import route, unroute
from .attention import attn_fwd, attn_bwd, attn_fwd_windows, attn_bwd_windows
from . import brute, planner, block

__all__ = [
    "Geometry", "window_extents", "token_table", "window_classes",
    "route", "unroute", "attn_fwd", "attn_bwd", "attn_fwd_windows",
    "attn_bwd_windows", "brute", "planner", "block",
]
