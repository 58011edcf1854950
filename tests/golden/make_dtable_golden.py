"""Write the oracle's bias-table gradient for the full-size grids.

Calls only the oracle (and the seeded input generator): route every input,
run the fp64 backward over every window, and store dT as float64 .npy files
dtable_<config>.npy next to this script.  The GPU parity test compares the
HIP path's dT with these files, because the full-size oracle backward takes
minutes.

    python tests/golden/make_dtable_golden.py [config ...]
"""

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import terra_synth as ts  # noqa: E402
from oracle import Geometry, route, attn_bwd  # noqa: E402

DEFAULT = ["c4_bf16_128x1080_w8x16", "c5_bf16_256x540_w24",
           "p1_f16_256x540_hd128_w8", "p2_f16_256x540_hd128_w32"]


def main(names):
    for name in names:
        cfg = ts.ALL[name]
        g = Geometry(**cfg.geom_kwargs())
        t0 = time.time()
        inp = ts.make_inputs(cfg)
        q, k, v, do = (route(inp[n], g) for n in ("q", "k", "v", "dout"))
        _, _, _, dt = attn_bwd(q, k, v, do, inp["table"], g)
        out = os.path.join(HERE, "dtable_%s.npy" % name)
        np.save(out, dt)
        print("%s: %s  (%.0f s)" % (name, out, time.time() - t0), flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or DEFAULT)
