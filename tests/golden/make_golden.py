"""Write the oracle regression fixtures in this folder.

Calls only the CPU oracle (and the seeded input generators) on small inputs
and stores inputs and outputs together, so that a later change to the
oracle's arithmetic shows up in tests/test_oracle_golden.py.  These are
regression fixtures, not pins: the paper prints no worked example.

    python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_1912_03203_amd import inputs  # noqa: E402

CASES = [
    # name, (N, H, W, C, E), density, seed
    ("block_2x8x9_c16_e32", (2, 8, 9, 16, 32), 0.3, 11),
    ("block_1x5x13_c8_e16", (1, 5, 13, 8, 16), 0.5, 12),
]


def make(name, shape, density, seed):
    N, H, W, C, E = shape
    rng = inputs.rng_for(seed)
    x = inputs.blob_features(rng, N, H, W, C).astype(np.float32)  # NHWC
    wts = inputs.block_weights(rng, C, E, dtype="f32")
    x_nchw = np.ascontiguousarray(x.transpose(0, 3, 1, 2))
    _, s = oracle.mask(x_nchw, wts["w_m"], 0.0)
    b_m = np.float32(inputs.percentile_bias(s, density))
    out = oracle.block_forward(x_nchw.astype(np.float64), wts, wts["w_m"], b_m)
    y_sparse, _, _ = oracle.block_sparse(x_nchw.astype(np.float64), wts, out["A"], out["D"], out["nbr"])
    assert np.array_equal(out["y"], y_sparse)
    np.savez_compressed(
        os.path.join(HERE, name + ".npz"),
        x_nchw=x_nchw, w1=wts["w1"], b1=wts["b1"], w2=wts["w2"], b2=wts["b2"], w3=wts["w3"],
        b3=wts["b3"], w_m=wts["w_m"], b_m=np.array(b_m, np.float32),
        G=out["G"], logits=out["logits"], Gd=out["Gd"], A=out["A"], D=out["D"], nbr=out["nbr"],
        y=out["y"])
    print("%s: P=%d P_d=%d" % (name, out["A"].size, out["D"].size))


if __name__ == "__main__":
    for case in CASES:
        make(*case)
