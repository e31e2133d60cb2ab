"""Regression check of the CPU oracle against the fixtures that
tests/golden/make_golden.py wrote with the oracle itself: the same inputs must
give the same masks, index maps and block outputs bit for bit.  Not a pin of
the oracle (the pins are the other test_oracle_* files); a guard against an
unintended change of its arithmetic."""
import glob
import os

import numpy as np
import pytest

import oracle

GOLDEN = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.npz")))


@pytest.mark.parametrize("path", GOLDEN, ids=[os.path.basename(p) for p in GOLDEN])
def test_oracle_matches_fixture(path):
    z = np.load(path)  # allow_pickle stays False
    x = z["x_nchw"]
    N, C, H, W = x.shape
    wts = {k: z[k] for k in ("w1", "b1", "w2", "b2", "w3", "b3")}
    G, logits = oracle.mask(x, z["w_m"], z["b_m"])
    assert G.tobytes() == z["G"].tobytes()
    assert logits.tobytes() == z["logits"].tobytes()
    Gd = oracle.dilate(G, N, H, W, 1)
    assert Gd.tobytes() == z["Gd"].tobytes()
    A, D, nbr = oracle.indices(G, Gd, N, H, W)
    for got, key in ((A, "A"), (D, "D"), (nbr, "nbr")):
        assert got.tobytes() == z[key].tobytes(), key
    y, _, _ = oracle.block_dense(x.astype(np.float64), wts, G)
    assert y.tobytes() == z["y"].tobytes()
    ys, _, _ = oracle.block_sparse(x.astype(np.float64), wts, A, D, nbr)
    assert ys.tobytes() == z["y"].tobytes()


def test_fixtures_present():
    assert len(GOLDEN) >= 2
