"""The library's offline commitment estimator (acceptmoe_commit_count /
_estimate, host side) against the oracle on synthetic verification traces of
trees and chains, bit for bit, and its argument checks."""
import ctypes

import numpy as np
import pytest

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import _lib as L
from paper_2608_02989_amd import ops
from paper_2608_02989_amd import workload as W

V = ctypes.c_void_p


@pytest.mark.parametrize("shape,D", [("tree", 9), ("chain", 12), ("tree", 4)])
def test_estimator_matches_oracle(shape, D):
    rng = np.random.default_rng(5)
    est = ops.CommitEstimator(D)
    m = np.zeros(D, np.int64)
    c = np.zeros(D, np.int64)
    for b in range(300):
        if shape == "tree":
            par, dep, sib = W.make_tree(np.random.default_rng(b), int(rng.integers(1, 40)), 8)
        else:
            par, dep, sib = W.chain(int(rng.integers(1, 16)))
        on = W.accepted_prefix(rng, par, sib)
        est.add(dep, on)
        mb, cb = O.commit_counts(dep, on, D)
        m += mb
        c += cb
    assert np.array_equal(est.m, m) and np.array_equal(est.c, c)
    p = est.estimate()
    assert np.array_equal(p.view(np.uint32), O.commit_estimate(m, c).view(np.uint32))


def test_estimator_rejects():
    lib = L.lib()
    m = np.array([2, 1], np.int64)
    c = np.array([1, 2], np.int64)
    p = np.zeros(2, np.float32)
    assert lib.acceptmoe_commit_estimate(V(m.ctypes.data), V(c.ctypes.data), 2, V(p.ctypes.data)) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_commit_estimate(V(m.ctypes.data), V(c.ctypes.data), 0, V(p.ctypes.data)) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_commit_count(None, None, 3, 2, V(m.ctypes.data), V(c.ctypes.data)) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_commit_count(None, None, 0, 2, V(m.ctypes.data), V(c.ctypes.data)) == L.OK
    assert lib.acceptmoe_commit_expand(None, 2, None, 0, None, None) == L.OK
    assert lib.acceptmoe_commit_expand(None, 2, None, 4, None, None) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_commit_expand(V(0x1000), 0, V(0x2000), 4, V(0x3000), None) == L.ERR_INVALID_ARG
