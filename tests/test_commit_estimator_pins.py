"""Pins for the offline commitment estimator of the oracle (Sec. 3.2,
p_hat_d = c_d / m_d): a hand-counted pair of blocks, and convergence to the
closed-form marginal of a synthetic acceptance process (law of large numbers,
within five standard deviations) for a tree and for a chain."""
import math

import numpy as np
import pytest

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import workload as W


def test_hand_counted_blocks():
    # block A: a chain of 4, prefix = first two nodes; block B: root, children a, b, a's child c; prefix root, b
    dA, onA = [0, 1, 2, 3], [1, 1, 0, 0]
    dB, onB = [0, 1, 1, 2], [1, 0, 1, 0]
    mA, cA = O.commit_counts(dA, onA, 4)
    mB, cB = O.commit_counts(dB, onB, 4)
    m, c = mA + mB, cA + cB
    assert m.tolist() == [2, 3, 2, 1] and c.tolist() == [2, 2, 0, 0]
    p = O.commit_estimate(m, c)
    assert p.dtype == np.float32 and p.tolist() == [1.0, np.float32(2.0 / 3.0), 0.0, 0.0]
    # positions outside the table are not counted; unobserved positions estimate 0
    m2, c2 = O.commit_counts([0, 5, -1], [1, 1, 1], 3)
    assert m2.tolist() == [1, 0, 0] and O.commit_estimate(m2, c2).tolist() == [1.0, 0.0, 0.0]
    assert O.commit_expand(np.float32([0.5, 0.25]), [0, 1, 1, 2, 0]).tolist() == [0.5, 0.25, 0.25, 0.0, 0.5]


def closed_form_marginals(parent, sib, q):
    pi = np.zeros(len(parent))
    for t in range(len(parent)):
        p, node = 1.0, t
        while parent[node] >= 0:
            r = int(sib[node])
            p *= q[r] if r < len(q) else 0.0
            node = int(parent[node])
        pi[t] = p
    return pi


@pytest.mark.parametrize("shape", ["tree", "chain"])
def test_converges_to_closed_form_marginal(shape):
    q = (0.55, 0.2, 0.1, 0.05)
    if shape == "tree":
        parent, depth, sib = W.make_tree(np.random.default_rng(4), 24, 5)
    else:
        parent, depth, sib = W.chain(8)
    D = int(depth.max()) + 1
    N = 20000
    rng = np.random.default_rng(11)
    m = np.zeros(D, np.int64)
    c = np.zeros(D, np.int64)
    for _ in range(N):
        on = W.accepted_prefix(rng, parent, sib, q)
        mb, cb = O.commit_counts(depth, on, D)
        m += mb
        c += cb
    p_hat = O.commit_estimate(m, c)
    pi = closed_form_marginals(parent, sib, q)
    for d in range(D):
        Nd = int((depth == d).sum())
        P = float(pi[depth == d].sum())          # at most one prefix node per depth: X_d ~ Bernoulli(P)
        want = P / Nd
        sd = math.sqrt(max(P * (1 - P), 1e-12) / N) / Nd
        assert abs(float(p_hat[d]) - want) <= 5 * sd + 1e-7, (d, p_hat[d], want)
    if shape == "chain":
        assert all(p_hat[d] > p_hat[d + 1] for d in range(D - 1))
