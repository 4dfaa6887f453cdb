"""Commitment probabilities from an estimated table on the GPU: the device
expansion p_t = p_hat[d_t] bit-exact against the oracle, and selection of
tree and chain blocks driven by an estimated table equal to the oracle's."""
import numpy as np
import pytest
import torch

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import ops
from paper_2608_02989_amd import workload as W

from _util import oracle_logits32

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def estimated_table(shape, D, n=400):
    rng = np.random.default_rng(21)
    est = ops.CommitEstimator(D)
    for b in range(n):
        if shape == "tree":
            par, dep, sib = W.make_tree(np.random.default_rng(1000 + b), 60, 8)
        else:
            par, dep, sib = W.chain(10)
        est.add(dep, W.accepted_prefix(rng, par, sib))
    return est.estimate()


def test_commit_expand_matches_oracle(gpu):
    p_hat = np.float32([1.0, 0.5, 0.3, 0.125])
    depth = np.array([0, 1, 3, 2, 7, -1, 1, 0] * 40, np.int32)
    got = ops.commit_expand(torch.from_numpy(p_hat).to(DEV), torch.from_numpy(depth).to(DEV)).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), O.commit_expand(p_hat, depth).view(np.uint32))


@pytest.mark.parametrize("shape", ["tree", "chain"])
def test_select_with_estimated_table(gpu, shape):
    cfg = W.CONFIGS["qwen3_30b_a3b"]
    D = 9 if shape == "tree" else 10
    p_hat = estimated_table(shape, D)
    say(f"estimated p_hat ({shape}): {np.round(p_hat, 4).tolist()}")
    assert p_hat[0] == 1.0 and np.all(np.diff(p_hat) <= 0)
    rw = W.router_weights(cfg)
    for b in range(3):
        if shape == "tree":
            blk = W.make_block(cfg, block=b)
            par, dep = blk.parent, blk.depth
            h32 = blk.hidden
        else:
            par, dep, _ = W.chain(10)
            rng = np.random.default_rng(b)
            h32 = W.correlated_hidden(rng, par, cfg.H, cfg.hidden_std, 0.9)
        h64 = O.widen_bf16(W.bf16_round(h32))
        z32 = oracle_logits32(h64, rw)
        prob_dev = ops.commit_expand(torch.from_numpy(p_hat).to(DEV), torch.from_numpy(dep).to(DEV))
        got = ops.select(torch.from_numpy(z32).to(DEV), torch.from_numpy(par).to(DEV), torch.from_numpy(dep).to(DEV),
                         prob_dev, None, cfg.k)
        ref = O.select(z32, par, dep, O.commit_expand(p_hat, dep), None, cfg.k)
        assert not ref["ambiguous"].any()
        torch.cuda.synchronize()
        assert np.array_equal(got["eligible"].cpu().numpy(), ref["eligible"]), (shape, b)
        assert np.array_equal(got["idx"].cpu().numpy(), ref["idx"]), (shape, b)
