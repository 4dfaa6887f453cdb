"""acceptmoe_select_noalloc (static per-device scratch, no workspace) against
acceptmoe_select (caller workspace) through the C ABI: two calls in a row on
the same device scratch, the second with a smaller input, every output equal
bit for bit (the same kernels run on the same inputs)."""
import numpy as np
import pytest
import torch

from paper_2608_02989_amd import _lib as L
from paper_2608_02989_amd import ops
from paper_2608_02989_amd import workload as W

pytestmark = pytest.mark.gpu

DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def trees(rng, sizes, depth_max=8):
    pars, deps, probs, offs = [], [], [], [0]
    for n in sizes:
        par, dep, sib = W.make_tree(rng, n, depth_max)
        pars.append(np.where(par < 0, -1, par + offs[-1]))
        deps.append(dep)
        probs.append((0.75 ** dep * 0.6 ** sib).astype(np.float32))
        offs.append(offs[-1] + n)
    return (np.concatenate(pars).astype(np.int32), np.concatenate(deps).astype(np.int32),
            np.concatenate(probs).astype(np.float32), offs)


def dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, dt)).to(DEV)


def both(z, par, dep, prob, offs, k, mode=L.MODE_SELF_SIZING, budget=0, resident=None):
    args = (dev(z, np.float32), dev(par, np.int32), dev(dep, np.int32), dev(prob, np.float32))
    res = None if resident is None else dev(resident, np.uint8)
    ref = ops.select(*args, offs, k, mode=mode, budget=budget, resident=res)
    got = ops.select_noalloc(*args, offs, k, mode=mode, budget=budget, resident=res)
    torch.cuda.synchronize()
    return ({n: t.cpu().numpy() for n, t in got.items()}, {n: t.cpu().numpy() for n, t in ref.items()})


def assert_same(got, ref, what):
    for name in ("eligible", "idx", "stats"):
        assert np.array_equal(got[name], ref[name]), (what, name)
    assert np.array_equal(got["gate"].view(np.uint32), ref["gate"].view(np.uint32)), (what, "gate")


@pytest.mark.parametrize("mode,budget", [(L.MODE_SELF_SIZING, 0), (L.MODE_MOESPEC, 30)])
def test_select_noalloc_matches_workspace_entry(gpu, mode, budget):
    rng = np.random.default_rng(1234 + mode)
    # call 1: 8 trees of 64 nodes, E = 128, k = 8, 25 % of the experts resident
    par, dep, prob, offs = trees(rng, [64] * 8)
    z = rng.standard_normal((offs[-1], 128)).astype(np.float32)
    resident = (rng.random(128) < 0.25).astype(np.uint8)
    say(f"noalloc call 1: T={offs[-1]} B=8 E=128 k=8 mode={mode}")
    got, ref = both(z, par, dep, prob, offs, 8, mode, budget, resident)
    assert_same(got, ref, "call 1")
    assert (ref["stats"][:, L.NUM_STATS - 2] == 0).all()
    # call 2, smaller: one tree of 21 nodes, E = 48, k = 4, no mask; the scratch
    # still holds call 1's contents
    par, dep, prob, offs = trees(rng, [21], depth_max=5)
    z = rng.standard_normal((21, 48)).astype(np.float32)
    say(f"noalloc call 2: T=21 B=1 E=48 k=4 mode={mode}")
    got, ref = both(z, par, dep, prob, offs, 4, mode, min(budget, 12))
    assert_same(got, ref, "call 2")
    assert (ref["idx"] >= 0).all()
