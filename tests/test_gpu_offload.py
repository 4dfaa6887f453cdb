"""Physical expert offload on the GPU (acceptmoe_pool_*, acceptmoe_copy_rows)
against the oracle loop: per block, the selection sees the oracle pool's
resident set, the routing, waves, hits and misses match exactly, the layer
output matches the oracle forward over the original experts, and every slot
holds the bytes of the expert the books say it holds."""
import numpy as np
import pytest
import torch

from oracle import acceptmoe_oracle as O
from oracle import offload_oracle as OO
from paper_2608_02989_amd import _lib as L
from paper_2608_02989_amd import ops
from paper_2608_02989_amd import workload as W

from _util import HostExperts, check_forward, hidden_for

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def dev_hidden(cfg, arr):
    if cfg.dtype == "bf16":
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).to(DEV)


# small layers whose routed unions exceed the pool: both misses and waves occur
CASES = [("bf16", L.MODE_SELF_SIZING, 10), ("bf16", L.MODE_ALL_EXPERTS, 10), ("f32", L.MODE_ALL_EXPERTS, 6)]


@pytest.mark.parametrize("dtype,mode,X", CASES)
def test_offload_layer_matches_oracle(gpu, dtype, mode, X):
    cfg = W.LayerConfig("offload_small", 120 + mode * 7 + X, dtype, T=20, B=1, H=256, E=24, k=4, I=128,
                        depth_max=5, commit_rule="depth_sibling", hidden_std=1.0)
    rw = W.router_weights(cfg)
    wg, wu, wd = W.expert_weights_torch(cfg, 0, DEV)
    layer = ops.OffloadLayer(torch.from_numpy(rw).to(DEV), wg, wu, wd, cfg.k, X, max_tokens=cfg.T, mode=mode)
    ref_pool = OO.LRUPool(X, cfg.E)
    hw = (HostExperts(wg), HostExperts(wu), HostExperts(wd))
    total_waves = 0
    for b in range(8):
        blk = W.make_block(cfg, block=b, rho=0.9)
        hdev, h64 = hidden_for(cfg, blk.hidden)
        mask = ref_pool.resident_mask()
        assert np.array_equal(layer.pool.resident_mask(), mask), b
        z32 = O.route(h64, rw.astype(np.float64)).astype(np.float32)
        ref = O.select(z32, blk.parent, blk.depth, blk.prob, None, cfg.k, mode=mode, resident=mask)
        assert not ref["ambiguous"].any()
        say(f"offload {dtype} mode={mode} X={X} block {b}")
        outs, out, wave_of = layer.step(dev_hidden(cfg, hdev), torch.from_numpy(blk.parent).to(DEV),
                                        torch.from_numpy(blk.depth).to(DEV), torch.from_numpy(blk.prob).to(DEV))
        torch.cuda.synchronize()
        assert np.array_equal(outs["idx"].cpu().numpy(), ref["idx"]), b
        rw_of, rn = OO.plan_waves(ref["idx"], X)
        assert np.array_equal(wave_of, rw_of), b
        for w in range(rn):
            ref_pool.serve_wave(OO.wave_experts(ref["idx"], rw_of, w))
        total_waves += rn
        y_ref = O.moe_forward_grouped(h64, *hw, ref["idx"], ref["gate"], cfg.dtype)
        check_forward(out.cpu().numpy(), y_ref, cfg.dtype, f"offload block {b}")
    st = layer.pool.stats
    assert st[L.POOL_HITS] == ref_pool.hits and st[L.POOL_MISSES] == ref_pool.misses
    assert st[L.POOL_WAVES] == total_waves
    assert st[L.POOL_H2D_BYTES] == ref_pool.misses * layer.pool.expert_bytes
    assert ref_pool.misses > 0 and ref_pool.hits > 0
    if mode == L.MODE_ALL_EXPERTS:
        assert total_waves > 8  # some block needed more than one wave
    # every slot holds the packed bytes of the expert the books name
    pool = layer.pool
    gu = pool.pool_gu.cpu().numpy().reshape(X, -1)
    dn = pool.pool_dn.cpu().numpy().reshape(X, -1)
    hg = pool.host_gu.numpy().reshape(cfg.E, -1)
    hd = pool.host_dn.numpy().reshape(cfg.E, -1)
    for s, e in enumerate(ref_pool.expert_in):
        if e >= 0:
            assert np.array_equal(gu[s], hg[e]) and np.array_equal(dn[s], hd[e]), (s, e)


def test_copy_rows(gpu):
    rng = np.random.default_rng(7)
    T, H = 37, 96
    src = torch.from_numpy(rng.standard_normal((T, H)).astype(np.float32)).to(DEV)
    dst0 = rng.standard_normal((T, H)).astype(np.float32)
    dst = torch.from_numpy(dst0.copy()).to(DEV)
    tag = rng.integers(0, 3, T).astype(np.int32)
    ops.copy_rows(src, dst, torch.from_numpy(tag).to(DEV), 1)
    torch.cuda.synchronize()
    want = np.where((tag == 1)[:, None], src.cpu().numpy(), dst0)
    assert np.array_equal(dst.cpu().numpy(), want)
