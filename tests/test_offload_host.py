"""Host side of the offload runtime (acceptmoe_pool_*), CPU only: the
library's planning and LRU bookkeeping (no weight pointers, so no copies)
against the offload oracle on random block traces, bit for bit, and the
argument checks of the offload entry points."""
import ctypes

import numpy as np
import pytest

from oracle import offload_oracle as OO
from paper_2608_02989_amd import _lib as L
from paper_2608_02989_amd import ops

V = ctypes.c_void_p


def random_blocks(rng, n, E, k, Tmax):
    blocks = []
    for _ in range(n):
        T = int(rng.integers(0, Tmax + 1))
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) if T else \
            np.zeros((0, k), np.int32)
        if T:
            idx[rng.random(idx.shape) < 0.08] = -1
            rep = rng.random(T) < 0.05
            idx[rep, -1] = idx[rep, 0]          # a repeated expert counts once
            idx[rng.random(idx.shape) < 0.02] = E + 3  # out of range: ignored
        blocks.append(idx)
    return blocks


@pytest.mark.parametrize("seed,E,k,X,Tmax", [(0, 16, 2, 4, 12), (1, 40, 4, 10, 30), (2, 128, 8, 48, 64),
                                            (3, 24, 3, 3, 9), (4, 64, 8, 8, 40)])
def test_pool_bookkeeping_matches_oracle(seed, E, k, X, Tmax):
    rng = np.random.default_rng(seed)
    blocks = random_blocks(rng, 40, E, k, Tmax)
    expert_bytes = 1000
    pool = ops.OffloadPool(X, E, expert_bytes=expert_bytes)
    ref = OO.LRUPool(X, E)
    waves = 0
    for b, idx in enumerate(blocks):
        assert np.array_equal(pool.resident_mask(), ref.resident_mask()), b
        clean = np.where((idx >= 0) & (idx < E), idx, -1)
        wave_of, nw = pool.plan_waves(idx)
        rw, rn = OO.plan_waves(clean, X)
        assert nw == rn and np.array_equal(wave_of, rw), b
        for w in range(nw):
            slot = pool.serve_wave(idx, wave_of, w)
            ref.serve_wave(OO.wave_experts(clean, rw, w))
            assert np.array_equal(slot, OO.slot_routing(clean, rw, w, ref)), (b, w)
        waves += nw
    st = pool.stats
    assert st[L.POOL_WAVES] == waves
    assert st[L.POOL_HITS] == ref.hits and st[L.POOL_MISSES] == ref.misses
    assert st[L.POOL_ACCESSES] == ref.hits + ref.misses
    assert st[L.POOL_H2D_BYTES] == ref.misses * expert_bytes


def test_pool_rejects():
    lib = L.lib()
    assert lib.acceptmoe_pool_state_bytes(0, 8) == 0 and lib.acceptmoe_pool_state_bytes(4, 0) == 0
    n = lib.acceptmoe_pool_state_bytes(4, 8)
    st = np.zeros(n // 8 + 1, np.int64)
    p = V(st.ctypes.data)
    assert lib.acceptmoe_pool_init(p, n - 1, 4, 8) == L.ERR_WORKSPACE
    assert lib.acceptmoe_pool_init(V(st.ctypes.data + 4), n, 4, 8) == L.ERR_INVALID_ARG  # misaligned
    assert lib.acceptmoe_pool_init(p, n, 0, 8) == L.ERR_INVALID_ARG
    junk = np.zeros_like(st)
    mask = np.zeros(8, np.uint8)
    assert lib.acceptmoe_pool_resident_mask(V(junk.ctypes.data), V(mask.ctypes.data)) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_pool_init(p, n, 4, 8) == L.OK
    # a token with more experts than slots cannot be planned
    idx = np.array([[0, 1, 2, 3, 4]], np.int32)
    wave_of = np.zeros(1, np.int32)
    nw = ctypes.c_int32(0)
    assert lib.acceptmoe_pool_plan_waves(V(idx.ctypes.data), 1, 5, 8, 4, V(wave_of.ctypes.data),
                                         ctypes.byref(nw)) == L.ERR_UNSUPPORTED
    # a wave whose union exceeds X is refused
    idx2 = np.array([[0, 1], [2, 3], [4, 5]], np.int32)
    w2 = np.zeros(3, np.int32)
    slot = np.zeros((3, 2), np.int32)
    stats = np.zeros(L.POOL_NUM_STATS, np.int64)
    args = (p, V(idx2.ctypes.data), V(w2.ctypes.data), 0, 3, 2)
    none = (V(0), V(0), V(0), V(0), 0, 0)
    assert lib.acceptmoe_pool_serve_wave(*args, *none, V(slot.ctypes.data), V(stats.ctypes.data), None) == \
        L.ERR_UNSUPPORTED
    # weight pointers: all four or none
    part = (V(0x1000), V(0), V(0x2000), V(0), 64, 64)
    w2[:] = [0, 0, 1]
    assert lib.acceptmoe_pool_serve_wave(*args, *part, V(slot.ctypes.data), V(stats.ctypes.data), None) == \
        L.ERR_INVALID_ARG
    assert lib.acceptmoe_pool_serve_wave(*args, *none, V(0), V(stats.ctypes.data), None) == L.ERR_INVALID_ARG
    assert lib.acceptmoe_pool_serve_wave(*args, *none, V(slot.ctypes.data), V(stats.ctypes.data), None) == L.OK
    assert stats[L.POOL_MISSES] == 4 and slot.tolist() == [[0, 1], [2, 3], [-1, -1]]
    # copy_rows checks run before any launch
    f = lib.acceptmoe_copy_rows
    assert f(V(0x1000), V(0x2000), V(0x3000), 0, 4, 6, None) == L.ERR_UNSUPPORTED   # H % 4
    assert f(V(0x1000), V(0x2000), V(0x3000), 0, 70000, 8, None) == L.ERR_UNSUPPORTED
    assert f(V(0x1008), V(0x2000), V(0x3000), 0, 4, 8, None) == L.ERR_INVALID_ARG  # misaligned
    assert f(None, V(0x2000), V(0x3000), 0, 4, 8, None) == L.ERR_INVALID_ARG
    assert f(None, None, None, 0, 0, 8, None) == L.OK
