"""Pins for the offload oracle (X-slot pool, LRU, waves): hand-worked traces,
the classic LRU page-fault count of a textbook reference string, a second LRU
written with an ordered dictionary for single-expert waves, and the invariants
the runtime must keep (every wave fits, every token in one wave, no expert
twice in a pool, loads = misses)."""
from collections import OrderedDict

import numpy as np
import pytest

from oracle import offload_oracle as OO


def single_expert_blocks(refs):
    # one block per reference: one token routed to one expert (k = 1)
    return [np.array([[e]], np.int32) for e in refs]


def test_textbook_reference_string_three_frames():
    # the classic 20-reference string on 3 frames: LRU takes 12 faults
    refs = [7, 0, 1, 2, 0, 3, 0, 4, 2, 3, 0, 3, 2, 1, 2, 0, 1, 7, 0, 1]
    rows, pool = OO.simulate(single_expert_blocks(refs), X=3, E=8)
    assert pool.misses == 12 and pool.hits == 8
    assert sorted(pool.expert_in) == [0, 1, 7]


def ordered_dict_lru(refs, X):
    cache, faults = OrderedDict(), 0
    for e in refs:
        if e in cache:
            cache.move_to_end(e)
        else:
            faults += 1
            if len(cache) == X:
                cache.popitem(last=False)
            cache[e] = True
    return faults, set(cache)


@pytest.mark.parametrize("seed", range(6))
def test_single_expert_waves_match_ordered_dict_lru(seed):
    rng = np.random.default_rng(seed)
    X, E = int(rng.integers(2, 9)), 24
    refs = rng.integers(0, E, 300).tolist()
    rows, pool = OO.simulate(single_expert_blocks(refs), X=X, E=E)
    faults, content = ordered_dict_lru(refs, X)
    assert pool.misses == faults and pool.hits == len(refs) - faults
    assert set(e for e in pool.expert_in if e >= 0) == content


def test_hand_waves():
    # X = 3, k = 2: {0,1} {1,2} fit together (union 3); {3,4} starts wave 1; {0,5} wave 2
    idx = np.array([[0, 1], [1, 2], [3, 4], [0, 5]], np.int32)
    wave_of, n = OO.plan_waves(idx, 3)
    assert n == 3 and wave_of.tolist() == [0, 0, 1, 2]
    assert OO.wave_experts(idx, wave_of, 0) == [0, 1, 2]
    # empty and repeated entries do not count
    idx2 = np.array([[4, -1], [4, 4], [-1, -1]], np.int32)
    w2, n2 = OO.plan_waves(idx2, 1)
    assert n2 == 1 and w2.tolist() == [0, 0, 0]


def test_hand_victims():
    # X = 4: wave {1,2,3} fills slots 0..2; wave {2,5}: 2 hits, 5 takes the empty slot 3;
    # wave {6,7}: slots 0 and 2 (stamp of the first wave) are the oldest -> 6 to slot 0, 7 to slot 2
    pool = OO.LRUPool(4, 8)
    assert pool.serve_wave([3, 1, 2]) == [(1, 0), (2, 1), (3, 2)]
    assert pool.serve_wave([5, 2]) == [(5, 3)]
    assert pool.serve_wave([7, 6]) == [(6, 0), (7, 2)]
    assert pool.expert_in == [6, 2, 7, 5]
    assert pool.hits == 1 and pool.misses == 6
    assert pool.resident_mask().tolist() == [0, 0, 1, 0, 0, 1, 1, 1]


@pytest.mark.parametrize("seed", range(5))
def test_wave_and_pool_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    E, k, X = 40, 4, 10
    blocks = []
    for _ in range(30):
        T = int(rng.integers(1, 20))
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
        idx[rng.random(idx.shape) < 0.1] = -1
        blocks.append(idx)
    pool = OO.LRUPool(X, E)
    for idx in blocks:
        wave_of, nw = OO.plan_waves(idx, X)
        # contiguous, every token once, each union fits, greedy maximal
        assert np.all(np.diff(wave_of) >= 0) and (nw == 0 or wave_of[-1] == nw - 1)
        for w in range(nw):
            ex = OO.wave_experts(idx, wave_of, w)
            assert len(ex) <= X
            if w + 1 < nw:
                first_next = int(np.argmax(wave_of == w + 1))
                assert len(set(ex) | set(OO.routed_experts(idx[first_next]))) > X
            m0 = pool.misses
            loads = pool.serve_wave(ex)
            assert len(loads) == pool.misses - m0
            held = [e for e in pool.expert_in if e >= 0]
            assert len(held) == len(set(held)) and set(ex) <= set(held)
            sr = OO.slot_routing(idx, wave_of, w, pool)
            for t in range(len(idx)):
                for j in range(k):
                    if wave_of[t] == w and idx[t, j] >= 0 and idx[t, j] not in idx[t, :j]:
                        assert pool.expert_in[sr[t, j]] == idx[t, j]
                    else:
                        assert sr[t, j] == -1
