"""Plain CPU oracle for the physical expert-offload runtime of AcceptMoE.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests and the benchmark use it.  It shares no
code with the HIP library or its host runtime.

What it models (arXiv 2608.02989, Sec. 3.4 offload paragraph and the offload
setup of Sec. 4): every MoE layer keeps an X-slot expert pool in GPU memory and
the complete expert weights in pinned host memory.  The pool limits residency,
not eligibility: the selector only sees the resident set as a mask (pruning of
Eq. 7), and any expert that receives a token while not resident is copied into
the pool synchronously.  When the routed union of a block does not fit in X
slots, the block's tokens are processed in several waves whose routed unions
each fit.  The resident set is managed least-recently-used.

Readings of points the paper leaves open (listed in the design notes too):
  O1  one slot holds one expert's complete FFN weights (gate, up and down) of
      one layer; pools of different layers are independent.
  O2  recency is kept per wave: every expert a wave uses is stamped with that
      wave's time (a per-layer counter advanced once per wave); the victim of
      a load is the slot with the oldest stamp among the slots whose expert the
      wave does not use, empty slots counting as oldest, ties going to the
      lower slot index.
  O3  the experts a wave uses are visited in ascending expert index: a
      resident one is a hit, a missing one is loaded into the next victim.
  O4  waves: tokens are taken in node order and join the current wave unless
      that would make its routed union exceed X, in which case a new wave
      starts with that token (needs X >= k, so a token always fits alone).
  O5  one access per (wave, routed expert); it is a hit when the expert is
      resident before the wave's loads.  Hit rate = hits / accesses.
  O6  host-to-device bytes = loads x the bytes of one expert's weights.
  O7  the residency mask handed to selection for a block is the layer's pool
      content before that block.
  O8  pools start empty.
"""
from __future__ import annotations

import numpy as np


def routed_experts(idx_row) -> list:
    """Distinct valid experts of one token's routing row (entries < 0 are empty slots)."""
    out = []
    for e in idx_row:
        e = int(e)
        if e >= 0 and e not in out:
            out.append(e)
    return out


def plan_waves(idx, X: int):
    """Token -> wave assignment by reading O4; returns (wave_of[T], n_waves)."""
    idx = np.asarray(idx)
    T = idx.shape[0]
    wave_of = np.zeros(T, np.int32)
    current = set()
    w = 0
    for t in range(T):
        mine = set(routed_experts(idx[t]))
        if len(mine) > X:
            raise ValueError("a single token routes to more experts than the pool holds")
        if current and len(current | mine) > X:
            w += 1
            current = set()
        current |= mine
        wave_of[t] = w
    return wave_of, (w + 1 if T > 0 else 0)


def wave_experts(idx, wave_of, w: int) -> list:
    """Sorted routed union of the tokens of wave w."""
    s = set()
    for t in range(len(wave_of)):
        if wave_of[t] == w:
            s |= set(routed_experts(idx[t]))
    return sorted(s)


class LRUPool:
    """X-slot pool of one layer under readings O2, O3, O5 and O8."""

    def __init__(self, X: int, E: int):
        self.X, self.E = X, E
        self.expert_in = [-1] * X      # slot -> expert (-1 empty)
        self.stamp = [-1] * X          # slot -> last wave that used it (-1 never)
        self.clock = 0
        self.hits = 0
        self.misses = 0

    def slot_of(self, e: int) -> int:
        return self.expert_in.index(e) if e in self.expert_in else -1

    def resident_mask(self) -> np.ndarray:
        m = np.zeros(self.E, np.uint8)
        for e in self.expert_in:
            if e >= 0:
                m[e] = 1
        return m

    def serve_wave(self, experts) -> list:
        """Make every expert of the wave resident; returns the loads [(expert, slot)] in order."""
        self.clock += 1
        needed = set(int(e) for e in experts)
        if len(needed) > self.X:
            raise ValueError("wave does not fit in the pool")
        loads = []
        for e in sorted(needed):
            s = self.slot_of(e)
            if s >= 0:
                self.hits += 1
            else:
                self.misses += 1
                # victim: oldest stamp among slots not holding an expert of this wave
                cands = [j for j in range(self.X) if self.expert_in[j] not in needed]
                s = min(cands, key=lambda j: (self.stamp[j], j))
                self.expert_in[s] = e
                loads.append((e, s))
            self.stamp[s] = self.clock
        return loads


def slot_routing(idx, wave_of, w: int, pool: LRUPool) -> np.ndarray:
    """Routing rows of wave w rewritten to pool slots (-1 for other waves' tokens and empty entries)."""
    idx = np.asarray(idx)
    out = np.full(idx.shape, -1, np.int32)
    for t in range(idx.shape[0]):
        if wave_of[t] != w:
            continue
        seen = set()
        for j, e in enumerate(idx[t]):
            e = int(e)
            if e >= 0 and e not in seen:
                seen.add(e)
                out[t, j] = pool.slot_of(e)
    return out


def simulate(idx_per_block, X: int, E: int):
    """Serve a sequence of routed blocks on one layer's pool.

    Returns per block: (n_waves, loads, hits, misses) and the pool.  The
    routing of each block must already have been chosen with the mask of the
    pool state before that block (O7)."""
    pool = LRUPool(X, E)
    rows = []
    for idx in idx_per_block:
        h0, m0 = pool.hits, pool.misses
        wave_of, nw = plan_waves(idx, X)
        loads = []
        for w in range(nw):
            loads += pool.serve_wave(wave_experts(idx, wave_of, w))
        rows.append((nw, loads, pool.hits - h0, pool.misses - m0))
    return rows, pool
