"""Shared helpers for the GPU parity tests: seeded inputs on both sides,
oracle-side preparation, tolerance checks.  Inputs come from the workload
generator; expected values come from oracle/ only."""
from __future__ import annotations

import numpy as np

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import workload as W

# Tolerances (the layer's contract): normwise max-relative error of outputs
FWD_TOL = {"f32": 1e-4, "bf16": 2e-2}
LOGIT_TOL = 1e-5          # router logits, fp32 accumulation vs fp64
GATE_RTOL = 1.2e-7        # gates: fp64 on both sides, one fp32 rounding each (<= 1 ulp)


def normwise_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    if scale == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref))) / scale


def hidden_for(cfg: W.LayerConfig, h32: np.ndarray):
    """(device-side array to upload, exact fp64 values the oracle sees)."""
    if cfg.dtype == "bf16":
        bits = W.bf16_round(h32)
        return bits, O.widen_bf16(bits)
    return h32.astype(np.float32), h32.astype(np.float64)


def oracle_logits32(h64: np.ndarray, router_w: np.ndarray) -> np.ndarray:
    """fp32 logits as the oracle computes them (fp64 product rounded once)."""
    return O.route(h64, router_w.astype(np.float64)).astype(np.float32)


class HostExperts:
    """Host view of a device weight stack, fetched one expert at a time."""

    def __init__(self, t):
        self.t = t
        self.cache = {}

    def __len__(self):
        return self.t.shape[0]

    def __getitem__(self, e):
        e = int(e)
        if e not in self.cache:
            if len(self.cache) > 8:
                self.cache.clear()
            self.cache[e] = W.to_bits(self.t[e])
        return self.cache[e]
