"""Shared helpers for the GPU parity tests: seeded inputs on both sides,
oracle-side preparation, tolerance checks.  Inputs come from the workload
generator; expected values come from oracle/ only."""
from __future__ import annotations

import json
import os

import numpy as np

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import workload as W

# Tolerances (the layer's contract): normwise max-relative error of outputs
FWD_TOL = {"f32": 1e-4, "bf16": 2e-2}
LOGIT_TOL = 1e-5          # router logits, fp32 accumulation vs fp64
GATE_RTOL = 1.2e-7        # gates: fp64 on both sides, one fp32 rounding each (<= 1 ulp)


# Per-row bound: max_h |y_th - yref_th| / max_h |yref_th| for every output row t
# (a row is one token's layer output).  bf16: the SwiGLU activation is stored
# in bf16 before the down projection, each element rounded with relative error
# <= u = 2^-9; summed over I terms of random sign that error stays near u of a
# row's largest output (measured 1.0-1.5 u at every workload shape, 2.5 u as
# the worst of 65,600 rows with only I = 32 terms); 1e-2 (~5 u) bounds it.
# fp32: accumulation over H or I <= 4096 terms, ~sqrt(H) 2^-24 of the row
# (measured <= 9.4e-7); 1e-5 bounds it.
ROW_TOL = {"f32": 1e-5, "bf16": 1e-2}


def normwise_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    if scale == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref))) / scale


def per_row_rel(got, ref) -> float:
    """Largest over rows t of max|got_t - ref_t| / max|ref_t|.  A row whose
    reference is all zero must come back exactly zero (else it counts as inf)."""
    got = np.asarray(got, np.float64).reshape(len(got), -1)
    ref = np.asarray(ref, np.float64).reshape(len(ref), -1)
    if ref.size == 0:
        return 0.0
    diff = np.max(np.abs(got - ref), axis=1)
    scale = np.max(np.abs(ref), axis=1)
    zero = scale == 0.0
    out = np.where(zero, np.where(diff == 0.0, 0.0, np.inf), diff / np.where(zero, 1.0, scale))
    return float(out.max())


def elementwise_rel(got, ref) -> float:
    """Largest |got - ref| / (|ref| + 1e-3 max|ref|) over all elements (reported
    beside the normwise figure; near-zero outputs make it large by nature)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    floor = 1e-3 * float(np.max(np.abs(ref)))
    den = np.abs(ref) + floor
    if floor == 0.0:
        return 0.0 if np.array_equal(got, ref) else float("inf")
    return float(np.max(np.abs(got - ref) / den))


def check_forward(got, ref, dtype: str, label: str) -> dict:
    """Asserts the forward contract on one output tensor (normwise and per-row
    bounds) and reports the three error figures (printed, and appended as a
    JSON line to $ACCEPTMOE_ERR_REPORT when that is set)."""
    figs = {"label": label, "dtype": dtype, "normwise": normwise_rel(got, ref),
            "per_row": per_row_rel(got, ref), "elementwise": elementwise_rel(got, ref)}
    line = json.dumps(figs)
    print(f"[errors] {line}", flush=True)
    path = os.environ.get("ACCEPTMOE_ERR_REPORT")
    if path:
        with open(path, "a") as f:
            f.write(line + "\n")
    assert np.isfinite(np.asarray(got)).all(), f"{label}: non-finite output"
    assert figs["normwise"] <= FWD_TOL[dtype], figs
    assert figs["per_row"] <= ROW_TOL[dtype], figs
    return figs


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
