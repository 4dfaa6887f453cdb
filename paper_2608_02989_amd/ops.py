"""Thin torch binding over the C ABI: argument marshalling only.

Every step runs in the HIP kernels of libacceptmoe.so; torch provides device
memory and the current stream.  Functions raise AcceptMoEError on any status
other than OK and RuntimeError when the library is missing.
"""
from __future__ import annotations

import copy
import ctypes

import numpy as np
import torch

from . import _lib as L
from ._lib import AcceptMoEError, check, lib  # noqa: F401


def _stream_ptr(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return L.BF16
    if t.dtype == torch.float32:
        return L.F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _need(t: torch.Tensor, name: str, dtype=None, dim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if dim is not None and t.dim() != dim:
        raise ValueError(f"{name} must have {dim} dims")


# ---------------------------------------------------------------------------
class PackedRouter:
    """Router matrix W_r [E, H] (fp32 as three bf16 planes) in the layout acceptmoe_route reads."""

    def __init__(self, data: torch.Tensor, E: int, H: int):
        self.data, self.E, self.H = data, E, H


def pack_router_weights(router_w: torch.Tensor, stream=None) -> PackedRouter:
    """[E, H] fp32 router matrix -> PackedRouter (acceptmoe_pack_router_weights)."""
    _need(router_w, "router_w", torch.float32, 2)
    E, H = router_w.shape
    n = int(lib().acceptmoe_packed_router_bytes(E, H))
    if n == 0:
        raise ValueError(f"unsupported router shape {tuple(router_w.shape)}")
    data = torch.empty(n // 2, dtype=torch.int16, device=router_w.device)
    check(lib().acceptmoe_pack_router_weights(_ptr(router_w), E, H, _ptr(data), _stream_ptr(stream)))
    return PackedRouter(data, E, H)


def route(hidden: torch.Tensor, router: PackedRouter, out: torch.Tensor | None = None,
          stream=None) -> torch.Tensor:
    """Router logits [T, E] fp32 (acceptmoe_route) from a packed router matrix."""
    _need(hidden, "hidden", dim=2)
    if not isinstance(router, PackedRouter):
        raise TypeError("route needs the router matrix packed by pack_router_weights")
    T, H = hidden.shape
    if router.H != H:
        raise ValueError(f"router packed for H={router.H}, hidden has H={H}")
    if out is None:
        out = torch.empty((T, router.E), dtype=torch.float32, device=hidden.device)
    check(lib().acceptmoe_route(_ptr(hidden), _dtype_code(hidden), _ptr(router.data), T, H, router.E, _ptr(out),
                                _stream_ptr(stream)))
    return out


def select_workspace(T: int, E: int, k: int, device) -> torch.Tensor:
    n = lib().acceptmoe_select_workspace_size(T, E, k)
    return torch.empty(max(int(n), 256), dtype=torch.uint8, device=device)


def select(logits: torch.Tensor, parent: torch.Tensor | None, depth: torch.Tensor, prob: torch.Tensor,
           tree_offsets=None, k: int = 8, beta: float = 0.5, mode: int = L.MODE_SELF_SIZING,
           budget: int = 0, removal_cap: int = -1, resident: torch.Tensor | None = None,
           workspace: torch.Tensor | None = None, outputs: dict | None = None, stream=None) -> dict:
    """Eligible sets, restricted top-k and gates (acceptmoe_select).

    tree_offsets: host sequence of B+1 ints, or None for one tree.
    Returns dict(eligible [B,E] uint8, idx [T,k] int32, gate [T,k] fp32, stats [B,10] int32).
    """
    _need(logits, "logits", torch.float32, 2)
    _need(depth, "depth", torch.int32, 1)
    _need(prob, "prob", torch.float32, 1)
    if parent is not None:
        _need(parent, "parent", torch.int32, 1)
    if resident is not None:
        _need(resident, "resident", torch.uint8, 1)
    T, E = logits.shape
    if tree_offsets is None:
        offs_arr, B = None, 1
    else:
        offs_np = np.ascontiguousarray(np.asarray(tree_offsets, dtype=np.int32))
        B = len(offs_np) - 1
        offs_arr = (ctypes.c_int32 * len(offs_np))(*offs_np.tolist())
    dev = logits.device
    if outputs is None:
        outputs = {
            "eligible": torch.empty((max(B, 1), E), dtype=torch.uint8, device=dev),
            "idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "gate": torch.empty((T, k), dtype=torch.float32, device=dev),
            "stats": torch.empty((max(B, 1), L.NUM_STATS), dtype=torch.int32, device=dev),
        }
    if workspace is None:
        workspace = select_workspace(T, E, k, dev)
    check(lib().acceptmoe_select(
        _ptr(logits), _ptr(parent), _ptr(depth), _ptr(prob), offs_arr, B, T, E, k, float(beta), int(mode),
        int(budget), int(removal_cap), _ptr(resident), _ptr(outputs["eligible"]), _ptr(outputs["idx"]),
        _ptr(outputs["gate"]), _ptr(outputs["stats"]), _ptr(workspace), workspace.numel(),
        _stream_ptr(stream)))
    return outputs


def select_noalloc(logits: torch.Tensor, parent: torch.Tensor | None, depth: torch.Tensor, prob: torch.Tensor,
                   tree_offsets=None, k: int = 8, beta: float = 0.5, mode: int = L.MODE_SELF_SIZING,
                   budget: int = 0, removal_cap: int = -1, resident: torch.Tensor | None = None,
                   outputs: dict | None = None, stream=None) -> dict:
    """select() through acceptmoe_select_noalloc: no workspace, the library's
    static per-device scratch (calls on one device must not overlap)."""
    _need(logits, "logits", torch.float32, 2)
    _need(depth, "depth", torch.int32, 1)
    _need(prob, "prob", torch.float32, 1)
    if parent is not None:
        _need(parent, "parent", torch.int32, 1)
    if resident is not None:
        _need(resident, "resident", torch.uint8, 1)
    T, E = logits.shape
    if tree_offsets is None:
        offs_arr, B = None, 1
    else:
        offs_np = np.ascontiguousarray(np.asarray(tree_offsets, dtype=np.int32))
        B = len(offs_np) - 1
        offs_arr = (ctypes.c_int32 * len(offs_np))(*offs_np.tolist())
    dev = logits.device
    if outputs is None:
        outputs = {
            "eligible": torch.empty((max(B, 1), E), dtype=torch.uint8, device=dev),
            "idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "gate": torch.empty((T, k), dtype=torch.float32, device=dev),
            "stats": torch.empty((max(B, 1), L.NUM_STATS), dtype=torch.int32, device=dev),
        }
    check(lib().acceptmoe_select_noalloc(
        _ptr(logits), _ptr(parent), _ptr(depth), _ptr(prob), offs_arr, B, T, E, k, float(beta), int(mode),
        int(budget), int(removal_cap), _ptr(resident), _ptr(outputs["eligible"]), _ptr(outputs["idx"]),
        _ptr(outputs["gate"]), _ptr(outputs["stats"]), _stream_ptr(stream)))
    return outputs


def pack_expert_weights(w: torch.Tensor, stream=None) -> torch.Tensor:
    """[E, N, K] row-major stack -> packed MFMA fragment layout (same shape and size)."""
    _need(w, "w", dim=3)
    E, N, K = w.shape
    out = torch.empty_like(w)
    check(lib().acceptmoe_pack_expert_weights(_ptr(w), _dtype_code(w), E, N, K, _ptr(out),
                                              _stream_ptr(stream)))
    return out


class PackedGateUp:
    """Gate and up stacks [E, I, H] packed together (acceptmoe_pack_gate_up_weights)."""

    def __init__(self, data: torch.Tensor, E: int, I: int, H: int):
        self.data, self.E, self.I, self.H = data, E, I, H
        self.dtype = data.dtype


def pack_gate_up_weights(w_gate: torch.Tensor, w_up: torch.Tensor, stream=None) -> PackedGateUp:
    """Gate and up [E, I, H] stacks -> one PackedGateUp buffer (tile pairs, gate/up adjacent)."""
    _need(w_gate, "w_gate", dim=3)
    _need(w_up, "w_up", w_gate.dtype, 3)
    if w_up.shape != w_gate.shape:
        raise ValueError("w_gate and w_up must have the same shape [E, I, H]")
    E, I, H = w_gate.shape
    code = _dtype_code(w_gate)
    n = int(lib().acceptmoe_packed_gate_up_bytes(code, E, I, H))
    if n == 0:
        raise ValueError(f"unsupported gate/up shape {tuple(w_gate.shape)}")
    data = torch.empty(n // w_gate.element_size(), dtype=w_gate.dtype, device=w_gate.device)
    check(lib().acceptmoe_pack_gate_up_weights(_ptr(w_gate), _ptr(w_up), code, E, I, H, _ptr(data),
                                               _stream_ptr(stream)))
    return PackedGateUp(data, E, I, H)


def forward_workspace(T: int, H: int, I: int, E: int, k: int, dtype: torch.dtype, device) -> torch.Tensor:
    code = L.BF16 if dtype == torch.bfloat16 else L.F32
    n = lib().acceptmoe_moe_forward_workspace_size(T, H, I, E, k, code)
    return torch.empty(max(int(n), 256), dtype=torch.uint8, device=device)


def moe_forward(hidden: torch.Tensor, w_gate_up: PackedGateUp, w_down_p: torch.Tensor,
                topk_idx: torch.Tensor, topk_gate: torch.Tensor, out: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Grouped SwiGLU expert FFN over packed weights (acceptmoe_moe_forward) -> [T, H] fp32."""
    _need(hidden, "hidden", dim=2)
    if not isinstance(w_gate_up, PackedGateUp):
        raise TypeError("w_gate_up must come from pack_gate_up_weights")
    _need(w_gate_up.data, "w_gate_up", hidden.dtype, 1)
    _need(w_down_p, "w_down", hidden.dtype, 3)
    _need(topk_idx, "topk_idx", torch.int32, 2)
    _need(topk_gate, "topk_gate", torch.float32, 2)
    T, H = hidden.shape
    E, I = w_gate_up.E, w_gate_up.I
    k = topk_idx.shape[1]
    if w_gate_up.H != H or tuple(w_down_p.shape) != (E, H, I):
        raise ValueError("weights must be gate/up packed from [E, I, H] stacks and down [E, H, I]")
    if tuple(topk_idx.shape) != (T, k) or tuple(topk_gate.shape) != (T, k):
        raise ValueError("topk_idx / topk_gate must be [T, k]")
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32, device=hidden.device)
    if workspace is None:
        workspace = forward_workspace(T, H, I, E, k, hidden.dtype, hidden.device)
    check(lib().acceptmoe_moe_forward(
        _ptr(hidden), _dtype_code(hidden), _ptr(w_gate_up.data), _ptr(w_down_p), T, H, I, E, k,
        _ptr(topk_idx), _ptr(topk_gate), _ptr(out), _ptr(workspace), workspace.numel(), _stream_ptr(stream)))
    return out


# ---------------------------------------------------------------------------
class VerifyLayer:
    """One MoE layer with packed expert weights and preallocated workspaces.

    step() runs route -> select -> forward for one verification block on the
    current stream, allocating nothing.
    """

    def __init__(self, router_w: torch.Tensor, w_gate: torch.Tensor, w_up: torch.Tensor,
                 w_down: torch.Tensor, k: int, max_tokens: int, max_trees: int = 1, beta: float = 0.5,
                 mode: int = L.MODE_SELF_SIZING, budget: int = 0, removal_cap: int = -1):
        self.router_w = router_w  # [E, H] fp32, kept for reference checks
        self.router = pack_router_weights(router_w)
        self.E, self.I, self.H = w_gate.shape
        self.k, self.beta, self.mode, self.budget, self.removal_cap = k, beta, mode, budget, removal_cap
        self.dtype = w_gate.dtype
        self.wgu = pack_gate_up_weights(w_gate, w_up)
        self.wd = pack_expert_weights(w_down)
        self._alloc(max_tokens, max_trees, w_gate.device)

    def _alloc(self, max_tokens: int, max_trees: int, dev):
        T, k = max_tokens, self.k
        self.max_tokens, self.max_trees = max_tokens, max_trees
        self.logits = torch.empty((T, self.E), dtype=torch.float32, device=dev)
        self.sel_ws = select_workspace(T, self.E, k, dev)
        self.fwd_ws = forward_workspace(T, self.H, self.I, self.E, k, self.dtype, dev)
        self.sel_out = {
            "eligible": torch.empty((max_trees, self.E), dtype=torch.uint8, device=dev),
            "idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "gate": torch.empty((T, k), dtype=torch.float32, device=dev),
            "stats": torch.empty((max_trees, L.NUM_STATS), dtype=torch.int32, device=dev),
        }
        self.out = torch.empty((T, self.H), dtype=torch.float32, device=dev)

    def twin(self) -> "VerifyLayer":
        """The same layer (shared packed weights) with its own workspaces and
        outputs, for a second block in flight on another stream."""
        other = copy.copy(self)
        other._alloc(self.max_tokens, self.max_trees, self.logits.device)
        return other

    def step(self, hidden, parent, depth, prob, tree_offsets=None, resident=None, stream=None):
        T = hidden.shape[0]
        B = 1 if tree_offsets is None else len(tree_offsets) - 1
        logits = self.logits[:T]
        route(hidden, self.router, out=logits, stream=stream)
        outs = {"eligible": self.sel_out["eligible"][:B], "idx": self.sel_out["idx"][:T],
                "gate": self.sel_out["gate"][:T], "stats": self.sel_out["stats"][:B]}
        select(logits, parent, depth, prob, tree_offsets, self.k, self.beta, self.mode, self.budget,
               self.removal_cap, resident, workspace=self.sel_ws, outputs=outs, stream=stream)
        out = self.out[:T]
        moe_forward(hidden, self.wgu, self.wd, outs["idx"], outs["gate"], out=out,
                    workspace=self.fwd_ws, stream=stream)
        return logits, outs, out


def residual_add(hidden: torch.Tensor, y: torch.Tensor, out: torch.Tensor | None = None,
                 stream=None) -> torch.Tensor:
    """out = hidden + y rounded to hidden's dtype (acceptmoe_residual_add)."""
    _need(hidden, "hidden", dim=2)
    _need(y, "y", torch.float32, 2)
    if y.shape != hidden.shape:
        raise ValueError("residual_add: hidden and y must have the same shape")
    if out is None:
        out = torch.empty_like(hidden)
    T, H = hidden.shape
    check(lib().acceptmoe_residual_add(_ptr(hidden), _dtype_code(hidden), _ptr(y), T, H, _ptr(out),
                                       _stream_ptr(stream)))
    return out


class VerifyStack:
    """Verify layers chained by the residual stream, h_{l+1} = h_l + y_l rounded
    to the layer dtype (attention between the MoE layers is not modelled).

    step() runs route -> select -> forward -> residual add for every layer on
    one stream and allocates nothing, so a whole pass can be captured in one
    HIP graph.  The input of every layer stays in `h[l]` and each layer's
    logits, routing and output in its own buffers (for teacher-forced checks).
    """

    def __init__(self, layers: list, max_tokens: int):
        self.layers = layers
        dev = layers[0].logits.device
        self.h = [torch.empty((max_tokens, layers[0].H), dtype=layers[0].dtype, device=dev)
                  for _ in range(len(layers) + 1)]

    def twin(self) -> "VerifyStack":
        """Same weights, own buffers (a second block in flight)."""
        return VerifyStack([ly.twin() for ly in self.layers], self.h[0].shape[0])

    def step(self, h0, parent, depth, prob, tree_offsets=None, stream=None) -> torch.Tensor:
        T = h0.shape[0]
        if h0.data_ptr() != self.h[0].data_ptr():
            with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
                self.h[0][:T].copy_(h0)
        for l, layer in enumerate(self.layers):
            _, _, y = layer.step(self.h[l][:T], parent, depth, prob, tree_offsets, stream=stream)
            residual_add(self.h[l][:T], y, out=self.h[l + 1][:T], stream=stream)
        return self.h[len(self.layers)][:T]


# ---------------------------------------------------------------------------
# physical expert offload (acceptmoe_pool_*, acceptmoe_copy_rows)
# ---------------------------------------------------------------------------
def _host_ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


class OffloadPool:
    """X-slot expert pool of one layer: LRU state in host memory (the library's),
    X packed expert slots in device memory, and the layer's E packed experts in
    pinned host memory.  Built without weights it keeps only the books (routing
    to slots, hits, misses, host-to-device bytes) and copies nothing."""

    def __init__(self, X: int, E: int, w_gate: torch.Tensor | None = None, w_up: torch.Tensor | None = None,
                 w_down: torch.Tensor | None = None, expert_bytes: int = 0):
        n = int(lib().acceptmoe_pool_state_bytes(X, E))
        if n == 0:
            raise ValueError(f"unsupported pool X={X} E={E}")
        self._state = np.zeros((n + 7) // 8, np.int64)  # 8-byte aligned
        check(lib().acceptmoe_pool_init(_host_ptr(self._state), n, X, E))
        self.X, self.E = X, E
        self.stats = np.zeros(L.POOL_NUM_STATS, np.int64)
        self.physical = w_gate is not None
        self.gu_bytes, self.dn_bytes = 0, 0
        if self.physical:
            gu = pack_gate_up_weights(w_gate, w_up)
            dn = pack_expert_weights(w_down)
            torch.cuda.synchronize()
            self.dtype, self.I, self.H = w_gate.dtype, w_gate.shape[1], w_gate.shape[2]
            gub = gu.data.view(torch.uint8)
            dnb = dn.view(torch.uint8).reshape(-1)
            self.gu_bytes, self.dn_bytes = gub.numel() // E, dnb.numel() // E
            # the full stacks live in pinned host memory; the device copies are dropped
            self.host_gu = torch.empty(gub.numel(), dtype=torch.uint8, pin_memory=True)
            self.host_dn = torch.empty(dnb.numel(), dtype=torch.uint8, pin_memory=True)
            self.host_gu.copy_(gub)
            self.host_dn.copy_(dnb)
            del gu, dn, gub, dnb
            dev = w_gate.device
            self.pool_gu = torch.empty(X * self.gu_bytes, dtype=torch.uint8, device=dev)
            self.pool_dn = torch.empty(X * self.dn_bytes, dtype=torch.uint8, device=dev)
            self.gate_up = PackedGateUp(self.pool_gu.view(self.dtype), X, self.I, self.H)
            self.down = self.pool_dn.view(self.dtype).view(X, self.H, self.I)
        self.expert_bytes = (self.gu_bytes + self.dn_bytes) if self.physical else int(expert_bytes)

    def resident_mask(self) -> np.ndarray:
        m = np.zeros(self.E, np.uint8)
        check(lib().acceptmoe_pool_resident_mask(_host_ptr(self._state), _host_ptr(m)))
        return m

    def plan_waves(self, idx: np.ndarray):
        idx = np.ascontiguousarray(idx, np.int32)
        T, k = idx.shape
        wave_of = np.zeros(max(T, 1), np.int32)
        n = ctypes.c_int32(0)
        check(lib().acceptmoe_pool_plan_waves(_host_ptr(idx), T, k, self.E, self.X, _host_ptr(wave_of),
                                              ctypes.byref(n)))
        return wave_of[:T], int(n.value)

    def serve_wave(self, idx: np.ndarray, wave_of: np.ndarray, wave: int, stream=None) -> np.ndarray:
        """Loads the wave's missing experts (stream-ordered) and returns its routing rewritten to slots."""
        idx = np.ascontiguousarray(idx, np.int32)
        wave_of = np.ascontiguousarray(wave_of, np.int32)
        T, k = idx.shape
        slot = np.full((max(T, 1), k), -1, np.int32)
        if self.physical:
            ptrs = (_ptr(self.host_gu), _ptr(self.host_dn), _ptr(self.pool_gu), _ptr(self.pool_dn))
            gub, dnb, s = self.gu_bytes, self.dn_bytes, _stream_ptr(stream)
        else:
            ptrs = (ctypes.c_void_p(0),) * 4
            gub, dnb, s = self.expert_bytes, 0, ctypes.c_void_p(0)
        check(lib().acceptmoe_pool_serve_wave(_host_ptr(self._state), _host_ptr(idx), _host_ptr(wave_of), wave, T, k,
                                              *ptrs, gub, dnb, _host_ptr(slot), _host_ptr(self.stats), s))
        return slot[:T]


def copy_rows(src: torch.Tensor, dst: torch.Tensor, row_tag: torch.Tensor, tag: int, stream=None):
    """dst[t] = src[t] where row_tag[t] == tag (acceptmoe_copy_rows)."""
    _need(src, "src", torch.float32, 2)
    _need(dst, "dst", torch.float32, 2)
    _need(row_tag, "row_tag", torch.int32, 1)
    T, H = src.shape
    if tuple(dst.shape) != (T, H) or row_tag.shape[0] != T:
        raise ValueError("copy_rows: shapes must match")
    check(lib().acceptmoe_copy_rows(_ptr(src), _ptr(dst), _ptr(row_tag), int(tag), T, H, _stream_ptr(stream)))


def stream_read(src: torch.Tensor, nbytes: int, sink: torch.Tensor, grid: int, stream=None):
    """Streams the first nbytes of the device tensor src with `grid`
    workgroups, one checksum word each into sink (acceptmoe_stream_read; a
    measurement of the attainable HBM read rate)."""
    if not src.is_cuda or not sink.is_cuda or sink.dtype != torch.int32 or sink.numel() < grid:
        raise ValueError("stream_read: src and an int32 sink of >= grid words on the GPU")
    if nbytes > src.numel() * src.element_size():
        raise ValueError("stream_read: nbytes exceeds src")
    check(lib().acceptmoe_stream_read(_ptr(src), int(nbytes), _ptr(sink), int(grid), _stream_ptr(stream)))


class OffloadLayer:
    """One MoE layer served from an X-slot pool (Sec. 3.4 offload paragraph).

    step(): route -> select with the pool's resident set as mask -> routing
    copied to the host -> waves planned -> per wave: missing experts loaded
    into slots, routing rewritten to slots, forward over the pool (E = X) ->
    wave outputs joined.  The host round trip after selection is the
    synchronous decision point of the offload path."""

    def __init__(self, router_w: torch.Tensor, w_gate: torch.Tensor, w_up: torch.Tensor, w_down: torch.Tensor,
                 k: int, X: int, max_tokens: int, beta: float = 0.5, mode: int = L.MODE_SELF_SIZING,
                 budget: int = 0, removal_cap: int = -1):
        self.router = pack_router_weights(router_w)
        self.E, self.I, self.H = w_gate.shape
        self.k, self.X, self.beta, self.mode, self.budget, self.removal_cap = k, X, beta, mode, budget, removal_cap
        self.pool = OffloadPool(X, self.E, w_gate, w_up, w_down)
        dev = w_gate.device
        T = max_tokens
        self.logits = torch.empty((T, self.E), dtype=torch.float32, device=dev)
        self.sel_ws = select_workspace(T, self.E, k, dev)
        self.sel_out = {
            "eligible": torch.empty((1, self.E), dtype=torch.uint8, device=dev),
            "idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "gate": torch.empty((T, k), dtype=torch.float32, device=dev),
            "stats": torch.empty((1, L.NUM_STATS), dtype=torch.int32, device=dev),
        }
        self.mask = torch.empty(self.E, dtype=torch.uint8, device=dev)
        self.slot_idx = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.wave_tag = torch.empty(T, dtype=torch.int32, device=dev)
        self.fwd_ws = forward_workspace(T, self.H, self.I, X, k, w_gate.dtype, dev)
        self.out = torch.empty((T, self.H), dtype=torch.float32, device=dev)
        self.out_wave = torch.empty((T, self.H), dtype=torch.float32, device=dev)

    def step(self, hidden, parent, depth, prob):
        """One block (one tree) through the layer on the current stream; returns (outs, out, wave_of)."""
        T = hidden.shape[0]
        logits = self.logits[:T]
        route(hidden, self.router, out=logits)
        self.mask.copy_(torch.from_numpy(self.pool.resident_mask()))
        outs = {"eligible": self.sel_out["eligible"], "idx": self.sel_out["idx"][:T],
                "gate": self.sel_out["gate"][:T], "stats": self.sel_out["stats"]}
        select(logits, parent, depth, prob, None, self.k, self.beta, self.mode, self.budget, self.removal_cap,
               self.mask, workspace=self.sel_ws, outputs=outs)
        idx = outs["idx"].cpu().numpy()
        wave_of, nw = self.pool.plan_waves(idx)
        out = self.out[:T]
        if nw > 1:
            self.wave_tag[:T].copy_(torch.from_numpy(wave_of))
        for w in range(nw):
            slot = self.pool.serve_wave(idx, wave_of, w)
            self.slot_idx[:T].copy_(torch.from_numpy(slot))
            target = out if nw == 1 else self.out_wave[:T]
            moe_forward(hidden, self.pool.gate_up, self.pool.down, self.slot_idx[:T], outs["gate"], out=target,
                        workspace=self.fwd_ws)
            if nw > 1:
                copy_rows(target, out, self.wave_tag[:T], w)
        return outs, out, wave_of


# ---------------------------------------------------------------------------
# offline commitment estimator (acceptmoe_commit_*)
# ---------------------------------------------------------------------------
class CommitEstimator:
    """Accumulates m_d / c_d over verification traces and turns them into the
    p_hat table (Sec. 3.2); host arrays, the library does the counting."""

    def __init__(self, D: int):
        self.D = D
        self.m = np.zeros(D, np.int64)
        self.c = np.zeros(D, np.int64)

    def add(self, depth, on_path):
        depth = np.ascontiguousarray(depth, np.int32)
        on_path = np.ascontiguousarray(on_path, np.uint8)
        check(lib().acceptmoe_commit_count(_host_ptr(depth), _host_ptr(on_path), len(depth), self.D,
                                           _host_ptr(self.m), _host_ptr(self.c)))

    def estimate(self) -> np.ndarray:
        p = np.zeros(self.D, np.float32)
        check(lib().acceptmoe_commit_estimate(_host_ptr(self.m), _host_ptr(self.c), self.D, _host_ptr(p)))
        return p


def commit_expand(p_hat: torch.Tensor, depth: torch.Tensor, out: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """Per-node commitment probabilities p_t = p_hat[d_t] on the device (acceptmoe_commit_expand)."""
    _need(p_hat, "p_hat", torch.float32, 1)
    _need(depth, "depth", torch.int32, 1)
    if out is None:
        out = torch.empty(depth.shape[0], dtype=torch.float32, device=depth.device)
    check(lib().acceptmoe_commit_expand(_ptr(p_hat), p_hat.shape[0], _ptr(depth), depth.shape[0], _ptr(out),
                                        _stream_ptr(stream)))
    return out
