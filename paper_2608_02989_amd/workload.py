"""Seeded synthetic inputs for verify-block MoE layers.

This module draws inputs only -- draft trees, hidden states, router and expert
weights, commitment probabilities and residency masks.  It holds none of the
selection or FFN arithmetic, so both the HIP path and the CPU oracle can be fed
from it.

Workload recipe (the paper evaluates real Qwen3-30B-A3B / GPT-OSS targets with
EAGLE-3 trees of 64 draft tokens, 5 draft steps, top-k 10 (Sec. 4); none of
those models or datasets is used here, seeded synthetic blocks of the same
shape stand in for them):

* tree: breadth-first expansion from the root; every popped node below the
  depth limit draws 1..4 children uniformly until T nodes exist, so nodes come
  in BFS order (parent[t] < t) and sibling ranks are 0-based child order.
* hidden states: root ~ N(0, s^2); a child is rho * parent + sqrt(1-rho^2) * eps
  (still marginally N(0, s^2)).  rho = 0.9 is the tree-correlated regime whose
  eligible-set sizes land near the paper's 23..34 experts; rho = 0 is the
  i.i.d. reading of the configuration text.
* router weights fp32 N(0, 0.02^2); expert weights N(0, 0.02^2) in the layer
  dtype (bf16 rounding is round-to-nearest-even by torch).
* commitment probabilities: per-depth p_d = 0.7^d * U(0.8, 1) expanded per node
  (small fp32 layer) or p_t = 0.75^d * 0.6^r with sibling rank r.
* residency mask: a fixed fraction of experts drawn without replacement.

Random streams: numpy ``default_rng(SeedSequence([cfg, block, layer, stream]))``
for small arrays; large weights use a seeded ``torch.Generator`` on the target
device (then copied to the host where the oracle needs them).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

STREAM_TREE, STREAM_HIDDEN, STREAM_ROUTER, STREAM_EXPERTS, STREAM_COMMIT, STREAM_MASK, STREAM_TRACE = range(7)


@dataclass(frozen=True)
class LayerConfig:
    name: str
    cfg_id: int
    dtype: str              # "f32" or "bf16" (expert weights and hidden states)
    T: int                  # nodes per tree
    B: int                  # trees per call
    H: int
    E: int
    k: int
    I: int
    depth_max: int
    commit_rule: str        # "per_depth_0.7" or "depth_sibling"
    hidden_std: float
    weight_std: float = 0.02
    router_std: float = 0.02
    resident_frac: float = 0.0
    layers: int = 1
    blocks: int = 1
    branch: tuple = (1, 4)
    extra: dict = field(default_factory=dict)

    @property
    def total_tokens(self) -> int:
        return self.T * self.B

    @property
    def wbytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def expert_bytes(self) -> int:
        """Bytes of one expert's gate, up and down matrices."""
        return 3 * self.H * self.I * self.wbytes


CONFIGS = {
    "fp32_small": LayerConfig("fp32_small", 1, "f32", T=8, B=1, H=256, E=16, k=2, I=128,
                              depth_max=3, commit_rule="per_depth_0.7", hidden_std=0.02),
    "qwen3_30b_a3b": LayerConfig("qwen3_30b_a3b", 2, "bf16", T=32, B=1, H=2048, E=128, k=8,
                                 I=768, depth_max=6, commit_rule="depth_sibling",
                                 hidden_std=1.0),
    "qwen3_30b_a3b_x48": LayerConfig("qwen3_30b_a3b_x48", 3, "bf16", T=60, B=1, H=2048, E=128,
                                     k=8, I=768, depth_max=8, commit_rule="depth_sibling",
                                     hidden_std=1.0, layers=48, blocks=256),
    "wide_offload": LayerConfig("wide_offload", 4, "bf16", T=64, B=1, H=4096, E=128, k=8,
                                I=1536, depth_max=8, commit_rule="depth_sibling",
                                hidden_std=1.0, resident_frac=0.25),
    "batched_8x64": LayerConfig("batched_8x64", 5, "bf16", T=64, B=8, H=4096, E=128, k=8,
                                I=1536, depth_max=8, commit_rule="depth_sibling",
                                hidden_std=1.0),
}


def rng_for(cfg_id: int, block: int, layer: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg_id, block, layer, stream]))


def torch_seed(cfg_id: int, block: int, layer: int, stream: int) -> int:
    return int(np.random.SeedSequence([cfg_id, block, layer, stream]).generate_state(1, np.uint64)[0]
               & 0x7FFFFFFFFFFFFFFF)


# ---------------------------------------------------------------------------
# draft trees
# ---------------------------------------------------------------------------
def make_tree(rng: np.random.Generator, T: int, depth_max: int, branch=(1, 4)):
    """BFS-ordered draft tree: (parent[T] int32 with -1 root, depth[T], sibling_rank[T])."""
    if T <= 0:
        z = np.zeros(0, np.int32)
        return z, z.copy(), z.copy()
    while True:
        parent, depth, sib = [-1], [0], [0]
        head = 0
        while len(parent) < T and head < len(parent):
            node = head
            head += 1
            if depth[node] >= depth_max:
                continue
            nb = int(rng.integers(branch[0], branch[1] + 1))
            for c in range(nb):
                if len(parent) >= T:
                    break
                parent.append(node)
                depth.append(depth[node] + 1)
                sib.append(c)
        if len(parent) == T:
            return (np.asarray(parent, np.int32), np.asarray(depth, np.int32),
                    np.asarray(sib, np.int32))


def chain(T: int):
    """A draft chain: node t has parent t-1 and depth t."""
    parent = np.arange(-1, T - 1, dtype=np.int32)
    depth = np.arange(T, dtype=np.int32)
    return parent, depth, np.zeros(T, np.int32)


def commit_probs(rng: np.random.Generator, rule: str, depth, sib) -> np.ndarray:
    depth = np.asarray(depth)
    if rule == "per_depth_0.7":
        dmax = int(depth.max()) if depth.size else 0
        table = np.array([0.7 ** d * rng.uniform(0.8, 1.0) for d in range(dmax + 1)])
        return table[depth].astype(np.float32)
    if rule == "depth_sibling":
        return (0.75 ** depth.astype(np.float64) * 0.6 ** np.asarray(sib, np.float64)).astype(np.float32)
    raise ValueError(rule)


def accepted_prefix(rng: np.random.Generator, parent, sib, q=(0.55, 0.2, 0.1, 0.05)) -> np.ndarray:
    """Synthetic verification outcome of one draft tree (or chain): starting at
    the root, the verifier takes the child of sibling rank r with probability
    q[r] (nothing with the remaining mass) and continues from it.  Returns a
    0/1 mask of the nodes on the accepted output prefix (the root included).
    One uniform draw per visited node; a node's marginal chance to be on the
    prefix is the product of q over the ranks along its path."""
    T = len(parent)
    on = np.zeros(T, np.uint8)
    if T == 0:
        return on
    kids = [[] for _ in range(T)]
    for t in range(T):
        if parent[t] >= 0:
            kids[int(parent[t])].append(t)
    node = 0
    on[0] = 1
    while kids[node]:
        u = rng.random()
        nxt, acc = -1, 0.0
        for c in sorted(kids[node], key=lambda c: sib[c]):
            r = int(sib[c])
            acc += q[r] if r < len(q) else 0.0
            if u < acc:
                nxt = c
                break
        if nxt < 0:
            break
        on[nxt] = 1
        node = nxt
    return on


def correlated_hidden(rng: np.random.Generator, parent, H: int, std: float, rho: float,
                      root=None) -> np.ndarray:
    """fp32 hidden states along the tree: child = rho*parent + sqrt(1-rho^2)*eps.

    root: optional unit-variance state [H] for the root (default: a fresh draw)."""
    T = len(parent)
    h = np.empty((T, H), np.float64)
    c = np.sqrt(max(0.0, 1.0 - rho * rho))
    for t in range(T):
        eps = rng.standard_normal(H)
        p = int(parent[t])
        if p < 0:
            h[t] = eps if root is None else root
        else:
            h[t] = rho * h[p] + c * eps
    return (h * std).astype(np.float32)


def trace_roots(cfg: LayerConfig, layer: int, n_blocks: int, rho_step: float) -> np.ndarray:
    """Unit-variance root states of consecutive blocks of a decode trace on one
    layer: root_b = rho_step * root_{b-1} + sqrt(1 - rho_step^2) * eps_b, so
    consecutive blocks route alike (the temporal locality an expert cache
    feeds on); rho_step = 0 makes blocks independent."""
    rng = rng_for(cfg.cfg_id, 0, layer, STREAM_TRACE)
    c = np.sqrt(max(0.0, 1.0 - rho_step * rho_step))
    out = np.empty((n_blocks, cfg.H), np.float64)
    r = rng.standard_normal(cfg.H)
    for b in range(n_blocks):
        if b > 0:
            r = rho_step * r + c * rng.standard_normal(cfg.H)
        out[b] = r
    return out


# ---------------------------------------------------------------------------
# a whole block: trees + probabilities + hidden states (+ mask)
# ---------------------------------------------------------------------------
@dataclass
class Block:
    parent: np.ndarray       # [T_total] int32, global ids, -1 for roots
    depth: np.ndarray        # [T_total] int32
    sib: np.ndarray          # [T_total] int32
    prob: np.ndarray         # [T_total] float32
    offsets: np.ndarray      # [B+1] int32
    hidden: np.ndarray       # [T_total, H] float32 (round to bf16 by the caller if needed)
    resident: np.ndarray | None  # [E] uint8 or None


def make_block(cfg: LayerConfig, block: int = 0, layer: int = 0, rho: float = 0.9,
               T: int | None = None, B: int | None = None, tree_layer: int | None = None,
               root=None) -> Block:
    """Trees, probabilities, hidden states (and mask) of one verification block.

    tree_layer selects the seed of the tree structure (default: layer); a
    block seen by every layer of a stack keeps one tree (tree_layer = 0) while
    each layer draws its own hidden states.  root: optional unit-variance root
    state (one tree; see trace_roots).
    """
    T = cfg.T if T is None else T
    B = cfg.B if B is None else B
    tl = layer if tree_layer is None else tree_layer
    parents, depths, sibs, probs, hid = [], [], [], [], []
    offsets = [0]
    for b in range(B):
        rt = rng_for(cfg.cfg_id, block, tl * 1000 + b, STREAM_TREE)
        par, dep, sib = make_tree(rt, T, cfg.depth_max, cfg.branch)
        pr = commit_probs(rng_for(cfg.cfg_id, block, tl * 1000 + b, STREAM_COMMIT),
                          cfg.commit_rule, dep, sib)
        hs = correlated_hidden(rng_for(cfg.cfg_id, block, layer * 1000 + b, STREAM_HIDDEN),
                               par, cfg.H, cfg.hidden_std, rho, root=root if b == 0 else None)
        base = offsets[-1]
        parents.append(np.where(par < 0, -1, par + base).astype(np.int32))
        depths.append(dep)
        sibs.append(sib)
        probs.append(pr)
        hid.append(hs)
        offsets.append(base + T)
    resident = None
    if cfg.resident_frac > 0.0:
        rm = rng_for(cfg.cfg_id, block, layer, STREAM_MASK)
        n_res = int(round(cfg.resident_frac * cfg.E))
        resident = np.zeros(cfg.E, np.uint8)
        resident[rm.choice(cfg.E, size=n_res, replace=False)] = 1
    cat = (lambda xs, dt: np.concatenate(xs).astype(dt)) if B else (lambda xs, dt: np.zeros(0, dt))
    return Block(parent=cat(parents, np.int32), depth=cat(depths, np.int32), sib=cat(sibs, np.int32),
                 prob=cat(probs, np.float32), offsets=np.asarray(offsets, np.int32),
                 hidden=(np.concatenate(hid) if B else np.zeros((0, cfg.H), np.float32)),
                 resident=resident)


def router_weights(cfg: LayerConfig, layer: int = 0) -> np.ndarray:
    rng = rng_for(cfg.cfg_id, 0, layer, STREAM_ROUTER)
    return (rng.standard_normal((cfg.E, cfg.H)) * cfg.router_std).astype(np.float32)


# ---------------------------------------------------------------------------
# expert weights (torch, any device)
# ---------------------------------------------------------------------------
def expert_weights_torch(cfg: LayerConfig, layer: int = 0, device="cpu", E: int | None = None):
    """(w_gate [E,I,H], w_up [E,I,H], w_down [E,H,I]) in the layer dtype, seeded per layer."""
    import torch
    E = cfg.E if E is None else E
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    out = []
    for i, shape in enumerate(((E, cfg.I, cfg.H), (E, cfg.I, cfg.H), (E, cfg.H, cfg.I))):
        g = torch.Generator(device=device)
        g.manual_seed(torch_seed(cfg.cfg_id, 0, layer * 8 + i, STREAM_EXPERTS))
        w = torch.empty(shape, dtype=torch.float32, device=device)
        # fill expert by expert to bound the fp32 staging memory
        for e in range(E):
            w[e].normal_(0.0, cfg.weight_std, generator=g)
        out.append(w.to(dt))
        del w
    return tuple(out)


def to_bits(t) -> np.ndarray:
    """Host copy of a torch tensor for the oracle: bf16 -> uint16 bits, fp32 -> float32."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (host-side input preparation)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16) \
        .view(torch.int16).numpy().view(np.uint16)
