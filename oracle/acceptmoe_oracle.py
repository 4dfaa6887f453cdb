"""Plain, slow, fp64 CPU oracle for the AcceptMoE verify-block MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library.

The method is "AcceptMoE: Commitment-Weighted Self-Sizing Verifier Expert
Sets for Efficient MoE Speculative Decoding" (arXiv 2608.02989).  Every step
below cites the section / equation of that paper it follows:

  Sec. 3.1  router distribution r_t = softmax(z_t), natural top-k K_t,
            natural union (Eq. 1), constrained routing (Eq. 2)
  Sec. 3.2  token importance alpha_t (Eq. 3), utility u_e (Eq. 4)
  Sec. 3.3  root anchor A (Eq. 5), effective-rank cardinality (Eq. 6),
            minimum set size |S| >= k, zero-residual rule
  Sec. 3.4  votes v_e, rerouting budget a(S), longest-prefix removal (Eq. 7)

Where the method reduces to a plain definition (top-k by rank, softmax, the
SwiGLU expert FFN) the definition is written out directly; the selection rule
itself is a heuristic and is followed step by step in the paper's order.

Readings of points the paper leaves open (each one is also listed in the
design notes of the repository):
  R1  r in Eq. 4 is the full softmax over all E experts, masked by e in K_t.
  R2  TopK ranks fp32 logits z (equivalent to ranking r in exact arithmetic);
      equal logits are broken toward the lower expert index, everywhere.
  R3  demand, entropy and gates are evaluated in fp64.
  R4  n_er = ceil(exp(H) - 1e-9), clamped to [1, #{e in R : u_e > 0}], so an
      exactly uniform demand over m experts gives m; Z = 0 gives n_er = 0.
  R6  the minimum-size fill takes the next experts of R in (u desc, index asc)
      order.
  R7  anchor tokens are the depth-0 nodes of each tree.
  R8  commitment probabilities arrive per node (p_t); a per-depth table is
      expanded by p_t = p_hat[d_t] by the caller.  N_d counts nodes by depth.
  R9  native post-top-k weighting = softmax over the k selected logits
      (Qwen3-style renormalisation).
  R10 pruning may remove nonresident anchor experts (Fig. 2 caption).
  R11 several independent trees in one call each get their own S'; the
      residency mask is shared.
  R12 the removal cap defaults to E (nonbinding).
  R13 the fixed-budget rows (AcceptMoE-B, MoE-Spec, Count-B) take |S| = B;
      AcceptMoE-B keeps the anchor and fills with the top of R by u;
      MoE-Spec ranks every expert by sum_t r_{t,e}; Count-B ranks by v_e;
      both baselines break ties toward the lower index, keep no anchor and
      are never pruned (residency pruning is a stage of AcceptMoE only).
"""
from __future__ import annotations

import itertools
import math

import numpy as np

# ---------------------------------------------------------------------------
# status codes written into stats[..., CODE]; identical meaning in the library
# ---------------------------------------------------------------------------
TREE_OK = 0
TREE_EMPTY = 1          # a tree with no node
TREE_BAD_ROOT = 2       # first node of a tree is not a root (parent -1, depth 0)
TREE_BAD_PARENT = 3     # a later node has no parent inside the tree before it
TREE_BAD_DEPTH = 4      # depth[t] != depth[parent[t]] + 1 (or out of range)
TREE_BAD_PROB = 5       # a commitment probability is negative or not finite

MODE_SELF_SIZING = 0    # AcceptMoE (Sec. 3.3)
MODE_ALL_EXPERTS = 1    # S = [E]: Standard SD / natural routing (Sec. 3.1)
MODE_FIXED_BUDGET = 2   # AcceptMoE-B: same utility and anchor, |S| = B (Sec. 4)
MODE_MOESPEC = 3        # MoE-Spec baseline: top-B by summed router mass (Sec. 4)
MODE_COUNT = 4          # Count-B baseline: top-B by natural votes (Sec. 4)

# stats columns
ST_T, ST_A, ST_NER, ST_S, ST_SP, ST_UNAT, ST_BUDGET, ST_MSTAR, ST_CODE, ST_ROUTED = range(10)
N_STATS = 10

EPS_CEIL = 1e-9         # reading R4
AMBIG_REL = 1e-10       # relative margin below which a decision is reported ambiguous


# ---------------------------------------------------------------------------
# number formats
# ---------------------------------------------------------------------------
def widen_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp64 values (bf16 is the top half of fp32)."""
    b = np.asarray(bits).astype(np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def as_f64(x, dtype: str) -> np.ndarray:
    """Operand in fp64: dtype 'bf16' means uint16 bit patterns, 'f32' means float32."""
    if dtype == "bf16":
        return widen_bf16(x)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Sec. 3.1: router
# ---------------------------------------------------------------------------
def route(hidden64: np.ndarray, router_w64: np.ndarray) -> np.ndarray:
    """Router logits z_t = W_r h_t for every node t (Sec. 3.1), exact-ish in fp64."""
    return np.asarray(hidden64, np.float64) @ np.asarray(router_w64, np.float64).T


def softmax64(z_row) -> np.ndarray:
    """r_t = softmax(z_t) in fp64 from fp32 logits (Sec. 3.1, reading R3)."""
    z = np.asarray(z_row, dtype=np.float32).astype(np.float64)
    m = z.max()
    w = np.exp(z - m)
    return w / w.sum()


def topk_by_rank(z_row, k: int, eligible=None) -> np.ndarray:
    """TopK_k as a rank count over fp32 logits (Sec. 3.1 Eq. 2, readings R2).

    Expert e is selected iff fewer than k eligible experts j beat it, where j
    beats e when z_j > z_e, or z_j == z_e and j < e.  Returns the selected
    experts in slot order: by that rank, i.e. (z desc, index asc).  With an
    eligibility mask this is TopK_k(z_t + M_S) of Eq. 2: experts outside S
    have logit -inf and are never chosen.
    """
    z = np.asarray(z_row, dtype=np.float32)
    E = z.shape[0]
    elig = np.ones(E, dtype=bool) if eligible is None else np.asarray(eligible, dtype=bool)
    cand = np.flatnonzero(elig)
    zc = z[cand]
    beats = (zc[None, :] > zc[:, None]) | ((zc[None, :] == zc[:, None])
                                             & (cand[None, :] < cand[:, None]))
    rank = beats.sum(axis=1)
    chosen = rank < k
    order = np.argsort(rank[chosen], kind="stable")
    return cand[chosen][order]


# ---------------------------------------------------------------------------
# tree checks (the block structure of Sec. 3.1: parents precede children)
# ---------------------------------------------------------------------------
def validate_tree(parent, depth, prob) -> int:
    """Smallest error code that applies to one tree (local node ids 0..T_b-1).

    parent may be None (then only depth ranges are checked).
    """
    Tb = len(depth)
    if Tb == 0:
        return TREE_EMPTY
    codes = []
    for t in range(Tb):
        d = int(depth[t])
        if t == 0:
            if d != 0 or (parent is not None and int(parent[0]) != -1):
                codes.append(TREE_BAD_ROOT)
            continue
        if parent is not None:
            p = int(parent[t])
            if p < 0 or p >= t:
                codes.append(TREE_BAD_PARENT)
            elif d != int(depth[p]) + 1:
                codes.append(TREE_BAD_DEPTH)
        else:
            if d < 1 or d >= Tb:
                codes.append(TREE_BAD_DEPTH)
    for t in range(Tb):
        pt = float(prob[t])
        if not math.isfinite(pt) or pt < 0.0:
            codes.append(TREE_BAD_PROB)
    return min(codes) if codes else TREE_OK


# ---------------------------------------------------------------------------
# Sec. 3.2: commitment-weighted demand
# ---------------------------------------------------------------------------
def depth_counts(depth) -> dict:
    """N_d = number of block tokens at draft position d (Sec. 3.2)."""
    counts: dict = {}
    for d in depth:
        counts[int(d)] = counts.get(int(d), 0) + 1
    return counts


def commit_counts(depth, on_path, D: int):
    """Offline counts behind p_hat (Sec. 3.2): m_d = proposed nodes at draft
    position d, c_d = those lying on the accepted output prefix.  Positions
    outside [0, D) are not counted."""
    m = np.zeros(D, np.int64)
    c = np.zeros(D, np.int64)
    for d, a in zip(depth, on_path):
        d = int(d)
        if 0 <= d < D:
            m[d] += 1
            c[d] += 1 if a else 0
    return m, c


def commit_estimate(m, c) -> np.ndarray:
    """p_hat_d = c_d / m_d (Sec. 3.2), rounded once to fp32 (the precision the
    selector takes); a position never observed (m_d = 0) gets 0."""
    out = np.zeros(len(m), np.float32)
    for d in range(len(m)):
        out[d] = np.float32(c[d] / m[d]) if m[d] > 0 else np.float32(0.0)
    return out


def commit_expand(p_hat, depth) -> np.ndarray:
    """Per-node commitment probabilities p_t = p_hat[d_t]; positions beyond the
    table get 0 (never observed)."""
    D = len(p_hat)
    return np.array([p_hat[int(d)] if 0 <= int(d) < D else 0.0 for d in depth], np.float32)


def importance(depth, prob, beta: float) -> np.ndarray:
    """alpha_t = p_{d_t}^beta * N_{d_t}^{-1/2}  (Sec. 3.2, Eq. 3)."""
    N = depth_counts(depth)
    alpha = np.empty(len(depth), dtype=np.float64)
    for t, d in enumerate(depth):
        p = float(np.float32(prob[t]))
        alpha[t] = (p ** beta) / math.sqrt(N[int(d)])
    return alpha


def utility(K_nat, r_nat, alpha, E: int) -> np.ndarray:
    """u_e = sum_t alpha_t r_{t,e} 1[e in K_t]  (Sec. 3.2, Eq. 4; reading R1).

    K_nat[t] lists the natural top-k experts of token t, r_nat[t] its full
    softmax row.  Tokens are visited in order, their selected experts in slot
    order.
    """
    u = np.zeros(E, dtype=np.float64)
    for t in range(len(K_nat)):
        for e in K_nat[t]:
            u[e] += alpha[t] * r_nat[t][e]
    return u


def votes(K_nat, E: int) -> np.ndarray:
    """v_e = sum_t 1[e in K_t], natural top-k assignment count (Sec. 3.4)."""
    v = np.zeros(E, dtype=np.int64)
    for Kt in K_nat:
        for e in Kt:
            v[e] += 1
    return v


# ---------------------------------------------------------------------------
# Sec. 3.3: anchor and self-sizing
# ---------------------------------------------------------------------------
def anchor(K_nat, depth) -> set:
    """A = union of K_t over the anchor tokens, the depth-0 root (Eq. 5, reading R7)."""
    A: set = set()
    for t, d in enumerate(depth):
        if int(d) == 0:
            A.update(int(e) for e in K_nat[t])
    return A


def effective_rank(u_R) -> tuple:
    """n_er of Eq. 6 for the residual utilities u_R (Sec. 3.3; reading R4).

    Returns (n_er, x, Z) with x = exp(H(q)), q_e = u_e^+ / Z.
    """
    up = np.maximum(np.asarray(u_R, dtype=np.float64), 0.0)
    Z = float(up.sum())
    if not Z > 0.0:
        return 0, 0.0, Z
    q = up / Z
    pos = q > 0.0
    Hq = -float(np.sum(q[pos] * np.log(q[pos])))
    x = math.exp(Hq)
    n = int(math.ceil(x - EPS_CEIL))
    n = max(1, min(n, int(np.count_nonzero(up > 0.0))))
    return n, x, Z


def order_desc(ids, score) -> list:
    """ids sorted by (score desc, id asc)."""
    return sorted((int(e) for e in ids), key=lambda e: (-score[e], e))


def order_asc(ids, score) -> list:
    """ids sorted by (score asc, id asc) -- the pruning order pi of Sec. 3.4."""
    return sorted((int(e) for e in ids), key=lambda e: (score[e], e))


def self_sized_set(u, A: set, E: int, k: int):
    """S = A u Top_{n_er}(U_R), then the |S| >= min(k, E) fill (Sec. 3.3)."""
    R = [e for e in range(E) if e not in A]
    n_er, x, Z = effective_rank(u[R]) if R else (0, 0.0, 0.0)
    ordR = order_desc(R, u)
    S = set(A) | set(ordR[:n_er])
    need = min(k, E)
    for e in ordR[n_er:]:
        if len(S) >= need:
            break
        S.add(e)
    return S, n_er, x, ordR


# ---------------------------------------------------------------------------
# Sec. 3.4: residency-aware pruning
# ---------------------------------------------------------------------------
def residency_prune(S: set, u, v, U_nat: set, resident, k: int, removal_cap: int):
    """Remove the longest prefix D* of pi allowed by Eq. 7.

    a(S) = sum of v_e over the natural union outside S; C = nonresident members
    of S ordered by (u asc, index asc); m* is the largest m with
    sum_{j<=m} v_{pi(j)} <= a(S), |S| - m >= k and m <= removal_cap.
    Returns (S', a(S), m*, pi).
    """
    a = int(sum(int(v[e]) for e in U_nat if e not in S))
    C = [e for e in S if not bool(resident[e])]
    pi = order_asc(C, u)
    limit = min(len(pi), max(0, len(S) - k), int(removal_cap))
    m, acc = 0, 0
    while m < limit and acc + int(v[pi[m]]) <= a:
        acc += int(v[pi[m]])
        m += 1
    D = set(pi[:m])
    return S - D, a, m, pi


def eq7_bruteforce(S: set, u, v, U_nat: set, resident, k: int, removal_cap: int) -> int:
    """m* straight from the max{} of Eq. 7 by trying every m (test helper)."""
    a = sum(int(v[e]) for e in U_nat if e not in S)
    pi = order_asc([e for e in S if not bool(resident[e])], u)
    best = 0
    for m in range(0, len(pi) + 1):
        if m <= removal_cap and sum(int(v[e]) for e in pi[:m]) <= a and len(S) - m >= k:
            best = max(best, m)
    return best


# ---------------------------------------------------------------------------
# one verification tree, Sec. 3.1-3.4 in order
# ---------------------------------------------------------------------------
def select_tree(z32, parent, depth, prob, k: int, beta: float = 0.5,
                mode: int = MODE_SELF_SIZING, resident=None, removal_cap=None,
                budget: int = 0) -> dict:
    """Eligible set, restricted routing and gates for one tree.

    z32: [T_b, E] float32 logits; parent (local ids, -1 for the root, or None),
    depth, prob: per-node arrays.  Returns a dict with the eligible mask,
    restricted indices (slot order) and gates, the stats row and decision
    margins used to flag near-ties.
    """
    z32 = np.asarray(z32, dtype=np.float32)
    Tb, E = z32.shape if z32.ndim == 2 else (0, 0)
    out = {"eligible": np.zeros(E, dtype=np.uint8),
           "idx": -np.ones((Tb, k), dtype=np.int32),
           "gate": np.zeros((Tb, k), dtype=np.float32),
           "stats": np.zeros(N_STATS, dtype=np.int64),
           "ambiguous": False, "margins": {}}
    out["stats"][ST_T] = Tb
    code = validate_tree(parent, depth, prob)
    out["stats"][ST_CODE] = code
    if code != TREE_OK:
        return out
    if removal_cap is None:
        removal_cap = E

    # Sec. 3.1: router distribution and natural top-k, Eq. 1 natural union
    r_nat = [softmax64(z32[t]) for t in range(Tb)]
    K_nat = [topk_by_rank(z32[t], k) for t in range(Tb)]
    v = votes(K_nat, E)
    U_nat = {e for e in range(E) if v[e] > 0}

    # Sec. 3.2: commitment-weighted demand
    alpha = importance(depth, prob, beta)
    u = utility(K_nat, r_nat, alpha, E)

    # Sec. 3.3: anchor + self-sizing (or one of the comparison rules)
    A = anchor(K_nat, depth)
    n_er, x, ordR = 0, 0.0, []
    if mode == MODE_SELF_SIZING:
        S, n_er, x, ordR = self_sized_set(u, A, E, k)
    elif mode == MODE_ALL_EXPERTS:
        S = set(range(E))
        n_er = E - len(A)
    elif mode == MODE_FIXED_BUDGET:
        B = max(min(int(budget), E), min(k, E))
        R = [e for e in range(E) if e not in A]
        ordR = order_desc(R, u)
        n_er = max(0, B - len(A))
        S = set(A) | set(ordR[:n_er])
    elif mode in (MODE_MOESPEC, MODE_COUNT):
        B = max(min(int(budget), E), min(k, E))
        score = np.sum(np.stack(r_nat), axis=0) if mode == MODE_MOESPEC else v.astype(np.float64)
        ordR = order_desc(range(E), score)
        S = set(ordR[:B])
        n_er = len(S - A)
    else:
        raise ValueError("unknown mode")

    # Sec. 3.4: rerouting budget a(S) (reported always) and residency-aware
    # pruning (only with a mask, and only for AcceptMoE's own selectors:
    # natural routing and the two baselines never prune)
    a_S = int(sum(int(v[e]) for e in U_nat if e not in S)) if mode != MODE_ALL_EXPERTS else 0
    m_star, pi = 0, []
    if resident is not None and mode in (MODE_SELF_SIZING, MODE_FIXED_BUDGET):
        Sp, a_S, m_star, pi = residency_prune(S, u, v, U_nat, resident, k, removal_cap)
    else:
        Sp = set(S)

    # Sec. 3.1 Eq. 2: restricted routing and native (renormalised) gates
    elig = np.zeros(E, dtype=bool)
    elig[list(Sp)] = True
    routed = set()
    for t in range(Tb):
        sel = topk_by_rank(z32[t], k, elig)
        zs = z32[t][sel].astype(np.float64)
        w = np.exp(zs - zs.max()) if len(sel) else zs
        g = w / w.sum() if len(sel) else w
        out["idx"][t, :len(sel)] = sel
        out["gate"][t, :len(sel)] = g.astype(np.float32)
        routed.update(int(e) for e in sel)

    out["eligible"][list(Sp)] = 1
    st = out["stats"]
    st[ST_A] = len(A)
    st[ST_NER] = n_er
    st[ST_S] = len(S)
    st[ST_SP] = len(Sp)
    st[ST_UNAT] = len(U_nat)
    st[ST_BUDGET] = a_S
    st[ST_MSTAR] = m_star
    st[ST_ROUTED] = len(routed)
    out.update(u=u, v=v, alpha=alpha, A=A, S=S, S_prime=Sp, K_nat=K_nat, r_nat=r_nat, x=x)

    # margins: how close each floating-point decision came to flipping
    marg = {}
    scale = float(np.max(u)) if E and np.max(u) > 0 else 1.0
    if mode in (MODE_SELF_SIZING, MODE_FIXED_BUDGET) and ordR:
        cut = len(S - A)
        if 0 < cut < len(ordR):
            marg["cut"] = (u[ordR[cut - 1]] - u[ordR[cut]]) / scale
        if mode == MODE_SELF_SIZING and x > 0.0:
            y = x - EPS_CEIL
            marg["ceil"] = abs(y - round(y)) / max(1.0, abs(y))
    if mode == MODE_MOESPEC and ordR:
        sc = np.sum(np.stack(r_nat), axis=0)
        B = len(S)
        if 0 < B < E:
            marg["cut"] = (sc[ordR[B - 1]] - sc[ordR[B]]) / max(float(sc.max()), 1e-300)
    if 0 < m_star < len(pi):
        marg["prune"] = (u[pi[m_star]] - u[pi[m_star - 1]]) / scale
    out["margins"] = marg
    out["ambiguous"] = any(0.0 < abs(g) < AMBIG_REL for g in marg.values())
    return out


def select(z32, parent, depth, prob, tree_offsets, k: int, beta: float = 0.5,
           mode: int = MODE_SELF_SIZING, resident=None, removal_cap=None,
           budget: int = 0) -> dict:
    """All trees of a call: per-tree eligible sets, restricted top-k and gates.

    tree_offsets: [B+1] host offsets (None = one tree of all T nodes).  parent
    holds global node ids (-1 for roots) or is None.  Returns eligible [B,E]
    uint8, idx [T,k] int32, gate [T,k] float32, stats [B,10] int64 and the
    per-tree ambiguity flags.
    """
    z32 = np.asarray(z32, dtype=np.float32)
    T, E = z32.shape
    offs = [0, T] if tree_offsets is None else [int(o) for o in tree_offsets]
    B = len(offs) - 1
    res = {"eligible": np.zeros((B, E), np.uint8), "idx": -np.ones((T, k), np.int32),
           "gate": np.zeros((T, k), np.float32), "stats": np.zeros((B, N_STATS), np.int64),
           "ambiguous": np.zeros(B, bool), "trees": []}
    for b in range(B):
        s, e = offs[b], offs[b + 1]
        par = None
        if parent is not None:
            pg = np.asarray(parent[s:e], dtype=np.int64)
            # global -> local ids; -1 stays the root marker, anything pointing
            # before this tree (or another negative value) becomes invalid (-2)
            loc = pg - s
            par = np.where(pg == -1, -1, np.where(loc >= 0, loc, -2))
        tr = select_tree(z32[s:e], par, np.asarray(depth[s:e]), np.asarray(prob[s:e]), k, beta,
                         mode, resident, removal_cap, budget)
        res["eligible"][b] = tr["eligible"]
        res["idx"][s:e] = tr["idx"]
        res["gate"][s:e] = tr["gate"]
        res["stats"][b] = tr["stats"]
        res["ambiguous"][b] = tr["ambiguous"]
        res["trees"].append(tr)
    return res


# ---------------------------------------------------------------------------
# expert FFN (SwiGLU, Qwen3-style) over the restricted routing
# ---------------------------------------------------------------------------
def silu(x):
    return x / (1.0 + np.exp(-x))


def moe_forward_grouped(hidden64, w_gate, w_up, w_down, idx, gate, dtype: str = "f32"):
    """y_t = sum_{e in K~_t} g_{t,e} W_d,e (silu(W_g,e x_t) * W_u,e x_t).

    Experts are visited one at a time (only the routed ones); each gathers its
    tokens.  Weight stacks are [E, I, H] (gate, up) and [E, H, I] (down) in
    nn.Linear orientation, given as fp32 arrays (dtype 'f32') or bf16 bit
    patterns (dtype 'bf16'); they are widened per expert.
    """
    x = np.asarray(hidden64, dtype=np.float64)
    T, H = x.shape
    idx = np.asarray(idx)
    gate = np.asarray(gate, dtype=np.float32).astype(np.float64)
    y = np.zeros((T, H), dtype=np.float64)
    E = len(w_gate)
    for e in range(E):
        tt, jj = np.nonzero(idx == e)
        if tt.size == 0:
            continue
        Xe = x[tt]
        G = Xe @ as_f64(w_gate[e], dtype).T
        U = Xe @ as_f64(w_up[e], dtype).T
        Y = (silu(G) * U) @ as_f64(w_down[e], dtype).T
        y[tt] += gate[tt, jj][:, None] * Y
    return y


def moe_forward_dense(hidden64, w_gate, w_up, w_down, idx, gate, dtype: str = "f32"):
    """Same layer evaluated densely: every expert on every token, weighted by a
    zero-filled [T, E] gate matrix.  Independent of the grouped variant; for
    tiny shapes only."""
    x = np.asarray(hidden64, dtype=np.float64)
    T, H = x.shape
    E = len(w_gate)
    full = np.zeros((T, E), dtype=np.float64)
    idx = np.asarray(idx)
    gate = np.asarray(gate, dtype=np.float32)
    for t in range(T):
        for j in range(idx.shape[1]):
            if idx[t, j] >= 0:
                full[t, idx[t, j]] += float(gate[t, j])
    y = np.zeros((T, H), dtype=np.float64)
    for t in range(T):
        for e in range(E):
            if full[t, e] == 0.0:
                continue
            g = as_f64(w_gate[e], dtype) @ x[t]
            u = as_f64(w_up[e], dtype) @ x[t]
            h = g * (1.0 / (1.0 + np.exp(-g))) * u
            y[t] += full[t, e] * (as_f64(w_down[e], dtype) @ h)
    return y


def moe_forward_rows(hidden64, w_gate, w_up, w_down, idx, gate, rows, dtype: str = "f32"):
    """Output rows y_t for the listed tokens only (sampled checks at full size)."""
    x = np.asarray(hidden64, dtype=np.float64)
    idx = np.asarray(idx)
    gate = np.asarray(gate, dtype=np.float32).astype(np.float64)
    H = x.shape[1]
    y = np.zeros((len(rows), H), dtype=np.float64)
    for i, t in enumerate(rows):
        for j in range(idx.shape[1]):
            e = int(idx[t, j])
            if e < 0:
                continue
            g = as_f64(w_gate[e], dtype) @ x[t]
            u = as_f64(w_up[e], dtype) @ x[t]
            y[i] += gate[t, j] * (as_f64(w_down[e], dtype) @ (silu(g) * u))
    return y


# ---------------------------------------------------------------------------
# brute-force helpers used by the pins
# ---------------------------------------------------------------------------
def topk_bruteforce(z_row, k: int, eligible=None) -> set:
    """Best k-subset of the eligible experts by summed logit (distinct logits only)."""
    z = np.asarray(z_row, dtype=np.float64)
    E = len(z)
    cand = [e for e in range(E) if eligible is None or eligible[e]]
    best, best_set = -np.inf, None
    for comb in itertools.combinations(cand, min(k, len(cand))):
        s = float(sum(z[list(comb)]))
        if s > best:
            best, best_set = s, set(comb)
    return best_set


def top_n_bruteforce(ids, score, n: int) -> set:
    """Best n-subset of ids by summed score (distinct scores only)."""
    ids = list(ids)
    best, best_set = -np.inf, set()
    for comb in itertools.combinations(ids, min(n, len(ids))):
        s = float(sum(score[list(comb)]))
        if s > best:
            best, best_set = s, set(comb)
    return best_set
