"""Verify-block MoE layer benchmark on one MI355X.

A step = one verification block through one MoE layer: route -> select ->
grouped SwiGLU FFN (acceptmoe_route / acceptmoe_select / acceptmoe_moe_forward),
inputs resident in HBM.  Steps rotate over several independently seeded
layers (weight sets) and blocks so consecutive steps never reuse expert
weights through the 256 MB Infinity Cache.

Prints one JSON line:
  value      eligible-expert weight bytes streamed per second (GB/s) over the
             whole step (route + select + forward)
  roofline   the expert FFN launch (acceptmoe_moe_forward) against HBM peak,
             its duration measured with HIP events around every timed launch
  cpu_baseline  the CPU oracle on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import itertools
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--config", default="qwen3_30b_a3b")
    ap.add_argument("--rho", type=float, default=0.9, help="tree correlation of hidden states")
    ap.add_argument("--sets", type=int, default=0, help="weight sets to rotate (0 = enough for >= 2 GiB)")
    ap.add_argument("--blocks", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle sample budget (0 = skip)")
    ap.add_argument("--no-alt", action="store_true", help="skip the i.i.d. (rho = 0) companion run")
    ap.add_argument("--graph", type=int, default=1, help="time HIP-graph replays of the step sequence (1/0)")
    ap.add_argument("--stack-blocks", type=int, default=8, help="blocks timed through a whole layer stack")
    ap.add_argument("--offload", action="store_true",
                    help="expert-offload report (X-slot pools, LRU, waves) on a synthetic decode trace")
    ap.add_argument("--pool-slots", type=int, default=48, help="X, expert slots per layer pool")
    ap.add_argument("--trace-blocks", type=int, default=96, help="blocks of the offload trace")
    ap.add_argument("--trace-warmup", type=int, default=16, help="leading trace blocks not counted")
    ap.add_argument("--rho-step", type=float, default=0.9, help="root correlation of consecutive trace blocks")
    ap.add_argument("--phys-layers", type=int, default=4, help="layers of the physical (copying) offload run")
    ap.add_argument("--estimate", action="store_true",
                    help="offline commitment estimator report (p_hat from synthetic traces, tree and chain blocks)")
    ap.add_argument("--tp-share", type=int, default=1, metavar="G",
                    help="time one GPU's share of a G-way tensor-parallel split over I: the same routing "
                         "(router, hidden states and trees as the full layer), experts with I/G rows")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                    help="only run a plain device copy of MB MiB (HBM counter calibration) and exit")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "moe_forward_qwen3_30b_a3b_traffic.md")
FFN_SOURCES = ["paper_2608_02989_amd/csrc/forward.hip", "paper_2608_02989_amd/csrc/common.hpp"]


def ffn_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in FFN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """Measured / algorithmic HBM bytes of a forward launch from the committed
    counter summary, or None when it is missing or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        if line.startswith("traffic:"):
            for kv in line[len("traffic:"):].split():
                k, _, v = kv.partition("=")
                vals[k] = v
    if vals.get("source_hash") != ffn_source_hash() or "ratio" not in vals:
        return None
    return float(vals["ratio"])


def copy_calibration(mb: int) -> None:
    import torch
    n = mb << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {mb} MiB five times", flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.offload:
        offload_report(args)
        return
    if args.estimate:
        estimate_report(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the layer runs on a single MI355X; "
              "sharding it over several GPUs is designed but not built", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_02989_amd import ops
    from paper_2608_02989_amd import workload as W

    dev = "cuda"
    cfg = W.CONFIGS[args.config]
    if cfg.layers > 1:
        stack_report(args, cfg)
        return
    full_I = cfg.I
    if args.tp_share > 1:
        # one GPU's shard: the seeds depend on the configuration id, not on I,
        # so routing is the full layer's and only the expert weights shrink
        G = args.tp_share
        if cfg.I % (32 * G) != 0:
            print(f"--tp-share {G}: I = {cfg.I} does not split into {G} multiples of 32", file=sys.stderr)
            sys.exit(2)
        cfg = W.LayerConfig(**{**cfg.__dict__, "I": cfg.I // G})
    Ttot = cfg.total_tokens
    ebytes = cfg.expert_bytes
    layer_bytes = cfg.E * ebytes
    n_sets = args.sets or max(4, int(np.ceil(2 * 2**30 / layer_bytes)))
    n_sets = min(n_sets, 16)
    t0 = time.time()

    def log(msg):
        print(f"[bench {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    log(f"config {cfg.name} T={Ttot} B={cfg.B} H={cfg.H} E={cfg.E} k={cfg.k} I={cfg.I} "
        f"dtype={cfg.dtype} sets={n_sets} blocks={args.blocks}")

    # ---- weights: n_sets independently seeded layers, packed once ----
    layers = []
    for s in range(n_sets):
        rw = torch.from_numpy(W.router_weights(cfg, s)).to(dev)
        wg, wu, wd = W.expert_weights_torch(cfg, s, dev)
        layers.append(ops.VerifyLayer(rw, wg, wu, wd, cfg.k, max_tokens=Ttot, max_trees=cfg.B))
        del wg, wu, wd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log("weights generated and packed")

    def make_blocks(rho):
        out = []
        for b in range(args.blocks):
            blk = W.make_block(cfg, block=b, layer=0, rho=rho)
            if cfg.dtype == "bf16":
                h = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(dev)
            else:
                h = torch.from_numpy(blk.hidden).to(dev)
            out.append(dict(
                h=h, parent=torch.from_numpy(blk.parent).to(dev), depth=torch.from_numpy(blk.depth).to(dev),
                prob=torch.from_numpy(blk.prob).to(dev), offs=blk.offsets.tolist(),
                resident=None if blk.resident is None else torch.from_numpy(blk.resident).to(dev), host=blk))
        return out

    def combos(n):
        return [(i % n_sets, i % args.blocks) for i in range(n)]

    def run_once(blocks, s, b, stream, ev=None):
        L_, B_ = layers[s], blocks[b]
        if ev is None:
            return L_.step(B_["h"], B_["parent"], B_["depth"], B_["prob"], B_["offs"], B_["resident"], stream)
        T = B_["h"].shape[0]
        logits = L_.logits[:T]
        ops.route(B_["h"], L_.router, out=logits, stream=stream)
        nb = len(B_["offs"]) - 1
        outs = {"eligible": L_.sel_out["eligible"][:nb], "idx": L_.sel_out["idx"][:T],
                "gate": L_.sel_out["gate"][:T], "stats": L_.sel_out["stats"][:nb]}
        ops.select(logits, B_["parent"], B_["depth"], B_["prob"], B_["offs"], L_.k, L_.beta, L_.mode,
                   L_.budget, L_.removal_cap, B_["resident"], workspace=L_.sel_ws, outputs=outs, stream=stream)
        ev[0].record(stream)
        ops.moe_forward(B_["h"], L_.wgu, L_.wd, outs["idx"], outs["gate"], out=L_.out[:T],
                        workspace=L_.fwd_ws, stream=stream)
        ev[1].record(stream)

    def measure(rho, steps, warmup):
        blocks = make_blocks(rho)
        stream = torch.cuda.Stream()
        # untimed pre-pass: the routed union of every (set, block) pair (selection is
        # deterministic) and its routing, kept for the forward-only timing below
        routed, sprime, unat, routing = {}, {}, {}, {}
        with torch.cuda.stream(stream):
            for s in range(n_sets):
                for b in range(args.blocks):
                    _, sel, _ = run_once(blocks, s, b, stream)
                    idx = sel["idx"]
                    routing[(s, b)] = (idx.clone(), sel["gate"].clone())
                    routed[(s, b)] = int(torch.unique(idx[idx >= 0]).numel())
                    st = sel["stats"].cpu().numpy()
                    sprime[(s, b)] = float(st[:, 4].mean())
                    unat[(s, b)] = float(st[:, 5].mean())
        torch.cuda.synchronize()
        seq = combos(warmup + steps)
        timed = seq[warmup:]
        r = np.array([routed[c] for c in timed], np.float64)
        weight_bytes = r * ebytes
        act_bytes = Ttot * cfg.H * (2 if cfg.dtype == "bf16" else 4) + Ttot * cfg.H * 4 + Ttot * cfg.k * 8
        fwd_bytes = weight_bytes + act_bytes

        # (1) eager launches, HIP events around every expert-FFN launch
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        with torch.cuda.stream(stream):
            for (s, b) in seq[:warmup]:
                run_once(blocks, s, b, stream)
            torch.cuda.synchronize()
            start = torch.cuda.Event(enable_timing=True)
            stop = torch.cuda.Event(enable_timing=True)
            start.record(stream)
            for i, (s, b) in enumerate(timed):
                run_once(blocks, s, b, stream, evs[i])
            stop.record(stream)
        torch.cuda.synchronize()
        eager_ms = start.elapsed_time(stop)
        fwd_ms = [a.elapsed_time(z) for a, z in evs]

        # (2) the same step sequence replayed from a HIP graph (no host launch cost)
        period = n_sets * args.blocks // int(np.gcd(n_sets, args.blocks))
        graph_ms = None
        if args.graph:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(stream):
                with torch.cuda.graph(g, stream=stream):
                    for (s, b) in combos(period):
                        run_once(blocks, s, b, stream)
            torch.cuda.synchronize()
            reps = max(1, (steps + period - 1) // period)
            for _ in range(2):
                g.replay()
            torch.cuda.synchronize()
            gs, ge = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            gs.record(stream)
            with torch.cuda.stream(stream):
                for _ in range(reps):
                    g.replay()
            ge.record(stream)
            torch.cuda.synchronize()
            graph_ms = gs.elapsed_time(ge) / (reps * period) * steps
            del g
        # (3) the forward launches alone, replayed from a HIP graph over the same
        # rotation (every (set, block) pair's routing from the pre-pass): the
        # average launch duration without the host launch cost that the eager
        # events around each launch include
        fwd_graph_us, fwd_graph_bytes = None, None
        if args.graph:
            pairs = combos(period)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(stream):
                with torch.cuda.graph(g, stream=stream):
                    for (s, b) in pairs:
                        L_, B_ = layers[s], blocks[b]
                        T = B_["h"].shape[0]
                        ops.moe_forward(B_["h"], L_.wgu, L_.wd, routing[(s, b)][0], routing[(s, b)][1],
                                        out=L_.out[:T], workspace=L_.fwd_ws, stream=stream)
            torch.cuda.synchronize()
            reps = max(1, (steps + period - 1) // period)
            for _ in range(2):
                g.replay()
            torch.cuda.synchronize()
            gs, ge = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            gs.record(stream)
            with torch.cuda.stream(stream):
                for _ in range(reps):
                    g.replay()
            ge.record(stream)
            torch.cuda.synchronize()
            fwd_graph_us = gs.elapsed_time(ge) * 1e3 / (reps * period)
            fwd_graph_bytes = float(np.mean([routed[c] * ebytes for c in pairs])) + act_bytes
            del g
        total_ms = graph_ms if graph_ms is not None else eager_ms
        return dict(
            ms_per_step=total_ms / steps,
            eager_us=eager_ms / steps * 1e3,
            graph_us=None if graph_ms is None else graph_ms / steps * 1e3,
            value=float(weight_bytes.sum() / (total_ms * 1e-3) / 1e9),
            fwd_us=float(np.mean(fwd_ms) * 1e3) if fwd_graph_us is None else fwd_graph_us,
            fwd_gbs=(float(fwd_bytes.sum() / (np.sum(fwd_ms) * 1e-3) / 1e9) if fwd_graph_us is None
                     else fwd_graph_bytes / (fwd_graph_us * 1e-6) / 1e9),
            fwd_bytes_per_launch=float(fwd_bytes.mean()) if fwd_graph_bytes is None else fwd_graph_bytes,
            fwd_eager_us=float(np.mean(fwd_ms) * 1e3),
            fwd_eager_gbs=float(fwd_bytes.sum() / (np.sum(fwd_ms) * 1e-3) / 1e9),
            fwd_timing="HIP graph of forward launches" if fwd_graph_us is not None else "eager HIP events",
            routed=float(r.mean()), sprime=float(np.mean([sprime[c] for c in timed])),
            unat=float(np.mean([unat[c] for c in timed])),
            flops=float(Ttot * cfg.k * 6 * cfg.H * cfg.I + 2 * Ttot * cfg.E * cfg.H),
            blocks=blocks, stream=stream,
        )

    main_m = measure(args.rho, args.steps, args.warmup)
    log(f"rho={args.rho}: {main_m['ms_per_step'] * 1e3:.1f} us/step (eager {main_m['eager_us']:.1f}), "
        f"{main_m['value']:.0f} GB/s, ffn {main_m['fwd_us']:.1f} us ({main_m['fwd_gbs']:.0f} GB/s), "
        f"routed {main_m['routed']:.1f}")

    alt = None
    if not args.no_alt and args.rho != 0.0:
        m0 = measure(0.0, args.steps, args.warmup)
        alt = {"rho": 0.0, "value": round(m0["value"], 1), "latency_us": round(m0["ms_per_step"] * 1e3, 2),
               "eager_latency_us": round(m0["eager_us"], 2),
               "ffn_us": round(m0["fwd_us"], 2), "ffn_gbs": round(m0["fwd_gbs"], 1),
               "routed_experts": round(m0["routed"], 2), "eligible": round(m0["sprime"], 2),
               "natural_union": round(m0["unat"], 2)}
        log(f"rho=0: {m0['ms_per_step'] * 1e3:.1f} us/step, {m0['value']:.0f} GB/s, routed {m0['routed']:.1f}")

    # ---- CPU oracle baseline on a bounded sample ----
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(cfg, layers, main_m["blocks"], args.cpu_seconds, ebytes, log)

    frac = main_m["fwd_gbs"] / HBM_PEAK_GBS
    line = {
        "metric": "verify-block MoE layer latency (us) + eligible-expert weight HBM GB/s, 1 GPU",
        "value": round(main_m["value"], 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_m["ms_per_step"], 5),
        "latency_us": round(main_m["ms_per_step"] * 1e3, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: 1 MoE layer, verify block T={Ttot} (B={cfg.B} trees), "
                               f"H={cfg.H} E={cfg.E} top-{cfg.k} I={cfg.I}, {cfg.dtype} experts, fp32 router, "
                               f"tree-correlated hidden rho={args.rho}"
                               + (f"; one GPU's I/{args.tp_share} shard of I={full_I} (tensor parallel over I)"
                                  if args.tp_share > 1 else ""),
                   "T": Ttot, "B": cfg.B, "H": cfg.H, "E": cfg.E, "k": cfg.k, "I": cfg.I,
                   "rho": args.rho, "weight_sets": n_sets, "blocks": args.blocks,
                   **({"tp_share": args.tp_share, "I_full": full_I} if args.tp_share > 1 else {}),
                   "routed_experts": round(main_m["routed"], 2), "eligible": round(main_m["sprime"], 2),
                   "natural_union": round(main_m["unat"], 2)},
        "roofline": {"bound": "hbm", "kernel": "acceptmoe_moe_forward (gate_up with per-item dispatch + down with in-LDS combine)",
                     "achieved": round(main_m["fwd_gbs"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(frac, 4),
                     "traffic": (None if measured_traffic() is None
                                 else round(measured_traffic() * main_m["fwd_bytes_per_launch"])),
                     "bytes_per_launch": round(main_m["fwd_bytes_per_launch"]),
                     "launch_us": round(main_m["fwd_us"], 2),
                     "launch_timing": main_m["fwd_timing"],
                     "eager_launch_us": round(main_m["fwd_eager_us"], 2),
                     "eager_achieved": round(main_m["fwd_eager_gbs"], 1),
                     "mfma_util": round(main_m["flops"] / (main_m["fwd_us"] * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 5)},
        "cpu_baseline": cpu,
        "alt_iid": alt,
        "timing": "HIP graph replay of the rotated step sequence" if main_m["graph_us"] is not None
                  else "eager launches",
        "eager_latency_us": round(main_m["eager_us"], 2),
    }
    print(json.dumps(line), flush=True)


def _dist(x):
    x = np.asarray(x, np.float64)
    return {"mean": round(float(x.mean()), 3), "p10": float(np.percentile(x, 10)),
            "p50": float(np.percentile(x, 50)), "p90": float(np.percentile(x, 90)),
            "min": float(x.min()), "max": float(x.max())}


def stack_report(args, cfg):
    """The 48-layer verify pass: layers chained by the residual stream
    (h_{l+1} = h_l + y_l rounded to bf16), each with its own router and
    experts (all 48 layers resident, 54 GiB).

    Part 1: eligible-set sizes of every (block, layer) pair over many seeded
    blocks run through the chained stack.  Part 2: latency of a whole pass per
    block -- eager launches, one HIP graph for the whole 48-layer pass, and two
    blocks in flight on two streams (one block's latency-bound selection chain
    overlapping the other's bandwidth-bound expert FFN).
    """
    import torch

    from paper_2608_02989_amd import _lib as L
    from paper_2608_02989_amd import ops
    from paper_2608_02989_amd import workload as W

    t0 = time.time()

    def log(msg):
        print(f"[stack {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    dev = "cuda"
    nblocks = args.blocks if args.blocks != 16 else cfg.blocks
    nl = cfg.layers
    T, k = cfg.T, cfg.k
    layers = []
    for l in range(nl):
        wg, wu, wd = W.expert_weights_torch(cfg, l, dev)
        layers.append(ops.VerifyLayer(torch.from_numpy(W.router_weights(cfg, l)).to(dev), wg, wu, wd, k,
                                      max_tokens=T))
        del wg, wu, wd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    stack = ops.VerifyStack(layers, T)
    log(f"{nl} layers packed")

    def block(b):
        blk = W.make_block(cfg, block=b, layer=0, rho=args.rho, tree_layer=0)
        h = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(dev)
        return (h,) + tuple(torch.from_numpy(a).to(dev) for a in (blk.parent, blk.depth, blk.prob))

    stats_all = torch.empty((nblocks, nl, L.NUM_STATS), dtype=torch.int32, device=dev)
    routed_bytes = []
    for b in range(nblocks):
        h, par, dep, prob = block(b)
        stack.step(h, par, dep, prob)
        for l in range(nl):
            stats_all[b, l].copy_(layers[l].sel_out["stats"][0])
        if b % 32 == 31:
            log(f"{b + 1} blocks through the chained stack")
    torch.cuda.synchronize()
    st = stats_all.cpu().numpy().reshape(-1, L.NUM_STATS).astype(np.float64)
    assert (st[:, 8] == 0).all(), "malformed synthetic tree"
    sp, un, routed, ner = st[:, 4], st[:, 5], st[:, 9], st[:, 2]
    report = {"report": "48-layer verify pass (residual-chained layers)", "config": cfg.name, "blocks": nblocks,
              "layers": nl, "samples": int(st.shape[0]), "T": T, "H": cfg.H, "E": cfg.E, "k": k,
              "rho": args.rho, "eligible_S_prime": _dist(sp), "natural_union": _dist(un),
              "ratio_S_prime_over_U_nat": _dist(sp / un), "routed_experts": _dist(routed),
              "n_er": _dist(ner)}
    log(f"|S'| mean {sp.mean():.2f}, |U_nat| mean {un.mean():.2f}")

    nb = args.stack_blocks
    inputs = [block(b) for b in range(nb)]
    pass_bytes = float(np.mean(routed[:nb * nl].reshape(nb, nl).sum(1))) * cfg.expert_bytes
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    # eager, one stream
    stack.step(*inputs[0])
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for b in range(nb):
        stack.step(*inputs[b])
    e1.record()
    torch.cuda.synchronize()
    eager_us = e0.elapsed_time(e1) * 1e3 / nb

    # one HIP graph per 48-layer pass; the block's inputs are copied into its buffers
    cap = tuple(torch.empty_like(x) for x in inputs[0])
    s = torch.cuda.Stream()
    for dst, src in zip(cap, inputs[0]):
        dst.copy_(src)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        stack.step(*cap)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        stack.step(*cap)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for b in range(nb):
        for dst, src in zip(cap, inputs[b]):
            dst.copy_(src)
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    graph_us = e0.elapsed_time(e1) * 1e3 / nb

    # two blocks in flight: two graphs over twin buffers, replayed on two streams
    twin = stack.twin()
    cap2 = tuple(torch.empty_like(x) for x in inputs[0])
    s2 = torch.cuda.Stream()
    for dst, src in zip(cap2, inputs[1 % nb]):
        dst.copy_(src)
    torch.cuda.synchronize()
    with torch.cuda.stream(s2):
        twin.step(*cap2)
    torch.cuda.synchronize()
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s2):
        twin.step(*cap2)
    torch.cuda.synchronize()
    main = torch.cuda.current_stream()
    e0, e1 = ev(), ev()
    e0.record()
    for b in range(0, nb - 1, 2):
        s.wait_stream(main)
        s2.wait_stream(main)
        with torch.cuda.stream(s):
            for dst, src in zip(cap, inputs[b]):
                dst.copy_(src)
            g.replay()
        with torch.cuda.stream(s2):
            for dst, src in zip(cap2, inputs[b + 1]):
                dst.copy_(src)
            g2.replay()
        main.wait_stream(s)
        main.wait_stream(s2)
    e1.record()
    torch.cuda.synchronize()
    pairs = (nb // 2) * 2
    two_us = e0.elapsed_time(e1) * 1e3 / max(pairs, 1)
    report.update({"stack_pass_blocks": nb, "eager_us_per_block": round(eager_us, 1),
                   "graph_us_per_block": round(graph_us, 1), "graph_us_per_layer": round(graph_us / nl, 2),
                   "two_stream_us_per_block": round(two_us, 1),
                   "routed_MB_per_pass": round(pass_bytes / 1e6, 1),
                   "graph_weight_GBs": round(pass_bytes / (graph_us * 1e-6) / 1e9, 1),
                   "two_stream_weight_GBs": round(pass_bytes / (two_us * 1e-6) / 1e9, 1),
                   "timing": "HIP events; 48 distinct resident layers per pass; two-stream figure is "
                             "throughput with two blocks in flight"})
    log(f"pass per block: eager {eager_us:.0f} us, graph {graph_us:.0f} us, two streams {two_us:.0f} us")
    print(json.dumps(report), flush=True)


def offload_report(args):
    """Physical expert offload on a synthetic decode trace (the traffic / hit-rate
    comparison of Sec. 4, Table 2, on stand-in inputs).

    Trace: the 48-layer Qwen3-30B-A3B stack shape (T = 60 draft trees, E = 128,
    k = 8); consecutive blocks' root states are correlated (--rho-step), every
    layer has its own router, hidden states and X-slot pool.  Methods, each on
    fresh pools: Vanilla AR (one token per step, natural routing), Standard SD
    (the whole draft tree, natural routing) and AcceptMoE (self-sized eligible
    set pruned against the pool's resident set).  Part 1 (all layers): routing
    on the GPU, pool bookkeeping without copies -> H2D MiB per block / per
    token and hit rate after a warm-up.  Part 2 (--phys-layers): the same trace
    with real pinned-host -> pool copies and the forward over the pool, timed.
    Tokens per block: AR 1; tree methods sum over depths d of the largest
    commitment probability at depth d (the chance the verified prefix reaches
    depth d, root = 1): the expected committed length of the synthetic trees.
    """
    import torch

    from paper_2608_02989_amd import _lib as L
    from paper_2608_02989_amd import ops
    from paper_2608_02989_amd import workload as W

    t0 = time.time()

    def log(msg):
        print(f"[offload {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    dev = "cuda"
    cfg = W.CONFIGS["qwen3_30b_a3b_x48"]
    X, nb, warm = args.pool_slots, args.trace_blocks, args.trace_warmup
    nl, T, E, k = cfg.layers, cfg.T, cfg.E, cfg.k
    methods = [("vanilla_ar", L.MODE_ALL_EXPERTS, True), ("standard_sd", L.MODE_ALL_EXPERTS, False),
               ("acceptmoe", L.MODE_SELF_SIZING, False)]
    routers = [ops.pack_router_weights(torch.from_numpy(W.router_weights(cfg, l)).to(dev)) for l in range(nl)]
    roots = [W.trace_roots(cfg, l, nb, args.rho_step) for l in range(nl)]
    # inputs of every (block, layer), shared by the methods
    inputs, tau = [], []
    for b in range(nb):
        per = []
        for l in range(nl):
            blk = W.make_block(cfg, block=b, layer=l, rho=args.rho, tree_layer=0, root=roots[l][b])
            h = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(dev)
            per.append((h,) + tuple(torch.from_numpy(a).to(dev) for a in (blk.parent, blk.depth, blk.prob)))
        inputs.append(per)
        pd = {}
        for d_, p_ in zip(blk.depth.tolist(), blk.prob.astype(np.float64).tolist()):
            pd[d_] = max(pd.get(d_, 0.0), p_)
        tau.append(float(sum(pd.values())))
        if b % 32 == 31:
            log(f"{b + 1} trace blocks generated")
    tau_tree = float(np.mean(tau[warm:]))
    logits = torch.empty((T, E), dtype=torch.float32, device=dev)
    ws = ops.select_workspace(T, E, k, dev)
    mask_dev = torch.empty(E, dtype=torch.uint8, device=dev)
    outs = {"eligible": torch.empty((1, E), dtype=torch.uint8, device=dev),
            "idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "gate": torch.empty((T, k), dtype=torch.float32, device=dev),
            "stats": torch.empty((1, L.NUM_STATS), dtype=torch.int32, device=dev)}

    def node_inputs(inp, single):
        h, par, dep, prob = inp
        return (h[:1], par[:1], dep[:1], prob[:1]) if single else inp

    results = {}
    for name, mode, single in methods:
        pools = [ops.OffloadPool(X, E, expert_bytes=cfg.expert_bytes) for _ in range(nl)]
        base = np.zeros(L.POOL_NUM_STATS, np.int64)
        routed = []
        for b in range(nb):
            if b == warm:
                base = sum(p.stats for p in pools)
            for l in range(nl):
                h, par, dep, prob = node_inputs(inputs[b][l], single)
                Tb = h.shape[0]
                ops.route(h, routers[l], out=logits[:Tb])
                mask_dev.copy_(torch.from_numpy(pools[l].resident_mask()))
                o = {"eligible": outs["eligible"], "idx": outs["idx"][:Tb], "gate": outs["gate"][:Tb],
                     "stats": outs["stats"]}
                ops.select(logits[:Tb], par, dep, prob, None, k, mode=mode, resident=mask_dev, workspace=ws,
                           outputs=o)
                idx = o["idx"].cpu().numpy()
                wave_of, n = pools[l].plan_waves(idx)
                for w in range(n):
                    pools[l].serve_wave(idx, wave_of, w)
                if b >= warm:
                    routed.append(len(np.unique(idx[idx >= 0])))
        st = sum(p.stats for p in pools) - base
        blocks = nb - warm
        tok = blocks * (1.0 if single else tau_tree)
        mib = st[L.POOL_H2D_BYTES] / 2**20
        results[name] = {"blocks": blocks, "tokens_per_block": round(1.0 if single else tau_tree, 3),
                         "h2d_MiB_per_block": round(float(mib) / blocks, 1),
                         "h2d_MiB_per_token": round(float(mib) / tok, 1),
                         "hit_rate": round(float(st[L.POOL_HITS]) / max(1, int(st[L.POOL_ACCESSES])), 4),
                         "loads_per_block_layer": round(float(st[L.POOL_MISSES]) / (blocks * nl), 2),
                         "routed_per_block_layer": round(float(np.mean(routed)), 2),
                         "waves_per_block_layer": round(float(st[L.POOL_WAVES]) / (blocks * nl), 3)}
        log(f"{name}: {results[name]}")

    # part 2: physical copies and the forward over the pools, timed (a few layers)
    npl = min(args.phys_layers, nl)
    phys_layers = []
    for l in range(npl):
        wg, wu, wd = W.expert_weights_torch(cfg, l, dev)
        phys_layers.append((wg, wu, wd))
    log(f"{npl} layers of weights generated")
    for name, mode, single in methods:
        layers = []
        for l in range(npl):
            wg, wu, wd = phys_layers[l]
            layers.append(ops.OffloadLayer(torch.from_numpy(W.router_weights(cfg, l)).to(dev), wg, wu, wd, k, X,
                                           max_tokens=T, mode=mode))
        torch.cuda.synchronize()
        base = np.zeros(L.POOL_NUM_STATS, np.int64)
        for b in range(nb):
            if b == warm:
                torch.cuda.synchronize()
                base = sum(ly.pool.stats for ly in layers)
                t_start = time.perf_counter()
            for l in range(npl):
                layers[l].step(*node_inputs(inputs[b][l], single))
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
        st = sum(ly.pool.stats for ly in layers) - base
        steps = (nb - warm) * npl
        results[name].update({
            "phys_layers": npl, "phys_us_per_block_layer": round(elapsed / steps * 1e6, 1),
            "phys_us_per_token_layer": round(elapsed / steps * 1e6 / (1.0 if single else tau_tree), 1),
            "phys_loads_per_block_layer": round(float(st[L.POOL_MISSES]) / steps, 2),
            "phys_h2d_GBs": round(float(st[L.POOL_H2D_BYTES]) / elapsed / 1e9, 2)})
        log(f"{name} physical: {results[name]}")
        del layers
        torch.cuda.empty_cache()
    sd, am = results["standard_sd"], results["acceptmoe"]
    report = {"report": "expert offload on a synthetic decode trace", "config": cfg.name, "X": X,
              "layers": nl, "E": E, "k": k, "T": T, "rho_tree": args.rho, "rho_step": args.rho_step,
              "trace_blocks": nb, "warmup_blocks": warm, "expert_MiB": round(cfg.expert_bytes / 2**20, 3),
              "methods": results,
              "acceptmoe_vs_sd": {
                  "h2d_per_token_change_pct": round(100.0 * (am["h2d_MiB_per_token"] / sd["h2d_MiB_per_token"] - 1), 1),
                  "hit_rate_change_pp": round(100.0 * (am["hit_rate"] - sd["hit_rate"]), 1)},
              "timing": "wall clock of eager steps (route, select, host round trip, loads, forward)",
              "data": "synthetic"}
    print(json.dumps(report), flush=True)


def estimate_report(args):
    """Offline commitment estimator (Sec. 3.2) on synthetic verification traces.

    Training split: 2000 draft trees (60 nodes, Qwen3-30B-A3B stack shape) and
    2000 chains of 8, each verified by the synthetic acceptance process (the
    verifier takes the sibling of rank r with probability (0.55, 0.2, 0.1,
    0.05)[r]); the library accumulates m_d, c_d and returns p_hat.  Held-out
    split: 64 blocks of each shape selected on the GPU with p_t = p_hat[d_t]
    (expanded on the device) and, for comparison, with the fixed synthetic
    probabilities 0.75^d 0.6^r; |S|, |S'| and routed experts are reported.
    """
    import torch

    from paper_2608_02989_amd import _lib as L
    from paper_2608_02989_amd import ops
    from paper_2608_02989_amd import workload as W

    t0 = time.time()

    def log(msg):
        print(f"[estimate {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    dev = "cuda"
    cfg = W.CONFIGS["qwen3_30b_a3b_x48"]
    shapes = {"tree": (9, lambda b: W.make_tree(np.random.default_rng(10_000 + b), cfg.T, cfg.depth_max)),
              "chain": (8, lambda b: W.chain(8))}
    n_train, n_eval = 2000, 64
    report = {"report": "offline commitment estimator on synthetic verification traces", "config": cfg.name,
              "acceptance_q": [0.55, 0.2, 0.1, 0.05], "train_blocks": n_train, "eval_blocks": n_eval, "shapes": {}}
    router = ops.pack_router_weights(torch.from_numpy(W.router_weights(cfg, 0)).to(dev))
    for name, (D, make) in shapes.items():
        est = ops.CommitEstimator(D)
        rng = np.random.default_rng(77)
        trees = [make(b) for b in range(n_train)]
        outcomes = [W.accepted_prefix(rng, par, sib) for par, dep, sib in trees]
        nodes = sum(len(t[0]) for t in trees)
        t1 = time.perf_counter()
        for (par, dep, sib), on in zip(trees, outcomes):
            est.add(dep, on)
        t_count = time.perf_counter() - t1
        p_hat = est.estimate()
        log(f"{name}: p_hat {np.round(p_hat, 4).tolist()}")
        p_hat_dev = torch.from_numpy(p_hat).to(dev)
        stats = {"estimated": [], "synthetic": []}
        for b in range(n_eval):
            par, dep, sib = make(n_train + b)
            h32 = W.correlated_hidden(W.rng_for(cfg.cfg_id, n_train + b, 0, W.STREAM_HIDDEN), par, cfg.H,
                                      cfg.hidden_std, args.rho)
            h = torch.from_numpy(W.bf16_round(h32).view(np.int16)).view(torch.bfloat16).to(dev)
            logits = ops.route(h, router)
            par_d, dep_d = torch.from_numpy(par).to(dev), torch.from_numpy(dep).to(dev)
            synth = torch.from_numpy(W.commit_probs(None, "depth_sibling", dep, sib)).to(dev)
            for kind, prob in (("estimated", ops.commit_expand(p_hat_dev, dep_d)), ("synthetic", synth)):
                out = ops.select(logits, par_d, dep_d, prob, None, cfg.k)
                stats[kind].append(out["stats"][0].cpu().numpy().copy())
        sh = {"D": D, "p_hat": [round(float(x), 5) for x in p_hat], "m": est.m.tolist(), "c": est.c.tolist(),
              "train_nodes": int(nodes), "count_ns_per_node": round(t_count / nodes * 1e9, 1)}
        for kind, rows in stats.items():
            st = np.asarray(rows, np.float64)
            sh[kind] = {"S": _dist(st[:, 3]), "S_prime": _dist(st[:, 4]), "natural_union": _dist(st[:, 5]),
                        "routed": _dist(st[:, 9]), "n_er": _dist(st[:, 2])}
        report["shapes"][name] = sh
        log(f"{name}: |S'| estimated {sh['estimated']['S_prime']['mean']} synthetic {sh['synthetic']['S_prime']['mean']}")
    report["data"] = "synthetic"
    print(json.dumps(report), flush=True)


def cpu_baseline(cfg, layers, blocks, budget_s, ebytes, log):
    """Oracle route + select + grouped forward per block, host cores, bounded sample."""
    import torch

    from oracle import acceptmoe_oracle as O
    from paper_2608_02989_amd import workload as W

    L0 = layers[0]
    rw = L0.router_w.cpu().numpy().astype(np.float64)
    # the oracle reads row-major weights: unpack by regenerating the same seeded layer on the host side
    wg, wu, wd = W.expert_weights_torch(cfg, 0, "cuda")
    host = [{}, {}, {}]

    def fetch(e):
        for j, w in enumerate((wg, wu, wd)):
            if e not in host[j]:
                host[j][e] = W.to_bits(w[e])

    class View:
        def __init__(self, j):
            self.j = j

        def __len__(self):
            return cfg.E

        def __getitem__(self, e):
            return host[self.j][int(e)]

    try:
        from threadpoolctl import threadpool_info
        threads = max([int(i.get("num_threads", 1)) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    elapsed, nbytes, n = 0.0, 0.0, 0
    prepared = set()
    # cycle over the blocks until the time budget is used (a bounded sample)
    for b in itertools.cycle(range(len(blocks))):
        blk = blocks[b]["host"]
        h64 = (O.widen_bf16(W.bf16_round(blk.hidden)) if cfg.dtype == "bf16"
               else blk.hidden.astype(np.float64))
        if b not in prepared:
            # weights needed by this block go to host memory before the clock starts
            z_pre = O.route(h64, rw).astype(np.float32)
            pre = O.select(z_pre, blk.parent, blk.depth, blk.prob, blk.offsets, cfg.k, resident=blk.resident)
            for e in np.unique(pre["idx"][pre["idx"] >= 0]):
                fetch(int(e))
            prepared.add(b)
        t1 = time.perf_counter()
        z = O.route(h64, rw).astype(np.float32)
        sel = O.select(z, blk.parent, blk.depth, blk.prob, blk.offsets, cfg.k, resident=blk.resident)
        O.moe_forward_grouped(h64, View(0), View(1), View(2), sel["idx"], sel["gate"], cfg.dtype)
        elapsed += time.perf_counter() - t1
        nbytes += len(np.unique(sel["idx"][sel["idx"] >= 0])) * ebytes
        n += 1
        if elapsed >= budget_s:
            break
    del wg, wu, wd
    log(f"cpu oracle: {n} blocks in {elapsed:.1f}s")
    return {"value": round(nbytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} block passes over {len(prepared)} seeded blocks of {cfg.name} (layer 0), "
                      f"route+select+grouped forward in fp64 numpy, {elapsed:.1f} s",
            "latency_us": round(elapsed / n * 1e6, 1)}


if __name__ == "__main__":
    main()
