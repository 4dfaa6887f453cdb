"""Verify-block MoE layer benchmark on one MI355X.

A step = one verification block through one MoE layer: route -> select ->
grouped SwiGLU FFN (acceptmoe_route / acceptmoe_select / acceptmoe_moe_forward),
inputs resident in HBM.  Steps rotate over several independently seeded
layers (weight sets) and blocks so consecutive steps never reuse expert
weights through the 256 MB Infinity Cache.

The headline workload is the largest single-tree configuration (H = 4096,
I = 1536, T = 64 nodes, 25 % residency mask); the Qwen3-30B-A3B-shaped layer
(T = 32) and the batched one (8 trees x 64 nodes) follow as companions, each
with its own roofline block, each measured by this script in a child process
(a fresh device allocator, as in a serving process).  Prints one JSON line:
  value      eligible-expert weight bytes streamed per second (GB/s) over the
             whole step (route + select + forward), bytes and time over the
             same timed steps
  roofline   the expert FFN launch (acceptmoe_moe_forward) against HBM peak,
             timed with HIP events around graph replays of the timed steps'
             forward launches; traffic from committed rocprofv3 counters;
             the rate a plain stream of the same bytes reaches
             (acceptmoe_stream_read) beside it
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


DEFAULT_CONFIG = "wide_offload"
COMPANIONS = "qwen3_30b_a3b,batched_8x64"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--config", default=DEFAULT_CONFIG,
                    help="headline workload (default: H=4096, I=1536, T=64 with a 25%% residency mask, the largest "
                         "single-tree configuration)")
    ap.add_argument("--companions", default=COMPANIONS,
                    help="comma-separated workloads timed after the headline, each with its own roofline "
                         "block ('' = none)")
    ap.add_argument("--rho", type=float, default=0.9, help="tree correlation of hidden states")
    ap.add_argument("--sets", type=int, default=0, help="weight sets to rotate (0 = enough for >= 2 GiB)")
    ap.add_argument("--blocks", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle sample budget (0 = skip)")
    ap.add_argument("--cpu-seconds-1t", type=float, default=8.0, help="single-thread oracle sample budget")
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
    ap.add_argument("--modes", action="store_true",
                    help="selector modes at a matched budget B_0 (AcceptMoE, AcceptMoE-B, MoE-Spec, Count-B, "
                         "natural routing): set sizes, routed experts and bytes, step latency")
    ap.add_argument("--modes-configs", default="qwen3_30b_a3b,wide_offload",
                    help="workloads of the --modes report")
    ap.add_argument("--tp-share", type=int, default=1, metavar="G",
                    help="time one GPU's share of a G-way tensor-parallel split over I: the same routing "
                         "(router, hidden states and trees as the full layer), experts with I/G rows")
    ap.add_argument("--ceiling", action="store_true",
                    help="reference rates of this GPU: read-only and copy streaming with plain torch kernels, "
                         "and the cost of an empty launch inside a HIP graph")
    ap.add_argument("--sweep-experts", default="",
                    help="comma-separated routed-expert counts n: forward time at --config with exactly n "
                         "experts routed (tokens spread evenly), e.g. 12,16,17,...")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                    help="only run a plain device copy of MB MiB (HBM counter calibration) and exit")
    return ap.parse_args()


# Measured HBM traffic of the forward per workload: one line per configuration,
# "traffic: config=NAME source_hash=H ratio=R ...", R = counted bytes /
# algorithmic bytes of one launch; a line applies only while the forward
# sources still hash to H.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "moe_forward_traffic.md")
FFN_SOURCES = ["paper_2608_02989_amd/csrc/forward.hip", "paper_2608_02989_amd/csrc/common.hpp"]


def ffn_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in FFN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(config: str):
    """Measured / algorithmic HBM bytes of a forward launch of `config` from the
    committed counter summary; None when that configuration was not measured
    or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    want = ffn_source_hash()
    for line in text.splitlines():
        if not line.startswith("traffic:"):
            continue
        vals = dict(kv.partition("=")[::2] for kv in line[len("traffic:"):].split())
        if vals.get("config") == config and vals.get("source_hash") == want and "ratio" in vals:
            return float(vals["ratio"])
    return None


def copy_calibration(mb: int) -> None:
    import torch
    n = mb << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {mb} MiB five times", flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def _pct(x, q):
    return round(float(np.percentile(np.asarray(x, np.float64), q)), 2)


class Workload:
    """One configuration's resident weight sets (VerifyLayer each) and seeded blocks."""

    def __init__(self, name, args, log, tp_share=1, sets=0):
        import torch

        from paper_2608_02989_amd import ops
        from paper_2608_02989_amd import workload as W

        self.dev = "cuda"
        cfg = W.CONFIGS[name]
        self.full_I = cfg.I
        if tp_share > 1:
            # one GPU's shard: the seeds depend on the configuration id, not on I,
            # so routing is the full layer's and only the expert weights shrink
            if cfg.I % (32 * tp_share) != 0:
                raise SystemExit(f"--tp-share {tp_share}: I = {cfg.I} does not split into multiples of 32")
            cfg = W.LayerConfig(**{**cfg.__dict__, "I": cfg.I // tp_share})
        self.cfg, self.tp_share, self.nblocks = cfg, tp_share, args.blocks
        self.T = cfg.total_tokens
        self.ebytes = cfg.expert_bytes
        layer_bytes = cfg.E * self.ebytes
        # enough independently seeded layers that consecutive steps never reuse
        # weights through the 256 MB Infinity Cache
        n = sets or max(2 if cfg.B > 1 else 4, int(np.ceil(2 * 2**30 / layer_bytes)))
        self.n_sets = min(n, 16)
        log(f"config {cfg.name} T={self.T} B={cfg.B} H={cfg.H} E={cfg.E} k={cfg.k} I={cfg.I} "
            f"dtype={cfg.dtype} sets={self.n_sets} blocks={self.nblocks}")
        self.layers = []
        for s in range(self.n_sets):
            rw = torch.from_numpy(W.router_weights(cfg, s)).to(self.dev)
            wg, wu, wd = W.expert_weights_torch(cfg, s, self.dev)
            self.layers.append(ops.VerifyLayer(rw, wg, wu, wd, cfg.k, max_tokens=self.T, max_trees=cfg.B))
            del wg, wu, wd
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        log("weights generated and packed")

    def blocks(self, rho):
        import torch

        from paper_2608_02989_amd import workload as W
        out = []
        for b in range(self.nblocks):
            blk = W.make_block(self.cfg, block=b, layer=0, rho=rho)
            if self.cfg.dtype == "bf16":
                h = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(self.dev)
            else:
                h = torch.from_numpy(blk.hidden).to(self.dev)
            out.append(dict(
                h=h, parent=torch.from_numpy(blk.parent).to(self.dev),
                depth=torch.from_numpy(blk.depth).to(self.dev), prob=torch.from_numpy(blk.prob).to(self.dev),
                offs=blk.offsets.tolist(),
                resident=None if blk.resident is None else torch.from_numpy(blk.resident).to(self.dev), host=blk))
        return out

    def free(self):
        import torch
        self.layers = []
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def measure(wl: Workload, rho, steps, warmup, graph=True, min_graph_steps=100):
    """Times `steps` steps (after `warmup` untimed ones) of one workload.

    A step is route -> select -> forward of one block through one weight set;
    steps rotate over (weight set, block) pairs.  The same timed sequence is
    (1) launched eagerly with HIP events around every step and every forward,
    (2) captured in one HIP graph and replayed (the headline time), and (3)
    its forward launches alone, with the routing of an untimed pre-pass, in a
    second graph (the forward's roofline).  Bytes are summed over exactly the
    timed steps.
    """
    import torch

    from paper_2608_02989_amd import ops

    cfg, layers = wl.cfg, wl.layers
    blocks = wl.blocks(rho)
    stream = torch.cuda.Stream()

    def run_once(s, b, ev=None):
        L_, B_ = layers[s], blocks[b]
        T = B_["h"].shape[0]
        nb = len(B_["offs"]) - 1
        outs = {"eligible": L_.sel_out["eligible"][:nb], "idx": L_.sel_out["idx"][:T],
                "gate": L_.sel_out["gate"][:T], "stats": L_.sel_out["stats"][:nb]}
        if ev is not None:
            ev[0].record(stream)
        ops.route(B_["h"], L_.router, out=L_.logits[:T], stream=stream)
        ops.select(L_.logits[:T], B_["parent"], B_["depth"], B_["prob"], B_["offs"], L_.k, L_.beta, L_.mode,
                   L_.budget, L_.removal_cap, B_["resident"], workspace=L_.sel_ws, outputs=outs, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        ops.moe_forward(B_["h"], L_.wgu, L_.wd, outs["idx"], outs["gate"], out=L_.out[:T],
                        workspace=L_.fwd_ws, stream=stream)
        if ev is not None:
            ev[2].record(stream)
        return outs

    # untimed pre-pass: routed union, |S'| and |U_nat| of every (set, block) pair
    # (selection is deterministic) and its routing, kept for the forward-only graph
    routed, ssize, sprime, unat, routing = {}, {}, {}, {}, {}
    with torch.cuda.stream(stream):
        for s in range(wl.n_sets):
            for b in range(wl.nblocks):
                sel = run_once(s, b)
                idx = sel["idx"]
                routing[(s, b)] = (idx.clone(), sel["gate"].clone())
                routed[(s, b)] = int(torch.unique(idx[idx >= 0]).numel())
                st = sel["stats"].cpu().numpy()
                ssize[(s, b)] = float(st[:, 3].mean())
                sprime[(s, b)] = float(st[:, 4].mean())
                unat[(s, b)] = float(st[:, 5].mean())
    torch.cuda.synchronize()
    seq = [(i % wl.n_sets, i % wl.nblocks) for i in range(warmup + steps)]
    timed = seq[warmup:]
    r = np.array([routed[c] for c in timed], np.float64)
    weight_bytes = float(r.mean()) * wl.ebytes
    eb = 2 if cfg.dtype == "bf16" else 4
    act_bytes = wl.T * cfg.H * eb + wl.T * cfg.H * 4 + wl.T * cfg.k * 8   # hidden in, out, routing in
    fwd_bytes = weight_bytes + act_bytes

    # (1) eager launches, HIP events around every step and every forward
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(steps)]
    with torch.cuda.stream(stream):
        for (s, b) in seq[:warmup]:
            run_once(s, b)
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for i, (s, b) in enumerate(timed):
            run_once(s, b, evs[i])
        stop.record(stream)
    torch.cuda.synchronize()
    eager_us = start.elapsed_time(stop) * 1e3 / steps
    step_eager = [a.elapsed_time(z) * 1e3 for a, _, z in evs]
    fwd_eager = [m.elapsed_time(z) * 1e3 for _, m, z in evs]

    def graph_time(body):
        """Average replay time of a graph of `body` (the timed sequence), replayed
        until at least min_graph_steps steps ran; per-replay times returned too."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(g, stream=stream):
                body()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        reps = max(1, -(-min_graph_steps // steps))
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        with torch.cuda.stream(stream):
            marks[0].record(stream)
            for i in range(reps):
                g.replay()
                marks[i + 1].record(stream)
        torch.cuda.synchronize()
        per = [marks[i].elapsed_time(marks[i + 1]) * 1e3 / steps for i in range(reps)]
        del g
        return marks[0].elapsed_time(marks[-1]) * 1e3 / (reps * steps), per, reps

    step_us, fwd_us, step_reps, fwd_reps, reps = None, None, None, None, 0
    if graph:
        step_us, step_reps, reps = graph_time(lambda: [run_once(s, b) for (s, b) in timed])

        def fwd_body():
            for (s, b) in timed:
                L_, B_ = layers[s], blocks[b]
                T = B_["h"].shape[0]
                ops.moe_forward(B_["h"], L_.wgu, L_.wd, routing[(s, b)][0], routing[(s, b)][1], out=L_.out[:T],
                                workspace=L_.fwd_ws, stream=stream)
        fwd_us, fwd_reps, _ = graph_time(fwd_body)
    headline_us = step_us if step_us is not None else eager_us
    fwd_time_us = fwd_us if fwd_us is not None else float(np.mean(fwd_eager))
    return dict(
        step_us=headline_us, eager_us=eager_us, graph=step_us is not None, graph_reps=reps,
        step_eager_p50=_pct(step_eager, 50), step_eager_p10=_pct(step_eager, 10), step_eager_p90=_pct(step_eager, 90),
        step_graph_replays=None if step_reps is None else [round(x, 2) for x in step_reps],
        value=weight_bytes / (headline_us * 1e-6) / 1e9,
        weight_bytes=weight_bytes, fwd_bytes=fwd_bytes, fwd_us=fwd_time_us,
        fwd_gbs=fwd_bytes / (fwd_time_us * 1e-6) / 1e9,
        fwd_eager_us=float(np.mean(fwd_eager)), fwd_eager_p50=_pct(fwd_eager, 50),
        fwd_eager_gbs=fwd_bytes / (float(np.mean(fwd_eager)) * 1e-6) / 1e9,
        fwd_timing="HIP graph of the timed steps' forward launches" if fwd_us is not None else "eager HIP events",
        routed=float(r.mean()), s_size=float(np.mean([ssize[c] for c in timed])),
        sprime=float(np.mean([sprime[c] for c in timed])),
        unat=float(np.mean([unat[c] for c in timed])),
        flops=float(wl.T * cfg.k * 6 * cfg.H * cfg.I + 2 * wl.T * cfg.E * cfg.H),
        blocks=blocks,
    )


def workload_text(wl: Workload, rho) -> str:
    cfg = wl.cfg
    txt = (f"{cfg.name}: 1 MoE layer, verify block T={wl.T} ({cfg.B} tree{'s' if cfg.B > 1 else ''} of "
           f"{cfg.T} nodes), H={cfg.H} E={cfg.E} top-{cfg.k} I={cfg.I}, {cfg.dtype} experts, fp32 router, "
           f"tree-correlated hidden rho={rho}")
    if cfg.resident_frac:
        txt += f", {int(round(cfg.resident_frac * 100))}% residency mask"
    if cfg.B > 1:
        txt += ", a separate eligible set per tree"
    if wl.tp_share > 1:
        txt += f"; one GPU's I/{wl.tp_share} shard of I={wl.full_I} (tensor parallel over I)"
    return txt


def attainable_read_gbs(nbytes: int) -> float:
    """The rate a plain stream of nbytes reaches on this GPU
    (acceptmoe_stream_read, best of 256 and 512 workgroups, each launch on a
    fresh window of an 8 GiB buffer so the Infinity Cache holds none of it)."""
    import torch

    from paper_2608_02989_amd import ops

    nbytes -= nbytes % 256
    big = max(8 << 30, 4 * nbytes)
    buf = torch.empty(big // 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(512, dtype=torch.int32, device="cuda")
    windows = big // nbytes
    best = 0.0
    for g in (256, 512):
        for i in range(3):
            ops.stream_read(buf[(i % windows) * nbytes // 4:], nbytes, sink, g)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        e0.record()
        for i in range(reps):
            ops.stream_read(buf[((i + 3) % windows) * nbytes // 4:], nbytes, sink, g)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3 / reps) / 1e9)
    del buf, sink
    torch.cuda.empty_cache()
    return best


def roofline_block(wl: Workload, m) -> dict:
    ratio = measured_traffic(wl.cfg.name) if wl.tp_share == 1 else None
    read = attainable_read_gbs(int(m["fwd_bytes"]))
    return {"bound": "hbm",
            "kernel": "acceptmoe_moe_forward (gate/up + down passes of the grouped SwiGLU FFN)",
            "achieved": round(m["fwd_gbs"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(m["fwd_gbs"] / HBM_PEAK_GBS, 4),
            "traffic": None if ratio is None else round(ratio * m["fwd_bytes"]),
            "traffic_ratio": ratio,
            "bytes_per_launch": round(m["fwd_bytes"]), "launch_us": round(m["fwd_us"], 2),
            "launch_timing": m["fwd_timing"],
            "eager_launch_us": round(m["fwd_eager_us"], 2), "eager_launch_p50_us": m["fwd_eager_p50"],
            "eager_achieved": round(m["fwd_eager_gbs"], 1),
            "mfma_util": round(m["flops"] / (m["fwd_us"] * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 5),
            "attainable_read_GBs": round(read, 1), "frac_of_attainable": round(m["fwd_gbs"] / read, 4)}


def summary(wl: Workload, m, rho) -> dict:
    return {"workload": workload_text(wl, rho), "value": round(m["value"], 1), "unit": "GB/s",
            "latency_us": round(m["step_us"], 2), "eager_latency_us": round(m["eager_us"], 2),
            "eager_step_p10_p50_p90_us": [m["step_eager_p10"], m["step_eager_p50"], m["step_eager_p90"]],
            "weight_MB_per_step": round(m["weight_bytes"] / 1e6, 1),
            "routed_experts": round(m["routed"], 2), "eligible": round(m["sprime"], 2),
            "natural_union": round(m["unat"], 2), "roofline": roofline_block(wl, m)}


def companion_run(name: str, args, log) -> dict:
    """One companion workload, measured by this script in a child process.
    Each workload gets a fresh device allocator: after a large allocation was
    freed in the same process, the Qwen3-30B-A3B forward measured 59.2 instead
    of 56.8 us (a 20 GB allocate-and-free before it sufficed), so weights are
    placed as a serving process would place them at start-up."""
    import subprocess
    cmd = [sys.executable, os.path.abspath(__file__), "--config", name, "--companions", "", "--no-alt",
           "--cpu-seconds", "0", "--steps", str(args.steps), "--warmup", str(args.warmup), "--rho", str(args.rho),
           "--graph", str(args.graph), "--blocks", str(args.blocks)]
    out = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, check=True)
    line = json.loads(out.stdout.strip().splitlines()[-1])
    c = line["config"]
    res = {"workload": c["workload"], "value": line["value"], "unit": line["unit"],
           "latency_us": line["latency_us"], "eager_latency_us": line["eager_latency_us"],
           "eager_step_p10_p50_p90_us": line["eager_step_p10_p50_p90_us"],
           "weight_MB_per_step": c["weight_MB_per_step"], "routed_experts": c["routed_experts"],
           "eligible": c["eligible"], "natural_union": c["natural_union"], "roofline": line["roofline"],
           "timing": line["timing"]}
    r = line["roofline"]
    log(f"{name}: {line['latency_us']:.1f} us/step, {line['value']:.0f} GB/s, ffn {r['launch_us']:.1f} us "
        f"({r['achieved']:.0f} GB/s), routed {c['routed_experts']:.1f} (child process)")
    return res


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
    if args.ceiling:
        ceiling_report(args)
        return
    if args.sweep_experts:
        sweep_experts_report(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the layer runs on a single MI355X; "
              "sharding it over several GPUs is designed but not built", file=sys.stderr)
        sys.exit(2)

    from paper_2608_02989_amd import workload as W

    if args.modes:
        modes_report(args)
        return
    if W.CONFIGS[args.config].layers > 1:
        stack_report(args, W.CONFIGS[args.config])
        return
    t0 = time.time()

    def log(msg):
        print(f"[bench {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    wl = Workload(args.config, args, log, tp_share=args.tp_share, sets=args.sets)
    cfg = wl.cfg
    main_m = measure(wl, args.rho, args.steps, args.warmup, graph=bool(args.graph))
    log(f"rho={args.rho}: {main_m['step_us']:.1f} us/step (eager {main_m['eager_us']:.1f}), "
        f"{main_m['value']:.0f} GB/s, ffn {main_m['fwd_us']:.1f} us ({main_m['fwd_gbs']:.0f} GB/s), "
        f"routed {main_m['routed']:.1f}")

    alt = None
    if not args.no_alt and args.rho != 0.0:
        m0 = measure(wl, 0.0, args.steps, args.warmup, graph=bool(args.graph))
        alt = {"rho": 0.0, "value": round(m0["value"], 1), "latency_us": round(m0["step_us"], 2),
               "eager_latency_us": round(m0["eager_us"], 2),
               "ffn_us": round(m0["fwd_us"], 2), "ffn_gbs": round(m0["fwd_gbs"], 1),
               "routed_experts": round(m0["routed"], 2), "eligible": round(m0["sprime"], 2),
               "natural_union": round(m0["unat"], 2)}
        log(f"rho=0: {m0['step_us']:.1f} us/step, {m0['value']:.0f} GB/s, routed {m0['routed']:.1f}")

    # ---- CPU oracle baseline on a bounded sample (headline workload only) ----
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(cfg, wl.layers, main_m["blocks"], args.cpu_seconds, args.cpu_seconds_1t, wl.ebytes, log)
    wl.free()

    companions = {}
    for name in [c for c in args.companions.split(",") if c and c != args.config]:
        companions[name] = companion_run(name, args, log)

    head = summary(wl, main_m, args.rho)
    line = {
        "metric": "verify-block MoE layer latency (us) + eligible-expert weight HBM GB/s, 1 GPU",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_m["step_us"] / 1e3, 5),
        "latency_us": head["latency_us"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": head["workload"],
                   "T": wl.T, "B": cfg.B, "H": cfg.H, "E": cfg.E, "k": cfg.k, "I": cfg.I,
                   "rho": args.rho, "weight_sets": wl.n_sets, "blocks": wl.nblocks,
                   **({"tp_share": wl.tp_share, "I_full": wl.full_I} if wl.tp_share > 1 else {}),
                   "routed_experts": head["routed_experts"], "eligible": head["eligible"],
                   "natural_union": head["natural_union"], "weight_MB_per_step": head["weight_MB_per_step"]},
        "roofline": head["roofline"],
        "cpu_baseline": cpu,
        "timing": (f"HIP graph of the {args.steps} timed steps, replayed {main_m['graph_reps']}x; value = routed "
                   "expert-weight bytes of those steps / their time" if main_m["graph"] else "eager launches"),
        "eager_latency_us": head["eager_latency_us"],
        "eager_step_p10_p50_p90_us": head["eager_step_p10_p50_p90_us"],
        "alt_iid": alt,
        "companions": companions,
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


def ceiling_report(args):
    """Reference rates of the GPU the bench runs on: the library's plain
    streaming read (acceptmoe_stream_read: contiguous shares, 16-byte
    non-temporal loads, no arithmetic) over the byte counts of the headline
    forward and its passes, each window moved through a 16 GiB buffer so no
    launch rereads what the previous one left in the Infinity Cache, best over
    workgroup counts; plain torch kernels for a read-only reduction and a
    device copy over 4 GiB buffers; and an empty launch inside a HIP graph (a
    one-element fill, 200 launches per graph)."""
    import torch

    from paper_2608_02989_amd import ops

    dev = "cuda"
    res = {"report": "streaming and launch reference rates"}
    big = 16 << 30
    buf = torch.ones(big // 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(65536, dtype=torch.int32, device=dev)
    sizes = {"wide_offload down pass (25.25 experts)": int(25.25 * 4096 * 1536 * 2),
             "wide_offload gate/up pass (25.25 experts)": int(25.25 * 2 * 4096 * 1536 * 2),
             "wide_offload forward (25.25 experts)": int(25.25 * 3 * 4096 * 1536 * 2),
             "1 GiB": 1 << 30, "batched_8x64 forward (116.4 experts)": int(116.4 * 3 * 4096 * 1536 * 2)}
    grids = [256, 512, 1024, 2048, 4096, 8192]
    reads = {}
    for name, nb in sizes.items():
        nb -= nb % 256
        windows = big // nb
        rates = {}
        for g in grids:
            def run(i, nb=nb, g=g):
                off = (i % windows) * nb
                ops.stream_read(buf[off // 4:], nb, sink, g)
            for i in range(3):
                run(i)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 20
            e0.record()
            for i in range(reps):
                run(i + 3)
            e1.record()
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) * 1e-3 / reps
            rates[g] = (round(t * 1e6, 2), round(nb / t / 1e9, 1))
        best = max(rates, key=lambda g: rates[g][1])
        reads[name] = {"bytes": nb, "best_grid": best, "us": rates[best][0], "GBs": rates[best][1],
                       "by_grid_GBs": {g: v[1] for g, v in rates.items()}}
        print(f"[ceiling] stream read {name}: {rates[best][1]} GB/s ({rates[best][0]} us, grid {best})",
              file=sys.stderr, flush=True)
    res["library_stream_read"] = reads
    del buf, sink
    torch.cuda.empty_cache()
    n = 2 << 30                                   # 2 Gi bf16 elements = 4 GiB
    a = torch.ones(n, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    acc = torch.zeros((), dtype=torch.float32, device=dev)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / reps

    t_read = timed(lambda: acc.copy_(a.sum(dtype=torch.float32)), 10)
    t_copy = timed(lambda: b.copy_(a), 10)
    res["torch_read_GBs"] = round(2 * n / t_read / 1e9, 1)
    res["torch_copy_GBs"] = round(2 * 2 * n / t_copy / 1e9, 1)
    del a, b
    tiny = torch.zeros(1, dtype=torch.float32, device=dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        tiny.fill_(1.0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for _ in range(200):
                tiny.fill_(1.0)
    g.replay()
    torch.cuda.synchronize()
    t_g = timed(g.replay, 20)
    res["graph_launch_us"] = round(t_g / 200 * 1e6, 2)
    res["bytes"] = {"read": 2 * n, "copy_read_plus_write": 4 * n}
    print(json.dumps(res), flush=True)


def sweep_experts_report(args):
    """Forward time against the exact number of routed experts n at one block
    shape: T tokens with k slots each, slot j of token t routed to expert
    (t k + j) mod n of a random n-subset (every token k distinct experts, the
    tokens spread evenly over the n experts); 4 weight sets rotate; each n
    timed as graph replays of the forward launches."""
    import torch

    from paper_2608_02989_amd import ops
    from paper_2608_02989_amd import workload as W

    dev = "cuda"
    cfg = W.CONFIGS[args.config]
    T, k, E = cfg.total_tokens, cfg.k, cfg.E
    sets = 4
    wl = []
    for s_ in range(sets):
        wg, wu, wd = W.expert_weights_torch(cfg, s_, dev)
        wl.append((ops.pack_gate_up_weights(wg, wu), ops.pack_expert_weights(wd)))
        del wg, wu, wd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    rng = np.random.default_rng(0)
    hb = W.bf16_round(rng.standard_normal((T, cfg.H)).astype(np.float32)).view(np.int16)
    h = torch.from_numpy(hb).view(torch.bfloat16).to(dev)
    out = torch.empty((T, cfg.H), dtype=torch.float32, device=dev)
    ws = ops.forward_workspace(T, cfg.H, cfg.I, E, k, torch.bfloat16, dev)
    gate = torch.full((T, k), 1.0 / k, dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()
    rows = []
    for n in [int(x) for x in args.sweep_experts.split(",")]:
        if n < k or n > E:
            raise SystemExit(f"--sweep-experts: n must be in [k, E] = [{k}, {E}] (got {n})")
        routs = []
        for s_ in range(sets):
            ex = rng.permutation(E)[:n]
            idx = np.array([[ex[(t * k + j) % n] for j in range(k)] for t in range(T)], np.int32)
            routs.append(torch.from_numpy(idx).to(dev))

        def run():
            for s_ in range(sets):
                ops.moe_forward(h, wl[s_][0], wl[s_][1], routs[s_], gate, out=out, workspace=ws, stream=stream)
        with torch.cuda.stream(stream):
            run()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(g, stream=stream):
                run()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        with torch.cuda.stream(stream):
            for _ in range(10):
                g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / (10 * sets)
        mb = n * cfg.expert_bytes / 1e6
        rows.append({"n": n, "forward_us": round(us, 2), "weight_MB": round(mb, 1), "TBs": round(mb / us, 3)})
        print(f"n={n} {us:.1f} us {mb / us:.2f} TB/s", file=sys.stderr, flush=True)
        del g
    print(json.dumps({"report": "forward time vs routed experts", "config": cfg.name, "T": T, "k": k,
                      "rows": rows}), flush=True)


def modes_report(args):
    """Selector rules at a matched budget (Sec. 4 baselines): natural routing
    (Standard SD), AcceptMoE (self-sizing), and at B_0 = the round-half-up mean
    of AcceptMoE's |S| over the same blocks (Sec. 4's budget rule) the
    fixed-budget rules AcceptMoE-B (anchor + utility), MoE-Spec (summed router
    mass) and Count-B (natural votes).  Per rule: mean |S|, |S'|, routed experts,
    routed weight bytes and the graph-replayed step time over the same timed
    step sequence.  With the residency mask (wide_offload) AcceptMoE and
    AcceptMoE-B prune against it; the baselines do not (they are evaluated at
    full residency)."""
    from paper_2608_02989_amd import _lib as L

    t0 = time.time()

    def log(msg):
        print(f"[modes {time.time() - t0:6.1f}s] {msg}", file=sys.stderr, flush=True)

    rules = [("standard_sd", L.MODE_ALL_EXPERTS), ("acceptmoe", L.MODE_SELF_SIZING),
             ("acceptmoe_b", L.MODE_FIXED_BUDGET), ("moe_spec", L.MODE_MOESPEC), ("count_b", L.MODE_COUNT)]
    report = {"report": "selector rules at a matched budget B_0", "steps": args.steps, "warmup": args.warmup,
              "blocks": args.blocks, "configs": {}}
    for name in [c for c in args.modes_configs.split(",") if c]:
        wl = Workload(name, args, log)
        per_cfg = {"workload": workload_text(wl, args.rho), "expert_MB": round(wl.ebytes / 1e6, 3)}
        for rho in (args.rho, 0.0):
            for ly in wl.layers:
                ly.mode, ly.budget = L.MODE_SELF_SIZING, 0
            base = measure(wl, rho, args.steps, args.warmup, graph=bool(args.graph))
            mean_s = base["s_size"]
            b0 = int(np.floor(mean_s + 0.5))
            rows = {}
            for rule, mode in rules:
                for ly in wl.layers:
                    ly.mode, ly.budget = mode, (b0 if mode >= L.MODE_FIXED_BUDGET else 0)
                m = base if mode == L.MODE_SELF_SIZING else measure(wl, rho, args.steps, args.warmup,
                                                                   graph=bool(args.graph))
                rows[rule] = {"S": round(m["s_size"], 2), "S_prime": round(m["sprime"], 2),
                              "routed": round(m["routed"], 2), "routed_MB": round(m["weight_bytes"] / 1e6, 1),
                              "step_us": round(m["step_us"], 2), "forward_us": round(m["fwd_us"], 2),
                              "weight_GBs": round(m["value"], 1)}
                log(f"{name} rho={rho} {rule}: {rows[rule]}")
            per_cfg[f"rho={rho}"] = {"B0": b0, "acceptmoe_mean_S": round(mean_s, 3),
                                     "natural_union": round(base["unat"], 2), "rules": rows}
        for ly in wl.layers:
            ly.mode, ly.budget = L.MODE_SELF_SIZING, 0
        report["configs"][name] = per_cfg
        wl.free()
    report["data"] = "synthetic"
    print(json.dumps(report), flush=True)


def cpu_baseline(cfg, layers, blocks, budget_s, budget_1t, ebytes, log):
    """Oracle route + select + grouped forward per block on the host cores, a
    bounded sample, with all BLAS threads and then with one thread."""
    from oracle import acceptmoe_oracle as O
    from paper_2608_02989_amd import workload as W

    L0 = layers[0]
    rw = L0.router_w.cpu().numpy().astype(np.float64)
    # the oracle reads row-major weights: regenerate the same seeded layer
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

    def blas_threads():
        try:
            from threadpoolctl import threadpool_info
            return max([int(i.get("num_threads", 1)) for i in threadpool_info()] or [1])
        except Exception:
            return os.cpu_count() or 1

    prepared = set()

    def sample(budget):
        elapsed, nbytes, n = 0.0, 0.0, 0
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
            if elapsed >= budget:
                return n, elapsed, nbytes

    threads = blas_threads()
    n, elapsed, nbytes = sample(budget_s)
    log(f"cpu oracle: {n} blocks in {elapsed:.1f}s ({threads} threads)")
    one = None
    if budget_1t > 0:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            n1, el1, nb1 = sample(budget_1t)
        log(f"cpu oracle, 1 thread: {n1} blocks in {el1:.1f}s")
        one = {"value": round(nb1 / el1 / 1e9, 4), "unit": "GB/s", "cores": 1,
               "latency_us": round(el1 / n1 * 1e6, 1), "sample": f"{n1} block passes, {el1:.1f} s"}
    del wg, wu, wd
    return {"value": round(nbytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"{n} block passes over {len(prepared)} seeded blocks of {cfg.name} (layer 0), "
                      f"route+select+grouped forward in fp64 numpy, {elapsed:.1f} s",
            "latency_us": round(elapsed / n * 1e6, 1), "one_thread": one}


if __name__ == "__main__":
    main()
