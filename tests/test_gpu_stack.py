"""A stack of verify layers chained by the residual stream (h_{l+1} = h_l + y_l
rounded to bf16), checked teacher-forced per layer against the oracle (each
oracle layer takes the GPU's input and logits, so fp drift cannot change later
routing), the residual add bit-exact, a HIP-graph capture of the whole pass
replayed against the eager result, and two blocks in flight on two streams."""
import numpy as np
import pytest
import torch

from oracle import acceptmoe_oracle as O
from paper_2608_02989_amd import ops
from paper_2608_02989_amd import workload as W

from _util import GATE_RTOL, LOGIT_TOL, HostExperts, check_forward, normwise_rel

pytestmark = pytest.mark.gpu
DEV = "cuda"
NL = 6


def say(*a):
    print(*a, flush=True)


def small_stack():
    cfg = W.LayerConfig("stack_small", 130, "bf16", T=20, B=1, H=256, E=32, k=4, I=128, depth_max=5,
                        commit_rule="depth_sibling", hidden_std=1.0)
    layers, host = [], []
    for l in range(NL):
        rw = W.router_weights(cfg, l)
        wg, wu, wd = W.expert_weights_torch(cfg, l, DEV)
        layers.append(ops.VerifyLayer(torch.from_numpy(rw).to(DEV), wg, wu, wd, cfg.k, max_tokens=cfg.T))
        host.append((rw, HostExperts(wg), HostExperts(wu), HostExperts(wd)))
    return cfg, ops.VerifyStack(layers, cfg.T), host


def block_inputs(cfg, b):
    blk = W.make_block(cfg, block=b, rho=0.9)
    h = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(DEV)
    return h, tuple(torch.from_numpy(a).to(DEV) for a in (blk.parent, blk.depth, blk.prob)), blk


def bits(t):
    return t.detach().cpu().view(torch.int16).numpy()


def test_stack_teacher_forced(gpu):
    cfg, stack, host = small_stack()
    h0, tree, blk = block_inputs(cfg, 0)
    say("stack of", NL, "layers, teacher-forced")
    stack.step(h0, *tree)
    torch.cuda.synchronize()
    for l, layer in enumerate(stack.layers):
        rw, wg, wu, wd = host[l]
        hb = bits(stack.h[l][:cfg.T]).view(np.uint16)
        h64 = O.widen_bf16(hb)
        z_gpu = layer.logits[:cfg.T].cpu().numpy()
        assert normwise_rel(z_gpu, O.route(h64, rw.astype(np.float64))) <= LOGIT_TOL, l
        ref = O.select(z_gpu, blk.parent, blk.depth, blk.prob, None, cfg.k)
        assert not ref["ambiguous"].any()
        idx = layer.sel_out["idx"][:cfg.T].cpu().numpy()
        assert np.array_equal(idx, ref["idx"]), l
        gate = layer.sel_out["gate"][:cfg.T].cpu().numpy()
        assert np.allclose(gate, ref["gate"], rtol=GATE_RTOL, atol=0), l
        y = layer.out[:cfg.T].cpu().numpy()
        y_ref = O.moe_forward_grouped(h64, wg, wu, wd, ref["idx"], ref["gate"], "bf16")
        check_forward(y, y_ref, "bf16", f"stack layer {l}")
        # residual: the fp32 sum rounded to nearest even, bit for bit
        want = W.bf16_round(O.widen_bf16(hb).astype(np.float32) + y)
        assert np.array_equal(bits(stack.h[l + 1][:cfg.T]).view(np.uint16), want), l


def test_stack_graph_replay_and_two_streams(gpu):
    cfg, stack, _ = small_stack()
    inputs = [block_inputs(cfg, b)[:2] for b in range(2)]
    eager = []
    for h0, tree in inputs:
        eager.append(bits(stack.step(h0, *tree)).copy())
    torch.cuda.synchronize()
    # one HIP graph for the whole pass; replays interleaved with eager work
    h_in = torch.empty_like(inputs[0][0])
    tree_in = tuple(torch.empty_like(t) for t in inputs[0][1])

    def load(b):
        h_in.copy_(inputs[b][0])
        for dst, src in zip(tree_in, inputs[b][1]):
            dst.copy_(src)

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    load(0)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        stack.step(h_in, *tree_in)  # warm-up on the capture stream
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        out_g = stack.step(h_in, *tree_in)
    for rep in range(3):
        say("graph replay", rep)
        load(rep % 2)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(out_g), eager[rep % 2]), rep
        stack.layers[0].step(inputs[1][0], *inputs[1][1])  # unrelated eager work between replays
        torch.cuda.synchronize()
    # two blocks in flight on two streams, each with its own buffers
    twin = stack.twin()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        o1 = stack.step(inputs[0][0], *inputs[0][1], stream=s1)
    with torch.cuda.stream(s2):
        o2 = twin.step(inputs[1][0], *inputs[1][1], stream=s2)
    torch.cuda.synchronize()
    assert np.array_equal(bits(o1), eager[0]) and np.array_equal(bits(o2), eager[1])


def test_stack_full_size_48_layers(gpu):
    """The 48-layer Qwen3-30B-A3B-shaped stack at its full size (T = 60 nodes,
    the pass bench.py times), teacher-forced per layer: logits, routing, gates
    and the residual add on every layer; the full expert output on four
    sampled layers (their weights regenerated from the same seeds)."""
    cfg = W.CONFIGS["qwen3_30b_a3b_x48"]
    T = cfg.T
    layers = []
    for l in range(cfg.layers):
        wg, wu, wd = W.expert_weights_torch(cfg, l, DEV)
        layers.append(ops.VerifyLayer(torch.from_numpy(W.router_weights(cfg, l)).to(DEV), wg, wu, wd, cfg.k,
                                      max_tokens=T))
        del wg, wu, wd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    stack = ops.VerifyStack(layers, T)
    blk = W.make_block(cfg, block=5, layer=0, rho=0.9, tree_layer=0)
    h0 = torch.from_numpy(W.bf16_round(blk.hidden).view(np.int16)).view(torch.bfloat16).to(DEV)
    tree = tuple(torch.from_numpy(a).to(DEV) for a in (blk.parent, blk.depth, blk.prob))
    say(f"full-size stack: {cfg.layers} layers, T={T}")
    stack.step(h0, *tree)
    torch.cuda.synchronize()
    sampled = {0, 16, 33, cfg.layers - 1}
    sizes = []
    for l, layer in enumerate(stack.layers):
        hb = bits(stack.h[l][:T]).view(np.uint16)
        h64 = O.widen_bf16(hb)
        z_gpu = layer.logits[:T].cpu().numpy()
        rw = W.router_weights(cfg, l)
        assert normwise_rel(z_gpu, O.route(h64, rw.astype(np.float64))) <= LOGIT_TOL, l
        ref = O.select(z_gpu, blk.parent, blk.depth, blk.prob, None, cfg.k)
        assert not ref["ambiguous"].any(), l
        assert np.array_equal(layer.sel_out["idx"][:T].cpu().numpy(), ref["idx"]), l
        assert np.array_equal(layer.sel_out["eligible"][:1].cpu().numpy(), ref["eligible"]), l
        assert np.allclose(layer.sel_out["gate"][:T].cpu().numpy(), ref["gate"], rtol=GATE_RTOL, atol=0), l
        sizes.append(int(ref["eligible"].sum()))
        y = layer.out[:T].cpu().numpy()
        if l in sampled:
            wg, wu, wd = W.expert_weights_torch(cfg, l, DEV)
            y_ref = O.moe_forward_grouped(h64, HostExperts(wg), HostExperts(wu), HostExperts(wd), ref["idx"],
                                          ref["gate"], "bf16")
            del wg, wu, wd
            figs = check_forward(y, y_ref, "bf16", f"48-layer stack layer {l}")
            say(f"  layer {l}: |S'| = {sizes[-1]}, output error {figs['normwise']:.2e}")
        want = W.bf16_round(h64.astype(np.float32) + y)
        assert np.array_equal(bits(stack.h[l + 1][:T]).view(np.uint16), want), l
    say(f"  |S'| over the layers: min {min(sizes)}, mean {np.mean(sizes):.1f}, max {max(sizes)}")
