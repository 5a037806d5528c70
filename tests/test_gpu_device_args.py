"""The decode step with budgets and lengths as device data
(pqhsa_decode_device_args): the same output as the host-argument call for the
same N_b and k_b, bit for bit, also when it is captured in a graph and
replayed with new values written between replays."""

import pytest
import torch

from gpu_util import context, make, say
from paper_2609_33746_amd import synth

pytestmark = pytest.mark.gpu

WORKLOADS = {
    "ragged-g4": synth.workload(4, max_seq=6000, ragged_min=3000, batch=3, n_q_heads=8,
                                n_kv_heads=2, n_list=37),
    "g8": synth.workload(3, max_seq=5000, batch=2, n_q_heads=16, n_kv_heads=2, n_list=64, topk=90),
    "128k": synth.workload(2),
}


def host_call(ctx, inp, lens, topk):
    ctx.set_lengths(lens)
    out = ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], topk)
    torch.cuda.synchronize()
    return out


def dev_i32(values):
    return torch.tensor(list(values), dtype=torch.int32, device="cuda")


def cases(inp, ctx_max_topk, max_seq):
    lens = [int(x) for x in inp["seq_lens"]]
    topk = [int(x) for x in inp["topk"]]
    grown = [min(n + 300, max_seq) for n in lens]
    return [
        ("indexed", lens, topk),
        ("half budget", lens, [t // 2 for t in topk]),
        ("no budget", lens, [0] * len(lens)),
        ("grown tail", grown, topk),
        ("full budget", grown, [ctx_max_topk] * len(lens)),
    ]


@pytest.mark.parametrize("name", ["ragged-g4", "g8", "128k"])
def test_device_args_match_host_args(name):
    wl = WORKLOADS[name]
    inp = make(wl, seed=5)
    ctx = context(inp)
    mt = ctx.shape.max_topk
    for label, lens, topk in cases(inp, mt, wl.max_seq):
        say(f"[device args] {name}: {label}")
        ref = host_call(ctx, inp, lens, topk)
        got = ctx.decode_device_args(inp["q"], inp["k_cache"], inp["v_cache"], dev_i32(lens),
                                     dev_i32(topk))
        torch.cuda.synchronize()
        assert torch.equal(got, ref), label
    # out-of-range budgets are clamped into [0, min(|R_b|, max_topk)]
    lens = [int(x) for x in inp["seq_lens"]]
    ref = host_call(ctx, inp, lens, [mt] * wl.batch)
    got = ctx.decode_device_args(inp["q"], inp["k_cache"], inp["v_cache"], dev_i32(lens),
                                 dev_i32([10 ** 6] * wl.batch))
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    ref = host_call(ctx, inp, lens, [0] * wl.batch)
    got = ctx.decode_device_args(inp["q"], inp["k_cache"], inp["v_cache"], dev_i32(lens),
                                 dev_i32([-7] * wl.batch))
    torch.cuda.synchronize()
    assert torch.equal(got, ref)


@pytest.mark.parametrize("name", ["ragged-g4", "128k"])
def test_device_args_graph_replays(name):
    wl = WORKLOADS[name]
    inp = make(wl, seed=6)
    ctx = context(inp)
    mt = ctx.shape.max_topk
    q, kc, vc = inp["q"], inp["k_cache"], inp["v_cache"]
    lens0 = [int(x) for x in inp["seq_lens"]]
    topk0 = [int(x) for x in inp["topk"]]
    lens_d, topk_d = dev_i32(lens0), dev_i32(topk0)
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    ctx.decode_device_args(q, kc, vc, lens_d, topk_d, out=out)   # eager warm-up
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ctx.decode_device_args(q, kc, vc, lens_d, topk_d, out=out)
    torch.cuda.synchronize()
    for label, lens, topk in cases(inp, mt, wl.max_seq) * 2:
        say(f"[graph] {name}: replay with {label}")
        lens_d.copy_(dev_i32(lens))
        topk_d.copy_(dev_i32(topk))
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ref = host_call(ctx, inp, lens, topk)   # eager work between the replays
        assert torch.equal(out, ref), label
