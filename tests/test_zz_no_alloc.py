"""The dense decode entry point that allocates nothing
(pqhsa_dense_decode_noalloc), through the C ABI: on two calls in a row, the
second smaller, and on a repeat of the first, its output equals the
context-based dense decode's bit for bit (the same kernels over the same
splits) and the oracle's within the operator's bar."""

import numpy as np
import pytest
import torch

from gpu_util import OUT_TOL, make, say
from oracle import pqhsa_ref as R
from paper_2609_33746_amd import pqhsa, synth

pytestmark = pytest.mark.gpu


def _against_context_and_oracle(inp, out):
    wl = inp["workload"]
    lens = inp["seq_lens"].tolist()
    ctx = pqhsa.context_for(inp)
    ref = ctx.dense_decode(inp["q"], inp["k_cache"], inp["v_cache"], lens)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    G = wl.n_q_heads // wl.n_kv_heads
    worst = 0.0
    for b in range(wl.batch):
        n = lens[b]
        for h in range(0, wl.n_q_heads, max(1, wl.n_q_heads // 4)):
            y = R.dense_attention_ref(inp["q"][b, h].double().cpu().numpy(),
                                      inp["k_cache"][b, h // G, :n].double().cpu().numpy(),
                                      inp["v_cache"][b, h // G, :n].double().cpu().numpy())
            got = out[b, h].double().cpu().numpy()
            err = float(np.max(np.abs(got - y)) / np.max(np.abs(y)))
            assert err <= OUT_TOL, (b, h, err)
            worst = max(worst, err)
    ctx.close()
    say(f"[noalloc] {wl.name}: equal to the context's dense decode, worst oracle error {worst:.2e}")


def test_noalloc_dense_two_calls_second_smaller():
    big = make(synth.workload(4, batch=3, max_seq=20000, ragged_min=9000, n_list=8), seed=3)
    small = make(synth.workload(4, batch=2, max_seq=6000, ragged_min=3000, n_q_heads=8,
                                n_kv_heads=2, n_list=8), seed=4)
    outs = []
    for inp in (big, small, big):
        lens = inp["seq_lens"].tolist()
        say(f"[noalloc] call: batch {len(lens)} lens {lens} heads {tuple(inp['q'].shape[1:2])}")
        out = pqhsa.dense_decode_noalloc(inp["q"], inp["k_cache"], inp["v_cache"], lens)
        torch.cuda.synchronize()
        outs.append(out)
    _against_context_and_oracle(big, outs[0])
    _against_context_and_oracle(small, outs[1])
    assert torch.equal(outs[2], outs[0])


def test_noalloc_dense_f32_single_head():
    inp = make(synth.workload(0), seed=5)
    out = pqhsa.dense_decode_noalloc(inp["q"], inp["k_cache"], inp["v_cache"],
                                     inp["seq_lens"].tolist())
    torch.cuda.synchronize()
    _against_context_and_oracle(inp, out)
