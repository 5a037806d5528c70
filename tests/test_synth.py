"""Seeded generator: shapes, determinism, budgets and list means."""

import numpy as np
import pytest
import torch

from oracle import pqhsa_ref as R
from paper_2609_33746_amd import synth


def small(idx, **kw):
    base = dict(max_seq=2048, n_list=8)
    base.update(kw)
    return synth.workload(idx, **base)


def test_workload_budgets():
    assert synth.WORKLOADS[0].topk == 64
    assert synth.WORKLOADS[1].topk == synth.ratio_topk(0.02, 32768) == 655
    assert synth.WORKLOADS[2].topk == synth.ratio_topk(0.01, 131072) == 1311
    assert synth.WORKLOADS[3].topk == synth.ratio_topk(0.02, 131072) == 2621


def test_shapes_and_dtypes():
    wl = small(1, batch=2, topk=20)
    inp = synth.make_inputs(wl, seed=3)
    B, Hq, Hkv, d, N = 2, 32, 8, 128, 2048
    assert inp["q"].shape == (B, Hq, d) and inp["q"].dtype == torch.bfloat16
    assert inp["k_cache"].shape == (B, Hkv, N, d) and inp["v_cache"].dtype == torch.bfloat16
    assert inp["codes"].shape == (B, Hkv, N, 16) and inp["codes"].dtype == torch.uint8
    assert inp["codebooks"].shape == (B, Hkv, 16, 256, 8)
    assert inp["list_ids"].dtype == torch.int32 and int(inp["list_ids"].max()) < 8
    assert inp["seq_lens"].tolist() == [N, N] and inp["topk"].tolist() == [20, 20]


def test_deterministic():
    wl = small(0)
    a = synth.make_inputs(wl, seed=5)
    b = synth.make_inputs(wl, seed=5)
    c = synth.make_inputs(wl, seed=6)
    for key in ("q", "k_cache", "v_cache", "list_ids", "codes", "list_means"):
        assert torch.equal(a[key], b[key])
    assert not torch.equal(a["k_cache"], c["k_cache"])


def test_ragged_lengths_and_budgets():
    wl = synth.workload(4, max_seq=4096, ragged_min=2048, n_list=8, batch=5, n_kv_heads=2)
    inp = synth.make_inputs(wl, seed=1)
    lens = inp["seq_lens"].numpy()
    assert np.all((lens >= 2048) & (lens <= 4096))
    assert inp["topk"].tolist() == [int(np.floor(0.01 * n + 0.5)) for n in lens]
    # entries past each sequence's end stay zero
    for b, n in enumerate(lens):
        assert float(inp["k_cache"][b, :, n:].abs().sum()) == 0.0


@pytest.mark.parametrize("kw", [dict(), dict(norm_variant=True), dict(list_constant_values=True)])
def test_list_means_are_means_over_indexed_members(kw):
    wl = small(1, n_q_heads=4, n_kv_heads=2, topk=10)
    inp = synth.make_inputs(wl, seed=2, **kw)
    for g in range(2):
        n = int(inp["seq_lens"][0])
        Rr = np.arange(wl.n_sink, n - wl.n_local)
        ref = R.list_means_ref(inp["v_cache"][0, g].double().numpy(),
                               inp["list_ids"][0, g].numpy(), wl.n_list, Rr)
        np.testing.assert_allclose(inp["list_means"][0, g].numpy(), ref, rtol=2e-7, atol=1e-7)


def test_keys_follow_the_index_recipe():
    wl = small(0, kv_dtype="f32")
    inp = synth.make_inputs(wl, seed=4, noise=0.0, norm_variant=True)
    a = inp["list_ids"][0, 0].long()
    z = inp["codes"][0, 0].long()
    cen = inp["centroids"][0, 0].double()
    cb = inp["codebooks"][0, 0].double()
    recon = cen[a] + torch.cat([cb[m][z[:, m]] for m in range(16)], dim=1)
    recon = recon * inp["norms"][0, 0].double()[:, None]
    torch.testing.assert_close(inp["k_cache"][0, 0].double(), recon, rtol=1e-5, atol=1e-5)


def test_pq4_workloads_use_the_papers_index_setting():
    wl = synth.pq4(2)
    assert (wl.pq_m, wl.pq_ksub, wl.n_list) == (8, 16, 512)
    small = synth.pq4(0, max_seq=600, topk=8)
    inp = synth.make_inputs(small, seed=0)
    assert inp["codes"].shape[-1] == 8 and int(inp["codes"].max()) < 16
    assert tuple(inp["codebooks"].shape[-3:]) == (8, 16, 16)
