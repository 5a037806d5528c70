"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Element-by-element at sizes the oracle finishes in seconds (several scan
tiles and a ragged tail), and on every query row of every workload, the
128K ones at full size in the launch configuration the benchmark times.
"""

import numpy as np
import pytest
import torch

from gpu_util import check_rows, context, make, run, say
from oracle import pqhsa_ref as R
from paper_2609_33746_amd import pqhsa, synth

pytestmark = pytest.mark.gpu


def small(idx, **kw):
    return synth.workload(idx, **kw)


# ---------------------------------------------------------------------------
# index preparation: list-major layout, bit-exact
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("wl", [
    small(0),
    small(4, max_seq=6000, ragged_min=3000, batch=3, n_q_heads=8, n_kv_heads=2, n_list=37),
], ids=["tiny", "ragged"])
def test_prepare_layout_is_stable_list_major_sort(wl):
    inp = make(wl, seed=1)
    ctx = context(inp)
    perm, offs = ctx.index_export()
    perm, offs = perm.cpu().numpy(), offs.cpu().numpy()
    ids = inp["list_ids"].cpu().numpy()
    for b in range(wl.batch):
        n = int(inp["seq_lens"][b])
        Rr = np.arange(wl.n_sink, n - wl.n_local)
        for g in range(wl.n_kv_heads):
            a = ids[b, g, Rr]
            order = np.argsort(a, kind="stable")
            np.testing.assert_array_equal(perm[b, g, :Rr.size], Rr[order])
            assert np.all(perm[b, g, Rr.size:] == -1)
            cnt = np.bincount(a, minlength=wl.n_list)
            np.testing.assert_array_equal(offs[b, g], np.concatenate([[0], np.cumsum(cnt)]))


# ---------------------------------------------------------------------------
# end to end, every row
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("idx", [0, 1])
def test_workload_every_row(idx):
    wl = synth.workload(idx)
    inp = make(wl)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


@pytest.mark.parametrize("idx", [0, 1])
def test_norm_variant(idx):
    """Key norms outside the quantizer (r_i != 1)."""
    wl = synth.workload(idx)
    inp = make(wl, seed=3, norm_variant=True)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(0, wl.n_q_heads, 3)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


# ---------------------------------------------------------------------------
# full-size workloads (the benchmark's launch configuration), every row
# ---------------------------------------------------------------------------
@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [2, 3, 4])
def test_full_size_workloads(idx):
    """Every (sequence, query head) row of the 128K workloads, score rows
    included: 32 rows of the Llama layer, 128 of the four-sequence group-8
    layer and 512 of the sixteen ragged sequences."""
    wl = synth.workload(idx)
    inp = make(wl)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)
    # properties that hold on every row
    assert torch.isfinite(out).all()
    for b in range(wl.batch):
        k = topk[b]
        s = sel[b, :, :k]
        assert bool((s[:, 1:] > s[:, :-1]).all()) if k > 1 else True
        n = int(inp["seq_lens"][b])
        assert int(s.min()) >= wl.n_sink and int(s.max()) < n - wl.n_local
        u = unsel[b].sum(dim=1)
        assert bool((u == n - wl.n_sink - wl.n_local - k).all())


# ---------------------------------------------------------------------------
# edge cases of the method
# ---------------------------------------------------------------------------
EDGE = {
    # several scan tiles and a ragged tail: |R| = 4868 = 19 x 256 + 4
    "ragged-tail-g4": (small(1, max_seq=5000, n_list=64, topk=97), {}),
    "g1-f32": (small(0, max_seq=3000, n_list=8, topk=30), {}),
    "g2": (small(1, max_seq=3000, n_q_heads=4, n_kv_heads=2, n_list=16, topk=50), {}),
    "g8": (small(3, batch=2, max_seq=3000, n_q_heads=16, n_kv_heads=2, n_list=16, topk=60), {}),
    "k0": (small(1, max_seq=3000, n_list=16, topk=0), {}),
    "k-all": (small(1, max_seq=2000, n_list=16, topk=2000 - 132), {}),
    "no-sink-no-window": (small(1, max_seq=3000, n_list=16, topk=40, n_sink=0, n_local=0), {}),
    "k0-no-window": (small(0, max_seq=3000, n_list=16, topk=0, n_sink=0, n_local=0), {}),
    "one-list": (small(1, max_seq=3000, n_list=1, topk=40), {}),
    "many-empty-lists": (small(1, max_seq=2000, n_list=4096, topk=40), {}),
    "tiny-lists": (small(1, max_seq=3000, n_list=1500, topk=40), {}),
    "diffuse-query": (small(1, max_seq=6000, n_list=64, topk=60, temp="0.3"), {}),
    "ragged-batch": (small(4, batch=5, max_seq=6000, ragged_min=2500, n_list=40), {}),
    "window-only": (small(1, max_seq=132, n_list=4, topk=0), {}),
    "list-constant-values": (small(0, max_seq=3000, n_list=8, topk=30), dict(list_constant_values=True, noise=0.0)),
}


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_cases(name):
    wl, kw = EDGE[name]
    inp = make(wl, seed=7, **kw)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


def test_k_all_is_dense_attention():
    """rho = 1: the background is empty and the output is dense attention."""
    wl = small(1, max_seq=2000, n_list=16, topk=2000 - 132)
    inp = make(wl, seed=2)
    ctx = context(inp)
    topk, out, *_ = run(ctx, inp)
    for h in range(wl.n_q_heads):
        y = R.dense_attention_ref(inp["q"][0, h].double().cpu().numpy(),
                                  inp["k_cache"][0, h // 4].double().cpu().numpy(),
                                  inp["v_cache"][0, h // 4].double().cpu().numpy())
        got = out[0, h].double().cpu().numpy()
        assert np.max(np.abs(got - y)) / np.max(np.abs(y)) <= 2e-3


# ---------------------------------------------------------------------------
# the exact re-scan path of the top-k stage
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["forced", "starved-threshold"])
@pytest.mark.parametrize("topk", [0, 37])
def test_rescan_path(mode, topk):
    wl = small(1, max_seq=5000, n_list=64, topk=topk)
    inp = make(wl, seed=11)
    ctx = context(inp)
    if mode == "forced":
        ctx.set_option(pqhsa.OPT_FORCE_FALLBACK, 1)
    else:
        ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, 1_000_000)   # +1000 on every threshold
    topk_l, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(0, h) for h in range(wl.n_q_heads)]
    check_rows(inp, topk_l, rows, out, sel, unsel, sc)
    ctx.set_option(pqhsa.OPT_FORCE_FALLBACK, 0)
    ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, 0)
    _, out2, sel2, *_ = run(ctx, inp)
    assert torch.equal(sel2, sel)
    assert float((out2 - out).abs().max()) <= 1e-4 * float(out.abs().max())


# ---------------------------------------------------------------------------
# every indexed token a candidate: the copy tiers of the top-k stage (up to
# 4, 8 and 12 candidates per thread) and its global-memory path beyond the
# LDS capacity (12288 candidates)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n_r", [3000, 6000, 10000, 14000])
def test_candidate_volume(n_r):
    wl = small(1, max_seq=n_r + 132, n_list=96, topk=n_r // 50)
    inp = make(wl, seed=13)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, -1_000_000)   # -1000 on every threshold
    topk_l, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(0, h) for h in range(0, wl.n_q_heads, 5)]
    check_rows(inp, topk_l, rows, out, sel, unsel, sc)
    ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, 0)
    _, out2, sel2, *_ = run(ctx, inp)
    assert torch.equal(sel2, sel)
    assert float((out2 - out).abs().max()) <= 1e-4 * float(out.abs().max())


# more rows than CUs (9 x 32 = 288): the top-k stage runs two workgroups per
# CU with room for 7168 candidates each; a flood of every token takes its
# global-memory path at about 8K tokens per row, and its widest in-LDS copy
# (4097 to 7168 candidates a row) at about 6K
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("flood,n_seq", [(False, 8192), (True, 8192), (True, 6144)],
                         ids=["sampled", "every-token", "every-token-in-lds"])
def test_many_rows_small_select(flood, n_seq):
    wl = small(1, batch=9, max_seq=n_seq + 132, n_list=96, topk=160)
    inp = make(wl, seed=17)
    ctx = context(inp)
    if flood:
        ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, -1_000_000)
    topk_l, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in (0, 13, 31)]
    check_rows(inp, topk_l, rows, out, sel, unsel, sc)
    if flood:
        ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, 0)
        _, out2, sel2, *_ = run(ctx, inp)
        assert torch.equal(sel2, sel)
        assert float((out2 - out).abs().max()) <= 1e-4 * float(out.abs().max())


# ---------------------------------------------------------------------------
# the paper's own index setting: 8 subspaces of 4-bit codes (Section 3.1)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("idx", [0, 1])
def test_pq4_every_row(idx):
    wl = synth.pq4(idx)
    inp = make(wl, seed=2)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("idx", [2, 3])
def test_pq4_full_size(idx):
    """128K with 512 lists of 4-bit codes (the paper's index), every row."""
    wl = synth.pq4(idx)
    inp = make(wl)
    ctx = context(inp)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


@pytest.mark.parametrize("case", ["g1-f32", "g8", "k0", "rescan", "all-candidates"])
def test_pq4_edge_cases(case):
    if case == "g1-f32":
        wl = synth.pq4(0, max_seq=3000, topk=50)
    elif case == "g8":
        wl = synth.pq4(3, batch=1, max_seq=6000, topk=120, n_list=64)
    elif case == "k0":
        wl = synth.pq4(1, max_seq=5000, n_list=64, topk=0)
    else:
        wl = synth.pq4(1, max_seq=9000, n_list=96, topk=150)
    inp = make(wl, seed=21)
    ctx = context(inp)
    if case == "rescan":
        ctx.set_option(pqhsa.OPT_FORCE_FALLBACK, 1)
    if case == "all-candidates":
        ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, -1_000_000)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(0, wl.n_q_heads, 3)]
    check_rows(inp, topk, rows, out, sel, unsel, sc)


# ---------------------------------------------------------------------------
# mechanism variants of the background term (Appendix B): the same exact set,
# background dropped (T), filled with the global value mean (C) or with the
# mean of each list's unselected members (Bx)
# ---------------------------------------------------------------------------
VARIANTS = {"T": pqhsa.VARIANT_T, "C": pqhsa.VARIANT_C, "Bx": pqhsa.VARIANT_BX}


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("idx", [0, 1])
def test_variant_every_row(idx, variant):
    wl = synth.workload(idx)
    inp = make(wl, seed=5)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, VARIANTS[variant])
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(0, wl.n_q_heads, 1 + idx)]
    check_rows(inp, topk, rows, out, sel, unsel, sc, variant=variant)


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_variant_full_size(variant):
    """128K tokens, 1024 lists, every row; then back to the default."""
    wl = synth.workload(2)
    inp = make(wl)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, VARIANTS[variant])
    topk, out, sel, unsel, _ = run(ctx, inp)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, variant=variant)
    ctx.set_option(pqhsa.OPT_VARIANT, pqhsa.VARIANT_B)
    topk, out_b, sel_b, unsel_b, _ = run(ctx, inp)
    assert torch.equal(sel_b, sel)
    check_rows(inp, topk, rows[:4], out_b, sel_b, unsel_b)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("variant", list(VARIANTS))
def test_variant_batched_full_size(variant):
    """Each variant at 128K with four sequences and groups of 8 query heads,
    every row: an attend grid of several rounds, which puts the background
    workgroups first (none for T)."""
    wl = synth.workload(3)
    inp = make(wl, seed=2)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, VARIANTS[variant])
    topk, out, sel, unsel, _ = run(ctx, inp)
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    check_rows(inp, topk, rows, out, sel, unsel, variant=variant)


@pytest.mark.parametrize("flood", [False, True], ids=["sampled", "every-token"])
def test_variant_bx_many_rows(flood):
    """Bx on more rows than CUs (9 x 32 = 288): the Bx weights of the
    two-workgroups-per-CU top-k stage, in LDS and, with every token a
    candidate (about 8K a row), on its global-memory path."""
    wl = small(1, batch=9, max_seq=8192 + 132, n_list=96, topk=160)
    inp = make(wl, seed=23)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, pqhsa.VARIANT_BX)
    if flood:
        ctx.set_option(pqhsa.OPT_THRESHOLD_BIAS, -1_000_000)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in (0, 13, 31)]
    check_rows(inp, topk, rows, out, sel, unsel, sc, variant="Bx")


VARIANT_EDGE = {
    "g8": (small(3, batch=2, max_seq=3000, n_q_heads=16, n_kv_heads=2, n_list=16, topk=60), {}),
    "k0": (small(1, max_seq=3000, n_list=16, topk=0), {}),
    "ragged-batch": (small(4, batch=5, max_seq=6000, ragged_min=2500, n_list=40), {}),
    "many-empty-lists": (small(1, max_seq=2000, n_list=4096, topk=40), {}),
    "rescan": (small(1, max_seq=5000, n_list=64, topk=97), {}),
    "pq4": (synth.pq4(1, max_seq=9000, n_list=96, topk=150), {}),
}


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("case", list(VARIANT_EDGE))
def test_variant_edge_cases(case, variant):
    wl, kw = VARIANT_EDGE[case]
    inp = make(wl, seed=9, **kw)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, VARIANTS[variant])
    if case == "rescan":
        ctx.set_option(pqhsa.OPT_FORCE_FALLBACK, 1)
    topk, out, sel, unsel, sc = run(ctx, inp, scores=True)
    rows = [(b, h) for b in range(wl.batch) for h in range(0, wl.n_q_heads, 2)]
    check_rows(inp, topk, rows, out, sel, unsel, sc, variant=variant)


# ---------------------------------------------------------------------------
# paged KV cache read in place (block table, interleaved K|V pages)
# ---------------------------------------------------------------------------
def paged_copy(k, v, page, seed, spare=5):
    """Scatter the [B, Hkv, N, d] caches into pages [n_pages, Hkv, page, 2d]
    (K in the first d, V in the last d) at a random page per logical block."""
    B, Hkv, N, d = k.shape
    nb = -(-N // page)
    gen = torch.Generator().manual_seed(seed)
    n_pages = B * nb + spare
    table = torch.randperm(n_pages, generator=gen)[:B * nb].reshape(B, nb)
    pages = torch.full((n_pages, Hkv, page, 2 * d), float("nan"), dtype=k.dtype, device=k.device)
    for half, src in ((slice(0, d), k), (slice(d, 2 * d), v)):
        x = torch.nn.functional.pad(src, (0, 0, 0, nb * page - N))
        x = x.reshape(B, Hkv, nb, page, d).permute(0, 2, 1, 3, 4).reshape(B * nb, Hkv, page, d)
        pages[table.reshape(-1).to(k.device), :, :, half] = x
    return pages[..., :d], pages[..., d:], table.to(torch.int32).to(k.device)


PAGED = {
    "tiny-p16": (small(0), 16, "B"),
    "32k-p16": (small(1), 16, "B"),
    "32k-p1": (small(1, max_seq=6000), 1, "B"),
    "ragged-p64": (small(4, batch=5, max_seq=6000, ragged_min=2500, n_list=40), 64, "B"),
    "g8-p32-bx": (small(3, batch=2, max_seq=3000, n_q_heads=16, n_kv_heads=2, n_list=16, topk=60), 32, "Bx"),
    "128k-p16": (small(2), 16, "B"),
}


@pytest.mark.parametrize("case", list(PAGED))
def test_paged_kv_matches_contiguous(case):
    wl, page, variant = PAGED[case]
    inp = make(wl, seed=4)
    ctx = context(inp)
    ctx.set_option(pqhsa.OPT_VARIANT, VARIANTS.get(variant, pqhsa.VARIANT_B))
    topk, out, sel, unsel, _ = run(ctx, inp)
    kp, vp, table = paged_copy(inp["k_cache"], inp["v_cache"], page, seed=len(case))
    say(f"[paged] page={page} pages={kp.shape[0]} table={tuple(table.shape)}")
    out_p = ctx.decode_paged(inp["q"], kp, vp, table, page, topk)
    torch.cuda.synchronize()
    assert torch.equal(out_p, out)
    rows = [(b, h) for b in range(wl.batch) for h in range(0, wl.n_q_heads, 5)][:12]
    check_rows(inp, topk, rows, out_p, sel, unsel, variant=variant)
    with pytest.raises(pqhsa.PQHSAError) as e:   # a table too short for the longest sequence
        n_max = int(inp["seq_lens"].max())
        ctx.decode_paged(inp["q"], kp, vp, table[:, :(n_max - 1) // page].contiguous(), page, topk)
    assert e.value.status == pqhsa.ERR_INVALID_ARGUMENT


# ---------------------------------------------------------------------------
# repeatability and the plain decode entry point
# ---------------------------------------------------------------------------
def test_repeatable_and_plain_decode_matches_debug():
    wl = small(1, max_seq=8192, n_list=64, topk=160)
    inp = make(wl, seed=5)
    ctx = context(inp)
    topk, out, sel, unsel, _ = run(ctx, inp)
    _, out_b, sel_b, unsel_b, _ = run(ctx, inp)
    assert torch.equal(sel, sel_b) and torch.equal(unsel, unsel_b)
    assert float((out - out_b).abs().max()) <= 1e-6 * float(out.abs().max())
    plain = ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], topk)
    torch.cuda.synchronize()
    assert float((plain - out).abs().max()) <= 1e-6 * float(out.abs().max())


def test_strided_cache_view():
    """A cache viewed through larger strides (padded token rows) is read in place."""
    wl = small(1, max_seq=3000, n_list=16, topk=40)
    inp = make(wl, seed=4)
    ctx = context(inp)
    topk, ref_out, *_ = run(ctx, inp)
    big_k = torch.zeros((1, 8, 3000, 256), dtype=torch.bfloat16, device="cuda")
    big_v = torch.zeros_like(big_k)
    big_k[..., 64:192] = inp["k_cache"]
    big_v[..., 64:192] = inp["v_cache"]
    out = ctx.decode(inp["q"], big_k[..., 64:192], big_v[..., 64:192], topk)
    torch.cuda.synchronize()
    assert float((out - ref_out).abs().max()) <= 1e-6 * float(ref_out.abs().max())


# ---------------------------------------------------------------------------
# dense baseline
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("wl", [small(0), small(1, max_seq=5000), small(4, batch=3, max_seq=6000,
                                                                         ragged_min=1000, n_list=8),
                                small(3, batch=1, max_seq=3000, n_list=8, topk=10)],
                         ids=["f32", "bf16", "ragged", "g8"])
def test_dense_decode(wl):
    inp = make(wl, seed=9)
    ctx = pqhsa.context_for(inp)
    lens = inp["seq_lens"].tolist()
    say(f"[dense] lens={lens}")
    out = ctx.dense_decode(inp["q"], inp["k_cache"], inp["v_cache"], lens)
    torch.cuda.synchronize()
    G = wl.n_q_heads // wl.n_kv_heads
    for b in range(wl.batch):
        n = lens[b]
        for h in range(wl.n_q_heads):
            y = R.dense_attention_ref(inp["q"][b, h].double().cpu().numpy(),
                                      inp["k_cache"][b, h // G, :n].double().cpu().numpy(),
                                      inp["v_cache"][b, h // G, :n].double().cpu().numpy())
            got = out[b, h].double().cpu().numpy()
            assert np.max(np.abs(got - y)) / np.max(np.abs(y)) <= 2e-3, (b, h)
    # cross-check against torch's attention in float32 for the first sequence
    b = 0
    n = lens[b]
    qf = inp["q"][b].float()[None, :, None, :]
    kf = inp["k_cache"][b, :, :n].float().repeat_interleave(G, dim=0)[None].contiguous()
    vf = inp["v_cache"][b, :, :n].float().repeat_interleave(G, dim=0)[None].contiguous()
    ref = torch.nn.functional.scaled_dot_product_attention(qf, kf, vf)[0, :, 0]
    assert float((ref - out[b]).abs().max()) <= 2e-3 * float(ref.abs().max())


def test_dense_decode_many_splits():
    """More than 64 splits of 2048 rows: the merge folds the partials in
    several thread groups at once (sampled rows, fp64 reference)."""
    wl = small(1, max_seq=135_000, n_q_heads=4, n_kv_heads=2, n_list=32, topk=100)
    inp = make(wl, seed=11)
    ctx = pqhsa.context_for(inp)
    lens = inp["seq_lens"].tolist()
    say(f"[dense many splits] lens={lens}")
    out = ctx.dense_decode(inp["q"], inp["k_cache"], inp["v_cache"], lens)
    torch.cuda.synchronize()
    G = wl.n_q_heads // wl.n_kv_heads
    n = lens[0]
    for h in (0, 3):
        y = R.dense_attention_ref(inp["q"][0, h].double().cpu().numpy(),
                                  inp["k_cache"][0, h // G, :n].double().cpu().numpy(),
                                  inp["v_cache"][0, h // G, :n].double().cpu().numpy())
        got = out[0, h].double().cpu().numpy()
        assert np.max(np.abs(got - y)) / np.max(np.abs(y)) <= 2e-3, h


# ---------------------------------------------------------------------------
# argument checks that need a device
# ---------------------------------------------------------------------------
def test_abi_errors_on_gpu():
    wl = small(1, max_seq=3000, n_list=16, topk=40)
    inp = make(wl, seed=1)
    ctx = pqhsa.context_for(inp)
    with pytest.raises(pqhsa.PQHSAError) as e:
        ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], [40])
    assert e.value.status == pqhsa.ERR_NOT_PREPARED
    # list ids of R are checked on the device; the first offending (b, g, i) is named
    bad = inp["list_ids"].clone()
    bad[0, 3, 500] = 16
    bad[0, 5, 7] = -2
    with pytest.raises(pqhsa.PQHSAError) as e:
        ctx.index_prepare([3000], bad, inp["codes"], inp["norms"], inp["centroids"],
                          inp["codebooks"], inp["list_means"])
    assert e.value.status == pqhsa.ERR_INVALID_ARGUMENT
    assert "list_ids[0][3][500] = 16" in str(e.value), str(e.value)
    bad[0, 3, 500] = 0
    with pytest.raises(pqhsa.PQHSAError) as e:
        ctx.index_prepare([3000], bad, inp["codes"], inp["norms"], inp["centroids"],
                          inp["codebooks"], inp["list_means"])
    assert "list_ids[0][5][7] = -2" in str(e.value), str(e.value)
    with pytest.raises(pqhsa.PQHSAError) as e:   # still unprepared
        ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], [40])
    assert e.value.status == pqhsa.ERR_NOT_PREPARED
    # ids outside R (sinks, local window, past N) are not part of the index
    bad = inp["list_ids"].clone()
    bad[0, :, :4] = 99
    bad[0, :, 3000 - 128:] = -5
    ctx.index_prepare([3000], bad, inp["codes"], inp["norms"], inp["centroids"],
                      inp["codebooks"], inp["list_means"])
    with pytest.raises(pqhsa.PQHSAError) as e:
        ctx.index_prepare([100], inp["list_ids"], inp["codes"], inp["norms"], inp["centroids"],
                          inp["codebooks"], inp["list_means"])
    assert e.value.status == pqhsa.ERR_INVALID_ARGUMENT
    pqhsa.prepare_from(ctx, inp)
    for k in (-1, 41, 3000):
        with pytest.raises(pqhsa.PQHSAError) as e:
            ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], [k])
        assert e.value.status == pqhsa.ERR_INVALID_ARGUMENT
    with pytest.raises(pqhsa.PQHSAError):
        ctx.dense_decode(inp["q"], inp["k_cache"], inp["v_cache"], [0])
    for v in (-1, 4):
        with pytest.raises(pqhsa.PQHSAError) as e:
            ctx.set_option(pqhsa.OPT_VARIANT, v)
        assert e.value.status == pqhsa.ERR_INVALID_ARGUMENT
    out = ctx.decode(inp["q"], inp["k_cache"], inp["v_cache"], [40])
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
