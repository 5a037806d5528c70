"""Benchmark of one PQ-HSA decode-attention call on one MI355X.

A step is one pqhsa_decode call (LUT build + threshold sample, code scan,
top-k select, exact attention + per-list background, merge) over the
Llama-3.1-8B-shaped 128K workload: batch 1, 32 query / 8 KV heads, d = 128,
N = 131072 bf16 K/V, 1024 lists, 16 x 8-bit PQ codes, k = 1311 (1%).
Inputs are synthetic and resident in HBM before timing. Between timed calls
a 1 GB buffer is read so that neither the 256 MB Infinity Cache nor L2 holds
the operator's data (a decode step of a real model runs the other layers in
between, whose traffic is mostly weight and KV reads); each call is
bracketed by HIP events on its stream. Overwriting the buffer instead would
leave the Infinity Cache full of dirty lines whose write-back competes with
the call's reads (a plain streaming read drops from 6.4 to 4.1 TB/s on
MI355X); that number is reported too, as us_per_call_write_flush.

Prints one JSON line (rank 0) with the per-call time, throughput forms, the
HBM roofline of the dominant (longest) kernel and of the whole call, the
same-chip dense decode and the CPU oracle baseline.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
FLUSH_BYTES = 1 << 30
COPY_CAL_BYTES = 256 << 20
WORKLOAD = 2


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(inp, topk, sel_union):
    """Bytes each stage must read (and the output it must write), per call.

    a1 LUT:    q (G d s_q) + centroids (n_list d 4) + codebooks (256 d 4) per (b, g)
    a2 scan:   codes + norms (M b / 8 + 4 per indexed token) + list offsets ((n_list+1) 4)
    a3 select: the selected ids (G k 4) per (b, g)
    a4 attend: the distinct gathered K and V rows (U 2 d s_kv) per (b, g)
    a5 bg:     list means (n_list d 4) per (b, g)
    a6 merge:  the fp32 output (B Hq d 4)
    """
    wl = inp["workload"]
    d = wl.head_dim
    s_kv = 2 if wl.kv_dtype == "bf16" else 4
    G = wl.n_q_heads // wl.n_kv_heads
    by = dict(lut=0, scan=0, select=0, attend=0, background=0, out=0)
    for b in range(wl.batch):
        n = int(inp["seq_lens"][b])
        n_r = n - wl.n_sink - wl.n_local
        for g in range(wl.n_kv_heads):
            by["lut"] += G * d * s_kv + wl.n_list * d * 4 + wl.pq_ksub * d * 4
            code_bytes = wl.pq_m * (wl.pq_ksub.bit_length() - 1) // 8
            by["scan"] += n_r * (code_bytes + 4) + (wl.n_list + 1) * 4
            by["select"] += G * topk[b] * 4
            by["attend"] += sel_union[b][g] * 2 * d * s_kv
            by["background"] += wl.n_list * d * 4
    by["out"] = wl.batch * wl.n_q_heads * d * 4
    return by


def config_sweep(args, dev) -> int:
    """Every synthetic workload (0-4) at its own shape: mean µs per call with
    the caches flushed between calls (as the bench line), the dense decode of
    the same cache, and the algorithmic bytes per stage (rooflines against the
    8 TB/s HBM peak). One JSON line per workload."""
    import numpy as np
    import torch

    from paper_2609_33746_amd import pqhsa, synth

    flush_buf = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def timed(fn, steps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        for i in range(steps):
            torch.sum(flush_buf)
            ev[i][0].record(stream)
            fn()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in ev])) * 1e3

    for idx in range(5):
        wl = synth.workload(idx)
        log(f"config {idx}: {wl.name}")
        inp = synth.make_inputs(wl, seed=args.seed, device=dev)
        topk = inp["topk"].tolist()
        lens = inp["seq_lens"].tolist()
        ctx = pqhsa.context_for(inp)
        pqhsa.prepare_from(ctx, inp)
        q, kc, vc = inp["q"], inp["k_cache"], inp["v_cache"]
        out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        out_d = torch.empty_like(out)
        steps = max(20, args.steps // 4)
        for _ in range(args.warmup):
            ctx.decode(q, kc, vc, topk, out=out)
        us = timed(lambda: ctx.decode(q, kc, vc, topk, out=out), steps)
        ctx.set_option(pqhsa.OPT_STAGE_TIMING, 1)
        acc = {}
        for _ in range(20):
            torch.sum(flush_buf)
            ctx.decode(q, kc, vc, topk, out=out)
            for k_, v_ in ctx.stage_times().items():
                acc.setdefault(k_, []).append(v_)
        ctx.set_option(pqhsa.OPT_STAGE_TIMING, 0)
        stage_us = {k_: float(np.mean(v_)) * 1e3 for k_, v_ in acc.items()}
        for _ in range(3):
            ctx.dense_decode(q, kc, vc, lens, out=out_d)
        dense_us = timed(lambda: ctx.dense_decode(q, kc, vc, lens, out=out_d), max(10, steps // 2))
        _, sel, _, _ = ctx.decode_debug(q, kc, vc, topk)
        torch.cuda.synchronize()
        G = wl.n_q_heads // wl.n_kv_heads
        sel_c = sel.cpu().numpy()
        union = [[int(np.unique(sel_c[b, g * G:(g + 1) * G, :topk[b]]).size) + wl.n_sink + wl.n_local
                  for g in range(wl.n_kv_heads)] for b in range(wl.batch)]
        by = algorithmic_bytes(inp, topk, union)
        total = sum(by.values())
        stage_bytes = dict(prologue=by["lut"], scan=by["scan"], select=by["select"],
                           attend=by["attend"] + by["background"], merge=by["out"])
        s_kv = 2 if wl.kv_dtype == "bf16" else 4
        dense_bytes = sum(n * wl.n_kv_heads * 2 * wl.head_dim * s_kv for n in lens)
        n_scanned = sum((n - wl.n_sink - wl.n_local) * wl.n_kv_heads for n in lens)
        print(json.dumps({
            "workload": wl.name, "batch": wl.batch, "n_q_heads": wl.n_q_heads,
            "n_kv_heads": wl.n_kv_heads, "max_seq": wl.max_seq, "seq_lens": [min(lens), max(lens)],
            "kv_dtype": wl.kv_dtype, "n_list": wl.n_list, "topk": [min(topk), max(topk)],
            "us_per_call": round(us, 3),
            "tokens_scanned_per_s": n_scanned / (us * 1e-6),
            "hbm_gbps_algorithmic": round(total / (us * 1e-6) / 1e9, 1),
            "call_roofline_frac": round(total / (us * 1e-6) / 8e12, 4),
            "stage_us": {k_: round(v_, 3) for k_, v_ in stage_us.items()},
            "stage_roofline_frac": {k_: round(stage_bytes[k_] / (stage_us[k_] * 1e-6) / 8e12, 4)
                                    for k_ in stage_us},
            "dense_us_per_call": round(dense_us, 3),
            "dense_hbm_gbps": round(dense_bytes / (dense_us * 1e-6) / 1e9, 1),
            "speedup_vs_dense": round(dense_us / us, 3),
        }), flush=True)
        ctx.close()
        del inp, q, kc, vc, out, out_d, sel
        torch.cuda.empty_cache()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-pq4", action="store_true",
                    help="skip the arm with the paper's 4-bit-code index setting")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--profile-only", action="store_true",
                    help="run the warm-up and timed decode calls only (for rocprofv3)")
    ap.add_argument("--all-configs", action="store_true",
                    help="instead of the bench line: one JSON line per synthetic workload "
                         "(µs per call, tokens scanned per second, algorithmic GB/s and "
                         "roofline fraction per stage, the same-chip dense decode beside it)")
    ap.add_argument("--profile-dense", action="store_true",
                    help="with --profile-only: time the dense decode instead of PQ-HSA")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="with --profile-only: also run a 256 MiB fp32 elementwise copy "
                         "(torch.neg) 5 times, whose FETCH_SIZE / WRITE_SIZE counters scale "
                         "the operator's counters to bytes")
    ap.add_argument("--profile-build", action="store_true",
                    help="run only the k-means index build of the bench workload (one coarse "
                         "and two subspace iterations), --warmup untimed then --steps timed "
                         "(for rocprofv3)")
    ap.add_argument("--summarize-build", nargs=2, metavar=("STATS_CSV", "COMMAND"),
                    help="print the index build's kernel summary (time per kernel, the "
                         "assignment passes' TFLOP/s against the fp32 peak) and exit")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("STATS_CSV", "COMMAND"),
                    help="print a summary of a rocprofv3 kernel_stats.csv and exit")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("STAGE", "FETCH_CSV", "WRITE_CSV", "COMMANDS"),
                    help="print the counter summary of one stage's kernel and exit")
    args = ap.parse_args()
    if args.summarize_trace:
        sys.stdout.write(summarize_trace(*args.summarize_trace))
        return 0
    if args.summarize_build:
        sys.stdout.write(summarize_build(*args.summarize_build))
        return 0
    if args.summarize_pmc:
        sys.stdout.write(summarize_pmc(*args.summarize_pmc))
        return 0
    if args.gpus != 1:
        print("bench.py measures one GPU: the operator is a single-GPU kernel path and this "
              "build has no multi-GPU mode (run with --gpus 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_33746_amd import pqhsa, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.all_configs:
        return config_sweep(args, dev)
    if args.profile_build:
        return build_only(args, dev)
    wl = synth.workload(WORKLOAD)
    log(f"generating {wl.name}")
    inp = synth.make_inputs(wl, seed=args.seed, device=dev)
    topk = inp["topk"].tolist()
    lens = inp["seq_lens"].tolist()
    ctx = pqhsa.context_for(inp)
    pqhsa.prepare_from(ctx, inp)
    q, kc, vc = inp["q"], inp["k_cache"], inp["v_cache"]
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    out_dense = torch.empty_like(out)
    flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    flush_buf.fill_(1.0)

    def flush():
        # a read of 4x the Infinity Cache: evicts the operator's data and
        # leaves clean lines behind
        torch.sum(flush_buf)

    def write_flush():
        flush_buf.fill_(1.0)

    def timed(fn, steps, do_flush=True, flush_fn=None):
        flush_fn = flush_fn or flush
        times = []
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            if do_flush:
                flush_fn()
            ev[i][0].record(stream)
            fn()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        times = [a.elapsed_time(b) for a, b in ev]
        return np.array(times), wall

    def pq_call():
        ctx.decode(q, kc, vc, topk, out=out)

    def dense_call():
        ctx.dense_decode(q, kc, vc, lens, out=out_dense)

    def copy_calibration():
        n = COPY_CAL_BYTES // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        log(f"copy calibration: 5 x {COPY_CAL_BYTES >> 20} MiB read + written")

    if args.profile_only and args.profile_dense:
        for _ in range(args.warmup):
            flush()
            dense_call()
        t_d, _ = timed(dense_call, args.steps)
        log(f"dense mean {t_d.mean() * 1e3:.2f} us")
        if args.copy_calibration:
            copy_calibration()
        return 0
    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        flush()
        pq_call()
    torch.cuda.synchronize()
    log(f"timing {args.steps} PQ-HSA calls")
    t_pq, wall_pq = timed(pq_call, args.steps)
    if args.profile_only:
        log(f"PQ-HSA mean {t_pq.mean() * 1e3:.2f} us")
        if args.copy_calibration:
            copy_calibration()
        return 0

    # per-stage durations, HIP events around each kernel on the same stream
    ctx.set_option(pqhsa.OPT_STAGE_TIMING, 1)
    stage_acc = {}
    n_stage = max(20, args.steps // 4)
    for _ in range(n_stage):
        flush()
        pq_call()
        for k_, v_ in ctx.stage_times().items():
            stage_acc.setdefault(k_, []).append(v_)
    ctx.set_option(pqhsa.OPT_STAGE_TIMING, 0)
    stage_us = {k_: float(np.mean(v_)) * 1e3 for k_, v_ in stage_acc.items()}

    log("timing hot (unflushed) calls")
    t_hot, _ = timed(pq_call, args.steps, do_flush=False)
    log("timing calls after a write flush (dirty Infinity Cache)")
    t_pq_wf, _ = timed(pq_call, max(20, args.steps // 4), flush_fn=write_flush)
    log("timing dense decode")
    for _ in range(5):
        dense_call()
    t_dense, _ = timed(dense_call, max(20, args.steps // 4))
    t_dense_wf, _ = timed(dense_call, 20, flush_fn=write_flush)
    # torch's own attention as a second dense reference (GQA-expanded bf16)
    sdpa_us = None
    try:
        G = wl.n_q_heads // wl.n_kv_heads
        qs = q[:, :, None, :]

        def sdpa_call():
            torch.nn.functional.scaled_dot_product_attention(qs, kc, vc, enable_gqa=True)
        sdpa_call()
        t_sdpa, _ = timed(sdpa_call, 20)
        sdpa_us = float(np.median(t_sdpa)) * 1e3
    except Exception as exc:  # noqa: BLE001 - reported, not fatal
        log(f"torch SDPA reference unavailable: {exc}")
    # a library dense decode: two batched GEMMs (hipBLASLt/rocBLAS) around a
    # softmax, bf16, K and V read once each (transposed operands are made
    # contiguous first; they are the small query and probability tensors)
    gemm_us = None
    try:
        BG = wl.batch * wl.n_kv_heads
        Kf = kc.reshape(BG, kc.shape[2], kc.shape[3])
        Vf = vc.reshape(BG, vc.shape[2], vc.shape[3])
        Qt = (q.reshape(BG, G, wl.head_dim) * (wl.head_dim ** -0.5)).transpose(1, 2).contiguous()

        def gemm_call():
            S = torch.bmm(Kf, Qt)                          # [BG, N, G]
            P = torch.softmax(S.float(), dim=1).to(Kf.dtype)
            return torch.bmm(P.transpose(1, 2).contiguous(), Vf)   # [BG, G, d]
        gemm_call()
        t_gemm, _ = timed(gemm_call, 20)
        gemm_us = float(np.median(t_gemm)) * 1e3
    except Exception as exc:  # noqa: BLE001 - reported, not fatal
        log(f"library dense reference unavailable: {exc}")

    # the mechanism variants of the background term (Appendix B) on the same
    # context: T drops the background workgroups, C reads one mean per (b, g),
    # Bx forms per-list weights in the top-k stage and weights the exact rows of T
    variant_us = {}
    for name, code in (("T", pqhsa.VARIANT_T), ("C", pqhsa.VARIANT_C), ("Bx", pqhsa.VARIANT_BX)):
        ctx.set_option(pqhsa.OPT_VARIANT, code)
        for _ in range(3):
            flush()
            pq_call()
        t_v, _ = timed(pq_call, max(20, args.steps // 4))
        variant_us[name] = round(float(np.mean(t_v)) * 1e3, 3)
    ctx.set_option(pqhsa.OPT_VARIANT, pqhsa.VARIANT_B)

    # the step with N_b and k_b as device data, eagerly and as a replayed
    # graph of the captured call (new values could be written between replays)
    lens_d = torch.tensor(lens, dtype=torch.int32, device=dev)
    topk_d = torch.tensor(topk, dtype=torch.int32, device=dev)

    def dev_call():
        ctx.decode_device_args(q, kc, vc, lens_d, topk_d, out=out)
    for _ in range(3):
        flush()
        dev_call()
    t_da, _ = timed(dev_call, max(20, args.steps // 4))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dev_call()
    for _ in range(3):
        flush()
        graph.replay()
    t_gr, _ = timed(graph.replay, max(20, args.steps // 4))
    device_args = {"us_per_call": round(float(np.mean(t_da)) * 1e3, 3),
                   "graph_replay_us_per_call": round(float(np.mean(t_gr)) * 1e3, 3)}
    del graph

    # the same call on a paged cache (pages of 16 tokens at random page
    # indices, K and V interleaved in each page as in vLLM's layout)
    paged_us = None
    if not args.no_pq4:
        B_, Hkv_, N_, d_ = kc.shape
        page = 16
        nb = -(-N_ // page)
        gen = torch.Generator().manual_seed(args.seed)
        table = torch.randperm(B_ * nb + 5, generator=gen)[:B_ * nb].reshape(B_, nb)
        pages = torch.zeros((B_ * nb + 5, Hkv_, page, 2 * d_), dtype=kc.dtype, device=dev)
        for lo, src in ((0, kc), (d_, vc)):
            x = torch.nn.functional.pad(src, (0, 0, 0, nb * page - N_))
            pages[table.reshape(-1).to(dev), :, :, lo:lo + d_] = \
                x.reshape(B_, Hkv_, nb, page, d_).permute(0, 2, 1, 3, 4).reshape(B_ * nb, Hkv_, page, d_)
        table = table.to(torch.int32).to(dev)
        kp, vp = pages[..., :d_], pages[..., d_:]

        def paged_call():
            ctx.decode_paged(q, kp, vp, table, page, topk, out=out)
        for _ in range(3):
            flush()
            paged_call()
        t_pg, _ = timed(paged_call, max(20, args.steps // 4))
        paged_us = {"page_size": page, "us_per_call": round(float(np.mean(t_pg)) * 1e3, 3)}
        del pages, kp, vp

    # the incremental index update: 256 tokens leave the local window and are
    # encoded into the lists (wall time of the call and its kernels: encode,
    # means, the list-major merge, the gather and the global means)
    update = None
    if not args.no_pq4:
        ctxu = pqhsa.context_for(inp)
        n0 = [int(x) - 5 * 256 for x in inp["seq_lens"]]
        pqhsa.prepare_from(ctxu, dict(inp, seq_lens=torch.tensor(n0, dtype=torch.int32)))
        t_up = []
        for i in range(1, 6):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ctxu.index_update([n + 256 * i for n in n0], kc, vc)
            torch.cuda.synchronize()
            t_up.append(time.perf_counter() - t0)
        ms_up = 1e3 * float(np.median(t_up))
        update = {"tokens_per_update": 256, "ms_per_update": round(ms_up, 3),
                  "us_per_step_amortized_over_256": round(ms_up * 1e3 / 256, 3)}
        ctxu.close()

    # the k-means index build of the same cache (one coarse and two subspace
    # iterations, the paper's setting), wall time of one call
    build = None
    if not args.no_pq4:
        ic_d, ip_d = build_seeds(inp, args.seed, dev)
        ctxb = pqhsa.context_for(inp)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctxb.index_build([int(x) for x in inp["seq_lens"]], kc, vc, ic_d, ip_d, *BUILD_ITERS)
        torch.cuda.synchronize()
        build = {"n_iter_coarse": BUILD_ITERS[0], "n_iter_pq": BUILD_ITERS[1],
                 "ms": round(1e3 * (time.perf_counter() - t0), 2)}
        log(f"index build {build['ms']} ms")
        ctxb.close()

    # the paper's own index setting on the same 128K shapes (8 subspaces of
    # 4-bit codes, 512 lists): a second PQ-HSA arm, reported beside the value
    pq4 = None
    if not args.no_pq4:
        log("timing the 4-bit-code index arm")
        wl4 = synth.pq4(WORKLOAD)
        inp4 = synth.make_inputs(wl4, seed=args.seed, device=dev)
        ctx4 = pqhsa.context_for(inp4)
        pqhsa.prepare_from(ctx4, inp4)
        q4, k4, v4 = inp4["q"], inp4["k_cache"], inp4["v_cache"]
        topk4 = inp4["topk"].tolist()
        out4 = torch.empty(q4.shape, dtype=torch.float32, device=dev)

        def pq4_call():
            ctx4.decode(q4, k4, v4, topk4, out=out4)
        for _ in range(args.warmup):
            flush()
            pq4_call()
        t_pq4, _ = timed(pq4_call, max(20, args.steps // 2))
        ctx4.set_option(pqhsa.OPT_STAGE_TIMING, 1)
        acc4 = {}
        for _ in range(20):
            flush()
            pq4_call()
            for k_, v_ in ctx4.stage_times().items():
                acc4.setdefault(k_, []).append(v_)
        ctx4.set_option(pqhsa.OPT_STAGE_TIMING, 0)
        us4 = float(np.mean(t_pq4)) * 1e3
        pq4 = {"workload": wl4.name, "pq_m": wl4.pq_m, "pq_ksub": wl4.pq_ksub,
               "n_list": wl4.n_list, "topk": topk4[0], "us_per_call": round(us4, 3),
               "stage_us": {k_: round(float(np.mean(v_)) * 1e3, 3) for k_, v_ in acc4.items()}}
        ctx4.close()
        del inp4, q4, k4, v4

    # distinct gathered rows per (b, g) for the byte model
    _, sel, _, _ = ctx.decode_debug(q, kc, vc, topk)
    torch.cuda.synchronize()
    G = wl.n_q_heads // wl.n_kv_heads
    sel_c = sel.cpu().numpy()
    union = []
    for b in range(wl.batch):
        row = []
        for g in range(wl.n_kv_heads):
            ids = np.unique(sel_c[b, g * G:(g + 1) * G, :topk[b]])
            row.append(int(ids.size) + wl.n_sink + wl.n_local)
        union.append(row)
    by = algorithmic_bytes(inp, topk, union)
    total_bytes = sum(by.values())

    us = float(np.mean(t_pq)) * 1e3
    us_med = float(np.median(t_pq)) * 1e3
    dense_us = float(np.mean(t_dense)) * 1e3
    # the fastest same-chip dense decode measured here is the comparison
    arms = [("hip_dense_kernel", dense_us)]
    if gemm_us is not None:
        arms.append(("torch_bmm_softmax_bmm", gemm_us))
    if sdpa_us is not None:
        arms.append(("torch_sdpa", sdpa_us))
    best_dense = min(arms, key=lambda a: a[1])
    n_scanned = sum((n - wl.n_sink - wl.n_local) * wl.n_kv_heads for n in lens)
    stage_bytes = dict(prologue=by["lut"], scan=by["scan"], select=by["select"],
                       attend=by["attend"] + by["background"], merge=by["out"])
    # the dominant kernel for the HBM roofline: the one that takes the longest
    # (every stage is a candidate; the whole call's fraction is reported beside it)
    dom = max(stage_us, key=lambda s_: stage_us[s_])
    dom_gbps = stage_bytes[dom] / (stage_us[dom] * 1e-6) / 1e9
    stage_roofline = {s_: round(stage_bytes[s_] / (stage_us[s_] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
                      for s_ in stage_us if stage_bytes.get(s_, 0) > 0}
    call_gbps = total_bytes / (us * 1e-6) / 1e9

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inp, topk, args.cpu_seconds)

    rec = {
        "metric": "PQ-HSA decode-attention µs/call and HBM GB/s at 128K vs dense decode, 1 MI355X",
        "value": round(us, 3),
        "unit": "us/call",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "storage": "bf16 K/V and query, uint8 PQ codes, fp32 index tables",
        "data": "synthetic (seeded clustered keys; no model weights or datasets)",
        "config": {"workload": wl.name, "batch": wl.batch, "n_q_heads": wl.n_q_heads,
                   "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim, "seq_len": wl.max_seq,
                   "n_list": wl.n_list, "pq_m": wl.pq_m, "pq_ksub": wl.pq_ksub, "topk": topk[0],
                   "n_sink": wl.n_sink, "n_local": wl.n_local, "parallelism": "single GPU"},
        "us_per_call_median": round(us_med, 3),
        "us_per_call_hot": round(float(np.mean(t_hot)) * 1e3, 3),
        "us_per_call_write_flush": round(float(np.mean(t_pq_wf)) * 1e3, 3),
        "timed_region_wall_s": round(wall_pq, 4),
        "tokens_scanned_per_s": n_scanned / (us * 1e-6),
        "score_evals_per_s": n_scanned * G / (us * 1e-6),
        "algorithmic_bytes": total_bytes,
        "algorithmic_bytes_by_stage": by,
        "hbm_gbps_algorithmic": round(call_gbps, 1),
        "call_roofline_frac": round(call_gbps / HBM_PEAK_GBPS, 4),
        "stage_us": {k_: round(v_, 3) for k_, v_ in stage_us.items()},
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": round(dom_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes": stage_bytes[dom], "traffic": pmc_traffic(dom)},
        "call_roofline": {"bound": "hbm", "achieved": round(call_gbps, 1), "peak": HBM_PEAK_GBPS,
                          "unit": "GB/s", "frac": round(call_gbps / HBM_PEAK_GBPS, 4),
                          "algorithmic_bytes": total_bytes, "us_per_call": round(us, 3)},
        "stage_roofline_frac": stage_roofline,
        "dense_us_per_call": round(dense_us, 3),
        "dense_us_per_call_write_flush": round(float(np.mean(t_dense_wf)) * 1e3, 3),
        "dense_hbm_gbps": round(sum(n * wl.n_kv_heads * 2 * wl.head_dim * 2 for n in lens)
                                / (dense_us * 1e-6) / 1e9, 1),
        "torch_sdpa_us_per_call": None if sdpa_us is None else round(sdpa_us, 3),
        "torch_bmm_softmax_bmm_us_per_call": None if gemm_us is None else round(gemm_us, 3),
        "dense_best_arm": best_dense[0],
        "speedup_vs_dense": round(best_dense[1] / us, 3),
        "cpu_baseline": cpu,
        "variant_us_per_call": variant_us,
        "paged_kv_arm": paged_us,
        "device_args_arm": device_args,
        "index_update": update,
        "index_build": build,
        "paper_index_arm": pq4 if pq4 is None else dict(
            pq4, speedup_vs_dense=round(best_dense[1] / pq4["us_per_call"], 3)),
    }
    print(json.dumps(rec), flush=True)
    ctx.close()
    return 0


# Kernel sources whose text decides each stage's memory traffic: a counter
# summary taken on other sources no longer describes the kernel.
STAGE_KERNEL = dict(prologue="prologue_kernel", scan="scan_kernel", select="select_kernel",
                    attend="attend_kernel", merge="merge_kernel", dense="dense_kernel")
STAGE_SOURCES = dict(
    prologue=["prologue.hip", "hist_select.h", "radix_select.h", "pq_score.h"],
    scan=["scan.hip", "pq_score.h"], select=["select.hip", "hist_select.h", "radix_select.h"],
    attend=["attend.hip"], merge=["attend.hip"], dense=["attend.hip"])
COMMON_SOURCES = ["device_common.h", "pqhsa_internal.h"]
PROFILES = os.path.join(ROOT, "profiles")


def source_hash(stage: str) -> str:
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_33746_amd", "csrc")
    for f in STAGE_SOURCES[stage] + COMMON_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def pmc_file(stage: str) -> str:
    return os.path.join(PROFILES, f"{STAGE_KERNEL[stage]}_llama8b_n128k_pmc.txt")


def pmc_traffic(stage: str):
    """HBM bytes per launch of `stage` from its committed counter summary, or
    None when there is none or it was taken on other kernel sources."""
    path = pmc_file(stage)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith(" "):
                k_, v_ = line.split(":", 1)
                vals[k_.strip()] = v_.strip()
    if vals.get("source_hash") != source_hash(stage):
        log(f"{os.path.basename(path)} was taken on other sources: traffic unknown")
        return None
    return int(float(vals["traffic_bytes_per_launch"]))


BUILD_ITERS = (1, 2)   # coarse and subspace k-means iterations of the measured build


def build_seeds(inp, seed, dev):
    """The starting tokens of the index build: distinct tokens of R_b drawn
    per (b, g) for the coarse centers and per subspace for the codewords."""
    import numpy as np
    import torch
    wl = inp["workload"]
    rng = np.random.default_rng(seed)
    ic = np.zeros((wl.batch, wl.n_kv_heads, wl.n_list), np.int32)
    ip = np.zeros((wl.batch, wl.n_kv_heads, wl.pq_m, wl.pq_ksub), np.int32)
    for b in range(wl.batch):
        Rb = np.arange(wl.n_sink, int(inp["seq_lens"][b]) - wl.n_local)
        for g in range(wl.n_kv_heads):
            ic[b, g] = rng.choice(Rb, wl.n_list, replace=False)
            for m in range(wl.pq_m):
                ip[b, g, m] = rng.choice(Rb, wl.pq_ksub, replace=False)
    return torch.from_numpy(ic).to(dev), torch.from_numpy(ip).to(dev)


def build_only(args, dev) -> int:
    """The index build of the bench workload alone, for the profiler."""
    import torch

    from paper_2609_33746_amd import pqhsa, synth
    wl = synth.workload(WORKLOAD)
    inp = synth.make_inputs(wl, seed=args.seed, device=dev)
    ic_d, ip_d = build_seeds(inp, args.seed, dev)
    ctx = pqhsa.context_for(inp)
    lens = [int(x) for x in inp["seq_lens"]]
    for i in range(args.warmup + args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctx.index_build(lens, inp["k_cache"], inp["v_cache"], ic_d, ip_d, *BUILD_ITERS)
        torch.cuda.synchronize()
        log(f"index build {i}: {1e3 * (time.perf_counter() - t0):.2f} ms")
    ctx.close()
    return 0


def build_flops() -> dict:
    """Distance arithmetic of one build of the bench workload: 3 flops per
    dimension of a squared distance (a subtraction and a fused multiply-add).
    Passes: the norm pass (subspace search against the zero model), each
    coarse iteration and the final lists (coarse + subspace search), each
    subspace iteration and the final codes (subspace search)."""
    from paper_2609_33746_amd import synth
    wl = synth.workload(WORKLOAD)
    n = wl.batch * wl.n_kv_heads * (wl.max_seq - wl.n_sink - wl.n_local)   # not ragged
    dsub = wl.head_dim // wl.pq_m
    coarse = 3.0 * n * wl.n_list * wl.head_dim
    sub = 3.0 * n * wl.pq_m * wl.pq_ksub * dsub
    n_coarse = BUILD_ITERS[0] + 1
    n_sub = 1 + (BUILD_ITERS[0] + 1) + BUILD_ITERS[1] + 1
    return {"tokens": n, "coarse_passes": n_coarse, "subspace_passes": n_sub,
            "flops": n_coarse * coarse + n_sub * sub}


FP32_PEAK_TFLOPS = 157.3


def summarize_build(stats_csv: str, command: str) -> str:
    """Kernel summary of index builds (rocprofv3 --kernel-trace --stats), with
    the assignment passes' arithmetic rate against the fp32 peak."""
    rows = [r for r in _csv_rows(stats_csv) if "pqhsa" in r["Name"]]
    fl = build_flops()
    out = [f"command: {command}",
           f"build: {BUILD_ITERS[0]} coarse and {BUILD_ITERS[1]} subspace iterations, "
           f"{fl['tokens']} tokens, {fl['coarse_passes']} coarse and {fl['subspace_passes']} "
           f"subspace assignment passes per build, {fl['flops'] / 1e12:.3f} TFLOP of distances",
           "kernel  calls  avg_us  min_us  max_us  total_us"]
    enc_ns, enc_calls, tot_ns = 0.0, 0, 0.0
    for r in rows:
        name = r["Name"].split("(")[0]
        calls, tot = int(r["Calls"]), float(r["TotalDurationNs"])
        out.append(f"{name}  {calls}  {float(r['AverageNs']) / 1e3:.2f}  {float(r['MinNs']) / 1e3:.2f}  "
                   f"{float(r['MaxNs']) / 1e3:.2f}  {tot / 1e3:.1f}")
        tot_ns += tot
        if "encode_kernel" in name or "assign_kernel" in name or "subspace_kernel" in name:
            enc_ns += tot
        if "encode_kernel" in name or "subspace_kernel" in name:
            enc_calls += calls
    # one subspace-search launch per subspace pass (the coarse searches are
    # separate launches on the matrix cores)
    builds = enc_calls / fl["subspace_passes"]
    if builds:
        per_build_ms = enc_ns / builds / 1e6
        tflops = fl["flops"] / (enc_ns / builds * 1e-9) / 1e12
        out.append(f"builds profiled: {builds:g}; kernel time per build {tot_ns / builds / 1e6:.2f} ms, "
                   f"of which assignment passes (coarse and subspace searches) {per_build_ms:.2f} ms")
        out.append(f"assignment passes: {tflops:.1f} TFLOP/s = {tflops / FP32_PEAK_TFLOPS:.3f} of "
                   f"the {FP32_PEAK_TFLOPS} TFLOP/s fp32 peak")
    return "\n".join(out) + "\n"


def _csv_rows(path):
    import csv
    with open(path) as fh:
        return list(csv.DictReader(fh))


def summarize_trace(stats_csv: str, command: str) -> str:
    """Text summary of a rocprofv3 --kernel-trace --stats run (kernel_stats.csv)."""
    out = [f"command: {command}", "kernel  calls  avg_us  min_us  max_us"]
    for r in _csv_rows(stats_csv):
        if "pqhsa" in r["Name"]:
            out.append(f"{r['Name'].split('(')[0]}  {r['Calls']}  {float(r['AverageNs']) / 1e3:.2f}  "
                       f"{float(r['MinNs']) / 1e3:.2f}  {float(r['MaxNs']) / 1e3:.2f}")
    return "\n".join(out) + "\n"


def summarize_pmc(stage: str, fetch_csv: str, write_csv: str, commands: str) -> str:
    """Counter summary of one stage's kernel: FETCH_SIZE and WRITE_SIZE (KiB
    per dispatch) from two runs, each scaled by what the same counter reads
    for the calibration copy (COPY_CAL_BYTES read and written)."""
    def per_kernel(path, counter):
        acc = {}
        for r in _csv_rows(path):
            if r["Counter_Name"] == counter:
                acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return {k_: sum(v_) / len(v_) for k_, v_ in acc.items()}
    fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    write = per_kernel(write_csv, "WRITE_SIZE")
    cal_f = [v_ for k_, v_ in fetch.items() if "neg_kernel" in k_]
    cal_w = [v_ for k_, v_ in write.items() if "neg_kernel" in k_]
    kib = COPY_CAL_BYTES / 1024
    f_scale = kib / cal_f[0]
    w_scale = kib / cal_w[0]
    name = STAGE_KERNEL[stage]
    kf = [v_ for k_, v_ in fetch.items() if f"pqhsa::{name}" in k_]
    kw = [v_ for k_, v_ in write.items() if f"pqhsa::{name}" in k_]
    traffic = (kf[0] * f_scale + kw[0] * w_scale) * 1024
    lines = [
        f"commands: {commands}",
        f"kernel: {name}",
        f"source_hash: {source_hash(stage)}",
        f"copy_fetch_kib_per_dispatch: {cal_f[0]:.1f} (expected {kib:.0f}; scale {f_scale:.4f})",
        f"copy_write_kib_per_dispatch: {cal_w[0]:.1f} (expected {kib:.0f}; scale {w_scale:.4f})",
        f"fetch_kib_per_dispatch: {kf[0]:.1f}",
        f"write_kib_per_dispatch: {kw[0]:.1f}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        "all pqhsa kernels (fetch KiB, write KiB per dispatch, unscaled):",
    ]
    for k_ in fetch:
        if "pqhsa" in k_:
            lines.append(f"  {k_.split('(')[0]}  {fetch[k_]:.1f}  {write.get(k_, float('nan')):.1f}")
    return "\n".join(lines) + "\n"


def cpu_baseline(inp, topk, budget_s: float):
    """The CPU oracle on the same workload: whole calls (all 32 query rows)
    repeated until `budget_s` of CPU time, BLAS limited to one thread."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import pqhsa_ref as R

    wl = inp["workload"]
    log("CPU oracle baseline")
    host = {k_: (v_.cpu() if hasattr(v_, "cpu") else v_) for k_, v_ in inp.items()}
    rows = [(b, h) for b in range(wl.batch) for h in range(wl.n_q_heads)]
    calls = 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1):
        while True:
            R.pqhsa_batch_ref(host, topk, rows)
            calls += 1
            el = time.perf_counter() - t0
            log(f"oracle call {calls}: {el:.1f} s")
            if el >= budget_s:
                break
    per_call_us = el / calls * 1e6
    return {"value": round(per_call_us, 1), "unit": "us/call", "cores": 1, "kind": "oracle",
            "sample": f"{calls} whole calls of the {wl.name} workload (all {len(rows)} query rows), "
                      f"float64 NumPy, one thread, {el:.1f} s",
            "host_cpus": os.cpu_count()}


if __name__ == "__main__":
    sys.exit(main())
