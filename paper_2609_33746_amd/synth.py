"""Seeded synthetic workloads for the PQ-HSA decode operator.

This module only draws random inputs; it holds none of the operator's
arithmetic. It stands in for the paper's long-context KV caches (RULER
prompts on Llama-3.1-8B / Qwen3-30B-A3B shapes, Section 4.1), which are not
available: clustered keys that an IVF-PQ index describes well, values with a
per-list offset, and queries aimed at one cached key.

Recipe, per (batch element b, KV head g), from one SeedSequence per workload:
  centroids c_j ~ N(0, I_d)                       [n_list, d]
  codebooks p_{m,z} ~ N(0, 0.3^2 I_{d/M})         [M, ksub, d/M]
  list ids a_i ~ U{0..n_list-1}, codes z_im ~ U{0..ksub-1}
  keys k_i = s_i * (c_{a_i} + concat_m p_{m,z_im} + N(0, noise^2 I_d))
  list offsets o_j ~ N(0, I_d); values v_i = N(0, I_d) + 0.5 o_{a_i}
  norms r_i = s_i, with s_i = 1 (key-space index) or, for the norm variant,
  s_i log-uniform in [0.5, 2]
  K/V rounded to the cache dtype; list means v_bar_j = mean over R_j of the
  stored (rounded) values, accumulated in float64 and stored as float32
  query of head h: q_h = t_h * k_{j_h}, j_h uniform over the indexed region of
  its own KV head, rounded to the cache dtype.
Draws use torch generators on the target device, so the largest workloads
(8.6 GB of K/V) are generated in place in device memory.
"""

from __future__ import annotations

import math
import zlib
from dataclasses import dataclass, replace

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "workload", "pq4", "make_inputs", "ratio_topk"]


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    max_seq: int
    kv_dtype: str            # "f32" or "bf16"
    n_list: int
    pq_m: int = 16
    pq_ksub: int = 256
    topk: int | None = None  # fixed top-k for every sequence
    rho: float | None = None  # or k_b = round(rho * N_b)
    ragged_min: int | None = None  # N_b ~ U[ragged_min, max_seq] when set
    temp: str = "3"          # "3" or "1to4" (t_h = 1 + 3h/(Hq-1))
    n_sink: int = 4
    n_local: int = 128


WORKLOADS = {
    0: Workload("tiny-1q1kv-n4096-f32", 1, 1, 1, 128, 4096, "f32", 16, topk=64),
    1: Workload("llama8b-layer-n32k-bf16", 1, 32, 8, 128, 32768, "bf16", 256,
                topk=655),
    2: Workload("llama8b-layer-n128k-bf16", 1, 32, 8, 128, 131072, "bf16", 1024,
                topk=1311, temp="1to4"),
    3: Workload("qwen3-30b-a3b-layer-b4-n128k-bf16", 4, 32, 4, 128, 131072,
                "bf16", 1024, topk=2621),
    4: Workload("llama8b-layer-b16-ragged-64k-128k-bf16", 16, 32, 8, 128, 131072,
                "bf16", 1024, rho=0.01, ragged_min=65536),
}


def workload(idx: int, **overrides) -> Workload:
    return replace(WORKLOADS[idx], **overrides)


def pq4(idx: int, **overrides) -> Workload:
    """Workload idx with the paper's own index setting (Section 3.1): 8
    subspaces of 4-bit codes (16 codewords of 16 dimensions) and at most 512
    lists. The name changes too, so the draws differ from workload idx."""
    wl = WORKLOADS[idx]
    kw = dict(name=wl.name + "-pq4", pq_m=8, pq_ksub=16, n_list=min(wl.n_list, 512))
    kw.update(overrides)
    return replace(wl, **kw)


def ratio_topk(rho: float, n: int) -> int:
    """k = round(rho * N), halves rounded up (the workloads' budget rule)."""
    return int(math.floor(rho * n + 0.5))


def _pair_seeds(root: np.random.SeedSequence, n: int) -> list[int]:
    return [int(c.generate_state(1, dtype=np.uint64)[0] >> 1) for c in root.spawn(n)]


def make_inputs(wl: Workload, seed: int = 0, *, device: str | torch.device = "cpu",
                noise: float = 0.05, norm_variant: bool = False,
                list_constant_values: bool = False, seq_lens=None) -> dict:
    """Draw one workload's inputs as torch tensors on `device`.

    The draws are a function of (seed, workload name, device type): torch's
    CPU and GPU generators differ, so the same seed gives different data on
    the two; within one device type the result is deterministic.

    Returns a dict with the ABI's token-major layouts:
      q [B, Hq, d]; k_cache, v_cache [B, Hkv, Nmax, d] (kv dtype);
      list_ids int32 [B, Hkv, Nmax]; codes uint8 [B, Hkv, Nmax, M];
      norms float32 [B, Hkv, Nmax]; centroids float32 [B, Hkv, n_list, d];
      codebooks float32 [B, Hkv, M, ksub, d/M]; list_means float32
      [B, Hkv, n_list, d]; seq_lens, topk int32 [B] (CPU); n_sink, n_local.
    """
    device = torch.device(device)
    B, Hq, Hkv, d = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    M, ksub, n_list, Nmax = wl.pq_m, wl.pq_ksub, wl.n_list, wl.max_seq
    if d % M:
        raise ValueError("head_dim must be a multiple of pq_m")
    G = Hq // Hkv
    dsub = d // M
    root = np.random.SeedSequence([seed, zlib.crc32(wl.name.encode())])
    seq_ss, pair_root = root.spawn(2)
    g0 = np.random.Generator(np.random.PCG64(seq_ss))
    if seq_lens is not None:
        lens = np.asarray(seq_lens, dtype=np.int64)
    elif wl.ragged_min is not None:
        lens = g0.integers(wl.ragged_min, Nmax + 1, size=B)
    else:
        lens = np.full(B, Nmax, dtype=np.int64)
    if wl.topk is not None:
        topk = np.full(B, wl.topk, dtype=np.int64)
    else:
        topk = np.array([ratio_topk(wl.rho, int(n)) for n in lens])
    if wl.temp == "1to4":
        temps = 1.0 + 3.0 * np.arange(Hq) / max(Hq - 1, 1)
    else:
        temps = np.full(Hq, float(wl.temp))
    seeds = _pair_seeds(pair_root, B * Hkv)

    kvt = torch.bfloat16 if wl.kv_dtype == "bf16" else torch.float32
    f32 = dict(dtype=torch.float32, device=device)
    k_cache = torch.zeros((B, Hkv, Nmax, d), dtype=kvt, device=device)
    v_cache = torch.zeros((B, Hkv, Nmax, d), dtype=kvt, device=device)
    q = torch.zeros((B, Hq, d), dtype=kvt, device=device)
    list_ids = torch.zeros((B, Hkv, Nmax), dtype=torch.int32, device=device)
    codes = torch.zeros((B, Hkv, Nmax, M), dtype=torch.uint8, device=device)
    norms = torch.ones((B, Hkv, Nmax), **f32)
    centroids = torch.zeros((B, Hkv, n_list, d), **f32)
    codebooks = torch.zeros((B, Hkv, M, ksub, dsub), **f32)
    list_means = torch.zeros((B, Hkv, n_list, d), **f32)
    m_idx = torch.arange(M, device=device)

    for pair in range(B * Hkv):
        b, g = divmod(pair, Hkv)
        n = int(lens[b])
        gen = torch.Generator(device=device)
        gen.manual_seed(seeds[pair])
        cen = torch.randn((n_list, d), generator=gen, **f32)
        cb = 0.3 * torch.randn((M, ksub, dsub), generator=gen, **f32)
        a = torch.randint(0, n_list, (n,), generator=gen, device=device)
        z = torch.randint(0, ksub, (n, M), generator=gen, device=device)
        key = cen[a] + cb[m_idx[None, :], z].reshape(n, d)
        if noise:
            key += noise * torch.randn((n, d), generator=gen, **f32)
        if norm_variant:
            lo_s, hi_s = math.log(0.5), math.log(2.0)
            s = torch.exp(lo_s + (hi_s - lo_s) * torch.rand((n,), generator=gen, **f32))
            key *= s[:, None]
            norms[b, g, :n] = s
        kt = key.to(kvt)
        del key
        off = torch.randn((n_list, d), generator=gen, **f32)
        if list_constant_values:
            vals = 0.5 * off[a]
        else:
            vals = torch.randn((n, d), generator=gen, **f32) + 0.5 * off[a]
        vt = vals.to(kvt)
        del vals
        k_cache[b, g, :n] = kt
        v_cache[b, g, :n] = vt
        list_ids[b, g, :n] = a.to(torch.int32)
        codes[b, g, :n] = z.to(torch.uint8)
        centroids[b, g] = cen
        codebooks[b, g] = cb
        # list value means over the indexed region R_j of the stored values
        lo, hi = wl.n_sink, n - wl.n_local
        list_means[b, g] = _list_means(vt[lo:hi], a[lo:hi], n_list)
        # queries of the G heads that share this KV head
        if hi > lo:
            js = torch.randint(lo, hi, (G,), generator=gen, device=device)
        else:
            js = torch.zeros(G, dtype=torch.long, device=device)
        for hh in range(G):
            h = g * G + hh
            q[b, h] = (kt[js[hh]].float() * float(temps[h])).to(kvt)

    return dict(
        q=q, k_cache=k_cache, v_cache=v_cache, list_ids=list_ids, codes=codes, norms=norms,
        centroids=centroids, codebooks=codebooks, list_means=list_means,
        seq_lens=torch.from_numpy(lens.astype(np.int32)),
        topk=torch.from_numpy(topk.astype(np.int32)),
        n_sink=wl.n_sink, n_local=wl.n_local, workload=wl)


def _list_means(v: torch.Tensor, a: torch.Tensor, n_list: int) -> torch.Tensor:
    """Float64 mean of the rows of v per list id (0 for an empty list), as float32.

    Sort-and-difference of a float64 prefix sum: deterministic on every device.
    """
    d = v.shape[1]
    if a.numel() == 0:
        return torch.zeros((n_list, d), dtype=torch.float32, device=v.device)
    order = torch.argsort(a, stable=True)
    cs = torch.cumsum(v[order].double(), dim=0)
    counts = torch.bincount(a, minlength=n_list)
    ends = torch.cumsum(counts, 0)
    starts = ends - counts
    zero = torch.zeros((1, d), dtype=torch.float64, device=v.device)
    csz = torch.cat([zero, cs], dim=0)
    tot = csz[ends] - csz[starts]
    means = tot / counts.clamp(min=1)[:, None].double()
    return means.float()
