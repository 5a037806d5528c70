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
"""

from __future__ import annotations

import math
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "workload", "make_inputs", "ratio_topk"]


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


def ratio_topk(rho: float, n: int) -> int:
    """k = round(rho * N), halves rounded up (the workloads' budget rule)."""
    return int(math.floor(rho * n + 0.5))


def _bits_to_dtype(x: np.ndarray, kv_dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16) if kv_dtype == "bf16" else t


def make_inputs(wl: Workload, seed: int = 0, *, noise: float = 0.05,
                norm_variant: bool = False, list_constant_values: bool = False,
                threads: int | None = None, seq_lens=None) -> dict:
    """Draw one workload's inputs (CPU torch tensors; see module docstring).

    Returns a dict with the ABI's token-major layouts:
      q [B, Hq, d]; k_cache, v_cache [B, Hkv, Nmax, d] (kv dtype);
      list_ids int32 [B, Hkv, Nmax]; codes uint8 [B, Hkv, Nmax, M];
      norms float32 [B, Hkv, Nmax]; centroids float32 [B, Hkv, n_list, d];
      codebooks float32 [B, Hkv, M, ksub, d/M]; list_means float32
      [B, Hkv, n_list, d]; seq_lens int32 [B]; topk int32 [B]; n_sink, n_local.
    """
    B, Hq, Hkv, d = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    M, ksub, n_list, Nmax = wl.pq_m, wl.pq_ksub, wl.n_list, wl.max_seq
    if d % M:
        raise ValueError("head_dim must be a multiple of pq_m")
    G = Hq // Hkv
    dsub = d // M
    root = np.random.SeedSequence([seed, zlib.crc32(wl.name.encode())])
    seq_ss, *pair_ss = root.spawn(1 + B * Hkv)
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

    kvt = torch.bfloat16 if wl.kv_dtype == "bf16" else torch.float32
    k_cache = torch.zeros((B, Hkv, Nmax, d), dtype=kvt)
    v_cache = torch.zeros((B, Hkv, Nmax, d), dtype=kvt)
    q = torch.zeros((B, Hq, d), dtype=kvt)
    list_ids = np.zeros((B, Hkv, Nmax), dtype=np.int32)
    codes = np.zeros((B, Hkv, Nmax, M), dtype=np.uint8)
    norms = np.ones((B, Hkv, Nmax), dtype=np.float32)
    centroids = np.zeros((B, Hkv, n_list, d), dtype=np.float32)
    codebooks = np.zeros((B, Hkv, M, ksub, dsub), dtype=np.float32)
    list_means = np.zeros((B, Hkv, n_list, d), dtype=np.float32)

    def one(pair: int):
        b, g = divmod(pair, Hkv)
        n = int(lens[b])
        rng = np.random.Generator(np.random.PCG64(pair_ss[pair]))
        cen = rng.standard_normal((n_list, d))
        cb = 0.3 * rng.standard_normal((M, ksub, dsub))
        a = rng.integers(0, n_list, size=n)
        z = rng.integers(0, ksub, size=(n, M))
        recon = cen[a].astype(np.float32)
        recon += cb[np.arange(M)[None, :], z].reshape(n, d).astype(np.float32)
        if noise:
            recon += np.float32(noise) * rng.standard_normal((n, d), dtype=np.float32)
        if norm_variant:
            s = np.exp(rng.uniform(math.log(0.5), math.log(2.0), size=n)).astype(np.float32)
            recon *= s[:, None]
        else:
            s = np.ones(n, dtype=np.float32)
        kt = _bits_to_dtype(recon, wl.kv_dtype)
        del recon
        off = rng.standard_normal((n_list, d)).astype(np.float32)
        if list_constant_values:
            vals = 0.5 * off[a]
        else:
            vals = rng.standard_normal((n, d), dtype=np.float32)
            vals += 0.5 * off[a]
        vt = _bits_to_dtype(vals, wl.kv_dtype)
        del vals
        k_cache[b, g, :n] = kt
        v_cache[b, g, :n] = vt
        list_ids[b, g, :n] = a
        codes[b, g, :n] = z
        norms[b, g, :n] = s
        centroids[b, g] = cen
        codebooks[b, g] = cb
        # list value means over the indexed region R_j of the stored values
        lo, hi = wl.n_sink, n - wl.n_local
        vr = vt[lo:hi].double().numpy()
        ar = a[lo:hi]
        sums = np.zeros((n_list, d))
        _segment_add(sums, ar, vr)
        cnt = np.bincount(ar, minlength=n_list)
        nz = cnt > 0
        means = np.zeros((n_list, d))
        means[nz] = sums[nz] / cnt[nz, None]
        list_means[b, g] = means
        # queries of the G heads that share this KV head
        for hh in range(G):
            h = g * G + hh
            j = int(rng.integers(lo, hi)) if hi > lo else 0
            q[b, h] = (kt[j].float() * float(temps[h])).to(kvt)

    nthreads = threads or min(8, os.cpu_count() or 1)
    if B * Hkv == 1 or nthreads == 1:
        for p in range(B * Hkv):
            one(p)
    else:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(one, range(B * Hkv)))

    return dict(
        q=q, k_cache=k_cache, v_cache=v_cache,
        list_ids=torch.from_numpy(list_ids), codes=torch.from_numpy(codes),
        norms=torch.from_numpy(norms), centroids=torch.from_numpy(centroids),
        codebooks=torch.from_numpy(codebooks), list_means=torch.from_numpy(list_means),
        seq_lens=torch.from_numpy(lens.astype(np.int32)),
        topk=torch.from_numpy(topk.astype(np.int32)),
        n_sink=wl.n_sink, n_local=wl.n_local, workload=wl)


def _segment_add(sums: np.ndarray, ids: np.ndarray, rows: np.ndarray) -> None:
    """sums[j] += sum of rows with ids == j (sort + reduceat, float64)."""
    if ids.shape[0] == 0:
        return
    order = np.argsort(ids, kind="stable")
    ids_s = ids[order]
    starts = np.flatnonzero(np.r_[True, ids_s[1:] != ids_s[:-1]])
    sums[ids_s[starts]] += np.add.reduceat(rows[order], starts, axis=0)
