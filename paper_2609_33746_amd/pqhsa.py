"""Thin ctypes binding of libpqhsa (include/pqhsa.h).

Argument marshalling only: torch tensors provide device pointers and the
current HIP stream; every step of the operator runs in the library's HIP
kernels. There is no fallback: if the library is missing or the device is
not a GPU, the calls raise.
"""

from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libpqhsa.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "pqhsa.h")

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_HIP, ERR_OUT_OF_MEMORY, ERR_NOT_PREPARED = range(6)
F32, BF16 = 0, 1
OPT_FORCE_FALLBACK, OPT_STAGE_TIMING, OPT_THRESHOLD_BIAS, OPT_VARIANT = 1, 2, 3, 4
VARIANT_B, VARIANT_T, VARIANT_C, VARIANT_BX = 0, 1, 2, 3
STAGES = ("prologue", "scan", "select", "attend", "merge")


class Shape(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "batch", "n_q_heads", "n_kv_heads", "head_dim", "max_seq", "n_list", "pq_m",
        "pq_ksub", "n_sink", "n_local", "max_topk", "kv_dtype")]


class PQHSAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status


_lib = None


def load_library(build_if_missing: bool = True) -> ctypes.CDLL:
    """Load the in-tree libpqhsa.so (building it once if it does not exist)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        if not build_if_missing:
            raise FileNotFoundError(LIB_PATH)
        from .build import build
        build()
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sigs = {
        "pqhsa_create": ([ctypes.POINTER(Shape), ctypes.POINTER(P)], I32),
        "pqhsa_destroy": ([P], None),
        "pqhsa_index_prepare": ([P] + [P] * 7 + [P], I32),
        "pqhsa_decode": ([P, P, P, P, P, P, P, P], I32),
        "pqhsa_decode_device_args": ([P, P, P, P, P, P, P, P, P], I32),
        "pqhsa_decode_paged": ([P, P, P, P, P, P, I32, I32, P, P, P], I32),
        "pqhsa_index_update": ([P, P, P, P, P, P], I32),
        "pqhsa_set_lengths": ([P, P], I32),
        "pqhsa_index_export_tokens": ([P, P, P, P, P, P, P, P], I32),
        "pqhsa_index_build": ([P, P, P, P, P, P, P, I32, I32, P], I32),
        "pqhsa_decode_debug": ([P, P, P, P, P, P, P, P, P, P, P], I32),
        "pqhsa_dense_decode": ([P, P, P, P, P, P, P, P], I32),
        "pqhsa_dense_decode_noalloc": ([I32, I32, I32, I32, I32, P, P, P, P, P, P, P], I32),
        "pqhsa_index_export": ([P, P, P, P], I32),
        "pqhsa_set_option": ([P, I32, I64], I32),
        "pqhsa_stage_times": ([P, P, I32, P], I32),
        "pqhsa_status_string": ([I32], ctypes.c_char_p),
        "pqhsa_last_error": ([P], ctypes.c_char_p),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def declared_functions() -> list[str]:
    """Names of the functions declared in include/pqhsa.h."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pqhsa_[a-z_]+)\s*\(", text)))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _host_i32(values):
    arr = (ctypes.c_int32 * len(values))(*[int(v) for v in values])
    return arr


class PQHSA:
    """One operator context: shape, prepared index and decode workspace."""

    def __init__(self, batch: int, n_q_heads: int, n_kv_heads: int, max_seq: int, n_list: int,
                 max_topk: int, kv_dtype: str = "bf16", head_dim: int = 128, pq_m: int = 16,
                 pq_ksub: int = 256, n_sink: int = 4, n_local: int = 128):
        self.lib = load_library()
        self.shape = Shape(batch, n_q_heads, n_kv_heads, head_dim, max_seq, n_list, pq_m, pq_ksub,
                           n_sink, n_local, max_topk, BF16 if kv_dtype == "bf16" else F32)
        self.dtype = torch.bfloat16 if kv_dtype == "bf16" else torch.float32
        self.ctx = ctypes.c_void_p()
        st = self.lib.pqhsa_create(ctypes.byref(self.shape), ctypes.byref(self.ctx))
        if st != OK:
            raise PQHSAError(st, self.lib.pqhsa_last_error(None).decode())

    # -- helpers -----------------------------------------------------------
    def _check(self, st):
        if st != OK:
            raise PQHSAError(st, self.lib.pqhsa_last_error(self.ctx).decode())

    def _dev(self, t, dtype, name):
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
            raise ValueError(f"{name} must be a GPU tensor")
        if t.dtype != dtype:
            raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return t

    def _kv(self, k_cache, v_cache):
        if k_cache.dtype != self.dtype or v_cache.dtype != self.dtype:
            raise ValueError("k_cache / v_cache dtype does not match the context")
        if k_cache.device.type != "cuda" or v_cache.device.type != "cuda":
            raise ValueError("k_cache / v_cache must be GPU tensors")
        if k_cache.stride() != v_cache.stride() or k_cache.stride(3) != 1:
            raise ValueError("k_cache and v_cache need equal strides and a contiguous last dim")
        st = k_cache.stride()
        return (ctypes.c_int64 * 3)(st[0], st[1], st[2])

    # -- ABI calls -----------------------------------------------------------
    def index_prepare(self, seq_lens, list_ids, codes, norms, centroids, codebooks, list_means):
        lens = _host_i32(list(seq_lens))
        self._check(self.lib.pqhsa_index_prepare(
            self.ctx, lens,
            _ptr(self._dev(list_ids, torch.int32, "list_ids")),
            _ptr(self._dev(codes, torch.uint8, "codes")),
            _ptr(self._dev(norms, torch.float32, "norms")),
            _ptr(self._dev(centroids, torch.float32, "centroids")),
            _ptr(self._dev(codebooks, torch.float32, "codebooks")),
            _ptr(self._dev(list_means, torch.float32, "list_means")), _stream()))

    def index_update(self, new_seq_lens, k_cache, v_cache):
        """Encode the tokens leaving the local window into the existing lists."""
        strides = self._kv(k_cache, v_cache)
        self._check(self.lib.pqhsa_index_update(self.ctx, _host_i32(list(new_seq_lens)),
                                                _ptr(k_cache), _ptr(v_cache), strides, _stream()))

    def set_lengths(self, seq_lens):
        """Current cache lengths: the tokens past the index stay exact."""
        self._check(self.lib.pqhsa_set_lengths(self.ctx, _host_i32(list(seq_lens))))

    def index_export_tokens(self):
        """The token-major index: list_ids, codes, norms [B, Hkv, max_seq(, M)] and
        list_means [B, Hkv, n_list, d] (entries outside R unspecified)."""
        sh = self.shape
        dev = torch.device("cuda", torch.cuda.current_device())
        ids = torch.empty((sh.batch, sh.n_kv_heads, sh.max_seq), dtype=torch.int32, device=dev)
        codes = torch.empty((sh.batch, sh.n_kv_heads, sh.max_seq, sh.pq_m), dtype=torch.uint8,
                            device=dev)
        norms = torch.empty((sh.batch, sh.n_kv_heads, sh.max_seq), dtype=torch.float32, device=dev)
        means = torch.empty((sh.batch, sh.n_kv_heads, sh.n_list, sh.head_dim), dtype=torch.float32,
                            device=dev)
        cen = torch.empty_like(means)
        cb = torch.empty((sh.batch, sh.n_kv_heads, sh.pq_m, sh.pq_ksub, sh.head_dim // sh.pq_m),
                         dtype=torch.float32, device=dev)
        self._check(self.lib.pqhsa_index_export_tokens(self.ctx, _ptr(ids), _ptr(codes),
                                                       _ptr(norms), _ptr(means), _ptr(cen),
                                                       _ptr(cb), _stream()))
        return dict(list_ids=ids, codes=codes, norms=norms, list_means=means, centroids=cen,
                    codebooks=cb)

    def index_build(self, seq_lens, k_cache, v_cache, init_coarse, init_pq, n_iter_coarse=1,
                    n_iter_pq=2):
        """k-means build of the index from the keys (starting tokens drawn by the caller)."""
        strides = self._kv(k_cache, v_cache)
        ic = self._dev(init_coarse, torch.int32, "init_coarse")
        ip = self._dev(init_pq, torch.int32, "init_pq")
        self._check(self.lib.pqhsa_index_build(
            self.ctx, _host_i32(list(seq_lens)), _ptr(k_cache), _ptr(v_cache), strides, _ptr(ic),
            _ptr(ip), int(n_iter_coarse), int(n_iter_pq), _stream()))

    def _out(self, q, out):
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        return self._dev(out, torch.float32, "out")

    def decode(self, q, k_cache, v_cache, topk, out=None):
        strides = self._kv(k_cache, v_cache)
        q = self._dev(q, self.dtype, "q")
        out = self._out(q, out)
        self._check(self.lib.pqhsa_decode(self.ctx, _ptr(q), _ptr(k_cache), _ptr(v_cache), strides,
                                          _host_i32(list(topk)), _ptr(out), _stream()))
        return out

    def decode_device_args(self, q, k_cache, v_cache, seq_lens, topk, out=None):
        """Decode with N_b and k_b read on the device from int32 GPU tensors
        [B] when the step runs (so a captured graph takes new values on every
        replay)."""
        strides = self._kv(k_cache, v_cache)
        q = self._dev(q, self.dtype, "q")
        lens = self._dev(seq_lens, torch.int32, "seq_lens")
        tk = self._dev(topk, torch.int32, "topk")
        if lens.numel() != self.shape.batch or tk.numel() != self.shape.batch:
            raise ValueError("seq_lens and topk must hold one entry per sequence")
        out = self._out(q, out)
        self._check(self.lib.pqhsa_decode_device_args(self.ctx, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                      strides, _ptr(lens), _ptr(tk), _ptr(out),
                                                      _stream()))
        return out

    def decode_paged(self, q, k_pages, v_pages, block_table, page_size, topk, out=None):
        """Decode from a paged cache: k_pages / v_pages [n_pages, Hkv, page_size, d]
        (views of one interleaved tensor allowed), block_table int32 [B, max_blocks]."""
        strides = self._kv(k_pages, v_pages)
        if k_pages.shape[2] != page_size:
            raise ValueError("k_pages.shape[2] must equal page_size")
        bt = self._dev(block_table, torch.int32, "block_table")
        if bt.dim() != 2 or bt.shape[0] != self.shape.batch:
            raise ValueError("block_table must be [batch, max_blocks]")
        q = self._dev(q, self.dtype, "q")
        out = self._out(q, out)
        self._check(self.lib.pqhsa_decode_paged(
            self.ctx, _ptr(q), _ptr(k_pages), _ptr(v_pages), strides, _ptr(bt), int(bt.shape[1]),
            int(page_size), _host_i32(list(topk)), _ptr(out), _stream()))
        return out

    def decode_debug(self, q, k_cache, v_cache, topk, out=None, want_scores=False):
        strides = self._kv(k_cache, v_cache)
        q = self._dev(q, self.dtype, "q")
        out = self._out(q, out)
        s = self.shape
        dev = q.device
        selected = torch.empty((s.batch, s.n_q_heads, max(s.max_topk, 1)), dtype=torch.int32, device=dev)
        unsel = torch.empty((s.batch, s.n_q_heads, s.n_list), dtype=torch.int32, device=dev)
        scores = (torch.empty((s.batch, s.n_q_heads, s.max_seq), dtype=torch.float32, device=dev)
                  if want_scores else None)
        self._check(self.lib.pqhsa_decode_debug(
            self.ctx, _ptr(q), _ptr(k_cache), _ptr(v_cache), strides, _host_i32(list(topk)),
            _ptr(out), _ptr(selected), _ptr(unsel), _ptr(scores), _stream()))
        return out, selected[..., :s.max_topk], unsel, scores

    def dense_decode(self, q, k_cache, v_cache, seq_lens, out=None):
        strides = self._kv(k_cache, v_cache)
        q = self._dev(q, self.dtype, "q")
        out = self._out(q, out)
        self._check(self.lib.pqhsa_dense_decode(self.ctx, _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                strides, _host_i32(list(seq_lens)), _ptr(out),
                                                _stream()))
        return out

    def index_export(self):
        s = self.shape
        dev = torch.device("cuda", torch.cuda.current_device())
        perm = torch.empty((s.batch, s.n_kv_heads, s.max_seq), dtype=torch.int32, device=dev)
        offs = torch.empty((s.batch, s.n_kv_heads, s.n_list + 1), dtype=torch.int32, device=dev)
        self._check(self.lib.pqhsa_index_export(self.ctx, _ptr(perm), _ptr(offs), _stream()))
        return perm, offs

    def set_option(self, option: int, value: int):
        self._check(self.lib.pqhsa_set_option(self.ctx, option, int(value)))

    def stage_times(self) -> dict:
        ms = (ctypes.c_float * 8)()
        n = ctypes.c_int32()
        self._check(self.lib.pqhsa_stage_times(self.ctx, ms, 8, ctypes.byref(n)))
        return {STAGES[i]: ms[i] for i in range(n.value)}

    def close(self):
        if self.ctx:
            self.lib.pqhsa_destroy(self.ctx)
            self.ctx = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dense_decode_noalloc(q, k_cache, v_cache, seq_lens, out=None):
    """Dense decode without a context: the library's fixed scratch array holds
    the split partials, and the call allocates no device memory (apart from
    `out` when it is not given). q [B, Hq, d]; k_cache, v_cache [B, Hkv, N, d]
    with equal strides and a contiguous last dimension; seq_lens: B ints."""
    lib = load_library()
    if q.device.type != "cuda" or k_cache.device.type != "cuda" or v_cache.device.type != "cuda":
        raise ValueError("q, k_cache and v_cache must be GPU tensors")
    if not q.is_contiguous() or k_cache.stride() != v_cache.stride() or k_cache.stride(3) != 1:
        raise ValueError("q must be contiguous; k_cache and v_cache need equal strides and a "
                         "contiguous last dimension")
    if q.dtype != k_cache.dtype or v_cache.dtype != k_cache.dtype:
        raise ValueError("q, k_cache and v_cache must share one dtype")
    dtype = {torch.bfloat16: BF16, torch.float32: F32}.get(k_cache.dtype)
    if dtype is None:
        raise ValueError("dtype must be bfloat16 or float32")
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 tensor")
    st = k_cache.stride()
    strides = (ctypes.c_int64 * 3)(st[0], st[1], st[2])
    status = lib.pqhsa_dense_decode_noalloc(
        int(q.shape[0]), int(q.shape[1]), int(k_cache.shape[1]), int(q.shape[2]), dtype, _ptr(q),
        _ptr(k_cache), _ptr(v_cache), strides, _host_i32(list(seq_lens)), _ptr(out), _stream())
    if status != OK:
        raise PQHSAError(status, lib.pqhsa_last_error(None).decode())
    return out


def context_for(inp: dict, max_topk: int | None = None) -> "PQHSA":
    """Context sized for a generated workload (see synth.make_inputs)."""
    wl = inp["workload"]
    return PQHSA(wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.max_seq, wl.n_list,
                 int(max_topk if max_topk is not None else int(inp["topk"].max())),
                 kv_dtype=wl.kv_dtype, head_dim=wl.head_dim, pq_m=wl.pq_m, pq_ksub=wl.pq_ksub,
                 n_sink=inp["n_sink"], n_local=inp["n_local"])


def prepare_from(ctx: "PQHSA", inp: dict):
    """Load a generated workload's index (its tensors must be on the GPU)."""
    ctx.index_prepare(inp["seq_lens"].tolist(), inp["list_ids"], inp["codes"], inp["norms"],
                      inp["centroids"], inp["codebooks"], inp["list_means"])
