"""Thin ctypes binding of libdpool (include/dpool.h).

Argument marshalling only: every step of the decode runs in the library's
HIP kernels, the pool and the router run in its C++ host code.  torch
tensors supply device pointers and the current HIP stream.  There is no
fallback: if libdpool.so is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# DPOOL_LIB selects another build of the same library (the host-sanitizer
# build of build_sanitize.py, for the CPU tests)
LIB_PATH = os.environ.get("DPOOL_LIB") or os.path.join(_PKG, "libdpool.so")

DP_OK = 0
DP_EIO = -5
DP_ENOMEM = -12
DP_EINVAL = -22
DP_ENOTSUP = -95
KV_BF16, KV_FP8_E4M3 = 0, 1
OUT_BF16, OUT_FP32 = 0, 1

# every function the header declares
EXPORTS = (
    "dp_last_error", "dp_version",
    "kv_pool_create", "kv_pool_info", "kv_pool_alloc_seq", "kv_pool_free_seq", "kv_pool_destroy",
    "route_default_params", "route_init", "route_requests", "route_on_response",
    "route_adapt_default_params", "route_adapt_threshold", "dp_cost_model",
    "paged_decode_workspace_size", "paged_decode_partition_tokens", "paged_decode_attention",
    "paged_decode_attention_noalloc",
    "kv_cache_append", "chunked_prefill_attention", "dp_hbm_read_probe",
)


class DpoolError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libdpool error {code}: {msg}")
        self.code = code


class PoolConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype_bytes", ctypes.c_int32), ("block_size", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("c_max", ctypes.c_int64), ("m_gpu_bytes", ctypes.c_double), ("util", ctypes.c_double),
                ("m_model_bytes", ctypes.c_double)]


class RouteParams(ctypes.Structure):
    _fields_ = [("b_short", ctypes.c_double), ("beta", ctypes.c_double), ("gamma", ctypes.c_double),
                ("c0", ctypes.c_double), ("c_min", ctypes.c_double), ("spill_theta", ctypes.c_double)]


class CatState(ctypes.Structure):
    _fields_ = [("c_hat", ctypes.c_double), ("sigma", ctypes.c_double)]


class PoolState(ctypes.Structure):
    _fields_ = [("c_max", ctypes.c_int64), ("capacity", ctypes.c_int64), ("in_flight", ctypes.c_int64)]


class PoolSignals(ctypes.Structure):
    _fields_ = [("admitted", ctypes.c_int64), ("preempted", ctypes.c_int64), ("oom", ctypes.c_int64),
                ("rejected", ctypes.c_int64)]


class AdaptParams(ctypes.Structure):
    _fields_ = [("w_preempt", ctypes.c_double), ("w_oom", ctypes.c_double), ("w_reject", ctypes.c_double),
                ("target", ctypes.c_double), ("step", ctypes.c_double), ("b_min", ctypes.c_double),
                ("b_max", ctypes.c_double)]


class CostResult(ctypes.Structure):
    _fields_ = [("g_homo", ctypes.c_int64), ("g_dual", ctypes.c_int64), ("rho", ctypes.c_double),
                ("savings_formula", ctypes.c_double), ("savings_fleet", ctypes.c_double)]


class DecodeShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("max_blocks_per_seq", ctypes.c_int32), ("max_context_len", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("partition_tokens", ctypes.c_int32), ("workgroups_per_cu", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("num_blocks", ctypes.c_int64)]


class PrefillShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("max_blocks_per_seq", ctypes.c_int32), ("max_context_len", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32), ("query_tile", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("total_q", ctypes.c_int64), ("num_blocks", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libdpool.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2604_08075_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        c_i32p, c_i64p, c_i8p = (ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
                                 ctypes.POINTER(ctypes.c_int8))
        L.dp_last_error.restype = ctypes.c_char_p
        L.dp_version.restype = ctypes.c_char_p
        L.kv_pool_create.argtypes = [ctypes.POINTER(PoolConfig), ctypes.c_uint64, ctypes.POINTER(ctypes.c_void_p)]
        L.kv_pool_info.argtypes = [ctypes.c_void_p, c_i64p, c_i64p, c_i64p, c_i64p, c_i64p]
        L.kv_pool_alloc_seq.argtypes = [ctypes.c_void_p, ctypes.c_int64, c_i32p]
        L.kv_pool_free_seq.argtypes = [ctypes.c_void_p, c_i32p, ctypes.c_int64]
        L.kv_pool_destroy.argtypes = [ctypes.c_void_p]
        L.kv_pool_destroy.restype = None
        L.route_default_params.argtypes = [ctypes.POINTER(RouteParams)]
        L.route_init.argtypes = [ctypes.POINTER(RouteParams), ctypes.POINTER(CatState), ctypes.c_int32]
        L.route_requests.argtypes = [ctypes.POINTER(RouteParams), ctypes.POINTER(CatState), ctypes.c_int32,
                                     ctypes.POINTER(PoolState), c_i64p, c_i32p, c_i64p, ctypes.c_int64, c_i8p, c_i64p]
        L.route_on_response.argtypes = [ctypes.POINTER(RouteParams), ctypes.POINTER(CatState), ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int64, ctypes.c_int64]
        L.route_adapt_default_params.argtypes = [ctypes.POINTER(AdaptParams)]
        L.route_adapt_threshold.argtypes = [ctypes.POINTER(AdaptParams), ctypes.POINTER(PoolSignals),
                                            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]
        L.dp_cost_model.argtypes = [ctypes.c_double] * 4 + [ctypes.POINTER(CostResult)]
        L.paged_decode_workspace_size.argtypes = [ctypes.POINTER(DecodeShape)]
        L.paged_decode_workspace_size.restype = ctypes.c_size_t
        L.paged_decode_partition_tokens.argtypes = [ctypes.POINTER(DecodeShape)]
        L.paged_decode_partition_tokens.restype = ctypes.c_int32
        L.paged_decode_attention.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_float] + [ctypes.c_void_p] * 3 + [
            ctypes.POINTER(DecodeShape), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.paged_decode_attention_noalloc.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_float] + [
            ctypes.c_void_p] * 3 + [ctypes.POINTER(DecodeShape), ctypes.c_void_p]
        L.kv_cache_append.argtypes = [ctypes.c_void_p] * 8 + [ctypes.POINTER(DecodeShape), ctypes.c_void_p]
        L.chunked_prefill_attention.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_float] + [ctypes.c_void_p] * 3 + [
            ctypes.POINTER(PrefillShape), ctypes.c_void_p]
        L.dp_hbm_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        _lib = L
    return _lib


def last_error() -> str:
    return lib().dp_last_error().decode()


def check(rc: int) -> int:
    if rc != DP_OK:
        raise DpoolError(rc, last_error())
    return rc


def version() -> str:
    return lib().dp_version().decode()


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


# ---------------------------------------------------------------- KV pool

@dataclass
class PoolInfo:
    m_seq_bytes: int
    n_seq: int
    blocks_per_seq: int
    num_blocks: int
    free_blocks: int


class KVPool:
    """Owner of a dp_kv_pool handle (host memory)."""

    def __init__(self, n_layers, n_kv_heads, head_dim, dtype_bytes, c_max, m_gpu_bytes, util, m_model_bytes,
                 block_size=16, seed=0):
        cfg = PoolConfig(n_layers, n_kv_heads, head_dim, dtype_bytes, block_size, 0, c_max, m_gpu_bytes, util,
                         m_model_bytes)
        h = ctypes.c_void_p()
        check(lib().kv_pool_create(ctypes.byref(cfg), ctypes.c_uint64(seed), ctypes.byref(h)))
        self._h = h
        self.block_size = block_size

    def info(self) -> PoolInfo:
        vals = [ctypes.c_int64() for _ in range(5)]
        check(lib().kv_pool_info(self._h, *[ctypes.byref(v) for v in vals]))
        return PoolInfo(*[v.value for v in vals])

    def alloc_seq(self, n_tokens: int) -> np.ndarray:
        n = -(-n_tokens // self.block_size) if n_tokens > 0 else 0
        out = np.empty(max(n, 1), dtype=np.int32)
        check(lib().kv_pool_alloc_seq(self._h, n_tokens, _ptr(out, ctypes.c_int32)))
        return out[:n]

    def free_seq(self, ids) -> None:
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        check(lib().kv_pool_free_seq(self._h, _ptr(ids, ctypes.c_int32), len(ids)))

    def close(self):
        if self._h:
            lib().kv_pool_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- router

def default_route_params() -> RouteParams:
    p = RouteParams()
    check(lib().route_default_params(ctypes.byref(p)))
    return p


def make_categories(params: RouteParams, n_cats: int):
    cats = (CatState * n_cats)()
    check(lib().route_init(ctypes.byref(params), cats, n_cats))
    return cats


def make_pools(short_c_max, short_capacity, long_c_max, long_capacity):
    pools = (PoolState * 2)()
    pools[0] = PoolState(short_c_max, short_capacity, 0)
    pools[1] = PoolState(long_c_max, long_capacity, 0)
    return pools


def route_requests(params, cats, pools, req_bytes, req_cat, req_max_out):
    """Route a batch in order; returns (pool ids int8 [n], L_total int64 [n])."""
    b = np.ascontiguousarray(req_bytes, dtype=np.int64)
    k = np.ascontiguousarray(req_cat, dtype=np.int32)
    m = np.ascontiguousarray(req_max_out, dtype=np.int64)
    n = len(b)
    if len(k) != n or len(m) != n:
        raise ValueError("request arrays differ in length")
    out_p = np.empty(max(n, 1), dtype=np.int8)
    out_l = np.empty(max(n, 1), dtype=np.int64)
    check(lib().route_requests(ctypes.byref(params), cats, len(cats), pools, _ptr(b, ctypes.c_int64),
                               _ptr(k, ctypes.c_int32), _ptr(m, ctypes.c_int64), n, _ptr(out_p, ctypes.c_int8),
                               _ptr(out_l, ctypes.c_int64)))
    return out_p[:n], out_l[:n]


def route_on_response(params, cats, cat: int, req_bytes: int, prompt_tokens: int) -> None:
    check(lib().route_on_response(ctypes.byref(params), cats, len(cats), cat, req_bytes, prompt_tokens))


def default_adapt_params() -> AdaptParams:
    p = AdaptParams()
    check(lib().route_adapt_default_params(ctypes.byref(p)))
    return p


def adapt_threshold(params: AdaptParams, short_signals, long_signals, b_short: float):
    """One control step; signals are (admitted, preempted, oom, rejected).  Returns (b_short, action)."""
    sig = (PoolSignals * 2)(PoolSignals(*short_signals), PoolSignals(*long_signals))
    b = ctypes.c_double(float(b_short))
    act = ctypes.c_int32(0)
    check(lib().route_adapt_threshold(ctypes.byref(params), sig, ctypes.byref(b), ctypes.byref(act)))
    return b.value, act.value


# ---------------------------------------------------------------- cost model

def cost_model(lam: float, alpha: float, mu_short: float, mu_long: float) -> CostResult:
    """Sec. 3 fleet sizing and savings (include/dpool.h, dp_cost_model)."""
    out = CostResult()
    check(lib().dp_cost_model(float(lam), float(alpha), float(mu_short), float(mu_long), ctypes.byref(out)))
    return out


# ---------------------------------------------------------------- decode

def decode_shape(batch, n_q_heads, n_kv_heads, max_blocks_per_seq, max_context_len, num_blocks, kv_fp8=False,
                 out_fp32=False, partition_tokens=0, workgroups_per_cu=0, head_dim=128,
                 block_size=16) -> DecodeShape:
    return DecodeShape(batch, n_q_heads, n_kv_heads, head_dim, block_size, max_blocks_per_seq, max_context_len,
                       KV_FP8_E4M3 if kv_fp8 else KV_BF16, OUT_FP32 if out_fp32 else OUT_BF16, partition_tokens,
                       workgroups_per_cu, 0, num_blocks)


def workspace_size(shape: DecodeShape) -> int:
    return int(lib().paged_decode_workspace_size(ctypes.byref(shape)))


def partition_tokens(shape: DecodeShape) -> int:
    return int(lib().paged_decode_partition_tokens(ctypes.byref(shape)))


_partition_tokens = partition_tokens


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ws(workspace):
    if workspace is None:
        return None, 0
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def paged_decode_attention(q, k_blocks, v_blocks, block_tables, context_lens, scale, out, shape: DecodeShape,
                           workspace=None, k_scale=None, v_scale=None, stream=None) -> None:
    """Enqueue the decode on `stream` (default: torch's current stream).  All tensors are
    device tensors laid out as include/dpool.h documents; nothing is copied or converted.
    The workspace must have been zero-filled before its first use."""
    ws_ptr, ws_bytes = _ws(workspace)
    check(lib().paged_decode_attention(
        q.data_ptr(), k_blocks.data_ptr(), v_blocks.data_ptr(), block_tables.data_ptr(), context_lens.data_ptr(),
        float(scale), k_scale.data_ptr() if k_scale is not None else None,
        v_scale.data_ptr() if v_scale is not None else None, out.data_ptr(), ctypes.byref(shape), ws_ptr, ws_bytes,
        _stream_ptr(stream)))


def paged_decode_attention_noalloc(q, k_blocks, v_blocks, block_tables, context_lens, scale, out,
                                   shape: DecodeShape, k_scale=None, v_scale=None, stream=None) -> None:
    """Enqueue the decode without a workspace (the library's fixed per-GPU scratch;
    include/dpool.h, paged_decode_attention_noalloc)."""
    check(lib().paged_decode_attention_noalloc(
        q.data_ptr(), k_blocks.data_ptr(), v_blocks.data_ptr(), block_tables.data_ptr(), context_lens.data_ptr(),
        float(scale), k_scale.data_ptr() if k_scale is not None else None,
        v_scale.data_ptr() if v_scale is not None else None, out.data_ptr(), ctypes.byref(shape),
        _stream_ptr(stream)))


def kv_cache_append(k_new, v_new, k_blocks, v_blocks, block_tables, positions, shape: DecodeShape, k_scale=None,
                    v_scale=None, stream=None) -> None:
    """Enqueue the append of one token per sequence (include/dpool.h, kv_cache_append)."""
    check(lib().kv_cache_append(
        k_new.data_ptr(), v_new.data_ptr(), k_blocks.data_ptr(), v_blocks.data_ptr(), block_tables.data_ptr(),
        positions.data_ptr(), k_scale.data_ptr() if k_scale is not None else None,
        v_scale.data_ptr() if v_scale is not None else None, ctypes.byref(shape), _stream_ptr(stream)))


def prefill_shape(batch, n_q_heads, n_kv_heads, max_blocks_per_seq, max_context_len, num_blocks, total_q,
                  kv_fp8=False, out_fp32=False, query_tile=0, head_dim=128, block_size=16) -> PrefillShape:
    return PrefillShape(batch, n_q_heads, n_kv_heads, head_dim, block_size, max_blocks_per_seq, max_context_len,
                        KV_FP8_E4M3 if kv_fp8 else KV_BF16, OUT_FP32 if out_fp32 else OUT_BF16, query_tile, 0,
                        total_q, num_blocks)


def chunked_prefill_attention(q, k_blocks, v_blocks, block_tables, context_lens, q_start, scale, out,
                              shape: PrefillShape, k_scale=None, v_scale=None, stream=None) -> None:
    """Enqueue the chunked-prefill attention (include/dpool.h, chunked_prefill_attention)."""
    check(lib().chunked_prefill_attention(
        q.data_ptr(), k_blocks.data_ptr(), v_blocks.data_ptr(), block_tables.data_ptr(), context_lens.data_ptr(),
        q_start.data_ptr(), float(scale), k_scale.data_ptr() if k_scale is not None else None,
        v_scale.data_ptr() if v_scale is not None else None, out.data_ptr(), ctypes.byref(shape),
        _stream_ptr(stream)))


def hbm_read_probe(buf, workgroups, sink, tile_ids=None, stream=None) -> None:
    """Enqueue one read of `buf` (contiguous, or its 4 KiB tiles in `tile_ids` order)."""
    nbytes = buf.numel() * buf.element_size()
    check(lib().dp_hbm_read_probe(buf.data_ptr(), nbytes, tile_ids.data_ptr() if tile_ids is not None else None,
                                  tile_ids.numel() if tile_ids is not None else 0, int(workgroups), sink.data_ptr(),
                                  sink.numel() * sink.element_size(), _stream_ptr(stream)))


class PagedDecoder:
    """Holds one decode shape and its workspace; calling it enqueues the decode.

    Device memory for the workspace comes from torch's allocator once, at
    construction, zero-filled as the library requires; each call only marshals
    pointers into paged_decode_attention.
    """

    def __init__(self, batch, n_q_heads, n_kv_heads, max_blocks_per_seq, max_context_len, num_blocks,
                 kv_fp8=False, out_fp32=False, partition_tokens=0, workgroups_per_cu=0, device="cuda"):
        import torch
        self.shape = decode_shape(batch, n_q_heads, n_kv_heads, max_blocks_per_seq, max_context_len, num_blocks,
                                  kv_fp8, out_fp32, partition_tokens, workgroups_per_cu)
        self.partition_tokens = _partition_tokens(self.shape)
        if self.partition_tokens <= 0:
            raise DpoolError(DP_EINVAL, last_error())
        ws = workspace_size(self.shape)
        self.workspace = torch.zeros(ws, dtype=torch.uint8, device=device) if ws else None
        self.out_dtype = torch.float32 if out_fp32 else torch.bfloat16

    def new_out(self, device="cuda"):
        import torch
        s = self.shape
        return torch.empty((s.batch, s.n_q_heads, s.head_dim), dtype=self.out_dtype, device=device)

    def __call__(self, q, k_blocks, v_blocks, block_tables, context_lens, scale, out, k_scale=None, v_scale=None,
                 stream=None):
        paged_decode_attention(q, k_blocks, v_blocks, block_tables, context_lens, scale, out, self.shape,
                               self.workspace, k_scale, v_scale, stream)
        return out
