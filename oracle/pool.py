"""Per-GPU KV-cache sizing (Sec. 1.1, Eq. 1 and Eq. 2) and the paged block pool.

Test infrastructure only (see the package header).

Eq. 1: KV bytes one sequence reserves, M_seq = 2 * n_l * n_h * d_h * b_dtype * C_max
       (K and V, every layer, every KV head on this GPU, C_max tokens).
Eq. 2: concurrent sequences one GPU holds,
       N_seq = floor((M_gpu * u - M_model) / M_seq), never below 0.

The paged pool backing a pool instance reserves C_max tokens per sequence in
16-token blocks (Sec. 3, effects 1 and 3): blocks_per_seq = ceil(C_max / bs)
and num_blocks = N_seq * blocks_per_seq.  A sequence of n cached tokens
holds ceil(n / bs) of them (pages are allocated on demand, Sec. 3 effect 1).

Order of the float64 operations in Eq. 2: (M_gpu * u), then minus M_model,
then divided by float(M_seq), then floor.  The C library uses the same order.

Parity: pinned by the paper's worked MI300X case (Sec. 4.7): 94 layers, one KV
head per GPU at TP=8, d_h 128, FP8 -> 23.5 KiB per token; 192 GB * 0.9 - 39.4 GB
= 133.4 GB for KV; N_seq = 676 at C_max 8K and 169 at 32K; the last-block
waste of 128 sequences, 15 tokens each, is about 46 MB (Sec. 3 effect 3).
"""
from __future__ import annotations

import math


def kv_bytes_per_token(n_layers: int, n_kv_heads: int, head_dim: int, dtype_bytes: int) -> int:
    """Eq. 1 with C_max = 1: 2 * n_l * n_h * d_h * b_dtype."""
    return 2 * n_layers * n_kv_heads * head_dim * dtype_bytes


def m_seq(n_layers: int, n_kv_heads: int, head_dim: int, dtype_bytes: int, c_max: int) -> int:
    """Eq. 1: KV-cache bytes reserved per sequence (exact integer)."""
    return 2 * n_layers * n_kv_heads * head_dim * dtype_bytes * c_max


def n_seq(m_gpu_bytes: float, util: float, m_model_bytes: float, m_seq_bytes: int) -> int:
    """Eq. 2: maximum concurrent sequences per GPU (clamped at 0)."""
    x = math.floor((m_gpu_bytes * util - m_model_bytes) / float(m_seq_bytes))
    return max(0, int(x))


def blocks_per_seq(c_max: int, block_size: int = 16) -> int:
    return -(-c_max // block_size)


def pool_blocks(n_seq_value: int, c_max: int, block_size: int = 16) -> int:
    """Physical blocks in the paged pool: N_seq sequences of ceil(C_max / bs) blocks."""
    return n_seq_value * blocks_per_seq(c_max, block_size)


def blocks_for_tokens(n_tokens: int, block_size: int = 16) -> int:
    """Blocks one sequence of n_tokens cached tokens holds (on-demand pages)."""
    return -(-n_tokens // block_size)


def size_pool(n_layers, n_kv_heads, head_dim, dtype_bytes, block_size, c_max,
              m_gpu_bytes, util, m_model_bytes):
    """All sizing outputs at once: (M_seq, N_seq, blocks_per_seq, num_blocks)."""
    ms = m_seq(n_layers, n_kv_heads, head_dim, dtype_bytes, c_max)
    ns = n_seq(m_gpu_bytes, util, m_model_bytes, ms)
    bps = blocks_per_seq(c_max, block_size)
    return ms, ns, bps, ns * bps
