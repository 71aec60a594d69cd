"""KV-cache append (one new token per sequence), written out from its definition.

Test infrastructure only (see the package header).

What is computed.  Every decode step adds the new token's key and value to
the cache before attention reads it (Sec. 4.4, "Why TPOT also improves": one
KV-cache lookup per layer per generated token); the cache is PagedAttention's
16-token blocks handed out on demand (Sec. 3, effects 1 and 3); the Sec. 4.7
deployment stores it in FP8.  For sequence s whose new token sits at position
t = positions[s], and KV head g:

    blk = block_tables[s, t // 16], slot = t % 16
    k_blocks[blk, g, slot, :] = enc(k_new[s, g, :], k_scale[g])   (token-major K tile)
    v_blocks[blk, g, :, slot] = enc(v_new[s, g, :], v_scale[g])   (dims-major V tile)

enc copies the bf16 bits for a bf16 cache.  For an e4m3 cache it divides the
bf16 value by the per-head scale in IEEE float32 (correctly rounded; this
quotient decides an integer code, so it is taken in the precision the kernel
uses), clamps it to [-448, 448] and rounds to the nearest OCP E4M3FN value,
ties to the even code (the one whose mantissa's last bit is 0); the sign of
the quotient is kept, zero included.  A position outside the block table or
a block id outside the pool writes nothing (the library's documented choice;
the paper never appends out of range).

Parity: ``e4m3_encode`` is pinned by torch's float8_e4m3fn cast on
clamped float32 values (a library routine), by the exact round trip of every
finite code, and by hand-worked ties and saturation; ``kv_cache_append`` by
an element-by-element scalar restatement on small pools.
"""
from __future__ import annotations

import numpy as np

from . import numerics

E4M3_MAX = 448.0


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """Nearest OCP E4M3FN code (uint8) of each finite value, saturating, ties to even."""
    x = np.asarray(x, dtype=np.float64)
    table = numerics.e4m3_table()
    mags = table[:0x7F]                     # codes 0x00..0x7E: 0 .. 448, increasing
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.clip(np.searchsorted(mags, a, side="left"), 0, 0x7E)  # first magnitude >= a
    lo = np.maximum(hi - 1, 0)
    d_lo = a - mags[lo]
    d_hi = mags[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    neg = np.signbit(x)
    return np.where(neg, code | 0x80, code).astype(np.uint8)


def encode(bits: np.ndarray, fmt: str, scale: float | None) -> np.ndarray:
    """The stored codes of bf16 bit patterns for a cache of format fmt."""
    bits = np.asarray(bits).view(np.uint16)
    if fmt == "bf16":
        return bits.copy()
    if fmt == "fp8_e4m3":
        q = numerics.decode_bf16(bits).astype(np.float32) / np.float32(scale)   # IEEE float32 division
        return e4m3_encode(q.astype(np.float64))
    raise ValueError(fmt)


def kv_cache_append(k_new_bits, v_new_bits, k_pool, v_pool, block_tables, positions, kv_format="bf16",
                    k_scale=None, v_scale=None, block_size=16):
    """New (k_pool, v_pool) arrays with each sequence's token written in.

    k_new_bits, v_new_bits : uint16 [B, Hkv, D] bf16 codes of the new token
    k_pool                 : [num_blocks, Hkv, bs, D] codes (uint16 bf16 / uint8 e4m3)
    v_pool                 : [num_blocks, Hkv, D, bs] codes
    block_tables           : int [B, max_blocks_per_seq];  positions : int [B]
    """
    k_out, v_out = np.array(k_pool, copy=True), np.array(v_pool, copy=True)
    B, Hkv, _ = np.asarray(k_new_bits).shape
    max_blocks = np.asarray(block_tables).shape[1]
    num_blocks = k_out.shape[0]
    for s in range(B):
        t = int(positions[s])
        if t < 0 or t >= max_blocks * block_size:
            continue
        blk = int(block_tables[s][t // block_size])
        if blk < 0 or blk >= num_blocks:
            continue
        slot = t % block_size
        for g in range(Hkv):
            ks = None if k_scale is None else k_scale[g]
            vs = None if v_scale is None else v_scale[g]
            k_out[blk, g, slot, :] = encode(k_new_bits[s, g], kv_format, ks)
            v_out[blk, g, :, slot] = encode(v_new_bits[s, g], kv_format, vs)
    return k_out, v_out
