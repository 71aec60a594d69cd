"""Paged decode attention, written out from its definition in float64.

Test infrastructure only (see the package header).

What is computed.  The paper's cost model names the per-step decode KV read
as the memory-bandwidth-bound part of serving (Sec. 3, effect 4 "KV-read
bandwidth"; Sec. 4.4 "Why TPOT also improves": one KV-cache lookup per layer
per generated token).  The KV cache is PagedAttention's: fixed 16-token
blocks (Sec. 3, effect 3), pages allocated on demand (Sec. 3, effect 1).  The
paper does not write the attention formula; it relies on PagedAttention
(Sec. 5, "LLM serving engines").  The definition restated here is the
textbook scaled-dot-product attention of one new query token per sequence,
with grouped-query heads and block-table indexing:

  for sequence s with T = context_lens[s] cached tokens (the token being
  decoded included) and query head h, whose KV head is g = h // G
  (G = n_q_heads / n_kv_heads, consecutive query heads share a KV head):

    blk_t = block_tables[s, t // bs],  slot_t = t % bs       (t = 0 .. T-1)
    K_t   = k_scale[g] * dec(k_blocks[blk_t, g, slot_t, :])
    V_t   = v_scale[g] * dec(v_blocks[blk_t, g, :, slot_t])
    z_t   = scale * sum_i dec(q[s, h, i]) * K_t[i]
    out[s, h, :] = sum_t exp(z_t - mu) V_t / sum_t exp(z_t - mu),  mu = max_t z_t

  dec() is the exact decode of the storage format (``numerics``); for bf16
  storage k_scale = v_scale = 1.  The tile layouts are the interface's (the
  paper fixes none): a K tile is token-major [bs, D], a V tile dims-major
  [D, bs].  Subtracting mu changes nothing
  mathematically; it only keeps exp() finite.  T = 0 gives a zero row
  (a reading: the paper never decodes an empty sequence).

Split-K.  ``partition_partials`` and ``lse_merge`` restate the split of one
sequence's tokens into partitions whose softmax partials are merged with
log-sum-exp weights - the decomposition the GPU path uses for long contexts.
They are pinned (tests/) to give the unsplit result to 1e-12.

Parity: pinned by closed forms (one-token context returns V; constant V
returns V; identical K rows give the mean of V; scale 0 gives the mean of V;
adding one vector to every K row changes nothing), by a library routine
(torch.nn.functional.scaled_dot_product_attention in float64 on the densely
gathered tensors) and by brute-force scalar loops on tiny cases.
"""
from __future__ import annotations

import numpy as np

from . import numerics


def _gather_rows(pool, block_ids: np.ndarray, g: int, T: int, bs: int, dims_major: bool) -> np.ndarray:
    """Raw storage codes of tokens 0..T-1 of one sequence for KV head g: [T, D]."""
    n_blocks = -(-T // bs)
    tiles = pool[block_ids[:n_blocks]][:, g]       # [n_blocks, bs, D] or [n_blocks, D, bs]
    if dims_major:
        tiles = tiles.transpose(0, 2, 1)
    rows = tiles.reshape(n_blocks * bs, -1)        # token-major
    return rows[:T]


def paged_decode_attention(q_bits, k_pool, v_pool, block_tables, context_lens, scale,
                           kv_format="bf16", k_scale=None, v_scale=None,
                           block_size=16, seqs=None):
    """float64 [B, Hq, D] attention output (rows not in ``seqs`` are left NaN).

    q_bits       : uint16 [B, Hq, D] bf16 codes of the new query token
    k_pool       : indexable by an int array of block ids -> [n, Hkv, bs, D]
    v_pool       : likewise -> [n, Hkv, D, bs]
                   (storage codes: uint16 bf16 or uint8 e4m3)
    block_tables : int [B, max_blocks_per_seq]
    context_lens : int [B]
    k_scale/v_scale: float [Hkv] per-KV-head dequantization scales (fp8 only)
    seqs         : optional iterable of sequence indices to compute
    """
    q = numerics.decode_bf16(q_bits)
    B, Hq, D = q.shape
    first = k_pool[np.zeros(1, dtype=np.int64)]
    Hkv = first.shape[1]
    G = Hq // Hkv
    ks = np.ones(Hkv) if k_scale is None else np.asarray(k_scale, dtype=np.float64)
    vs = np.ones(Hkv) if v_scale is None else np.asarray(v_scale, dtype=np.float64)
    out = np.full((B, Hq, D), np.nan)
    for s in (range(B) if seqs is None else seqs):
        T = int(context_lens[s])
        if T == 0:
            out[s] = 0.0
            continue
        bt = np.asarray(block_tables[s])
        for g in range(Hkv):
            K = ks[g] * numerics.decode(_gather_rows(k_pool, bt, g, T, block_size, False), kv_format)
            V = vs[g] * numerics.decode(_gather_rows(v_pool, bt, g, T, block_size, True), kv_format)
            for h in range(g * G, (g + 1) * G):
                z = scale * (K @ q[s, h])
                w = np.exp(z - z.max())
                out[s, h] = (w @ V) / w.sum()
    return out


def partition_partials(q_vec, K, V, scale, part_tokens):
    """Softmax partials of one (sequence, query head) over token partitions.

    q_vec [D], K/V [T, D] already decoded (float64).  Partition p covers
    tokens [p*part_tokens, (p+1)*part_tokens).  Returns (o [P, D], m [P], l [P])
    with m_p the partition's max score, l_p = sum exp(z - m_p) and
    o_p = sum exp(z - m_p) V / l_p.
    """
    T = K.shape[0]
    z = scale * (K @ q_vec)
    os_, ms, ls = [], [], []
    for start in range(0, T, part_tokens):
        zp = z[start:start + part_tokens]
        m = zp.max()
        w = np.exp(zp - m)
        ls.append(w.sum())
        ms.append(m)
        os_.append((w @ V[start:start + part_tokens]) / w.sum())
    return np.array(os_), np.array(ms), np.array(ls)


def lse_merge(o, m, l):
    """Merge softmax partials: M = max m_p, w_p = l_p exp(m_p - M), out = sum w_p o_p / sum w_p."""
    M = m.max()
    w = l * np.exp(m - M)
    return (w[:, None] * o).sum(axis=0) / w.sum()
