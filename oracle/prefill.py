"""Chunked-prefill attention over the paged KV cache, written out from its definition in float64.

Test infrastructure only (see the package header).

What is computed.  Each pool runs chunked prefill internally: a long prompt
is split into fixed-size chunks (2,048 tokens by default) that are
interleaved with decode steps (Sec. 1.2, "Chunked Prefill: Necessary but
Insufficient").  A chunk's attention is causal self-attention of its query
tokens over everything cached so far - earlier chunks and the chunk itself,
whose K and V are written into the block-paged cache before attention runs
(the same cache and 16-token blocks as decode, Sec. 3 effects 1 and 3).
The paper does not write the formula; the definition restated here is
textbook causal scaled-dot-product attention with grouped-query heads and
block-table indexing:

  for sequence s with T = context_lens[s] cached tokens (the chunk
  included) and n = q_start[s+1] - q_start[s] query tokens, query row
  r = q_start[s] + i (i = 0 .. n-1) sits at absolute position p_i = T - n + i;
  for query head h with KV head g = h // G:

    K_t, V_t as for decode (block-table gather, per-head fp8 scales)
    z_t   = scale * sum_k dec(q[r, h, k]) * K_t[k]            (t = 0 .. p_i)
    out[r, h, :] = sum_{t <= p_i} exp(z_t - mu) V_t / sum_{t <= p_i} exp(z_t - mu)

  Decode is the case n = 1.  A sequence with n > T is invalid input
  (ValueError here); n = 0 contributes no rows.

Parity: pinned by the decode oracle (n = 1 for every sequence gives the same
rows), by a library routine (torch's scaled_dot_product_attention in float64
with an explicit causal mask on the densely gathered tensors), by brute-force
scalar loops on tiny cases, by causality (tokens after p_i may hold NaN
without reaching row i), by chunk consistency (a prompt attended as one
chunk or as two gives the same rows) and by closed forms (the first token
of a fresh prompt returns V_0; constant V returns V).
"""
from __future__ import annotations

import numpy as np

from . import numerics
from .attention import _gather_rows


def chunked_prefill_attention(q_bits, k_pool, v_pool, block_tables, context_lens, q_start, scale,
                              kv_format="bf16", k_scale=None, v_scale=None, block_size=16, seqs=None, rows=None):
    """float64 [total_q, Hq, D] (rows not computed are left NaN).

    q_bits  : uint16 [total_q, Hq, D] bf16 codes, sequences packed by q_start
    q_start : int [B + 1], non-decreasing, q_start[0] = 0, q_start[B] = total_q
    seqs    : optional sequences to compute; rows: optional global row indices
              to compute (a sample; each row is computed exactly as in full)
    other arguments as for attention.paged_decode_attention
    """
    want = None if rows is None else set(int(r) for r in rows)
    q = numerics.decode_bf16(q_bits)
    total_q, Hq, D = q.shape
    q_start = np.asarray(q_start, dtype=np.int64)
    B = len(q_start) - 1
    first = k_pool[np.zeros(1, dtype=np.int64)]
    Hkv = first.shape[1]
    G = Hq // Hkv
    ks = np.ones(Hkv) if k_scale is None else np.asarray(k_scale, dtype=np.float64)
    vs = np.ones(Hkv) if v_scale is None else np.asarray(v_scale, dtype=np.float64)
    out = np.full((total_q, Hq, D), np.nan)
    for s in (range(B) if seqs is None else seqs):
        r0, r1 = int(q_start[s]), int(q_start[s + 1])
        n, T = r1 - r0, int(context_lens[s])
        if n == 0:
            continue
        if n > T:
            raise ValueError(f"sequence {s}: {n} query tokens but only {T} cached tokens")
        sel = np.arange(r0, r1) if want is None else np.array(sorted(r for r in want if r0 <= r < r1), np.int64)
        if len(sel) == 0:
            continue
        pos = T - n + (sel - r0)                         # absolute position of each query row
        future = np.arange(T)[None, :] > pos[:, None]    # [rows, T]: token after the query
        bt = np.asarray(block_tables[s])
        for g in range(Hkv):
            K = ks[g] * numerics.decode(_gather_rows(k_pool, bt, g, T, block_size, False), kv_format)
            V = vs[g] * numerics.decode(_gather_rows(v_pool, bt, g, T, block_size, True), kv_format)
            for h in range(g * G, (g + 1) * G):
                z = scale * (q[sel, h] @ K.T)             # [rows, T]
                z[future] = -np.inf
                w = np.exp(z - z.max(axis=1, keepdims=True))
                out[sel, h] = (w @ V) / w.sum(axis=1, keepdims=True)
    return out
