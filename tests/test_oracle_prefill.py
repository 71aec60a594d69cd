"""Pins of the oracle's chunked-prefill attention over the paged cache.

Checked against: the (separately pinned) decode oracle for one-token chunks,
a library routine (torch scaled_dot_product_attention in float64 with an
explicit causal mask on densely gathered tensors), brute-force scalar loops,
causality with poisoned future tokens, chunk consistency, and closed forms.
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import attention, numerics, prefill
from test_oracle_attention import SCALE, codes_bf16, dense_case, dense_gather

def prefill_case(rng, Hq, Hkv, ctx, qlen, kv="bf16"):
    """Dense pool (as for decode) plus packed queries: qlen[s] rows per sequence."""
    B = len(ctx)
    _, kb, vb, bt, ctx = dense_case(rng, B, Hq, Hkv, ctx)
    q_start = np.concatenate([[0], np.cumsum(qlen)]).astype(np.int32)
    qb = codes_bf16(rng.standard_normal((int(q_start[-1]), Hq, 128)).astype(np.float32))
    return qb, kb, vb, bt, ctx, q_start


def sdpa_causal(qb, kb, vb, bt, ctx, q_start, scale, fmt="bf16", ks=None, vs=None):
    Hq = qb.shape[1]
    Hkv = kb.shape[1]
    G = Hq // Hkv
    out = np.zeros(qb.shape)
    for s in range(len(ctx)):
        r0, r1 = int(q_start[s]), int(q_start[s + 1])
        n, T = r1 - r0, int(ctx[s])
        if n == 0:
            continue
        kmul = [1.0] * Hkv if ks is None else [float(x) for x in ks]
        vmul = [1.0] * Hkv if vs is None else [float(x) for x in vs]
        K = np.stack([kmul[g] * dense_gather(kb, bt, s, g, T, fmt) for g in range(Hkv)])
        V = np.stack([vmul[g] * dense_gather(vb, bt, s, g, T, fmt, dims_major=True) for g in range(Hkv)])
        Kt = torch.from_numpy(K).repeat_interleave(G, dim=0)[None]          # [1, Hq, T, D]
        Vt = torch.from_numpy(V).repeat_interleave(G, dim=0)[None]
        Qt = torch.from_numpy(numerics.decode_bf16(qb[r0:r1])).permute(1, 0, 2)[None]   # [1, Hq, n, D]
        allowed = torch.arange(T)[None, :] <= (T - n + torch.arange(n))[:, None]
        o = torch.nn.functional.scaled_dot_product_attention(Qt, Kt, Vt, attn_mask=allowed, scale=scale)
        out[r0:r1] = o[0].permute(1, 0, 2).numpy()
    return out


def brute(qb, kb, vb, bt, ctx, q_start, scale):
    Hq = qb.shape[1]
    Hkv = kb.shape[1]
    G = Hq // Hkv
    out = np.zeros(qb.shape)
    for s in range(len(ctx)):
        r0, r1, T = int(q_start[s]), int(q_start[s + 1]), int(ctx[s])
        for i in range(r1 - r0):
            p = T - (r1 - r0) + i
            for h in range(Hq):
                g = h // G
                z = []
                for t in range(p + 1):
                    blk, slot = int(bt[s][t // 16]), t % 16
                    acc = 0.0
                    for d in range(128):
                        acc += numerics.bf16_value(int(qb[r0 + i, h, d])) * numerics.bf16_value(int(kb[blk, g, slot, d]))
                    z.append(scale * acc)
                mu = max(z)
                w = [math.exp(x - mu) for x in z]
                for d in range(128):
                    num = 0.0
                    for t in range(p + 1):
                        num += w[t] * numerics.bf16_value(int(vb[int(bt[s][t // 16]), g, d, t % 16]))
                    out[r0 + i, h, d] = num / sum(w)
    return out


def run(qb, kb, vb, bt, ctx, q_start, **kw):
    return prefill.chunked_prefill_attention(qb, kb, vb, bt, ctx, q_start, SCALE, **kw)


def test_brute_force_tiny():
    rng = np.random.default_rng(1)
    case = prefill_case(rng, 4, 2, [19, 5, 3], [4, 5, 1])
    np.testing.assert_allclose(run(*case), brute(*case, SCALE), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("Hq,Hkv,ctx,qlen", [(8, 2, [300, 64, 1000, 17], [100, 64, 33, 17]),
                                             (16, 1, [250, 48], [250, 1]), (8, 8, [77], [40])])
def test_library_sdpa_causal(Hq, Hkv, ctx, qlen):
    rng = np.random.default_rng(2)
    case = prefill_case(rng, Hq, Hkv, ctx, qlen)
    np.testing.assert_allclose(run(*case), sdpa_causal(*case, SCALE), rtol=1e-10, atol=1e-12)


def test_library_sdpa_causal_gqa16_fp8():
    """An e4m3 cache with per-head K and V scales (Sec. 4.7's FP8 serving): the
    oracle against torch SDPA on the decoded, scaled tensors."""
    w = workloads.make_prefill([(40, 100), (17, 17), (5, 70)], 16, 1, c_max=128, kv_format="fp8_e4m3", seed=17)
    kb, vb = w.k_store.dense(), w.v_store.dense()
    got = prefill.chunked_prefill_attention(w.q_bits, kb, vb, w.block_tables, w.context_lens, w.meta["q_start"],
                                            SCALE, kv_format="fp8_e4m3", k_scale=w.k_scale, v_scale=w.v_scale)
    ref = sdpa_causal(w.q_bits, kb, vb, w.block_tables, w.context_lens, w.meta["q_start"], SCALE, fmt="fp8_e4m3",
                      ks=w.k_scale, vs=w.v_scale)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)


def test_one_token_chunks_are_decode():
    rng = np.random.default_rng(3)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 8, 2, [40, 129, 1, 500], [1, 1, 1, 1])
    dec = attention.paged_decode_attention(qb, kb, vb, bt, ctx, SCALE)
    np.testing.assert_allclose(run(qb, kb, vb, bt, ctx, q_start), dec, rtol=1e-12, atol=1e-13)


def test_future_tokens_never_reach_a_row():
    rng = np.random.default_rng(4)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 4, 2, [90], [30])
    clean = run(qb, kb, vb, bt, ctx, q_start)
    T = int(ctx[0])
    blk, slot = int(bt[0][(T - 1) // 16]), (T - 1) % 16
    kb2, vb2 = kb.copy(), vb.copy()
    kb2[blk, :, slot, :] = codes_bf16(np.zeros(128, np.float32))   # rewrite the chunk's last token
    vb2[blk, :, :, slot] = codes_bf16(np.full(128, 1000.0, np.float32))
    got = run(qb, kb2, vb2, bt, ctx, q_start)
    np.testing.assert_array_equal(got[:29], clean[:29])   # rows before it never see it (bit for bit)
    assert np.abs(got[29] - clean[29]).min() > 1.0        # the last row attends it


def test_one_chunk_equals_two_chunks():
    rng = np.random.default_rng(5)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 8, 2, [150], [150])   # whole prompt as one chunk
    whole = run(qb, kb, vb, bt, ctx, q_start)
    first = run(qb[:61], kb, vb, bt, np.array([61]), np.array([0, 61]))      # chunk 1: tokens 0..60
    second = run(qb[61:], kb, vb, bt, ctx, np.array([0, 89]))                # chunk 2 over the full cache
    np.testing.assert_allclose(np.concatenate([first, second]), whole, rtol=1e-12, atol=1e-13)


def test_fresh_prompt_first_row_returns_v0():
    rng = np.random.default_rng(6)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 4, 2, [33], [33])
    out = run(qb, kb, vb, bt, ctx, q_start)
    for h in range(4):
        np.testing.assert_array_equal(out[0, h], numerics.decode_bf16(vb[bt[0][0], h // 2, :, 0]))


def test_constant_v_returns_v():
    rng = np.random.default_rng(7)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 4, 1, [70, 20], [50, 20])
    vb[:] = codes_bf16(np.linspace(-2, 2, 128, dtype=np.float32))[None, None, :, None]
    out = run(qb, kb, vb, bt, ctx, q_start)
    np.testing.assert_allclose(out, np.broadcast_to(numerics.decode_bf16(vb[0, 0, :, 0]), out.shape), rtol=1e-14)


def test_more_queries_than_cached_tokens_is_rejected():
    rng = np.random.default_rng(8)
    qb, kb, vb, bt, ctx, q_start = prefill_case(rng, 4, 2, [10], [10])
    with pytest.raises(ValueError):
        run(qb, kb, vb, bt, np.array([9]), q_start)


def test_sampled_rows_equal_full_rows():
    rng = np.random.default_rng(9)
    case = prefill_case(rng, 8, 2, [200, 90], [120, 90])
    full = run(*case)
    rows = [0, 5, 119, 120, 150, 209]
    got = run(*case, rows=rows)
    np.testing.assert_allclose(got[rows], full[rows], rtol=1e-12, atol=1e-15)   # BLAS blocking may differ
    others = np.setdiff1d(np.arange(210), rows)
    assert np.isnan(got[others]).all()
