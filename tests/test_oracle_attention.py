"""Pins of the oracle's paged decode attention.

Checked against: closed forms of softmax attention, a library routine
(torch scaled_dot_product_attention in float64 on the densely gathered
tensors), brute-force scalar loops on tiny cases, the split-K / log-sum-exp
merge identity, and paging invariances (block permutation, poisoned slots).
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import attention, numerics


def codes_bf16(x):
    return workloads.to_bf16_codes(np.asarray(x, dtype=np.float32))


def dense_case(rng, B, Hq, Hkv, ctx, nb_pool=None, vals=None, kv="bf16"):
    """Small dense pool with a shuffled block table; values N(0,1) unless given.

    K and V are drawn token-major [nb, Hkv, 16, 128]; V is returned in the
    interface's dims-major tile layout [nb, Hkv, 128, 16]."""
    nblk = [-(-c // 16) for c in ctx]
    used = sum(nblk)
    nb_pool = nb_pool or max(used * 2, 1)
    perm = rng.permutation(nb_pool)
    bt = np.full((B, max(max(nblk), 1)), -1, np.int32)
    off = 0
    for s in range(B):
        bt[s, :nblk[s]] = perm[off:off + nblk[s]]
        off += nblk[s]
    q = rng.standard_normal((B, Hq, 128)).astype(np.float32)
    k = rng.standard_normal((nb_pool, Hkv, 16, 128)).astype(np.float32)
    v = rng.standard_normal((nb_pool, Hkv, 16, 128)).astype(np.float32)
    if vals:
        q, k, v = vals(q, k, v, bt)
    vt = np.ascontiguousarray(codes_bf16(v).transpose(0, 1, 3, 2))
    return codes_bf16(q), codes_bf16(k), vt, bt, np.asarray(ctx, np.int32)


def dense_gather(pool_codes, bt, s, g, T, fmt="bf16", dims_major=False):
    """Token rows 0..T-1 of (sequence s, KV head g), one element lookup per row."""
    rows = []
    for t in range(T):
        tile = pool_codes[bt[s, t // 16], g]
        rows.append(numerics.decode(tile[:, t % 16] if dims_major else tile[t % 16], fmt))
    return np.array(rows).reshape(T, -1)


def sdpa_reference(qb, kb, vb, bt, ctx, scale, fmt="bf16", ks=None, vs=None):
    """torch SDPA in float64 over explicitly gathered K/V (GQA by head repeat)."""
    B, Hq, D = qb.shape
    Hkv = kb.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, D))
    for s in range(B):
        T = int(ctx[s])
        if T == 0:
            continue
        K = np.stack([dense_gather(kb, bt, s, g, T, fmt) * (1 if ks is None else ks[g]) for g in range(Hkv)])
        V = np.stack([dense_gather(vb, bt, s, g, T, fmt, dims_major=True) * (1 if vs is None else vs[g])
                      for g in range(Hkv)])
        Kt = torch.from_numpy(K).repeat_interleave(G, dim=0)[None]   # [1, Hq, T, D]
        Vt = torch.from_numpy(V).repeat_interleave(G, dim=0)[None]
        Qt = torch.from_numpy(numerics.decode_bf16(qb[s]))[None, :, None, :]  # [1, Hq, 1, D]
        o = torch.nn.functional.scaled_dot_product_attention(Qt, Kt, Vt, scale=scale)
        out[s] = o[0, :, 0, :].numpy()
    return out


def brute_force(qb, kb, vb, bt, ctx, scale):
    """Scalar loops, math.exp, per-element decode: no numpy arithmetic at all."""
    B, Hq, D = qb.shape
    Hkv = kb.shape[1]
    G = Hq // Hkv
    out = [[[0.0] * D for _ in range(Hq)] for _ in range(B)]
    for s in range(B):
        T = int(ctx[s])
        for h in range(Hq):
            g = h // G
            z = []
            for t in range(T):
                blk, slot = int(bt[s][t // 16]), t % 16
                acc = 0.0
                for i in range(D):
                    acc += numerics.bf16_value(int(qb[s, h, i])) * numerics.bf16_value(int(kb[blk, g, slot, i]))
                z.append(scale * acc)
            if T == 0:
                continue
            mu = max(z)
            w = [math.exp(x - mu) for x in z]
            den = sum(w)
            for i in range(D):
                num = 0.0
                for t in range(T):
                    blk, slot = int(bt[s][t // 16]), t % 16
                    num += w[t] * numerics.bf16_value(int(vb[blk, g, i, slot]))
                out[s][h][i] = num / den
    return np.array(out)


SCALE = 1.0 / math.sqrt(128)


def run_oracle(qb, kb, vb, bt, ctx, scale=SCALE, **kw):
    return attention.paged_decode_attention(qb, kb, vb, bt, ctx, scale, **kw)


def test_brute_force_tiny_cases():
    rng = np.random.default_rng(11)
    for ctx in ([1, 17, 33], [16, 40], [15, 32, 2]):
        B = len(ctx)
        qb, kb, vb, bt, cl = dense_case(rng, B, 4, 2, ctx)
        got = run_oracle(qb, kb, vb, bt, cl)
        ref = brute_force(qb, kb, vb, bt, cl, SCALE)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_library_sdpa_random():
    rng = np.random.default_rng(12)
    ctx = [1, 16, 17, 100, 255, 300]
    qb, kb, vb, bt, cl = dense_case(rng, len(ctx), 8, 2, ctx)
    got = run_oracle(qb, kb, vb, bt, cl)
    ref = sdpa_reference(qb, kb, vb, bt, cl, SCALE)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_library_sdpa_gqa16_fp8():
    rng = np.random.default_rng(13)
    ctx = [5, 48, 129]
    B, Hq, Hkv = len(ctx), 16, 1
    w = workloads.make_workload(B, Hq, Hkv, ctx, c_max=256, kv_format="fp8_e4m3", seed=5)
    kb, vb = w.k_store.dense(), w.v_store.dense()
    got = run_oracle(w.q_bits, kb, vb, w.block_tables, w.context_lens, kv_format="fp8_e4m3",
                     k_scale=w.k_scale, v_scale=w.v_scale)
    ref = sdpa_reference(w.q_bits, kb, vb, w.block_tables, w.context_lens, SCALE, fmt="fp8_e4m3",
                         ks=w.k_scale, vs=w.v_scale)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_one_token_returns_v0():
    rng = np.random.default_rng(1)
    qb, kb, vb, bt, cl = dense_case(rng, 3, 8, 2, [1, 1, 1])
    got = run_oracle(qb, kb, vb, bt, cl)
    for s in range(3):
        for h in range(8):
            assert np.array_equal(got[s, h], numerics.decode_bf16(vb[bt[s, 0], h // 4, :, 0]))


def test_constant_v_returns_v():
    rng = np.random.default_rng(2)

    def vals(q, k, v, bt):
        v[:] = rng.standard_normal((1, v.shape[1], 1, 128)).astype(np.float32)
        return q, k, v
    qb, kb, vb, bt, cl = dense_case(rng, 2, 4, 2, [37, 64], vals=vals)
    got = run_oracle(qb, kb, vb, bt, cl)
    for h in range(4):
        np.testing.assert_allclose(got[:, h], np.broadcast_to(numerics.decode_bf16(vb[0, h // 2, :, 0]), (2, 128)),
                                   rtol=0, atol=1e-14)


def test_identical_k_rows_give_mean_of_v():
    rng = np.random.default_rng(3)

    def vals(q, k, v, bt):
        k[:] = rng.standard_normal((1, k.shape[1], 1, 128)).astype(np.float32)
        return q, k, v
    ctx = [23, 50]
    qb, kb, vb, bt, cl = dense_case(rng, 2, 4, 2, ctx, vals=vals)
    got = run_oracle(qb, kb, vb, bt, cl)
    for s, T in enumerate(ctx):
        for h in range(4):
            mean = dense_gather(vb, bt, s, h // 2, T, dims_major=True).mean(axis=0)
            np.testing.assert_allclose(got[s, h], mean, rtol=0, atol=1e-13)


def test_zero_scale_gives_mean_of_v():
    rng = np.random.default_rng(4)
    ctx = [9, 77]
    qb, kb, vb, bt, cl = dense_case(rng, 2, 4, 1, ctx)
    got = run_oracle(qb, kb, vb, bt, cl, scale=0.0)
    for s, T in enumerate(ctx):
        mean = dense_gather(vb, bt, s, 0, T, dims_major=True).mean(axis=0)
        for h in range(4):
            np.testing.assert_allclose(got[s, h], mean, rtol=0, atol=1e-13)


def test_shifting_every_key_by_one_vector_changes_nothing():
    rng = np.random.default_rng(5)

    def ints(q, k, v, bt):
        return (np.rint(q * 2).astype(np.float32), np.rint(k * 2).astype(np.float32), v)
    qb, kb, vb, bt, cl = dense_case(rng, 2, 4, 2, [30, 70], vals=ints)
    base = run_oracle(qb, kb, vb, bt, cl)
    u = np.rint(rng.standard_normal((1, 2, 1, 128)) * 3).astype(np.float32)
    kb2 = codes_bf16(numerics.decode_bf16(kb).astype(np.float32) + u)   # small integers: exact in bf16
    assert np.array_equal(numerics.decode_bf16(kb2), numerics.decode_bf16(kb) + u)
    shifted = run_oracle(qb, kb2, vb, bt, cl)
    np.testing.assert_allclose(shifted, base, rtol=0, atol=1e-12)


def test_block_permutation_with_table_fixup_is_exact():
    rng = np.random.default_rng(6)
    qb, kb, vb, bt, cl = dense_case(rng, 3, 8, 2, [20, 64, 90])
    base = run_oracle(qb, kb, vb, bt, cl)
    pi = rng.permutation(kb.shape[0])
    kb2 = np.empty_like(kb)
    vb2 = np.empty_like(vb)
    kb2[pi] = kb
    vb2[pi] = vb
    bt2 = np.where(bt >= 0, pi[np.maximum(bt, 0)], -1).astype(np.int32)
    assert np.array_equal(run_oracle(qb, kb2, vb2, bt2, cl), base)


def test_poisoned_tail_and_unused_blocks_are_never_read():
    w = workloads.make_workload(3, 8, 2, [5, 16, 33], c_max=64, seed=9, poison=True)
    out = run_oracle(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens)
    assert np.isfinite(out).all()


def test_empty_context_gives_zero_row():
    rng = np.random.default_rng(8)
    qb, kb, vb, bt, cl = dense_case(rng, 2, 4, 2, [0, 5])
    out = run_oracle(qb, kb, vb, bt, cl)
    assert np.array_equal(out[0], np.zeros((4, 128)))
    assert np.isfinite(out[1]).all()


@pytest.mark.parametrize("P", [1, 16, 17, 64, 500])
def test_split_k_lse_merge_equals_unsplit(P):
    rng = np.random.default_rng(100 + P)
    T = 333
    q = rng.standard_normal(128)
    K = rng.standard_normal((T, 128)) * 2
    V = rng.standard_normal((T, 128))
    z = (K @ q) / math.sqrt(128)
    w = np.exp(z - z.max())
    direct = w @ V / w.sum()
    o, m, l = attention.partition_partials(q, K, V, 1 / math.sqrt(128), P)
    assert len(m) == -(-T // P)
    np.testing.assert_allclose(attention.lse_merge(o, m, l), direct, rtol=0, atol=1e-12)


def test_sampled_sequences_only():
    w = workloads.make_workload(4, 8, 2, [10, 20, 30, 40], c_max=64, seed=3)
    full = run_oracle(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens)
    part = run_oracle(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens, seqs=[1, 3])
    assert np.array_equal(part[[1, 3]], full[[1, 3]])
    assert np.isnan(part[[0, 2]]).all()
