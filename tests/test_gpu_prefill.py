"""GPU parity of chunked_prefill_attention (through the C ABI) against the fp64 oracle.

Same bar as decode: max abs error 1.5e-2 with bf16 KV, 3e-2 with fp8 e4m3 KV
(bf16 output; the fp32 output to the same bar).  Small cases are compared
row by row in full; the benchmark workloads at full size on every row of their
first chunk and on sampled rows of the others, which the oracle computes one
by one.  Causality, untouched rows and determinism are
checked bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import workloads
from oracle import prefill

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1.5e-2, "fp8_e4m3": 3e-2}


def note(msg):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def oracle_rows(w, rows=None):
    return prefill.chunked_prefill_attention(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens,
                                             w.meta["q_start"], w.scale, kv_format=w.kv_format, k_scale=w.k_scale,
                                             v_scale=w.v_scale, rows=rows)


def gpu_rows(lib, w, dev=None, out_fp32=False, query_tile=0, out=None):
    d = dev if dev is not None else workloads.to_device(w)
    total_q = int(w.meta["q_start"][-1])
    shape = lib.prefill_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq,
                              max(w.max_context_len, 0), w.num_blocks, total_q,
                              kv_fp8=w.kv_format == "fp8_e4m3", out_fp32=out_fp32, query_tile=query_tile)
    if out is None:
        out = torch.full((total_q, w.n_q_heads, 128), float("nan"), device="cuda",
                         dtype=torch.float32 if out_fp32 else torch.bfloat16)
    lib.chunked_prefill_attention(d["q"], d["k"][0], d["v"][0], d["block_tables"], d["context_lens"], d["q_start"],
                                  w.scale, out, shape, d["k_scale"], d["v_scale"])
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


SMALL = [
    # (chunks [(n, T)], Hq, Hkv, kv)
    ([(100, 300), (64, 64), (33, 1000), (17, 17)], 8, 2, "bf16"),
    ([(1, 40), (1, 129), (1, 1), (1, 500)], 16, 2, "bf16"),          # one-token chunks: decode
    ([(130, 130), (77, 205), (5, 37)], 4, 4, "bf16"),                # G = 1
    ([(96, 300), (31, 31), (200, 700)], 32, 2, "fp8_e4m3"),          # G = 16
    ([(64, 96), (40, 40)], 12, 2, "bf16"),                           # G = 6: one quad partly idle
]


@pytest.mark.parametrize("case", range(len(SMALL)))
@pytest.mark.parametrize("query_tile", [0, 32])
def test_small_parity(gpu_lib, case, query_tile):
    chunks, hq, hkv, kv = SMALL[case]
    note(f"prefill small case {case} tile {query_tile}: {chunks} {hq}/{hkv} {kv}")
    w = workloads.make_prefill(chunks, hq, hkv, c_max=1024, kv_format=kv, seed=10 + case)
    ref = oracle_rows(w)
    dev = workloads.to_device(w)
    got = gpu_rows(gpu_lib, w, dev, query_tile=query_tile)
    err = float(np.abs(got - ref).max())
    note(f"  max abs err {err:.3e}")
    assert np.isfinite(got).all() and err <= TOL[kv]
    got32 = gpu_rows(gpu_lib, w, dev, out_fp32=True, query_tile=query_tile)
    assert float(np.abs(got32 - ref).max()) <= TOL[kv]


@pytest.mark.parametrize("name", sorted(workloads.PREFILL_CONFIGS))
def test_benchmark_workload(gpu_lib, name):
    """The benchmark workloads at full size: every row of the first chunk (2,048
    query tokens at context 2,048), and sampled rows of the deeper chunks, which
    the oracle computes one by one exactly as in full."""
    note(f"prefill {name}: building")
    w = workloads.make_prefill_config(name)
    qs = w.meta["q_start"]
    rng = np.random.default_rng(99)
    rows = set(range(int(qs[0]), int(qs[1])))
    for s in range(1, w.batch):
        r0, r1 = int(qs[s]), int(qs[s + 1])
        rows.update({r0, r0 + 1, r0 + 63, r0 + 64, r1 - 1})
        rows.update(int(x) for x in rng.integers(r0, r1, 6))
    rows = sorted(rows)
    dev = workloads.to_device(w)
    got = gpu_rows(gpu_lib, w, dev)
    del dev
    torch.cuda.empty_cache()
    note(f"prefill {name}: oracle on {len(rows)} rows")
    ref = oracle_rows(w, rows)
    err = float(np.abs(got[rows] - ref[rows]).max())
    note(f"prefill {name}: max abs err {err:.3e}")
    assert np.isfinite(got).all() and err <= TOL[w.kv_format]


def test_rows_of_other_sequences_and_empty_chunks_untouched(gpu_lib):
    w = workloads.make_prefill([(40, 90), (0, 50), (25, 25)], 8, 2, c_max=256, seed=21)
    dev = workloads.to_device(w)
    total_q = int(w.meta["q_start"][-1])
    out = torch.full((total_q + 8, 8, 128), 7.0, device="cuda", dtype=torch.bfloat16)   # 8 rows past the end
    got = gpu_rows(gpu_lib, w, dev, out=out)
    assert (got[total_q:] == 7.0).all()
    ref = oracle_rows(w)
    assert float(np.abs(got[:total_q] - ref).max()) <= TOL["bf16"]


def test_future_tokens_never_reach_earlier_rows(gpu_lib):
    w = workloads.make_prefill([(150, 400)], 8, 2, c_max=512, seed=22)
    dev = workloads.to_device(w)
    base = gpu_rows(gpu_lib, w, dev)
    T = int(w.context_lens[0])
    blk, slot = int(w.block_tables[0][(T - 1) // 16]), (T - 1) % 16
    dev["k"][0, blk, :, slot, :] = 0
    dev["v"][0, blk, :, :, slot] = int(np.uint16(0x447A).view(np.int16))   # 1000.0 in bf16
    got = gpu_rows(gpu_lib, w, dev)
    np.testing.assert_array_equal(got[:149], base[:149])
    assert np.abs(got[149] - base[149]).max() > 1.0


def test_random_chunks_every_row(gpu_lib):
    """Forty seeded random prefill shapes (cache format, GQA group 1-16 including
    groups that leave a head quad partly idle, 1-4 KV heads, 1-5 chunks of
    1-1,500 context tokens each, fresh prompts and chunks over a cached
    prefix, both query tiles, bf16 and fp32 output), every row against the
    oracle; a second call must equal the first bit for bit."""
    rng = np.random.default_rng(2605)
    for case in range(40):
        kv = ["bf16", "fp8_e4m3"][int(rng.integers(0, 2))]
        G = int(rng.choice([1, 2, 4, 6, 8, 12, 16]))
        Hkv = int(rng.choice([1, 2, 4]))
        chunks = []
        for _ in range(int(rng.integers(1, 6))):
            T = int(rng.integers(1, 1500))
            chunks.append((int(rng.integers(1, T + 1)) if rng.random() < 0.7 else T, T))
        qt = int(rng.choice([0, 32]))
        seed = int(rng.integers(0, 1 << 30))
        note(f"case {case}: kv={kv} G={G} Hkv={Hkv} chunks={chunks} tile={qt} seed={seed}")
        w = workloads.make_prefill(chunks, G * Hkv, Hkv, c_max=1536, kv_format=kv, seed=seed)
        dev = workloads.to_device(w)
        got = gpu_rows(gpu_lib, w, dev, query_tile=qt, out_fp32=bool(case % 2))
        assert np.array_equal(gpu_rows(gpu_lib, w, dev, query_tile=qt, out_fp32=bool(case % 2)), got)
        err = float(np.abs(got - oracle_rows(w)).max())
        assert np.isfinite(got).all() and err <= TOL[kv], f"case {case}: max abs err {err:.3e}"


def test_deterministic(gpu_lib):
    w = workloads.make_prefill_config("chunked_prefill_llama70b")
    dev = workloads.to_device(w)
    a = gpu_rows(gpu_lib, w, dev)
    b = gpu_rows(gpu_lib, w, dev)
    np.testing.assert_array_equal(a, b)


def test_longest_context(gpu_lib):
    """A chunk at the end of a 65,536-token context (the longest the kernel stages
    block ids for), with a ragged last query tile; sampled rows against the oracle."""
    note("prefill at context 65536")
    w = workloads.make_prefill([(77, 65536), (40, 1000)], 16, 2, c_max=65536, seed=23)
    qs = w.meta["q_start"]
    rows = sorted({0, 1, 31, 32, 63, 64, 76, int(qs[1]), int(qs[2]) - 1})
    got = gpu_rows(gpu_lib, w)
    ref = oracle_rows(w, rows)
    err = float(np.abs(got[rows] - ref[rows]).max())
    note(f"  max abs err {err:.3e}")
    assert np.isfinite(got).all() and err <= TOL["bf16"]


@pytest.mark.parametrize("chunks,hq,hkv", [
    ([(2048, 2048), (2200, 4096)], 8, 2),     # 266 items: a partial second (backward) round
    ([(3000, 3000), (1500, 2000)], 8, 4),     # 564 items: a partial third (forward) round
])
def test_item_rounds_with_a_partial_last_round(gpu_lib, chunks, hq, hkv):
    """More (query tile, head group) items than workgroups, not a multiple of them:
    every row is written (the output starts as NaN) and sampled rows match the oracle."""
    note(f"prefill rounds {chunks} {hq}/{hkv}")
    w = workloads.make_prefill(chunks, hq, hkv, c_max=4096, seed=29)
    total_q = int(w.meta["q_start"][-1])
    rows = sorted(set(range(0, total_q, 97)) | {total_q - 1, int(w.meta["q_start"][1]) - 1, int(w.meta["q_start"][1])})
    got = gpu_rows(gpu_lib, w)
    ref = oracle_rows(w, rows)
    err = float(np.abs(got[rows] - ref[rows]).max())
    note(f"  max abs err {err:.3e}")
    assert np.isfinite(got).all() and err <= TOL["bf16"]
