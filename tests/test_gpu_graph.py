"""The hot path under HIP graph capture.

A serving loop replays its per-step launches from a captured graph.  Decode,
KV append and chunked prefill allocate nothing, record no memset and leave
the decode workspace reusable, so each can be captured once and replayed:
every replay, with eager work and synchronisations in between, must give
exactly the eager call's result.
"""
import sys

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


def note(msg):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def capture(fn):
    """Warm fn up on a side stream (default priority), then capture it."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_decode_replays_match_eager(gpu_lib, kv):
    note(f"decode graph, {kv}")
    w = workloads.make_workload(6, 32, 4, [1, 77, 300, 1500, 4096, 0], c_max=4096, kv_format=kv, seed=51)
    d = workloads.to_device(w)
    dec = gpu_lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                               w.num_blocks, kv_fp8=kv == "fp8_e4m3")
    args = (d["q"], d["k"][0], d["v"][0], d["block_tables"], d["context_lens"], w.scale)
    eager = dec.new_out()
    dec(*args, eager, d["k_scale"], d["v_scale"])
    torch.cuda.synchronize()
    out = dec.new_out()
    g = capture(lambda: dec(*args, out, d["k_scale"], d["v_scale"]))
    other = dec.new_out()
    for i in range(5):
        out.fill_(float("nan"))
        dec(*args, other, d["k_scale"], d["v_scale"])   # an eager call on the same workspace between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i}"
        assert torch.equal(other, eager)


def test_prefill_replays_match_eager(gpu_lib):
    note("prefill graph")
    w = workloads.make_prefill([(100, 300), (33, 1000), (64, 64)], 16, 2, c_max=1024, seed=52)
    d = workloads.to_device(w)
    total_q = int(w.meta["q_start"][-1])
    shape = gpu_lib.prefill_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                                  w.num_blocks, total_q)

    def run(out):
        gpu_lib.chunked_prefill_attention(d["q"], d["k"][0], d["v"][0], d["block_tables"], d["context_lens"],
                                          d["q_start"], w.scale, out, shape)

    eager = torch.empty((total_q, w.n_q_heads, 128), dtype=torch.bfloat16, device="cuda")
    run(eager)
    torch.cuda.synchronize()
    out = torch.empty_like(eager)
    g = capture(lambda: run(out))
    for i in range(5):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i}"


def test_append_replays_match_eager(gpu_lib):
    note("append graph")
    B, Hkv, nb = 8, 2, 64
    rng = np.random.default_rng(53)
    bt = torch.from_numpy(rng.permutation(nb).astype(np.int32).reshape(B, nb // B)).cuda()
    pos = torch.from_numpy(rng.integers(0, 16 * (nb // B), B).astype(np.int32)).cuda()
    k_new = torch.randn(B, Hkv, 128, device="cuda").to(torch.bfloat16)
    v_new = torch.randn(B, Hkv, 128, device="cuda").to(torch.bfloat16)
    shape = gpu_lib.decode_shape(B, 2 * Hkv, Hkv, nb // B, 16 * (nb // B), nb)
    pools = [torch.zeros((nb, Hkv, 16, 128), dtype=torch.int16, device="cuda") for _ in range(2)]
    gpu_lib.kv_cache_append(k_new, v_new, pools[0], pools[1], bt, pos, shape)
    torch.cuda.synchronize()
    eager = [p.clone() for p in pools]
    for p in pools:
        p.zero_()
    g = capture(lambda: gpu_lib.kv_cache_append(k_new, v_new, pools[0], pools[1], bt, pos, shape))
    for i in range(5):
        for p in pools:
            p.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(pools[0], eager[0]) and torch.equal(pools[1], eager[1]), f"replay {i}"
