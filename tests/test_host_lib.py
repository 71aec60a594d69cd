"""Host-side checks of libdpool: exports, router bit-exactness, pool sizing and allocator, shape validation.

No GPU is touched: the decode entry points are only called with arguments
that the host-side validation rejects before any HIP call.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import pool as opool
from oracle import route as oroute

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    txt = open(os.path.join(ROOT, "include", "dpool.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w]*\s*\**\s+\**\s*([A-Za-z_]\w*)\s*\(", txt, flags=re.M)
    return sorted(set(names))


def test_library_loads_and_exports_every_header_symbol(host_lib):
    names = header_functions()
    assert len(names) >= 14
    assert sorted(host_lib.EXPORTS) == names
    lib = host_lib.lib()
    for n in names:
        assert getattr(lib, n) is not None
    assert "gfx950" in host_lib.version()


# ---------------------------------------------------------------- router

def c_state(host_lib, p_py, n_cats):
    p = host_lib.RouteParams(p_py.b_short, p_py.beta, p_py.gamma, p_py.c0, p_py.c_min, p_py.spill_theta)
    return p, host_lib.make_categories(p, n_cats)


@pytest.mark.parametrize("nbytes,max_out,want_l,want_pool", [
    (32000, 0, 8000, 0), (32772, 0, 8193, 1), (4001, 7191, 8192, 0), (4001, 7192, 8193, 1)])
def test_route_cold_start_vectors(host_lib, nbytes, max_out, want_l, want_pool):
    p = host_lib.default_route_params()
    cats = host_lib.make_categories(p, 1)
    pools = host_lib.make_pools(8192, 128, 65536, 16)
    got_p, got_l = host_lib.route_requests(p, cats, pools, [nbytes], [0], [max_out])
    assert (int(got_p[0]), int(got_l[0])) == (want_pool, want_l)
    assert pools[want_pool].in_flight == 1



def test_route_bit_exact_against_oracle_1e6_requests(host_lib):
    rng = np.random.default_rng(2024)
    n_cats = 3
    py_p = oroute.RouteParams(spill_theta=0.9)
    p, cats = c_state(host_lib, py_p, n_cats)
    py_cats = oroute.init_categories(py_p, n_cats)
    pools = host_lib.make_pools(8192, 64, 65536, 8)
    py_pools = [oroute.PoolState(8192, 64), oroute.PoolState(65536, 8)]
    true_ratio = np.array([3.5, 2.0, 4.5])   # code / CJK / prose (Sec. 2.1 "Why per-category")
    total = 0
    while total < 1_000_000:
        n = 1000
        k = rng.integers(0, n_cats, n).astype(np.int32)
        toks = np.rint(rng.lognormal(np.log(600), 1.3, n)).astype(np.int64) + 1
        b = np.rint(toks * true_ratio[k] * rng.uniform(0.8, 1.2, n)).astype(np.int64)
        mo = rng.integers(0, 9000, n).astype(np.int64)
        cp, cl = host_lib.route_requests(p, cats, pools, b, k, mo)
        pp, pl = oroute.route_requests(py_p, py_cats, py_pools, b, k, mo)
        assert np.array_equal(cp.astype(np.int64), np.array(pp)), f"pool decisions differ after {total}"
        assert np.array_equal(cl, np.array(pl, dtype=np.int64))
        for i in range(0, n, 3):
            host_lib.route_on_response(p, cats, int(k[i]), int(b[i]), int(toks[i]))
            oroute.on_response(py_p, py_cats, int(k[i]), int(b[i]), int(toks[i]))
        for c in range(n_cats):   # bit-for-bit equal doubles
            assert cats[c].c_hat == py_cats[c].c_hat and cats[c].sigma == py_cats[c].sigma
        for j in range(2):
            assert pools[j].in_flight == py_pools[j].in_flight
            drop = int(rng.integers(0, pools[j].in_flight + 1))
            pools[j].in_flight -= drop
            py_pools[j].in_flight -= drop
        total += n


def test_route_closed_form_after_observations(host_lib):
    p = host_lib.default_route_params()
    cats = host_lib.make_categories(p, 1)
    for n in range(1, 101):
        host_lib.route_on_response(p, cats, 0, 2500, 1000)
        assert abs(cats[0].c_hat - (2.5 + 0.95 ** n * 1.5)) < 1e-13
        assert abs(cats[0].sigma - n * 0.05 * 0.95 ** n * 1.5) < 1e-13


def test_route_errors_leave_state_unchanged(host_lib):
    p = host_lib.default_route_params()
    cats = host_lib.make_categories(p, 2)
    pools = host_lib.make_pools(8192, 128, 65536, 16)
    with pytest.raises(host_lib.DpoolError) as e:
        host_lib.route_requests(p, cats, pools, [100, 200], [0, 2], [1, 1])
    assert e.value.code == host_lib.DP_EINVAL
    assert pools[0].in_flight == 0 and pools[1].in_flight == 0
    with pytest.raises(host_lib.DpoolError):
        host_lib.route_requests(p, cats, pools, [-1], [0], [1])
    with pytest.raises(host_lib.DpoolError):
        host_lib.route_on_response(p, cats, 0, 100, 0)
    assert (cats[0].c_hat, cats[0].sigma) == (4.0, 0.0)
    with pytest.raises(host_lib.DpoolError):
        host_lib.route_on_response(p, cats, 5, 100, 10)


def test_route_forced_spill_and_safety(host_lib):
    p = host_lib.default_route_params()
    cats = host_lib.make_categories(p, 1)
    pools = host_lib.make_pools(8192, 128, 65536, 16)
    pools[0].in_flight = 128
    got, _ = host_lib.route_requests(p, cats, pools, [400], [0], [10])
    assert got[0] == 1
    pools[1].in_flight = 16   # both overloaded: stay in the preferred pool
    got, _ = host_lib.route_requests(p, cats, pools, [400], [0], [10])
    assert got[0] == 0
    got, l = host_lib.route_requests(p, cats, pools, [40000], [0], [30000])
    assert got[0] == 1 and l[0] == 40000   # over C_max(short): always long


# ---------------------------------------------------------------- pool

def test_pool_sizing_matches_oracle_and_paper(host_lib):
    cases = [
        (94, 1, 128, 1, 8192, 192e9, 0.9, 39.4e9),    # Sec. 4.7: 676 sequences
        (94, 1, 128, 1, 32768, 192e9, 0.9, 39.4e9),   # 169
        (80, 8, 128, 2, 8192, 288e9, 0.9, 0.0),       # config 2 pool: 49,152 blocks
        (80, 8, 128, 2, 65536, 288e9, 0.9, 0.0),      # configs 3/4
        (94, 4, 128, 1, 8192, 288e9, 0.9, 0.0),       # config 5: 167,936 blocks
        (80, 8, 128, 2, 8192, 10e9, 0.9, 20e9),       # no room: 0
    ]
    for nl, nh, dh, b, cmax, mg, u, mm in cases:
        pool = host_lib.KVPool(nl, nh, dh, b, cmax, mg, u, mm, seed=1)
        inf = pool.info()
        want = opool.size_pool(nl, nh, dh, b, 16, cmax, mg, u, mm)
        assert (inf.m_seq_bytes, inf.n_seq, inf.blocks_per_seq, inf.num_blocks) == want
        assert inf.free_blocks == inf.num_blocks
    assert host_lib.KVPool(94, 1, 128, 1, 8192, 192e9, 0.9, 39.4e9).info().n_seq == 676
    assert host_lib.KVPool(94, 1, 128, 1, 32768, 192e9, 0.9, 39.4e9).info().n_seq == 169


def test_pool_allocator_invariants(host_lib):
    pool = host_lib.KVPool(1, 1, 128, 2, 1024, 1024 * 512 * 40, 1.0, 0.0, seed=3)   # 40 seqs x 64 blocks
    inf = pool.info()
    assert inf.n_seq == 40 and inf.num_blocks == 40 * 64
    rng = np.random.default_rng(0)
    held = []
    seen = set()
    for _ in range(200):
        if held and rng.random() < 0.4:
            ids = held.pop(int(rng.integers(0, len(held))))
            pool.free_seq(ids)
            for i in ids:
                seen.discard(int(i))
            continue
        n = int(rng.integers(0, 1025))
        try:
            ids = pool.alloc_seq(n)
        except host_lib.DpoolError as e:
            assert e.code == host_lib.DP_ENOMEM
            assert pool.info().free_blocks < -(-n // 16)
            continue
        assert len(ids) == -(-n // 16)
        assert ((ids >= 0) & (ids < inf.num_blocks)).all()
        for i in ids:
            assert int(i) not in seen
            seen.add(int(i))
        held.append(ids)
        assert pool.info().free_blocks == inf.num_blocks - len(seen)


def test_pool_scatters_blocks_and_errors(host_lib):
    pool = host_lib.KVPool(1, 1, 128, 2, 1024, 1024 * 512 * 40, 1.0, 0.0, seed=3)
    ids = pool.alloc_seq(1024)
    assert not np.array_equal(np.sort(ids), ids)   # shuffled free list
    with pytest.raises(host_lib.DpoolError) as e:
        pool.alloc_seq(1025)                          # over C_max
    assert e.value.code == host_lib.DP_EINVAL
    with pytest.raises(host_lib.DpoolError):
        pool.free_seq([ids[0], ids[0]])               # repeated id
    pool.free_seq(ids)
    with pytest.raises(host_lib.DpoolError):
        pool.free_seq(ids[:1])                        # already free
    free_before = pool.info().free_blocks
    with pytest.raises(host_lib.DpoolError):
        pool.free_seq([10 ** 8])
    assert pool.info().free_blocks == free_before
    # exhaustion: the OOM analogue
    got = [pool.alloc_seq(1024) for _ in range(40)]
    assert pool.info().free_blocks == 0
    with pytest.raises(host_lib.DpoolError) as e:
        pool.alloc_seq(1)
    assert e.value.code == host_lib.DP_ENOMEM
    all_ids = np.concatenate(got)
    assert len(np.unique(all_ids)) == len(all_ids) == 40 * 64
    with pytest.raises(host_lib.DpoolError):
        host_lib.KVPool(0, 1, 128, 2, 1024, 1e9, 0.9, 0.0)
    with pytest.raises(host_lib.DpoolError):
        host_lib.KVPool(1, 1, 128, 2, 1024, 1e9, 1.5, 0.0)


# ---------------------------------------------------------------- decode shape validation (host only)

def shape(host_lib, **kw):
    base = dict(batch=4, n_q_heads=8, n_kv_heads=2, max_blocks_per_seq=64, max_context_len=1000, num_blocks=300)
    base.update(kw)
    return host_lib.decode_shape(**base)


def test_workspace_and_partition_sizes(host_lib):
    s = shape(host_lib)
    P = host_lib.partition_tokens(s)
    assert P > 0 and P % 32 == 0
    ws = host_lib.workspace_size(s)
    assert ws > 0 and ws % 256 == 0
    # per wave: two arrival counters + three partial records of G heads x 130 floats
    s2 = shape(host_lib, partition_tokens=32)
    assert host_lib.partition_tokens(s2) == 32
    assert host_lib.workspace_size(s2) >= 8 + 3 * 4 * 130 * 4
    s3 = shape(host_lib, kv_fp8=True, partition_tokens=64)
    assert host_lib.partition_tokens(s3) == 64
    big = shape(host_lib, batch=4096, max_context_len=1000)
    assert host_lib.workspace_size(big) > 0
    assert host_lib.workspace_size(shape(host_lib, batch=4097)) == 0   # unit prefix is kept in LDS


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=64), -95), (dict(block_size=32), -95), (dict(n_q_heads=12, n_kv_heads=8), -22),
    (dict(n_q_heads=64, n_kv_heads=2), -95), (dict(max_context_len=64 * 16 + 1), -22),
    (dict(partition_tokens=24), -22), (dict(partition_tokens=16), -22),
    (dict(kv_fp8=True, partition_tokens=32), -22), (dict(workgroups_per_cu=9), -22),
    (dict(workgroups_per_cu=-1), -22), (dict(num_blocks=0), -22), (dict(batch=-1), -22),
    (dict(batch=5000), -95), (dict(partition_tokens=32 * 257), -22),
    # unit prefix + scales no longer fit in LDS beside the kernel's static arrays
    (dict(batch=4096, n_q_heads=16384, n_kv_heads=16384, num_blocks=16, max_blocks_per_seq=1, max_context_len=16), -95),
])
def test_invalid_shapes_rejected_on_host(host_lib, kw, code):
    s = shape(host_lib, **kw)
    assert host_lib.workspace_size(s) == 0
    L = host_lib.lib()
    rc = L.paged_decode_attention(16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), None, 0, None)
    assert rc == code
    assert host_lib.last_error() != ""


def test_bad_pointers_rejected_on_host(host_lib):
    L = host_lib.lib()
    s = shape(host_lib)
    ws = host_lib.workspace_size(s)
    assert L.paged_decode_attention(None, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), None, 0, None) == -22
    assert L.paged_decode_attention(17, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), 256, ws, None) == -22
    assert L.paged_decode_attention(16, 16, 16, 16, 16, 1.0, 16, 16, 16, ctypes.byref(s), 256, ws, None) == -22
    sf = shape(host_lib, kv_fp8=True)
    assert L.paged_decode_attention(16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(sf), 256, 10 ** 9,
                                    None) == -22
    s32 = shape(host_lib, partition_tokens=32)
    assert L.paged_decode_attention(16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s32), None, 0,
                                    None) == -12
    assert L.paged_decode_attention(16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), 256, ws - 1,
                                    None) == -12
    assert L.paged_decode_attention(16, 16, 16, 16, 16, float("nan"), None, None, 16, ctypes.byref(s), 256, ws,
                                    None) == -22


def test_decoder_wrapper_constructs_on_host(host_lib):
    dec = host_lib.PagedDecoder(4, 8, 2, 64, 1000, 300, partition_tokens=64, device="cpu")
    assert dec.partition_tokens == 64
    assert callable(dec)
    assert dec.workspace is not None and dec.workspace.numel() == host_lib.workspace_size(dec.shape)
    assert int(dec.workspace.count_nonzero()) == 0     # the library needs a zero-filled workspace
    assert tuple(dec.new_out("cpu").shape) == (4, 8, 128)
    with pytest.raises(host_lib.DpoolError):
        host_lib.PagedDecoder(4, 8, 2, 64, 1000, 300, partition_tokens=24, device="cpu")


# ---------------------------------------------------------------- chunked prefill (host-side validation only)

def pshape(host_lib, **kw):
    args = dict(batch=4, n_q_heads=8, n_kv_heads=2, max_blocks_per_seq=64, max_context_len=1000, num_blocks=300,
                total_q=100)
    args.update({k: kw.pop(k) for k in list(kw) if k in args})
    s = host_lib.prefill_shape(**args, **{k: v for k, v in kw.items() if k in ("kv_fp8", "out_fp32", "query_tile")})
    for k, v in kw.items():
        if k not in ("kv_fp8", "out_fp32", "query_tile"):
            setattr(s, k, v)
    return s


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=64), -95), (dict(block_size=32), -95), (dict(n_q_heads=12, n_kv_heads=8), -22),
    (dict(max_context_len=64 * 16 + 1), -22), (dict(query_tile=48), -22), (dict(query_tile=64), -22), (dict(num_blocks=0), -22),
    (dict(batch=-1), -22), (dict(batch=5000), -95), (dict(total_q=-1), -22), (dict(reserved=1), -22),
    (dict(kv_dtype=2), -95), (dict(out_dtype=3), -95),
])
def test_prefill_invalid_shapes_rejected_on_host(host_lib, kw, code):
    s = pshape(host_lib, **kw)
    L = host_lib.lib()
    assert L.chunked_prefill_attention(16, 16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), None) == code
    assert host_lib.last_error() != ""


def test_prefill_bad_pointers_and_scale_rejected_on_host(host_lib):
    L = host_lib.lib()
    s = pshape(host_lib)
    assert L.chunked_prefill_attention(None, 16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), None) == -22
    assert L.chunked_prefill_attention(8, 16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(s), None) == -22
    assert L.chunked_prefill_attention(16, 16, 16, 16, 16, 16, 1.0, 16, 16, 16, ctypes.byref(s), None) == -22
    sf = pshape(host_lib, kv_fp8=True)
    assert L.chunked_prefill_attention(16, 16, 16, 16, 16, 16, 1.0, None, None, 16, ctypes.byref(sf), None) == -22
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert L.chunked_prefill_attention(16, 16, 16, 16, 16, 16, bad, None, None, 16, ctypes.byref(s), None) == -22
    empty = pshape(host_lib, total_q=0)
    assert L.chunked_prefill_attention(None, None, None, None, None, None, 1.0, None, None, None,
                                       ctypes.byref(empty), None) == 0   # nothing to do, nothing enqueued


# ---------------------------------------------------------------- KV append validation (host only)

@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=64), -95), (dict(block_size=32), -95), (dict(batch=-1), -22), (dict(num_blocks=0), -22),
    (dict(n_q_heads=0, n_kv_heads=0), -22), (dict(max_blocks_per_seq=0, max_context_len=0), -22),
    (dict(batch=1 << 20, n_q_heads=1 << 10, n_kv_heads=1 << 10), -22),
])
def test_append_invalid_shapes_rejected_on_host(host_lib, kw, code):
    s = shape(host_lib, **kw)
    L = host_lib.lib()
    rc = L.kv_cache_append(16, 16, 16, 16, 16, 16, None, None, ctypes.byref(s), None)
    assert rc == code
    assert host_lib.last_error() != ""


def test_append_bad_pointers_rejected_on_host(host_lib):
    L = host_lib.lib()
    s = shape(host_lib)
    assert L.kv_cache_append(16, 16, 16, None, 16, 16, None, None, ctypes.byref(s), None) == -22   # null tensor
    assert L.kv_cache_append(16, 16, 16, 16, 16, 18, None, None, ctypes.byref(s), None) == -22   # misaligned
    one = (ctypes.c_float * 2)(1.0, 1.0)
    assert L.kv_cache_append(16, 16, 16, 16, 16, 16, one, one, ctypes.byref(s), None) == -22     # scales on bf16
    s8 = shape(host_lib, kv_fp8=True)
    assert L.kv_cache_append(16, 16, 16, 16, 16, 16, None, None, ctypes.byref(s8), None) == -22  # fp8 without scales
    assert L.kv_cache_append(None, None, None, None, None, None, None, None, None, None) == -22   # null shape
    s0 = shape(host_lib, batch=0)
    assert L.kv_cache_append(None, None, None, None, None, None, None, None, ctypes.byref(s0), None) == 0  # nothing to do


# ---------------------------------------------------------------- benchmark batches from the pool

def test_benchmark_batches_take_their_blocks_from_the_library_pool(host_lib):
    """Configs 2-5 lay out their batch with the library's allocator (Sec. 3
    effect 1: pages on demand from a shuffled per-GPU pool); the values drawn
    do not depend on where the block ids come from."""
    import workloads
    w = workloads.make_config(4, poison=False)
    ref = workloads.make_config(4, poison=False, block_source="numpy")
    assert w.meta["block_source"] == "pool" and ref.meta["block_source"] == "numpy"
    assert (w.context_lens == ref.context_lens).all()
    assert (w.q_bits == ref.q_bits).all() and (w.k_store.tiles == ref.k_store.tiles).all()
    assert (w.v_store.tiles == ref.v_store.tiles).all()
    # the same pool, seeded alike, hands out exactly these ids
    c = workloads.CONFIGS[4]
    pool = host_lib.KVPool(c["n_layers"], c["n_kv_heads"], 128, 2, c["c_max"], workloads.POOL_M_GPU_BYTES,
                           workloads.POOL_UTIL, 0.0, seed=4)
    assert pool.info().num_blocks == w.num_blocks == 49152
    nblk = -(-w.context_lens.astype(np.int64) // 16)
    for s in range(w.batch):
        assert (w.block_tables[s, :nblk[s]] == pool.alloc_seq(int(w.context_lens[s]))).all()
        assert (w.block_tables[s, nblk[s]:] == -1).all()
    used = np.concatenate([w.block_tables[s, :nblk[s]] for s in range(w.batch)])
    assert len(np.unique(used)) == len(used) and used.min() >= 0 and used.max() < w.num_blocks


def test_workload_rejects_bad_block_ids():
    import workloads
    with pytest.raises(ValueError):
        workloads.make_workload(2, 8, 2, [20, 16], c_max=64, seed=1, num_blocks=8, block_ids=[1, 2, 2])
    with pytest.raises(ValueError):
        workloads.make_workload(2, 8, 2, [20, 16], c_max=64, seed=1, num_blocks=8, block_ids=[1, 2, 8])
    with pytest.raises(ValueError):
        workloads.make_workload(2, 8, 2, [20, 16], c_max=64, seed=1, num_blocks=8, block_ids=[1, 2])
    w = workloads.make_workload(2, 8, 2, [20, 16], c_max=64, seed=1, num_blocks=8, block_ids=[5, 0, 7])
    assert w.block_tables[0, :2].tolist() == [5, 0] and w.block_tables[1, :1].tolist() == [7]
