"""GPU parity of paged_decode_attention (through the C ABI) against the fp64 oracle.

Tolerances are fixed by the target: max abs error 1.5e-2 with bf16 KV and
3e-2 with fp8 e4m3 KV, on the bf16 output the library ships (the fp32
output variant is checked to the same bar).  Integer-like properties
(block permutation, poisoned unused blocks, determinism, workspace reuse)
are checked bit for bit; different split-K slicings (partition length,
workgroups per compute unit) are checked against the bound the rounding of
the probabilities gives.
"""
import math
import sys

import numpy as np
import pytest
import torch

import workloads
from oracle import attention, numerics

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1.5e-2, "fp8_e4m3": 3e-2}


def note(msg):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def oracle_out(w, seqs=None):
    return attention.paged_decode_attention(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens, w.scale,
                                            kv_format=w.kv_format, k_scale=w.k_scale, v_scale=w.v_scale, seqs=seqs)


def gpu_out(lib, w, dev=None, out_fp32=False, P=0, wgs=0, layer=0, dec=None):
    d = dev if dev is not None else workloads.to_device(w)
    if dec is None:
        dec = lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, max(w.max_context_len, 0),
                               w.num_blocks, kv_fp8=w.kv_format == "fp8_e4m3", out_fp32=out_fp32,
                               partition_tokens=P, workgroups_per_cu=wgs)
    out = dec.new_out()
    dec(d["q"], d["k"][layer], d["v"][layer], d["block_tables"], d["context_lens"], w.scale, out, d["k_scale"],
        d["v_scale"])
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


def max_err(got, ref, seqs):
    return float(np.abs(got[seqs] - ref[seqs]).max())


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_parity(gpu_lib, cfg):
    """Every row of every benchmark configuration against the oracle, bf16 and fp32 output."""
    note(f"config {cfg}: building workload")
    w = workloads.make_config(cfg)
    rows = list(range(w.batch))
    note(f"config {cfg}: B={w.batch} max_ctx={w.max_context_len}, all rows")
    dev = workloads.to_device(w)
    got = gpu_out(gpu_lib, w, dev)
    got32 = gpu_out(gpu_lib, w, dev, out_fp32=True)
    del dev
    torch.cuda.empty_cache()
    ref = oracle_out(w)
    assert np.isfinite(ref).all()
    err = max_err(got, ref, rows)
    note(f"config {cfg}: max abs err {err:.3e} (bf16 out)")
    assert np.isfinite(got).all()
    assert err <= TOL[w.kv_format]
    err32 = max_err(got32, ref, rows)
    note(f"config {cfg}: max abs err {err32:.3e} (fp32 out)")
    assert err32 <= TOL[w.kv_format]


@pytest.mark.parametrize("cfg", [3, 4])
def test_repeated_calls_bit_identical(gpu_lib, cfg):
    """200 calls on shapes whose long segments are merged on two levels (groups of
    pieces, then the groups): each output equals the first bit for bit."""
    w = workloads.make_config(cfg, poison=False)
    dev = workloads.to_device(w, poison_unused=False)
    dec = gpu_lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                               w.num_blocks)
    ref, out = dec.new_out(), dec.new_out()
    args = (dev["q"], dev["k"][0], dev["v"][0], dev["block_tables"], dev["context_lens"], w.scale)
    dec(*args, ref)
    torch.cuda.synchronize()
    note(f"config {cfg}: 200 repeated calls")
    for i in range(200):
        out.fill_(float("nan"))
        dec(*args, out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"call {i} differs from the first"


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("G", [1, 4, 8, 16])
@pytest.mark.parametrize("P", [0, 64, 128, 512])
def test_random_shapes_ragged(gpu_lib, kv, G, P):
    ctx = [1, 15, 16, 17, 31, 33, 64, 100, 513, 1000, 2049]
    Hkv = 2
    note(f"random shapes kv={kv} G={G} P={P}")
    w = workloads.make_workload(len(ctx), G * Hkv, Hkv, ctx, c_max=2560, kv_format=kv, seed=G * 100 + P)
    got = gpu_out(gpu_lib, w, P=P, out_fp32=True)
    ref = oracle_out(w)
    err = max_err(got, ref, list(range(len(ctx))))
    note(f"  max abs err {err:.3e}")
    assert err <= TOL[kv]


def test_random_batches_every_row(gpu_lib):
    """Sixty seeded random decode shapes (cache format, GQA group 1-16, 1-8 KV
    heads, 1-130 sequences with empty ones among them, C_max 64-5000, minimum
    slice and workgroups per compute unit), every row against the oracle.  Each
    shape is called twice on one workspace: the second call starts its first
    unit from the tiles the first call kept, and must equal it bit for bit."""
    rng = np.random.default_rng(2604)
    for case in range(60):
        kv = ["bf16", "fp8_e4m3"][int(rng.integers(0, 2))]
        G = int(rng.choice([1, 2, 4, 8, 16]))
        Hkv = int(rng.choice([1, 2, 4, 8]))
        B = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 130]))
        cmax = int(rng.choice([64, 700, 2048, 5000]))
        ctx = rng.integers(0, cmax + 1, B)
        if rng.random() < 0.3:
            ctx[rng.random(B) < 0.5] = 0
        if ctx.max() == 0:
            ctx[0] = 1
        P = int(rng.choice([0, 0, 64, 128, 512]))
        wgs = int(rng.choice([0, 0, 1, 2]))
        seed = int(rng.integers(0, 1 << 30))
        note(f"case {case}: kv={kv} G={G} Hkv={Hkv} B={B} C_max={cmax} P={P} wgs={wgs} seed={seed}")
        w = workloads.make_workload(B, G * Hkv, Hkv, list(ctx), c_max=cmax, kv_format=kv, seed=seed)
        d = workloads.to_device(w)
        dec = gpu_lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                                   w.num_blocks, kv_fp8=kv == "fp8_e4m3", out_fp32=True, partition_tokens=P,
                                   workgroups_per_cu=wgs)
        first = gpu_out(gpu_lib, w, d, dec=dec)
        assert np.array_equal(gpu_out(gpu_lib, w, d, dec=dec), first), "the second call differs from the first"
        err = max_err(first, oracle_out(w), list(range(B)))
        assert np.isfinite(first).all() and err <= TOL[kv], f"case {case}: max abs err {err:.3e}"


def test_partition_invariance(gpu_lib):
    """Different split-K partitionings agree to the bound the arithmetic gives.

    The probabilities are rounded to bf16 (relative error <= 2^-9) relative to
    the running max, and that max depends on where partitions start.  Each
    output row is a convex combination of V rows, so perturbing every weight by
    a relative 2^-9 moves it by at most 2^-9 * max_t |v_t - out| (first order);
    two partitionings differ by at most twice that (plus fp32 rounding).
    """
    note("partition invariance")
    ctx = [3000, 1, 700, 4096, 2500]
    w = workloads.make_workload(len(ctx), 32, 4, ctx, c_max=4096, seed=77)
    dev = workloads.to_device(w)
    ref = oracle_out(w)
    bound = np.zeros((w.batch, w.n_q_heads, 1))
    for s_, T in enumerate(ctx):
        for h in range(w.n_q_heads):
            V = np.concatenate([numerics.decode_bf16(w.v_store[np.array([b])][0, h // 8].T)
                                for b in w.block_tables[s_, :-(-T // 16)]])[:T]
            bound[s_, h] = 2 * 2.0 ** -9 * np.abs(V - ref[s_, h]).max() + 1e-6
    outs = [gpu_out(gpu_lib, w, dev, out_fp32=True, P=P) for P in (32, 64, 256, 512, 1024, 4096)]
    outs += [gpu_out(gpu_lib, w, dev, out_fp32=True, wgs=k) for k in (1, 2, 4)]
    for o in outs[1:]:
        diff = np.abs(o - outs[0])
        note(f"  max diff {diff.max():.3e}, mean diff {diff.mean():.3e}")
        assert (diff <= bound).all()


def test_one_token_context_returns_v_exactly(gpu_lib):
    note("ctx=1 returns V")
    w = workloads.make_workload(5, 16, 2, [1] * 5, c_max=64, seed=4)
    got = gpu_out(gpu_lib, w)
    for s in range(5):
        blk = w.block_tables[s, 0]
        for h in range(16):
            v = numerics.decode_bf16(w.v_store[np.array([blk])][0, h // 8, :, 0])
            assert np.array_equal(got[s, h], v)


def test_empty_context_gives_zero_rows(gpu_lib):
    note("ctx=0 rows")
    w = workloads.make_workload(4, 8, 2, [0, 40, 0, 7], c_max=64, seed=5)
    for fp32 in (False, True):
        got = gpu_out(gpu_lib, w, out_fp32=fp32)
        assert np.array_equal(got[[0, 2]], np.zeros((2, 8, 128)))
        ref = oracle_out(w, [1, 3])
        assert max_err(got, ref, [1, 3]) <= TOL["bf16"]


def renumbered(ctx, seed, perm_seed):
    """The workload of make_workload(6, 64, 8, ctx, seed) with every physical
    block b moved to pi[b] and the block table fixed up."""
    w = workloads.make_workload(6, 64, 8, ctx, c_max=2048, seed=seed, num_blocks=600)
    pi = np.random.default_rng(perm_seed).permutation(w.num_blocks)
    for st in (w.k_store, w.v_store):
        st.used_ids = pi[st.used_ids]
        st.slot = np.full(st.num_blocks, -1, dtype=np.int64)
        st.slot[st.used_ids] = np.arange(len(st.used_ids))
    w.block_tables = np.where(w.block_tables >= 0, pi[np.maximum(w.block_tables, 0)], -1).astype(np.int32)
    return w


def test_block_permutation_is_bit_exact(gpu_lib):
    note("block permutation")
    ctx = [5, 300, 1024, 17, 2000, 64]
    w = workloads.make_workload(6, 64, 8, ctx, c_max=2048, seed=6, num_blocks=600)
    base = gpu_out(gpu_lib, w)
    moved = gpu_out(gpu_lib, renumbered(ctx, 6, 0))
    assert np.array_equal(moved, base)


def test_first_unit_hint_follows_changed_inputs(gpu_lib):
    """A wave issues its first unit's loads from the tiles the previous call on the
    same workspace used, and loads the unit again when the true tiles differ.
    One workspace, calls alternating between the same contexts with the blocks
    renumbered and different context lengths (other slices): every call equals
    its result on a fresh workspace bit for bit."""
    note("first-unit hint: alternating inputs on one workspace")
    ctx = [5, 300, 1024, 17, 2000, 64]
    ws = [workloads.make_workload(6, 64, 8, ctx, c_max=2048, seed=6, num_blocks=600), renumbered(ctx, 6, 0),
          workloads.make_workload(6, 64, 8, [700, 1, 1500, 2048, 90, 333], c_max=2048, seed=16, num_blocks=600)]
    assert len({(w.max_blocks_per_seq, w.num_blocks) for w in ws}) == 1
    devs = [workloads.to_device(w) for w in ws]

    def decoder():  # one shape for every call: C_max 2048
        return gpu_lib.PagedDecoder(6, 64, 8, ws[0].max_blocks_per_seq, 2048, ws[0].num_blocks)

    fresh = [gpu_out(gpu_lib, w, d, dec=decoder()) for w, d in zip(ws, devs)]
    dec = decoder()
    for i in (0, 0, 1, 1, 0, 2, 2, 1, 0):
        got = gpu_out(gpu_lib, ws[i], devs[i], dec=dec)
        assert np.array_equal(got, fresh[i]), f"call on input {i} differs from its fresh-workspace result"


def test_unused_blocks_never_read(gpu_lib):
    note("poisoned vs junk unused blocks")
    w = workloads.make_workload(4, 16, 2, [33, 700, 5, 129], c_max=1024, seed=7, num_blocks=400)
    a = gpu_out(gpu_lib, w, workloads.to_device(w, poison_unused=True))
    dev = workloads.to_device(w, poison_unused=True)
    used = torch.zeros(w.num_blocks, dtype=torch.bool, device="cuda")
    used[torch.from_numpy(w.k_store.used_ids).cuda()] = True
    for name in ("k", "v"):
        junk = torch.randint(-30000, 30000, dev[name].shape, dtype=torch.int16, device="cuda")
        dev[name][:, ~used] = junk[:, ~used]
    b = gpu_out(gpu_lib, w, dev)
    assert np.isfinite(a).all()
    assert np.array_equal(a, b)


def test_deterministic(gpu_lib):
    note("determinism")
    for kv in ("bf16", "fp8_e4m3"):
        w = workloads.make_workload(8, 64, 4, [1, 100, 900, 3000, 17, 4096, 256, 2222], c_max=4096, kv_format=kv,
                                    seed=8)
        dev = workloads.to_device(w)
        ref = gpu_out(gpu_lib, w, dev)
        for _ in range(3):
            assert np.array_equal(gpu_out(gpu_lib, w, dev), ref)


def test_longest_context_and_gqa16_bf16(gpu_lib):
    note("C_max 65536 sequence, GQA 16 bf16")
    w = workloads.make_workload(2, 32, 2, [65536, 40000], c_max=65536, seed=9)
    got = gpu_out(gpu_lib, w)
    ref = oracle_out(w)
    err = max_err(got, ref, [0, 1])
    note(f"  max abs err {err:.3e}")
    assert err <= TOL["bf16"]


def test_rotated_layers_read_their_own_pool(gpu_lib):
    note("layer rotation")
    w = workloads.make_workload(3, 16, 2, [100, 200, 300], c_max=512, seed=10)
    dev = workloads.to_device(w, layers=3)
    outs = [gpu_out(gpu_lib, w, dev, layer=l) for l in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_workspace_reused_across_shapes(gpu_lib):
    """One zero-filled workspace serves calls of different shapes in turn, including
    grids of very different widths (a few waves; two workgroups per compute unit;
    a grid wider than eight workgroups per compute unit, whose counters reach past
    the fixed counter region): every call equals its fresh-workspace result bit for
    bit, and every call leaves the counter region at zero."""
    note("workspace reuse")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rng = np.random.default_rng(12)
    wide_ctx = rng.integers(0, 40, 4096)
    wide_ctx[[5, 900, 4000]] = [3000, 700, 1500]
    cases = [  # (workload, decoder kwargs)
        (workloads.make_workload(3, 8, 2, [300, 17, 90], c_max=320, seed=11), {}),
        (workloads.make_workload(5, 32, 4, [3000, 1, 700, 4096, 2500], c_max=4096, seed=12), {"workgroups_per_cu": 2}),
        (workloads.make_workload(3, 64, 4, [9000, 33, 5000], c_max=16384, kv_format="fp8_e4m3", seed=13), {}),
        (workloads.make_workload(4096, 4, 2, wide_ctx, c_max=65536, seed=14), {}),
    ]
    devs, decs, refs = [], [], []
    for w, kw in cases:
        d = workloads.to_device(w)
        dec = gpu_lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                                   w.num_blocks, kv_fp8=w.kv_format == "fp8_e4m3", **kw)
        devs.append(d)
        decs.append(dec)
        refs.append(gpu_out(gpu_lib, w, d, dec=dec))
    sizes = [dec.workspace.numel() for dec in decs]
    note(f"  workspace sizes {sizes}")
    assert sizes[3] > sizes[0]
    shared = torch.zeros(max(sizes), dtype=torch.uint8, device="cuda")
    for dec, n in zip(decs, sizes):
        dec.workspace = shared[:n]
    counter_bytes = 2 * 4 * 8 * 4 * cus   # two int32 counters per wave, up to 8 four-wave workgroups per CU
    for order in ([0, 1, 2, 3], [3, 0, 3, 1, 2, 0, 3], [2, 1, 0]):
        for i in order:
            w, _ = cases[i]
            assert np.array_equal(gpu_out(gpu_lib, w, devs[i], dec=decs[i]), refs[i]), f"case {i} in {order}"
            assert int(shared[:counter_bytes].count_nonzero()) == 0
    for (w, _), ref in zip(cases, refs):
        rows = list(range(w.batch))
        assert max_err(ref, oracle_out(w), rows) <= TOL[w.kv_format]


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_largest_batch(gpu_lib, kv):
    """4,096 sequences (the most one call takes): short and empty contexts, every
    slice crossing many segments; every row against the oracle, empty rows zero."""
    note(f"batch 4096, {kv}")
    rng = np.random.default_rng(31)
    ctx = rng.integers(0, 97, 4096)
    ctx[rng.integers(0, 4096, 64)] = 0
    w = workloads.make_workload(4096, 16, 2, ctx, c_max=128, kv_format=kv, seed=14)
    got = gpu_out(gpu_lib, w)
    seqs = list(range(w.batch))
    err = max_err(got, oracle_out(w), seqs)
    note(f"  max abs err {err:.3e}")
    assert err <= TOL[kv]
    empty = np.nonzero(w.context_lens == 0)[0]
    assert len(empty) > 0 and np.all(got[empty] == 0.0)
