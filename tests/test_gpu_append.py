"""GPU parity of kv_cache_append (through the C ABI) against the oracle.

The stored codes are integers, so the bar is bit-exact: the whole K and V
pools after the append must equal the oracle's, untouched slots included.
The e4m3 path is swept over a wide range of magnitudes (subnormals, ties,
saturation) because the hardware conversion decides those codes.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import append, attention

pytestmark = pytest.mark.gpu


def note(msg):
    print(f"[gpu-test] {msg}", flush=True)


def bf16_bits(rng, shape, spread=False):
    if spread:   # magnitudes 2^-16 .. 2^12, both signs: exercises subnormal, tie and saturating e4m3 codes
        x = (rng.random(shape) + 1.0) * np.exp2(rng.integers(-16, 13, shape)) * np.where(rng.random(shape) < .5, -1, 1)
    else:
        x = rng.standard_normal(shape)
    return workloads.to_bf16_codes(x.astype(np.float32))


def random_pools(rng, fmt, nb, Hkv):
    if fmt == "bf16":
        k = bf16_bits(rng, (nb, Hkv, 16, 128))
        v = bf16_bits(rng, (nb, Hkv, 128, 16))
    else:
        k = rng.integers(0, 256, (nb, Hkv, 16, 128)).astype(np.uint8)
        v = rng.integers(0, 256, (nb, Hkv, 128, 16)).astype(np.uint8)
    return k, v


def to_dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def run_append(lib, knew, vnew, kp, vp, bt, pos, fmt, ks, vs, num_blocks):
    B, Hkv, _ = knew.shape
    shape = lib.decode_shape(B, Hkv, Hkv, bt.shape[1], bt.shape[1] * 16, num_blocks, kv_fp8=fmt != "bf16")
    dk, dv = to_dev(kp), to_dev(vp)
    lib.kv_cache_append(to_dev(knew), to_dev(vnew), dk, dv, to_dev(bt), to_dev(pos), shape,
                        to_dev(ks) if ks is not None else None, to_dev(vs) if vs is not None else None)
    torch.cuda.synchronize()
    conv = (lambda t: t.cpu().numpy().view(np.uint16)) if fmt == "bf16" else (lambda t: t.cpu().numpy())
    return conv(dk), conv(dv)


@pytest.mark.parametrize("fmt", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("spread", [False, True])
def test_append_bit_exact(gpu_lib, fmt, spread):
    note(f"append {fmt} spread={spread}")
    rng = np.random.default_rng(31 + spread)
    B, Hkv, nb, mbps = 40, 4, 400, 8
    kp, vp = random_pools(rng, fmt, nb, Hkv)
    knew, vnew = bf16_bits(rng, (B, Hkv, 128), spread), bf16_bits(rng, (B, Hkv, 128), spread)
    bt = rng.permutation(nb)[:B * mbps].reshape(B, mbps).astype(np.int32)
    bt[5, 2] = -1                      # a hole in the table: that position writes nothing
    bt[6, 0] = nb + 7                  # an id outside the pool: writes nothing
    pos = rng.integers(0, mbps * 16, B).astype(np.int32)
    pos[:8] = [0, 15, 16, mbps * 16 - 1, -1, 2 * 16 + 3, 5, mbps * 16]  # boundaries and invalid positions
    ks = vs = None
    if fmt != "bf16":
        ks = (rng.random(Hkv) * 0.05 + 0.001).astype(np.float32)
        vs = (rng.random(Hkv) * 0.05 + 0.001).astype(np.float32)
    gk, gv = run_append(gpu_lib, knew, vnew, kp, vp, bt, pos, fmt, ks, vs, nb)
    rk, rv = append.kv_cache_append(knew, vnew, kp, vp, bt, pos, fmt, ks, vs)
    assert np.array_equal(gk, rk)
    assert np.array_equal(gv, rv)
    assert not np.array_equal(rk, kp)  # something was written


@pytest.mark.parametrize("fmt", ["bf16", "fp8_e4m3"])
def test_append_then_decode(gpu_lib, fmt):
    """The token appended at position ctx is read by the next decode over ctx + 1 tokens."""
    note(f"append then decode {fmt}")
    ctx = [1, 15, 16, 31, 200, 1000]
    w = workloads.make_workload(len(ctx), 32, 4, ctx, c_max=2048, kv_format=fmt, seed=33, poison=True)
    dev = workloads.to_device(w, poison_unused=True)   # tail slots and unused blocks hold NaN codes on both sides
    rng = np.random.default_rng(34)
    knew, vnew = bf16_bits(rng, (w.batch, 4, 128)), bf16_bits(rng, (w.batch, 4, 128))
    # the new token needs its block: sequences at a block boundary get a fresh block from the unused ids
    bt = w.block_tables.copy()
    free = np.setdiff1d(np.arange(w.num_blocks), w.k_store.used_ids)
    for s, T in enumerate(ctx):
        if T % 16 == 0:
            bt[s, T // 16] = free[s]
    pos = np.array(ctx, np.int32)
    shape = gpu_lib.decode_shape(w.batch, 32, 4, w.max_blocks_per_seq, w.c_max, w.num_blocks, kv_fp8=fmt != "bf16")
    dbt = to_dev(bt)
    gpu_lib.kv_cache_append(to_dev(knew), to_dev(vnew), dev["k"][0], dev["v"][0], dbt, to_dev(pos), shape,
                            dev["k_scale"], dev["v_scale"])
    dec = gpu_lib.PagedDecoder(w.batch, 32, 4, w.max_blocks_per_seq, max(ctx) + 1, w.num_blocks, kv_fp8=fmt != "bf16",
                               out_fp32=True)
    out = dec.new_out()
    dec(dev["q"], dev["k"][0], dev["v"][0], dbt, to_dev(pos + 1), w.scale, out, dev["k_scale"], dev["v_scale"])
    torch.cuda.synchronize()
    kpool = dev["k"][0].cpu().numpy()
    vpool = dev["v"][0].cpu().numpy()
    if fmt == "bf16":
        kpool, vpool = kpool.view(np.uint16), vpool.view(np.uint16)
    ref = attention.paged_decode_attention(w.q_bits, kpool, vpool, bt, pos + 1, w.scale, kv_format=fmt,
                                           k_scale=w.k_scale, v_scale=w.v_scale)
    err = float(np.abs(out.cpu().numpy() - ref).max())
    note(f"  max abs err {err:.3e}")
    assert err <= (1.5e-2 if fmt == "bf16" else 3e-2)
    # and the appended slots hold exactly the oracle's codes
    rk, rv = append.kv_cache_append(knew, vnew, w.k_store.dense(), w.v_store.dense(), bt, pos, fmt, w.k_scale,
                                    w.v_scale)
    used = np.unique(bt[bt >= 0])
    assert np.array_equal(kpool[used], rk[used]) and np.array_equal(vpool[used], rv[used])
