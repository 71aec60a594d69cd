"""paged_decode_attention_noalloc (through the C ABI) against paged_decode_attention.

The entry point without a workspace runs the same decode launch on the
library's fixed per-GPU scratch array, so its output must equal the
workspace entry point's bit for bit, call after call: the array keeps the
previous call's contents, and a later, smaller call must not be disturbed by
them.  Shapes whose workspace exceeds the array are rejected on the host.
"""
import sys

import numpy as np
import pytest
import torch

import workloads
from oracle import attention

pytestmark = pytest.mark.gpu


def note(msg):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def both(lib, w, dev, out_fp32=False):
    """(noalloc output, workspace output) as numpy float32."""
    fp8 = w.kv_format == "fp8_e4m3"
    dec = lib.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                           w.num_blocks, kv_fp8=fp8, out_fp32=out_fp32)
    args = (dev["q"], dev["k"][0], dev["v"][0], dev["block_tables"], dev["context_lens"], w.scale)
    ref = dec.new_out()
    dec(*args, ref, dev["k_scale"], dev["v_scale"])
    got = torch.full_like(ref, float("nan"))
    lib.paged_decode_attention_noalloc(*args, got, dec.shape, dev["k_scale"], dev["v_scale"])
    torch.cuda.synchronize()
    return got.float().cpu().numpy(), ref.float().cpu().numpy()


def test_noalloc_equals_workspace_entry_point(gpu_lib):
    cases = [
        ("short pool (config 2)", workloads.make_config(2), False),
        ("tiny (config 1), smaller", workloads.make_config(1), False),
        ("split segments, fp8 GQA 16", workloads.make_workload(3, 64, 4, [9000, 33, 5000], c_max=16384,
                                                               kv_format="fp8_e4m3", seed=13), True),
        ("short pool again", workloads.make_config(2), False),
    ]
    for name, w, fp32 in cases:
        note(f"noalloc: {name}: B={w.batch} {w.n_q_heads}q/{w.n_kv_heads}kv {w.kv_format}")
        dev = workloads.to_device(w)
        got, ref = both(gpu_lib, w, dev, out_fp32=fp32)
        assert np.isfinite(got).all()
        assert np.array_equal(got, ref), name
        del dev
        torch.cuda.empty_cache()
    # and to the oracle's bar on the small case
    w = cases[1][1]
    got, _ = both(gpu_lib, w, workloads.to_device(w))
    exp = attention.paged_decode_attention(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens, w.scale)
    assert float(np.abs(got - exp).max()) <= 1.5e-2


def test_noalloc_rejects_shapes_beyond_its_scratch(gpu_lib):
    # 4096 sequences of up to 65,536 tokens over one KV head with GQA 16: the
    # grid, and with it the partial-record area, grows past the fixed array
    shape = gpu_lib.decode_shape(4096, 16, 1, 4096, 65536, 1 << 20)
    assert gpu_lib.workspace_size(shape) > 32 << 20
    dummy = torch.zeros(16, dtype=torch.int16, device="cuda")
    with pytest.raises(gpu_lib.DpoolError) as e:
        gpu_lib.paged_decode_attention_noalloc(dummy, dummy, dummy, dummy, dummy, 0.1, dummy, shape)
    assert e.value.code == gpu_lib.DP_ENOMEM
    assert "scratch" in gpu_lib.last_error()
