#!/usr/bin/env python3
"""Paged decode-attention benchmark on one MI355X.

One "step" is one decode step of one layer for the whole batch: one launch
of the decode kernel, which streams every cached K and V element once and
merges split-K partials inside the same launch - every stage of the hot
path, with the inputs already resident in HBM.  Successive steps rotate over R independent copies
of the layer's KV pool (R * KV bytes >= 1 GiB), so the 256 MB Infinity
Cache cannot serve a step from the previous one.

The headline workload is the short pool (B=128, Llama-3-70B layer shape,
bf16 KV, C_max 8192); the long pool (B=16, C_max 65536) is reported beside
it in the same line, as the metric compares the two.

Output: one JSON line on stdout.  Progress goes to stderr.

  python bench.py [--gpus 1] [--steps 100] [--warmup 10] [--all] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn achieved HBM GB/s (% of peak) + seq-steps/s, short vs long pool"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, published
KERNEL_SRC = os.path.join(ROOT, "paper_2604_08075_amd", "csrc", "paged_decode.hip")
PROFILES = os.path.join(ROOT, "profiles")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_sha() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload_name: str):
    """HBM bytes per launch of the decode kernel from the committed rocprofv3
    counter summary, if it was taken on the kernel source as it is now."""
    path = os.path.join(PROFILES, f"traffic_paged_decode_{workload_name}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != kernel_sha():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def describe(w) -> str:
    return (f"{w.name}: B={w.batch}, {w.n_q_heads}q/{w.n_kv_heads}kv heads, head_dim {w.head_dim}, "
            f"{w.kv_format} KV, block {w.block_size}, C_max {w.c_max}, seed {w.config}, "
            f"sum ctx {int(w.context_lens.sum())}, max ctx {w.max_context_len}, pool {w.num_blocks} blocks")


def measure(cfg: int, steps: int, warmup: int, partition_tokens: int, wgs: int):
    import torch

    import workloads
    from paper_2604_08075_amd import binding

    t0 = time.time()
    w = workloads.make_config(cfg, poison=False)
    layers = max(1, math.ceil((1 << 30) / w.kv_bytes))
    log(f"config {cfg}: {describe(w)}; generated in {time.time() - t0:.1f}s; rotating over {layers} layer copies")
    dev = workloads.to_device(w, layers=layers, poison_unused=False)
    fp8 = w.kv_format == "fp8_e4m3"
    dec = binding.PagedDecoder(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                               w.num_blocks, kv_fp8=fp8, partition_tokens=partition_tokens,
                               workgroups_per_cu=wgs)
    out = dec.new_out()
    q, bt, cl, ks, vs = dev["q"], dev["block_tables"], dev["context_lens"], dev["k_scale"], dev["v_scale"]
    kl, vl = dev["k"], dev["v"]

    def step(i):
        dec(q, kl[i % layers], vl[i % layers], bt, cl, w.scale, out, ks, vs)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    # timed region: exactly `steps` steps between two events on the launch stream
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        step(i)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / steps

    # kernel duration: the same steps with events around each launch, on the
    # launch stream (torch's current stream, which the binding passes down)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record()
        step(i)
        ev[i][1].record()
    torch.cuda.synchronize()
    kern_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / steps
    res = dict(
        workload=describe(w), name=w.name, batch=w.batch, kv_bytes=w.kv_bytes, kv_format=w.kv_format,
        ms_per_step=ms_step, gbs=w.kv_bytes / (ms_step * 1e-3) / 1e9,
        seq_steps_per_s=w.batch / (ms_step * 1e-3), kernel_ms=kern_ms,
        kernel_gbs=w.kv_bytes / (kern_ms * 1e-3) / 1e9, partition_tokens=dec.partition_tokens,
        layers_rotated=layers, sum_ctx=int(w.context_lens.sum()),
        flops=4 * w.head_dim * w.n_q_heads * int(w.context_lens.sum()))
    log(f"config {cfg}: {ms_step * 1e3:.1f} us/step, {res['gbs']:.0f} GB/s "
        f"({100 * res['gbs'] / PEAK_HBM_GBS:.1f}% of 8 TB/s), kernel {kern_ms * 1e3:.1f} us "
        f"({100 * res['kernel_gbs'] / PEAK_HBM_GBS:.1f}%), min slice {dec.partition_tokens} tokens")
    del dev
    torch.cuda.empty_cache()
    return res, w


def cpu_baseline(w, budget_s=10.0):
    """The fp64 oracle, unchanged, timed on this host over whole passes of the same batch."""
    from threadpoolctl import threadpool_limits

    from oracle import attention
    done_bytes = 0
    done_seqs = 0
    passes = 0
    t0 = time.time()
    with threadpool_limits(limits=1):
        while True:
            for s in range(w.batch):
                attention.paged_decode_attention(w.q_bits, w.k_store, w.v_store, w.block_tables, w.context_lens,
                                                 w.scale, kv_format=w.kv_format, k_scale=w.k_scale,
                                                 v_scale=w.v_scale, seqs=[s])
                done_bytes += int(w.context_lens[s]) * w.n_kv_heads * w.head_dim * 2 * (
                    1 if w.kv_format == "fp8_e4m3" else 2)
                done_seqs += 1
            passes += 1
            if time.time() - t0 >= budget_s or passes >= 20:
                break
    dt = time.time() - t0
    return {"value": done_bytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{passes} full pass(es) over the {w.name} batch ({w.batch} sequences, "
                      f"{int(w.context_lens.sum())} tokens) in {dt:.1f} s, one sequence per oracle call, "
                      f"BLAS limited to 1 thread",
            "seq_steps_per_s": done_seqs / dt, "seconds": dt}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="headline workload (2 = short pool)")
    ap.add_argument("--long-config", type=int, default=3, help="long-pool workload reported beside it (0 = none)")
    ap.add_argument("--all", action="store_true", help="also report configs 1, 4 and 5")
    ap.add_argument("--partition-tokens", type=int, default=0)
    ap.add_argument("--wgs-per-cu", type=int, default=0, help="resident workgroups per CU (0 = library choice)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB 10 times (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "launches": 10}))
        return
    from paper_2604_08075_amd import binding
    log(f"libdpool {binding.version()} on {torch.cuda.get_device_name(0)}")

    head, w_head = measure(args.config, args.steps, args.warmup, args.partition_tokens, args.wgs_per_cu)
    extra = {}
    if args.long_config:
        r, _ = measure(args.long_config, args.steps, args.warmup, args.partition_tokens, args.wgs_per_cu)
        extra["long_pool"] = r
    if args.all:
        for c in (1, 4, 5):
            if c not in (args.config, args.long_config):
                r, _ = measure(c, args.steps, args.warmup, args.partition_tokens, args.wgs_per_cu)
                extra[f"config_{c}"] = r

    traffic = measured_traffic(head["name"])
    roof = {"bound": "hbm", "achieved": head["kernel_gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": head["kernel_gbs"] / PEAK_HBM_GBS, "traffic": traffic,
            "kernel": "paged_decode_kernel", "algorithmic_bytes_per_launch": head["kv_bytes"],
            "avg_launch_ms": head["kernel_ms"]}
    line = {
        "metric": METRIC, "value": head["gbs"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": head["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": head["workload"], "batch": head["batch"], "kv_dtype": head["kv_format"],
                   "partition_tokens": head["partition_tokens"], "layers_rotated": head["layers_rotated"]},
        "pct_of_peak_hbm": 100.0 * head["gbs"] / PEAK_HBM_GBS,
        "seq_steps_per_s": head["seq_steps_per_s"],
        "roofline": roof,
    }
    line.update(extra)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on the same workload")
        line["cpu_baseline"] = cpu_baseline(w_head)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
