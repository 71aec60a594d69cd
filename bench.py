#!/usr/bin/env python3
"""Paged decode-attention benchmark on one MI355X.

One "step" is one decode step of one layer for the whole batch: one launch
of the decode kernel, which streams every cached K and V element once and
merges split-K partials inside the same launch - every stage of the hot
path, with the inputs already resident in HBM.  Successive steps rotate
over R independent copies of the layer's KV pool (R * KV bytes >= 1 GiB),
so the 256 MB Infinity Cache cannot serve a step from the previous one.

The headline workload is the short pool (B=128, Llama-3-70B layer shape,
bf16 KV, C_max 8192); the long pool (B=16, C_max 65536), the homogeneous
pool (B=16, mixed lengths, C_max 65536) and the Qwen3-shaped fp8 short pool
are reported beside it in the same line, as the metric compares the pools.
Each pool also times the KV-cache append of its batch (one new token per
sequence).  The line also carries:
  roofline      the decode kernel against 8 TB/s, with HBM traffic from the
                committed rocprofv3 counter summary when it matches the source;
  cpu_baseline  the fp64 oracle timed on this host over the same batch;
  cost_model    the paper's fleet cost model with the throughput ratio
                measured here (context only);
  router        the host router's dispatch rate and one adaptive-threshold step;
  chunked_prefill  the chunked-prefill attention on its two workloads, against
                the dense bf16 MFMA peak.

Output: one JSON line on stdout.  Progress goes to stderr.

  python bench.py [--gpus 1] [--steps 100] [--warmup 10] [--config 2] [--configs 3,4,5]
                  [--no-cpu-baseline] [--no-prefill] [--prefill-only]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

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

    # KV-cache append of one token per sequence, into the slot of each
    # sequence's last cached token (a position that always has its block)
    gen = torch.Generator(device="cuda").manual_seed(cfg)
    knew = torch.randn((w.batch, w.n_kv_heads, w.head_dim), device="cuda", generator=gen).to(torch.bfloat16)
    vnew = torch.randn((w.batch, w.n_kv_heads, w.head_dim), device="cuda", generator=gen).to(torch.bfloat16)
    pos = (cl - 1).clamp(min=0).to(torch.int32)
    ashape = binding.decode_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                                  w.num_blocks, kv_fp8=fp8)

    def app(i):
        binding.kv_cache_append(knew, vnew, kl[i % layers], vl[i % layers], bt, pos, ashape, ks, vs)

    for i in range(warmup):
        app(i)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record()
        app(i)
        ev[i][1].record()
    torch.cuda.synchronize()
    app_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / steps
    app_bytes = w.batch * w.n_kv_heads * w.head_dim * (2 * (1 if fp8 else 2) + 2 * 2)  # cache writes + bf16 inputs
    res["kv_append"] = {"us_per_launch": app_ms * 1e3, "bytes": app_bytes,
                        "gbs": app_bytes / (app_ms * 1e-3) / 1e9, "tokens": w.batch}
    log(f"config {cfg}: kv append {app_ms * 1e3:.1f} us for {w.batch} tokens x {w.n_kv_heads} heads")
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


PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA peak


def prefill_flops(w) -> int:
    """Algorithmic flops of causal chunked-prefill attention: 4 * D * Hq per attended (query, token) pair."""
    qs = w.meta["q_start"]
    pairs = 0
    for s in range(w.batch):
        n, T = int(qs[s + 1] - qs[s]), int(w.context_lens[s])
        pairs += n * (T - n) + n * (n + 1) // 2
    return 4 * w.head_dim * w.n_q_heads * pairs


def measure_prefill(name, steps, warmup, query_tile=0):
    """Time chunked_prefill_attention on one of the prefill workloads (HIP events, current stream)."""
    import torch

    import workloads
    from paper_2604_08075_amd import binding
    w = workloads.make_prefill_config(name, poison=False)
    dev = workloads.to_device(w, poison_unused=False)
    fp8 = w.kv_format == "fp8_e4m3"
    total_q = int(w.meta["q_start"][-1])
    shape = binding.prefill_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.max_blocks_per_seq, w.max_context_len,
                                  w.num_blocks, total_q, kv_fp8=fp8, query_tile=query_tile)
    out = torch.empty((total_q, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")

    def call():
        binding.chunked_prefill_attention(dev["q"], dev["k"][0], dev["v"][0], dev["block_tables"],
                                          dev["context_lens"], dev["q_start"], w.scale, out, shape, dev["k_scale"],
                                          dev["v_scale"])

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    flops = prefill_flops(w)
    tfs = flops / (ms * 1e-3) / 1e12
    chunks = ", ".join(f"{int(w.meta['q_start'][s + 1] - w.meta['q_start'][s])}@{int(w.context_lens[s])}"
                       for s in range(w.batch))
    log(f"prefill {name}: {ms * 1e3:.1f} us/launch, {tfs:.1f} TFLOP/s ({100 * tfs / PEAK_BF16_TFLOPS:.1f}% of "
        f"bf16 MFMA peak)")
    del dev
    torch.cuda.empty_cache()
    return {"workload": f"{name}: chunks (query tokens @ context) {chunks}, {w.n_q_heads}q/{w.n_kv_heads}kv, "
                        f"head_dim 128, {w.kv_format} KV, block 16",
            "us_per_launch": ms * 1e3, "flops": flops, "tflops": tfs,
            "roofline": {"bound": "mfma", "achieved": tfs, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": tfs / PEAK_BF16_TFLOPS, "kernel": "prefill_kernel"},
            "query_tile": 32}


def router_rate(binding, n=1 << 20, intervals=20000):
    """Host-side dispatch (Algorithm 1 Route, one C call over n requests) and the
    adaptive-threshold step, timed on this host (no GPU)."""
    rng = np.random.default_rng(11)
    params = binding.default_route_params()
    cats = binding.make_categories(params, 8)
    pools = binding.make_pools(8192, 1 << 40, 65536, 1 << 40)
    req_bytes = (np.clip(rng.lognormal(np.log(600.0), 1.2, n), 16, 60000) * 4).astype(np.int64)
    req_cat = rng.integers(0, 8, n).astype(np.int32)
    req_max_out = rng.integers(16, 2048, n).astype(np.int64)
    t0 = time.perf_counter()
    pool_ids, _ = binding.route_requests(params, cats, pools, req_bytes, req_cat, req_max_out)
    t_route = time.perf_counter() - t0
    ap = binding.default_adapt_params()
    b = 8192.0
    t0 = time.perf_counter()
    for i in range(intervals):
        b, _ = binding.adapt_threshold(ap, (1000, i % 30, 0, 0), (100, (i // 7) % 5, 0, 0), b)
    t_adapt = time.perf_counter() - t0
    return {"route_requests_per_s": n / t_route, "requests": n, "short_fraction": float(np.mean(pool_ids == 0)),
            "adapt_threshold_us_per_call": 1e6 * t_adapt / intervals,
            "note": "host C calls through ctypes; the adapt figure includes the ctypes call overhead"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="headline workload (2 = short pool)")
    ap.add_argument("--configs", default="3,4,5",
                    help="workloads reported beside it (3 long pool, 4 homogeneous pool, 5 Qwen3 fp8, 1 tiny)")
    ap.add_argument("--long-config", type=int, default=None, help="only this one beside the headline (0 = none)")
    ap.add_argument("--partition-tokens", type=int, default=0)
    ap.add_argument("--wgs-per-cu", type=int, default=0, help="resident workgroups per CU (0 = library choice)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true", help="skip the chunked-prefill attention timing")
    ap.add_argument("--prefill-tile", type=int, default=0, help="query tokens per prefill work item (0 or 32)")
    ap.add_argument("--prefill-only", action="store_true", help="only time the chunked-prefill attention")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB 10 times (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
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

    if args.prefill_only:
        res = {n: measure_prefill(n, max(args.steps // 5, 5), 3, args.prefill_tile)
               for n in ("chunked_prefill_llama70b", "chunked_prefill_qwen3_fp8")}
        print(json.dumps({"chunked_prefill": res}), flush=True)
        return
    head, w_head = measure(args.config, args.steps, args.warmup, args.partition_tokens, args.wgs_per_cu)
    others = [int(c) for c in args.configs.split(",") if c.strip()] if args.long_config is None else (
        [args.long_config] if args.long_config else [])
    extra = {}
    names = {3: "long_pool", 4: "homogeneous_pool", 5: "qwen3_fp8_short_pool", 1: "tiny", 2: "short_pool"}
    for c in others:
        if c != args.config:
            r, _ = measure(c, args.steps, args.warmup, args.partition_tokens, args.wgs_per_cu)
            extra[names.get(c, f"config_{c}")] = r

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
        "kv_append": head["kv_append"],
        "roofline": roof,
    }
    line.update(extra)
    homog = extra.get("homogeneous_pool")
    if head["name"] == "short_pool_llama70b" and homog:
        # decode-attention throughput ratio of the short pool over the
        # homogeneous pool (one layer, per GPU), into the Sec. 3 cost model
        rho = head["seq_steps_per_s"] / homog["seq_steps_per_s"]
        alpha = 0.80  # the paper's short-traffic fraction for its Azure trace at B_short = 8192
        cm = binding.cost_model(1000.0, alpha, rho, 1.0)
        line["cost_model"] = {
            "rho_decode_attention": rho, "alpha": alpha, "savings_formula": cm.savings_formula,
            "definition": "rho = (B / t_step) short pool / (B / t_step) homogeneous pool, decode attention only; "
                          "savings = alpha (1 - 1/rho) (Sec. 3); the paper's Table 1 rho = 4.0 gives 60%",
            "context_only": True}
    line["router"] = router_rate(binding)
    if not args.no_prefill:
        line["chunked_prefill"] = {n: measure_prefill(n, max(args.steps // 5, 5), 3, args.prefill_tile)
                                   for n in ("chunked_prefill_llama70b", "chunked_prefill_qwen3_fp8")}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on the same workload")
        line["cpu_baseline"] = cpu_baseline(w_head)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
