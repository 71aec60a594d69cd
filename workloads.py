"""Seeded synthetic decode workloads shaped like the paper's pools.

This module only draws inputs: sequence lengths, a scattered block table,
and the bf16 / fp8 codes of Q, K and V.  It holds none of the method's
arithmetic (no attention, no sizing equation, no routing), so both the CPU
oracle and the HIP path may use it.

The paper's traces (Azure LLM inference, LMSYS-Chat-1M; Sec. 4.1 "Traces")
are not available; these draws stand in for them with the shape statistics
the paper quotes: 80% of requests under 2K tokens with a tail to 64K
(Sec. 1.1, Sec. 4.1), mean generated length 214.5 tokens (Sec. 4.1), pools
with C_max 8K (short) and 65K (long, homogeneous) (Table 1), and a
Qwen3-235B-A22B layer with 64 query / 4 KV heads in FP8 (Sec. 4.7).

Config table (index -> shape):
  1 tiny         B=4,   8q/2kv,  bf16, C_max 512,   ctx ~ U{1..512}
  2 short pool   B=128, 64q/8kv, bf16, C_max 8192,  ctx = min(prompt + gen, 8192),
                 prompt = clip(rint(lognormal(ln 600, 1.2)), 16, 8192), gen ~ U{1..428}
  3 long pool    B=16,  64q/8kv, bf16, C_max 65536, ctx = floor(8192 / (1 - U (1 - 8^-1.5))^(1/1.5))
                 (Pareto alpha 1.5 truncated to [8192, 65536], inverse CDF)
  4 homogeneous  B=16,  64q/8kv, bf16, C_max 65536, per sequence 15% config-3 draw,
                 else config-2 draw
  5 Qwen3 short  B=256, 64q/4kv, fp8 e4m3 + per-KV-head fp32 scales, C_max 8192,
                 lengths as config 2

Pool sizes (blocks of 16 tokens): 49,152 for configs 2-4 and 167,936 for
config 5 (the per-layer share of a KV-only 288 GB GPU; the derivation is
checked in the tests against both sizing implementations); config 1 uses
4x the blocks it needs.  Block ids of configs 2-5 come from the library's
own block pool (kv_pool_create with the config's model shape and the
config index as shuffle seed, then kv_pool_alloc_seq per sequence in batch
order), so the allocator that serves the paper's on-demand pages is the one
that lays out every benchmark and parity batch; the ids it returns are
checked here (distinct, inside the pool) before use.  Elsewhere, and for
block_source="numpy", they are a seeded permutation of the pool (a shuffled
free list), handed out in order.  Either way every sequence's blocks are
scattered.  The numpy permutation is drawn in both cases, so Q, K and V do
not depend on the block source.

Draw order within one numpy Generator(seed): lengths, block-id permutation,
Q, K, V.  Values are N(0, 1) float32 rounded to bf16 (round-to-nearest-even).
Storage layout of one (block, KV head) tile: K token-major [16, 128], V
dims-major [128, 16] (each head dimension's 16 tokens contiguous), as the
library's interface specifies; the values are drawn token-major and V is
transposed after rounding, so the draw does not depend on the layout.
FP8 keys and values get one scale per KV head, amax / 448 over that head's
live tokens, and are clamped to +-448 before rounding to e4m3 (torch's cast
does not saturate).  With poison=True the slots past each sequence's last
token in its final block are filled with NaN codes, as are unused pool
blocks when materialised, so any read of them shows.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

BLOCK = 16
HEAD_DIM = 128
BF16_NAN = np.uint16(0x7FC0)
E4M3_NAN = np.uint8(0x7F)
E4M3_MAX = 448.0

CONFIGS = {
    1: dict(name="tiny", batch=4, n_q_heads=8, n_kv_heads=2, c_max=512, kv="bf16", lengths="uniform"),
    2: dict(name="short_pool_llama70b", batch=128, n_q_heads=64, n_kv_heads=8, c_max=8192, kv="bf16",
            lengths="lognormal", num_blocks=49152, n_layers=80),
    3: dict(name="long_pool_llama70b", batch=16, n_q_heads=64, n_kv_heads=8, c_max=65536, kv="bf16",
            lengths="pareto", num_blocks=49152, n_layers=80),
    4: dict(name="homogeneous_pool_llama70b", batch=16, n_q_heads=64, n_kv_heads=8, c_max=65536, kv="bf16",
            lengths="mixture", num_blocks=49152, n_layers=80),
    5: dict(name="short_pool_qwen3_fp8", batch=256, n_q_heads=64, n_kv_heads=4, c_max=8192, kv="fp8_e4m3",
            lengths="lognormal", num_blocks=167936, n_layers=94),
}
# The pool of configs 2-5 is one GPU's KV share: 288 GB of HBM, 90% usable,
# no weights counted (the whole budget goes to KV), model layer count and KV
# heads as above.
POOL_M_GPU_BYTES = 288e9
POOL_UTIL = 0.9


def _lognormal_ctx(rng, n, c_max=8192):
    prompt = np.clip(np.rint(rng.lognormal(math.log(600.0), 1.2, n)), 16, 8192)
    gen = rng.integers(1, 429, n)
    return np.minimum(prompt + gen, min(c_max, 8192)).astype(np.int64)


def _pareto_ctx(rng, n, lo=8192, hi=65536, alpha=1.5):
    u = rng.random(n)
    x = lo / (1.0 - u * (1.0 - (lo / hi) ** alpha)) ** (1.0 / alpha)
    return np.minimum(np.floor(x), hi).astype(np.int64)


def draw_lengths(rng, kind, n, c_max):
    if kind == "uniform":
        return rng.integers(1, c_max + 1, n).astype(np.int64)
    if kind == "lognormal":
        return _lognormal_ctx(rng, n, c_max)
    if kind == "pareto":
        return _pareto_ctx(rng, n, hi=c_max)
    if kind == "mixture":
        is_long = rng.random(n) < 0.15
        short = _lognormal_ctx(rng, n)
        long_ = _pareto_ctx(rng, n, hi=c_max)
        return np.where(is_long, long_, short).astype(np.int64)
    raise ValueError(kind)


def to_bf16_codes(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def to_e4m3_codes(x: np.ndarray) -> np.ndarray:
    """float32 -> OCP e4m3 bit patterns (uint8), saturating at +-448, round to nearest even."""
    x = np.clip(np.ascontiguousarray(x, dtype=np.float32), -E4M3_MAX, E4M3_MAX)
    t = torch.from_numpy(x).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


class BlockStore:
    """Read-only view of a paged pool [num_blocks, Hkv, ...tile] of codes that only
    materialises the blocks in use; unused blocks read back as NaN codes."""

    def __init__(self, used_ids: np.ndarray, tiles: np.ndarray, num_blocks: int, nan_code):
        self.used_ids = used_ids
        self.tiles = tiles
        self.num_blocks = num_blocks
        self.slot = np.full(num_blocks, -1, dtype=np.int64)
        self.slot[used_ids] = np.arange(len(used_ids))
        self._nan_tile = np.full((1,) + tiles.shape[1:], nan_code, dtype=tiles.dtype)
        self.dtype = tiles.dtype
        self.shape = (num_blocks,) + tiles.shape[1:]

    def __getitem__(self, ids):
        ids = np.asarray(ids, dtype=np.int64)
        slots = self.slot[ids]
        out = self.tiles[np.maximum(slots, 0)]
        if (slots < 0).any():
            out = out.copy()
            out[slots < 0] = self._nan_tile
        return out

    def dense(self) -> np.ndarray:
        """Full pool array (only for small pools)."""
        return self[np.arange(self.num_blocks)]


@dataclass
class Workload:
    config: int
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    c_max: int
    kv_format: str
    num_blocks: int
    max_blocks_per_seq: int
    context_lens: np.ndarray      # int32 [B]
    block_tables: np.ndarray      # int32 [B, max_blocks_per_seq], -1 past each sequence's blocks
    q_bits: np.ndarray            # uint16 [B, Hq, D]
    k_store: BlockStore
    v_store: BlockStore
    k_scale: np.ndarray | None    # float32 [Hkv] (fp8 only)
    v_scale: np.ndarray | None
    scale: float
    head_dim: int = HEAD_DIM
    block_size: int = BLOCK
    meta: dict = field(default_factory=dict)

    @property
    def max_context_len(self) -> int:
        return int(self.context_lens.max()) if self.batch else 0

    @property
    def kv_bytes(self) -> int:
        """Bytes of K and V one decode step must read (every cached element once)."""
        eb = 1 if self.kv_format == "fp8_e4m3" else 2
        return int(self.context_lens.astype(np.int64).sum()) * self.n_kv_heads * self.head_dim * 2 * eb


def make_workload(batch, n_q_heads, n_kv_heads, context_lens, c_max, kv_format="bf16",
                  num_blocks=None, seed=0, poison=True, config=0, name="custom", rng=None, block_ids=None):
    """Build a workload for given lengths (the rest of the draw order as documented).

    block_ids, if given, are the pool block ids of every sequence's blocks in
    batch order (as an allocator handed them out); else the seeded permutation
    supplies them."""
    rng = np.random.default_rng(seed) if rng is None else rng
    ctx = np.asarray(context_lens, dtype=np.int64)
    nblk = -(-ctx // BLOCK)
    used = int(nblk.sum())
    if num_blocks is None:
        num_blocks = max(4 * used, 1)
    if used > num_blocks:
        raise ValueError(f"batch needs {used} blocks, pool has {num_blocks}")
    max_blocks = -(-c_max // BLOCK)
    perm = rng.permutation(num_blocks).astype(np.int64)
    used_ids = perm[:used]
    if block_ids is not None:
        used_ids = np.asarray(block_ids, dtype=np.int64)
        if used_ids.shape != (used,):
            raise ValueError(f"block_ids: {used_ids.shape[0]} ids for {used} blocks")
        if used and (used_ids.min() < 0 or used_ids.max() >= num_blocks or len(np.unique(used_ids)) != used):
            raise ValueError("block_ids must be distinct ids inside the pool")
    bt = np.full((batch, max_blocks), -1, dtype=np.int32)
    off = 0
    for s in range(batch):
        bt[s, :nblk[s]] = used_ids[off:off + nblk[s]]
        off += nblk[s]
    q = rng.standard_normal((batch, n_q_heads, HEAD_DIM), dtype=np.float32)
    q_bits = to_bf16_codes(q)
    tile_shape = (used, n_kv_heads, BLOCK, HEAD_DIM)
    k = rng.standard_normal(tile_shape, dtype=np.float32)
    v = rng.standard_normal(tile_shape, dtype=np.float32)
    # live-slot mask per used tile: [used, bs]
    live = np.zeros((used, BLOCK), dtype=bool)
    off = 0
    for s in range(batch):
        for b in range(nblk[s]):
            n_live = min(BLOCK, int(ctx[s]) - b * BLOCK)
            live[off + b, :n_live] = True
        off += nblk[s]
    k_scale = v_scale = None
    if kv_format == "bf16":
        k_codes, v_codes = to_bf16_codes(k), to_bf16_codes(v)
        nan = BF16_NAN
    elif kv_format == "fp8_e4m3":
        lv = live[:, None, :, None]
        ka = np.where(lv, np.abs(k), 0).max(axis=(0, 2, 3)) if used else np.ones(n_kv_heads)
        va = np.where(lv, np.abs(v), 0).max(axis=(0, 2, 3)) if used else np.ones(n_kv_heads)
        k_scale = (np.maximum(ka, 1e-30) / E4M3_MAX).astype(np.float32)
        v_scale = (np.maximum(va, 1e-30) / E4M3_MAX).astype(np.float32)
        k_codes = to_e4m3_codes(k / k_scale[None, :, None, None])
        v_codes = to_e4m3_codes(v / v_scale[None, :, None, None])
        nan = E4M3_NAN
    else:
        raise ValueError(kv_format)
    del k, v
    v_codes = np.ascontiguousarray(v_codes.transpose(0, 1, 3, 2))   # [used, Hkv, D, bs]: dims-major V tiles
    if poison and used:
        dead_blk, dead_slot = np.nonzero(~live)
        k_codes[dead_blk, :, dead_slot, :] = nan
        v_codes[dead_blk, :, :, dead_slot] = nan
    return Workload(
        config=config, name=name, batch=batch, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
        c_max=c_max, kv_format=kv_format, num_blocks=int(num_blocks), max_blocks_per_seq=max_blocks,
        context_lens=ctx.astype(np.int32), block_tables=bt, q_bits=q_bits,
        k_store=BlockStore(used_ids, k_codes, num_blocks, nan),
        v_store=BlockStore(used_ids, v_codes, num_blocks, nan),
        k_scale=k_scale, v_scale=v_scale, scale=1.0 / math.sqrt(HEAD_DIM),
        meta=dict(used_blocks=used, seed=seed, poison=poison))


def pool_block_ids(i: int, context_lens, seed: int) -> np.ndarray:
    """Block ids of a config-i batch as the library's block pool hands them out:
    one pool sized for the config's model on one GPU, shuffled with `seed`, one
    kv_pool_alloc_seq per sequence in batch order (ids concatenated)."""
    from paper_2604_08075_amd import binding
    c = CONFIGS[i]
    pool = binding.KVPool(c["n_layers"], c["n_kv_heads"], HEAD_DIM, 1 if c["kv"] == "fp8_e4m3" else 2, c["c_max"],
                          POOL_M_GPU_BYTES, POOL_UTIL, 0.0, block_size=BLOCK, seed=seed)
    try:
        nb = pool.info().num_blocks
        if nb != c["num_blocks"]:
            raise ValueError(f"config {i}: the library's pool has {nb} blocks, expected {c['num_blocks']}")
        ids = [pool.alloc_seq(int(t)) for t in context_lens]
    finally:
        pool.close()
    return np.concatenate(ids) if ids else np.zeros(0, dtype=np.int32)


def make_config(i: int, seed: int | None = None, poison: bool = True, block_source: str | None = None) -> Workload:
    """The five benchmark configurations, seeded by their index unless told otherwise.
    block_source: "pool" (the library's block pool; default for configs 2-5) or
    "numpy" (the seeded permutation; default for config 1)."""
    c = CONFIGS[i]
    seed = i if seed is None else seed
    if block_source is None:
        block_source = "pool" if "n_layers" in c else "numpy"
    if block_source not in ("pool", "numpy"):
        raise ValueError(block_source)
    rng = np.random.default_rng(seed)
    ctx = draw_lengths(rng, c["lengths"], c["batch"], c["c_max"])
    ids = pool_block_ids(i, ctx, seed) if block_source == "pool" else None
    w = make_workload(c["batch"], c["n_q_heads"], c["n_kv_heads"], ctx, c["c_max"], c["kv"],
                      num_blocks=c.get("num_blocks"), seed=seed, poison=poison, config=i,
                      name=c["name"], rng=rng, block_ids=ids)
    w.meta["block_source"] = block_source
    return w


# Chunked-prefill workloads: each sequence's chunk is the last n tokens of its
# context (its K and V already cached).  name -> (heads, KV format, C_max, pool
# blocks, [(chunk tokens n, context tokens T)]).  The 2,048-token chunk is
# vLLM's default chunk size (Sec. 1.2); the contexts place one chunk at the
# start of a prompt and others deep into long prompts of the long pool.
PREFILL_CONFIGS = {
    "chunked_prefill_llama70b": dict(n_q_heads=64, n_kv_heads=8, kv="bf16", c_max=65536, num_blocks=49152,
                                     chunks=[(2048, 2048), (2048, 8192), (2048, 16384), (2048, 32768)]),
    "chunked_prefill_qwen3_fp8": dict(n_q_heads=64, n_kv_heads=4, kv="fp8_e4m3", c_max=8192, num_blocks=167936,
                                      chunks=[(2048, 2048), (2048, 4096), (2048, 6144), (2048, 8192)]),
}


def make_prefill(chunks, n_q_heads, n_kv_heads, c_max, kv_format="bf16", num_blocks=None, seed=0,
                 poison=True, name="custom_prefill") -> Workload:
    """A workload whose q_bits are the packed chunk queries [total_q, Hq, D] and whose
    meta["q_start"] holds the row offsets [B + 1]; contexts and KV as make_workload draws
    them (same generator, the chunk queries drawn after V)."""
    chunks = [(int(n), int(t)) for n, t in chunks]
    if any(n > t or n < 0 for n, t in chunks):
        raise ValueError("each chunk needs 0 <= n <= T")
    rng = np.random.default_rng(seed)
    w = make_workload(len(chunks), n_q_heads, n_kv_heads, [t for _, t in chunks], c_max, kv_format,
                      num_blocks=num_blocks, seed=seed, poison=poison, name=name, rng=rng)
    q_start = np.concatenate([[0], np.cumsum([n for n, _ in chunks])]).astype(np.int32)
    q = rng.standard_normal((int(q_start[-1]), n_q_heads, HEAD_DIM), dtype=np.float32)
    w.q_bits = to_bf16_codes(q)
    w.meta["q_start"] = q_start
    return w


def make_prefill_config(name: str, seed: int = 7, poison: bool = True) -> Workload:
    c = PREFILL_CONFIGS[name]
    return make_prefill(c["chunks"], c["n_q_heads"], c["n_kv_heads"], c["c_max"], c["kv"], c["num_blocks"],
                        seed=seed, poison=poison, name=name)


def to_device(w: Workload, device="cuda", layers: int = 1, poison_unused: bool = True):
    """Place a workload in device memory (torch tensors; plumbing only).

    Returns a dict with q [B, Hq, D] (bf16 codes as int16), k pools
    [layers, num_blocks, Hkv, bs, D] and v pools [layers, num_blocks, Hkv, D, bs]
    (int16 bf16 codes or uint8 e4m3 codes; every layer holds the same tiles at
    the same block ids), block_tables,
    context_lens (int32) and the fp8 scales.  Unused pool blocks are NaN codes
    when poison_unused, else left unwritten.
    """
    fp8 = w.kv_format == "fp8_e4m3"
    tdt = torch.uint8 if fp8 else torch.int16
    nan = int(E4M3_NAN) if fp8 else int(np.int16(np.uint16(BF16_NAN).view(np.int16)))
    ids = torch.from_numpy(w.k_store.used_ids).to(device)
    out = {}
    for name, store in (("k", w.k_store), ("v", w.v_store)):
        shape = (layers,) + tuple(store.shape)
        pool = torch.full(shape, nan, dtype=tdt, device=device) if poison_unused else torch.empty(
            shape, dtype=tdt, device=device)
        tiles = torch.from_numpy(store.tiles.view(np.int16) if not fp8 else store.tiles).to(device)
        for l in range(layers):
            pool[l].index_copy_(0, ids, tiles)
        out[name] = pool
        del tiles
    out["q"] = torch.from_numpy(w.q_bits.view(np.int16)).to(device)
    out["block_tables"] = torch.from_numpy(w.block_tables).to(device)
    out["context_lens"] = torch.from_numpy(w.context_lens).to(device)
    if "q_start" in w.meta:
        out["q_start"] = torch.from_numpy(w.meta["q_start"]).to(device)
    out["k_scale"] = torch.from_numpy(w.k_scale).to(device) if fp8 else None
    out["v_scale"] = torch.from_numpy(w.v_scale).to(device) if fp8 else None
    return out
