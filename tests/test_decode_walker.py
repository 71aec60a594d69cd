"""CPU check of the decode kernel's index arithmetic (no GPU).

The decode kernel walks a flat stream of 16 KiB units (every cached token of
every (sequence, KV head) segment) in equal per-wave slices, prefetches the
query group of the unit after next, and merges the pieces of segments that
slices cut through arrival counters and record slots in its workspace.  This
module restates that arithmetic in Python, step for step as the kernel and
its host launcher do it, and checks on random batches that

  * every query row the kernel loads (including look-ahead prefetches past the
    end of the stream) lies inside the [batch, n_q_heads, 128] query buffer;
  * every block-table entry read is one of the sequence's own live blocks, and
    every tile index lies inside the pool;
  * the slices cover every unit exactly once, the walker's position always
    equals the position of the unit it computes, and no slice exceeds the
    kernel's tile list;
  * every piece of a cut segment writes the record slot its merger reads, the
    arrival counters and record slots stay inside the workspace, and no two
    (segment, group) pairs share a counter;
  * the end-of-slice protocol (counters read first, records published before
    they are counted, the last arrival merging) writes every cut segment once,
    never reads an unpublished record and leaves every counter at zero, under
    any interleaving of the waves' steps.

A kernel change to any of these must be mirrored here.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

WAVES = 4               # waves per workgroup
MAX_UNITS_PER_WAVE = 256
FAN_IN = 8              # pieces per merge group


def host_plan(ctx, hkv, fp8, max_ctx, partition_tokens=0, wgs_per_cu=0, cus=256, resident=2):
    """Grid and minimum slice length as the launcher chooses them."""
    unit = 64 if fp8 else 32
    min_chunk = partition_tokens // unit if partition_tokens else 1
    max_units = -(-max_ctx // unit) * len(ctx) * hkv
    per_cu = min(wgs_per_cu, resident) if wgs_per_cu else 1
    grid = cus * per_cu
    need = -(-max_units // (WAVES * MAX_UNITS_PER_WAVE))
    useful = -(-max_units // (WAVES * min_chunk))
    return max(1, max(need, min(grid, useful))), min_chunk, unit


class Walk:
    __slots__ = ("s", "g", "j", "nus")

    def __init__(self, s, g, j, nus):
        self.s, self.g, self.j, self.nus = s, g, j, nus

    def copy(self):
        return Walk(self.s, self.g, self.j, self.nus)

    def key(self):
        return (self.s, self.g, self.j)


def simulate(ctx, hkv, fp8, max_ctx, max_blocks_per_seq, partition_tokens=0, wgs_per_cu=0, cus=256):
    """Run the kernel's index arithmetic; returns what it touched."""
    B = len(ctx)
    grid, min_chunk, UT = host_plan(ctx, hkv, fp8, max_ctx, partition_tokens, wgs_per_cu, cus)
    UB = UT // 16
    ctx = [min(max(int(c), 0), max_ctx) for c in ctx]
    pre = [0]
    for c in ctx:
        pre.append(pre[-1] + -(-c // UT))
    U = hkv * pre[B]
    TW = grid * WAVES
    C = max(-(-U // TW), min_chunk)

    def locate(u):  # binary search of the kernel: largest s with Hkv * pre[s] <= u
        lo, hi = 0, B - 1
        while lo < hi:
            mid = (lo + hi + 1) >> 1
            if hkv * pre[mid] <= u:
                lo = mid
            else:
                hi = mid - 1
        s = lo
        nus = pre[s + 1] - pre[s]
        r = u - hkv * pre[s]
        return Walk(s, r // nus, r % nus, nus)

    def advance(wk):
        wk.j += 1
        if wk.j == wk.nus:
            wk.j = 0
            wk.g += 1
            if wk.g == hkv:
                wk.g = 0
                while True:
                    wk.s += 1
                    if not (wk.s < B - 1 and pre[wk.s + 1] == pre[wk.s]):
                        break
                wk.s = min(wk.s, B - 1)
            wk.nus = pre[wk.s + 1] - pre[wk.s]

    q_rows, bt_reads, computed = [], [], []
    records = {}        # record slot -> (s, g, piece index r)
    pieces = {}         # (s, g) -> list of (wave, slot)
    staged = {}         # wave -> its staging entries in order: ("row", None) or ("rec", slot)
    for gw in range(TW):
        u0 = gw * C
        u1 = min(u0 + C, U)
        if u0 >= u1:
            continue
        n = u1 - u0
        assert n <= MAX_UNITS_PER_WAVE
        # tile list
        for i in range(n):
            p = locate(u0 + i)
            nb = -(-ctx[p.s] // 16)
            for b in range(UB):
                blk = p.j * UB + (b if p.j * UB + b < nb else 0)
                bt_reads.append((p.s, blk, nb))
        # walk
        cs = locate(u0)
        w1 = cs.copy()
        advance(w1)
        w2 = w1.copy()
        advance(w2)
        q_rows += [(cs.s, cs.g), (w1.s, w1.g)]
        state = {"piece_first": True, "piece_j0": 0}

        def compute(ui, cs):
            assert cs.key() == locate(u0 + ui).key()
            computed.append(u0 + ui)
            if ui == 0 or cs.j == 0:
                state["piece_first"] = ui == 0
                state["piece_j0"] = cs.j
            seg_end = cs.j == cs.nus - 1
            if not (seg_end or ui == n - 1):
                return
            if state["piece_j0"] == 0 and seg_end:
                staged.setdefault(gw, []).append(("row", None))
                return  # whole segment: its rows, staged then written to the output
            slot = 2 * gw + (0 if state["piece_first"] else 1)
            staged.setdefault(gw, []).append(("rec", slot))
            assert slot not in records
            records[slot] = (cs.s, cs.g)
            pieces.setdefault((cs.s, cs.g), []).append((gw, slot))

        ui = 0
        while ui + 2 < n:
            for d in (0, 1):
                compute(ui + d, cs)
                if w2.j == 0:
                    q_rows.append((w2.s, w2.g))
                cs, w1 = w1, w2.copy()
                advance(w2)
            ui += 2
        if ui + 1 < n:
            compute(ui, cs)
            if w2.j == 0:
                q_rows.append((w2.s, w2.g))
            cs, w1 = w1, w2.copy()
            advance(w2)
            ui += 1
        compute(ui, cs)
    return dict(B=B, TW=TW, C=C, U=U, pre=pre, q_rows=q_rows, bt_reads=bt_reads, computed=computed,
                records=records, pieces=pieces, max_blocks_per_seq=max_blocks_per_seq, staged=staged)


STAGE_BYTES, MAX_STAGED = 24 * 1024, 6      # a wave's LDS staging area: bytes and entries
ROW_BYTES, REC_BYTES = 4096, 8192 + 512     # one (sequence, KV head)'s bf16 rows; one record (o, m, l)


def flushed_mid_loop(entries, row_bytes=ROW_BYTES):
    """Record slots a wave's staging writes out before its slice ends: the
    kernel flushes every staged entry when the next one would not fit."""
    out, st_n, st_off, pending = set(), 0, 0, []
    for kind, slot in entries:
        size = row_bytes if kind == "row" else REC_BYTES
        if st_n == MAX_STAGED or st_off + size > STAGE_BYTES:
            out |= {x for x in pending if x is not None}
            st_n, st_off, pending = 0, 0, []
        st_n, st_off = st_n + 1, st_off + size
        pending.append(slot)
    return out


def check(sim, hkv):
    B, TW, C, pre = sim["B"], sim["TW"], sim["C"], sim["pre"]
    for s, g in sim["q_rows"]:
        assert 0 <= s < B and 0 <= g < hkv, (s, g)
    for s, blk, nb in sim["bt_reads"]:
        assert 0 <= blk < nb <= sim["max_blocks_per_seq"], (s, blk, nb)
    assert sorted(sim["computed"]) == list(range(sim["U"]))
    counters_group, counters_seg = set(), set()
    for (s, g), got in sim["pieces"].items():
        nus = pre[s + 1] - pre[s]
        a0 = hkv * pre[s] + g * nus
        k0, kend = a0 // C, (a0 + nus - 1) // C
        np_ = kend - k0 + 1
        assert np_ >= 2 and len(got) == np_
        first_slot = 2 * k0 + (1 if a0 > k0 * C else 0)
        by_wave = dict(got)
        assert sorted(by_wave) == list(range(k0, kend + 1))
        for r in range(np_):
            assert by_wave[k0 + r] == (first_slot if r == 0 else 2 * (k0 + r))
        for gfirst in range(0, np_, FAN_IN):
            gn = min(np_, gfirst + FAN_IN) - gfirst
            kg = k0 + gfirst + gn - 1
            assert 0 <= kg < TW and 2 * TW + kg < 3 * TW
            assert kg not in counters_group
            counters_group.add(kg)
        assert 0 <= kend < TW and kend not in counters_seg
        counters_seg.add(kend)
    for slot in sim["records"]:
        assert 0 <= slot < 2 * TW


def draw(rng, B, max_ctx, p_empty):
    ctx = rng.integers(1, max_ctx + 1, B)
    ctx[rng.random(B) < p_empty] = 0
    return ctx


def test_reported_case_stays_in_bounds():
    """Four sequences, two KV heads, whose last wave ends on the last sequence's
    last unit: its look-ahead positions stay on that sequence."""
    ctx = [100, 300, 50, 700]
    sim = simulate(ctx, 2, False, 700, 44)
    check(sim, 2)
    assert max(s for s, _ in sim["q_rows"]) == 3


@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("trial", range(40))
def test_random_batches(fp8, trial):
    rng = np.random.default_rng(1000 + trial + 100 * fp8)
    B = int(rng.choice([1, 2, 3, 5, 17, 64, 300]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    max_ctx = int(rng.choice([16, 64, 200, 2048, 9000]))
    ctx = draw(rng, B, max_ctx, float(rng.choice([0.0, 0.3, 0.9])))
    unit = 64 if fp8 else 32
    P = int(rng.choice([0, unit, 4 * unit, 64 * unit]))
    cus = int(rng.choice([1, 3, 8, 256]))
    wgs = int(rng.choice([0, 1, 2]))
    sim = simulate(ctx, hkv, fp8, max_ctx, -(-max_ctx // 16), P, wgs, cus)
    check(sim, hkv)


@pytest.mark.parametrize("ctx", [[0], [0, 0, 5], [7, 0, 0], [1], [16] * 9, [33, 0, 64, 0]])
def test_empty_and_tiny_batches(ctx):
    for fp8 in (False, True):
        for cus in (1, 256):
            sim = simulate(ctx, 2, fp8, max(max(ctx), 1), 8, cus=cus)
            check(sim, 2)


def test_benchmark_shapes():
    """The short, long, homogeneous and fp8 pools' length recipes at full batch size."""
    rng = np.random.default_rng(5)
    for B, hkv, fp8, cmax in ((128, 8, False, 8192), (16, 8, False, 65536), (256, 4, True, 8192)):
        prompt = np.clip(np.rint(rng.lognormal(math.log(600.0), 1.2, B)), 16, 8192)
        ctx = np.minimum(prompt + rng.integers(1, 429, B), cmax).astype(int)
        if cmax == 65536:
            ctx = np.maximum(ctx, rng.integers(8192, 42000, B))
        sim = simulate(ctx, hkv, fp8, int(ctx.max()), cmax // 16)
        check(sim, hkv)


# ---------------------------------------------------------------- end-of-slice merge protocol

def run_merge_protocol(sim, rng, p_staged=0.8):
    """Play the kernel's end-of-slice protocol for every split piece, with the
    waves' steps interleaved in a random order, and check that every cut
    segment is written exactly once, that no merge reads a record before it
    is published, and that every counter is zero afterwards.

    Per wave, as the kernel orders it: read both group counters (atomic
    loads) for pieces whose record is still staged in LDS; publish and count
    the pieces that were not found to be the group's last; count the pieces
    of segments that lie inside one workgroup on that workgroup's counter
    (their last arrival writes the segment, and they touch no global
    counter); then, piece by
    piece, the group's last arrival merges the group and either writes the
    segment or goes through the segment counter (load, then group record and
    increment unless every other group is done); last, after a step of its
    own, the wave returns to zero every counter it was the last arrival of.
    No wave may read or count a counter between its last arrival and that
    reset."""
    C, pre = sim["C"], sim["pre"]
    hkv = sim["hkv"]
    seg_of_piece = {}
    waves = {}
    for (s, g), got in sim["pieces"].items():
        nus = pre[s + 1] - pre[s]
        a0 = hkv * pre[s] + g * nus
        k0, kend = a0 // C, (a0 + nus - 1) // C
        np_ = kend - k0 + 1
        for r in range(np_):
            gfirst = r - r % FAN_IN
            gn = min(np_, gfirst + FAN_IN) - gfirst
            info = dict(seg=(s, g), r=r, gfirst=gfirst, gn=gn, kg=k0 + gfirst + gn - 1, ngroups=-(-np_ // FAN_IN),
                        kend=kend, np=np_, k0=k0, local=k0 // WAVES == kend // WAVES)
            w = k0 + r
            seg_of_piece[(w, r == 0)] = info
            waves.setdefault(w, []).append(info)
    group_cnt, seg_cnt, wg_cnt = {}, {}, {}
    published, group_published, written = set(), set(), {}
    published_local = set()  # pieces of segments merged inside their workgroup
    done_group, done_seg = set(), set()  # counters whose last arrival has come, not yet reset

    def read(cnt, done, k):
        assert k not in done, f"counter {k} read after its last arrival"
        return cnt.get(k, 0)

    def merge_group(info, own):
        seg = info["seg"]
        for u in range(info["gn"]):
            r = info["gfirst"] + u
            if not (own and r == info["r"]):
                assert (seg, r) in published, f"merge of {seg} read piece {r} before it was published"
        done_group.add(info["kg"])

    def steps_of(w):
        pieces = sorted(waves[w], key=lambda i: i["r"] != 0)  # the slice's first piece, then its last
        staged = [bool(rng.random() < p_staged) for _ in pieces]
        mine = [False] * len(pieces)
        # 1. atomic loads of the group counters (records still in LDS); pieces
        # of segments inside one workgroup take no part in the global protocol
        for x, info in enumerate(pieces):
            if staged[x] and not info["local"]:
                mine[x] = read(group_cnt, done_group, info["kg"]) == info["gn"] - 1
        yield
        # 2. publish and count the others
        last = [False] * len(pieces)
        for x, info in enumerate(pieces):
            if not mine[x] and not info["local"]:
                published.add((info["seg"], info["r"]))
                old = read(group_cnt, done_group, info["kg"])
                group_cnt[info["kg"]] = old + 1
                last[x] = old == info["gn"] - 1
                yield
        # 2b. segments inside the workgroup: publish the record's place, count
        # on the workgroup's counter (keyed by the segment's first wave); the
        # last arrival folds every piece and writes the segment
        for x, info in enumerate(pieces):
            if not info["local"]:
                continue
            seg = info["seg"]
            published_local.add((seg, info["r"]))
            key = (info["k0"] // WAVES, info["k0"])
            old = wg_cnt.get(key, 0)
            wg_cnt[key] = old + 1
            if old == info["np"] - 1:
                for r in range(info["np"]):
                    assert (seg, r) in published_local, f"local merge of {seg} read piece {r} before it was published"
                written[seg] = written.get(seg, 0) + 1
            yield
        # 3. merges
        resets = []
        for x, info in enumerate(pieces):
            if info["local"] or not (mine[x] or last[x]):
                continue
            merge_group(info, mine[x])
            resets.append((group_cnt, done_group, info["kg"]))
            yield
            seg = info["seg"]
            if info["ngroups"] == 1:
                written[seg] = written.get(seg, 0) + 1
                continue
            c_own = info["gfirst"] // FAN_IN
            if read(seg_cnt, done_seg, info["kend"]) == info["ngroups"] - 1:
                for c in range(info["ngroups"]):
                    if c != c_own:
                        assert (seg, c) in group_published, f"{seg}: group {c} read before it was published"
                done_seg.add(info["kend"])
                resets.append((seg_cnt, done_seg, info["kend"]))
                written[seg] = written.get(seg, 0) + 1
                continue
            group_published.add((seg, c_own))
            old = read(seg_cnt, done_seg, info["kend"])
            seg_cnt[info["kend"]] = old + 1
            yield
            if old == info["ngroups"] - 1:
                for c in range(info["ngroups"]):
                    assert (seg, c) in group_published
                done_seg.add(info["kend"])
                resets.append((seg_cnt, done_seg, info["kend"]))
                written[seg] = written.get(seg, 0) + 1
        # 4. the counters this wave was the last arrival of return to zero
        yield
        for cnt, done, k in resets:
            cnt[k] = 0
            done.discard(k)

    live = {w: steps_of(w) for w in waves}
    while live:
        w = list(live)[int(rng.integers(0, len(live)))]
        try:
            next(live[w])
        except StopIteration:
            del live[w]
    assert written == {seg: 1 for seg in sim["pieces"]}, "a cut segment was written other than once"
    assert all(v == 0 for v in group_cnt.values()) and all(v == 0 for v in seg_cnt.values())
    assert not done_group and not done_seg
    # every local counter saw exactly its segment's pieces (no reset needed:
    # the counters live in LDS for one launch)
    for (wg, k0), v in wg_cnt.items():
        assert v == next(i["np"] for ws in waves.values() for i in ws if i["k0"] == k0 and i["local"])


@pytest.mark.parametrize("fp8", [False, True])
def test_largest_batch_reaches_both_local_merge_sources(fp8):
    """The GPU test of the largest batch (4,096 short contexts, 2 KV heads)
    merges segments cut inside one workgroup from both places a piece's record
    can be: still in its owner's LDS staging area, and in its global slot after
    a mid-loop flush.  Replays that batch's slices and staging here."""
    rng = np.random.default_rng(31)
    ctx = rng.integers(0, 97, 4096)
    ctx[rng.integers(0, 4096, 64)] = 0
    sim = simulate(list(ctx), 2, fp8, int(ctx.max()), 8)  # the workload's max_context_len and table width
    check(sim, 2)
    flushed = set()
    for entries in sim["staged"].values():
        flushed |= flushed_mid_loop(entries)
    C, pre = sim["C"], sim["pre"]
    in_lds = in_slot = 0
    for (s_, g), got in sim["pieces"].items():
        nus = pre[s_ + 1] - pre[s_]
        a0 = 2 * pre[s_] + g * nus
        k0, kend = a0 // C, (a0 + nus - 1) // C
        if k0 // WAVES != kend // WAVES:
            continue
        for _, slot in got:
            if slot in flushed:
                in_slot += 1
            else:
                in_lds += 1
    assert in_lds > 0 and in_slot > 0, (in_lds, in_slot)


@pytest.mark.parametrize("trial", range(30))
def test_merge_protocol_any_arrival_order(trial):
    """Random batches (including long segments cut into more than eight pieces,
    which merge on two levels) under random interleavings of the waves' steps."""
    rng = np.random.default_rng(7000 + trial)
    fp8 = bool(trial % 2)
    B = int(rng.choice([2, 5, 16, 40]))
    hkv = int(rng.choice([1, 2, 4]))
    max_ctx = int(rng.choice([300, 3000, 20000]))
    ctx = draw(rng, B, max_ctx, 0.2)
    cus = int(rng.choice([2, 8, 32]))
    sim = simulate(ctx, hkv, fp8, max_ctx, -(-max_ctx // 16), 0, 0, cus)
    sim["hkv"] = hkv
    for rep in range(3):
        run_merge_protocol(sim, np.random.default_rng(rep + 10 * trial), p_staged=float(rng.choice([0.0, 0.5, 1.0])))
