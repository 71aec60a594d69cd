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
FAN_IN = 16             # workgroup pieces per merge group


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
                return  # whole segment: written straight to the output
            slot = 2 * gw + (0 if state["piece_first"] else 1)
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
                records=records, pieces=pieces, max_blocks_per_seq=max_blocks_per_seq)


def check(sim, hkv):
    B, TW, C, pre = sim["B"], sim["TW"], sim["C"], sim["pre"]
    for s, g in sim["q_rows"]:
        assert 0 <= s < B and 0 <= g < hkv, (s, g)
    for s, blk, nb in sim["bt_reads"]:
        assert 0 <= blk < nb <= sim["max_blocks_per_seq"], (s, blk, nb)
    assert sorted(sim["computed"]) == list(range(sim["U"]))
    counters_group, counters_seg = set(), set()
    nwg = TW // WAVES
    CW = WAVES * C
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
        # stage 2: workgroup pieces, groups of FAN_IN, device-wide counters per workgroup
        bk0, bkend = a0 // CW, (a0 + nus - 1) // CW
        nwp = bkend - bk0 + 1
        if nwp == 1:
            continue
        first_wslot = 2 * bk0 + (1 if a0 > bk0 * CW else 0)
        assert 2 * TW + first_wslot < 2 * TW + 2 * nwg and 2 * TW + 2 * bkend < 2 * TW + 2 * nwg
        for gfirst in range(0, nwp, FAN_IN):
            gn = min(nwp, gfirst + FAN_IN) - gfirst
            kg = bk0 + gfirst + gn - 1
            assert 0 <= kg < nwg and 2 * TW + 2 * nwg + kg < 3 * TW
            assert kg not in counters_group
            counters_group.add(kg)
        assert 0 <= bkend < nwg and bkend not in counters_seg
        counters_seg.add(bkend)
    for slot in sim["records"]:
        assert 0 <= slot < 2 * TW
    # stage 1: every share of a workgroup goes to exactly one of its waves, no
    # wave gets more than two (the kernel holds two), and the first and last
    # shares, the only ones that can cross the workgroup's edges, go to
    # different waves
    for b, entries in workgroup_entries(sim).items():
        segs = [e for e in entries if e is not None]
        runs = [seg for i, seg in enumerate(segs) if i == 0 or seg != segs[i - 1]]
        assert len(runs) == len(set(runs)) <= WAVES + 1
        got = assign_shares(entries)
        assert sorted(x for v in got.values() for x in v) == sorted(runs)
        assert all(len(v) <= 2 for v in got.values())
        if len(runs) >= 2:
            assert [w for w, v in got.items() if runs[0] in v] != [w for w, v in got.items() if runs[-1] in v]
        for seg in runs:  # a share that crosses an edge of the workgroup is its first or last
            others = [k for k, _ in sim["pieces"][seg] if k // WAVES != b]
            if others:
                assert seg in (runs[0], runs[-1])


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

def assign_shares(entries):
    """The kernel's split of a workgroup's shares over its waves.  entries[2w + x]
    is the segment of wave w's first (x = 0) or last (x = 1) split piece, or
    None.  Shares are the runs of equal segments among the entries, in order;
    share i goes to wave min(pos, WAVES - 1), pos = 0 for the first, 1 for the
    last, i + 1 for the others."""
    starts, prev = [], None
    for e, seg in enumerate(entries):
        if seg is None:
            continue
        if seg != prev:
            starts.append(e)
        prev = seg
    out = {w: [] for w in range(WAVES)}
    for i, e in enumerate(starts):
        pos = 0 if i == 0 else (1 if i == len(starts) - 1 else i + 1)
        out[min(pos, WAVES - 1)].append(entries[e])
    return out


def workgroup_entries(sim):
    """entries (as assign_shares takes them) of every workgroup that has units."""
    C, U = sim["C"], sim["U"]
    nwg = sim["TW"] // WAVES
    ents = {b: [None] * (2 * WAVES) for b in range(nwg) if b * WAVES * C < U}
    for seg, got in sim["pieces"].items():
        for k, slot in got:
            ents[k // WAVES][2 * (k % WAVES) + (slot & 1)] = seg
    return ents


def run_merge_protocol(sim, rng):
    """Play the kernel's end-of-slice protocol for every split piece, with the
    waves' steps interleaved in a random order, and check that every cut
    segment is written exactly once, that no merge reads a record before it
    is published, and that every counter is zero afterwards.

    Per wave, as the kernel orders it.  Stage 1: each split piece's record is
    in its owner's LDS; the workgroup's waves meet at a barrier (a wave
    without units too); then each share of a cut segment is merged by the
    wave assign_shares gives it, which folds the share's pieces.  A segment
    inside the workgroup is then written.  Stage 2, for a share of a segment
    that crosses workgroups: read the group counter (an atomic load); unless
    it shows every other workgroup piece of the group arrived, publish the
    workgroup piece and count it; the group's last arrival folds the group
    and either writes the segment or goes through the segment counter (load,
    then group record and increment unless every other group is done).  Last,
    after a step of its own, the wave returns to zero every device-wide
    counter it was the last arrival of.  No wave may read or count a counter
    between its last arrival and that reset."""
    C, pre, hkv = sim["C"], sim["pre"], sim["hkv"]
    CW = WAVES * C
    info_of = {}  # (workgroup, segment) -> the share's stage-2 facts
    pieces_of = {}  # wave -> its split pieces' segments
    for (s, g), got in sim["pieces"].items():
        nus = pre[s + 1] - pre[s]
        a0 = hkv * pre[s] + g * nus
        bk0, bkend = a0 // CW, (a0 + nus - 1) // CW
        nwp = bkend - bk0 + 1
        for k, _ in got:
            b = k // WAVES
            rb = b - bk0
            gfirst = rb - rb % FAN_IN
            gn = min(nwp, gfirst + FAN_IN) - gfirst
            info_of[(b, (s, g))] = dict(seg=(s, g), nwp=nwp, rb=rb, gfirst=gfirst, gn=gn,
                                        kg=bk0 + gfirst + gn - 1, ngroups=-(-nwp // FAN_IN), bkend=bkend)
            pieces_of.setdefault(k, []).append((s, g))
    ents = workgroup_entries(sim)
    group_cnt, seg_cnt = {}, {}
    published_local, wg_published, group_published, written = set(), set(), set(), {}
    done_group, done_seg = set(), set()  # counters whose last arrival has come, not yet reset
    at_barrier = {b: 0 for b in ents}

    def read(cnt, done, k):
        assert k not in done, f"counter {k} read after its last arrival"
        return cnt.get(k, 0)

    def steps_of(w):
        b = w // WAVES
        for seg in pieces_of.get(w, []):
            published_local.add((seg, w))
            yield
        at_barrier[b] += 1
        while at_barrier[b] < WAVES:
            yield
        resets = []
        for seg in assign_shares(ents[b])[w % WAVES]:
            info = info_of[(b, seg)]
            for k in range(b * WAVES, b * WAVES + WAVES):
                if seg in pieces_of.get(k, []):
                    assert (seg, k) in published_local, f"share of {seg} read piece of wave {k} before it was published"
            yield
            if info["nwp"] == 1:
                written[seg] = written.get(seg, 0) + 1
                continue
            c = read(group_cnt, done_group, info["kg"])
            yield
            if c != info["gn"] - 1:
                wg_published.add((seg, info["rb"]))
                old = read(group_cnt, done_group, info["kg"])
                group_cnt[info["kg"]] = old + 1
                yield
                if old != info["gn"] - 1:
                    continue
            for u in range(info["gn"]):
                rb = info["gfirst"] + u
                if rb != info["rb"]:
                    assert (seg, rb) in wg_published, f"group of {seg} read workgroup piece {rb} before it was published"
            done_group.add(info["kg"])
            resets.append((group_cnt, done_group, info["kg"]))
            if info["ngroups"] == 1:
                written[seg] = written.get(seg, 0) + 1
                continue
            c_own = info["gfirst"] // FAN_IN
            if read(seg_cnt, done_seg, info["bkend"]) != info["ngroups"] - 1:
                group_published.add((seg, c_own))
                old = read(seg_cnt, done_seg, info["bkend"])
                seg_cnt[info["bkend"]] = old + 1
                yield
                if old != info["ngroups"] - 1:
                    continue
            for c in range(info["ngroups"]):
                if c != c_own:
                    assert (seg, c) in group_published, f"{seg}: group {c} read before it was published"
            done_seg.add(info["bkend"])
            resets.append((seg_cnt, done_seg, info["bkend"]))
            written[seg] = written.get(seg, 0) + 1
        # the device-wide counters this wave was the last arrival of return to zero
        yield
        for cnt, done, k in resets:
            cnt[k] = 0
            done.discard(k)

    live = {w: steps_of(w) for b in ents for w in range(b * WAVES, b * WAVES + WAVES)}
    while live:
        w = list(live)[int(rng.integers(0, len(live)))]
        try:
            next(live[w])
        except StopIteration:
            del live[w]
    assert written == {seg: 1 for seg in sim["pieces"]}, "a cut segment was written other than once"
    assert all(v == 0 for v in group_cnt.values()) and all(v == 0 for v in seg_cnt.values())
    assert not done_group and not done_seg


@pytest.mark.parametrize("trial", range(30))
def test_merge_protocol_any_arrival_order(trial):
    """Random batches (segments inside one workgroup, across a few, and across
    more than sixteen, which merge on two levels) under random interleavings
    of the waves' steps."""
    rng = np.random.default_rng(7000 + trial)
    fp8 = bool(trial % 2)
    B = int(rng.choice([2, 5, 16, 40]))
    hkv = int(rng.choice([1, 2, 4]))
    max_ctx = int(rng.choice([300, 3000, 20000]))
    ctx = draw(rng, B, max_ctx, 0.2)
    cus = int(rng.choice([2, 8, 32, 96]))
    sim = simulate(ctx, hkv, fp8, max_ctx, -(-max_ctx // 16), 0, 0, cus)
    sim["hkv"] = hkv
    for rep in range(3):
        run_merge_protocol(sim, np.random.default_rng(rep + 10 * trial))


@pytest.mark.parametrize("trial", range(6))
def test_merge_protocol_two_levels(trial):
    """One long sequence cut across 64 workgroups (groups of sixteen workgroup
    pieces, then the groups) beside short ones, under random interleavings."""
    rng = np.random.default_rng(7100 + trial)
    ctx = [60000] + list(rng.integers(1, 3000, 7))
    sim = simulate(ctx, 1, bool(trial % 2), 60000, 3750, 0, 0, 64)
    sim["hkv"] = 1
    C, pre = sim["C"], sim["pre"]
    assert -(-(pre[1] - pre[0]) // (WAVES * C)) > FAN_IN  # the long segment spans more than one group
    for rep in range(3):
        run_merge_protocol(sim, np.random.default_rng(rep + 10 * trial))


def div_small(a, d):
    """The kernel's a / d for quotients below 2^22: the float32 product of a
    and the rounded reciprocal, truncated, then one correction step."""
    rd = np.float32(1.0) / np.float32(d)
    q = int(np.float32(np.float32(a) * rd))
    r = a - q * d
    return q + (1 if r >= d else 0) - (1 if r < 0 else 0)


def test_div_small_exact():
    """Exact for every divisor and dividend the merge uses: slice sizes C and
    4C up to the largest streams (4096 sequences of 65,536 tokens, 16 KV heads
    is 2^27 units), quotients up to the number of waves; edges at exact
    multiples, one below and one above them included."""
    rng = np.random.default_rng(11)
    cases = []
    for d in list(range(1, 300)) + [int(x) for x in rng.integers(1, 1 << 27, 3000)]:
        qmax = min((1 << 27) // d + 1, (1 << 22) - 1)
        for q in [0, 1, 2, qmax - 1, qmax] + [int(x) for x in rng.integers(0, qmax + 1, 8)]:
            for a in (q * d - 1, q * d, q * d + 1, q * d + d - 1):
                if 0 <= a < (1 << 31) and a // d < (1 << 22):
                    cases.append((a, d))
    for a, d in cases:
        assert div_small(a, d) == a // d, (a, d)
