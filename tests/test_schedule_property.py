"""Property test of the block-skip scheduler (host only, no GPU): for random
valid descriptors -- packed segments of random lengths (empty ones
included) with random position bases (neat packing, Section 3.2; ring-style
offsets, Section 2.1), pieces of one sequence (zigzag chunks), causal or
not, padding rows and keys, GQA groups and dummy head slots (Section 4.1)
-- the forward and dK/dV work lists cover every allowed (row, key) pair of
every real head exactly once and no other pair, tile every row (key) of a
real head exactly once, name no dummy slot, and come longest first.  The
allowed set is the oracle's mask."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle.attention as A
import paper_2505_22296_amd as sp
from tests.helpers import lib_desc, make_shard, oracle_kw
from tests.test_abi import _coverage_from_schedule


@st.composite
def shards(draw):
    n = draw(st.integers(0, 6))
    single = n >= 1 and draw(st.booleans())
    causal = draw(st.booleans())
    lq = draw(st.lists(st.integers(0, 70), min_size=n, max_size=n))
    same = not single and draw(st.booleans())
    lk = list(lq) if same else draw(st.lists(st.integers(0, 70), min_size=n, max_size=n))
    T_q = sum(lq) + draw(st.integers(0, 20))
    T_k = sum(lk) + draw(st.integers(0, 20))

    def positions(lens, T):
        pos = np.zeros(T, np.int64)
        at, nxt = 0, draw(st.integers(0, 50))
        for ln in lens:
            base = nxt + draw(st.integers(0, 40)) if single else draw(st.integers(0, 300))
            pos[at:at + ln] = base + np.arange(ln)
            at += ln
            nxt = base + ln
        if single:  # padding after the pieces keeps rising
            pos[at:] = nxt + np.arange(T - at)
        return pos.astype(np.int32)

    pos_q, pos_k = positions(lq, T_q), positions(lk, T_k)
    spn = draw(st.sampled_from([1, 2, 4]))
    H = draw(st.integers(1, 4))
    padded = spn * H
    g = draw(st.sampled_from([1, 2, 3, 4]))
    reals = [r for r in range(max(1, padded - spn + 1), padded + 1) if r % g == 0]
    if not reals:
        g = 1
        reals = list(range(max(1, padded - spn + 1), padded + 1))
    real = draw(st.sampled_from(reals))
    rank = draw(st.integers(0, spn - 1))
    off = rank * H
    if off < real:
        last = min(off + H, real) - 1
        kv_off, Hkv = off // g, last // g - off // g + 1
    else:  # an all-dummy rank
        kv_off, Hkv = 0, 1
    D = draw(st.sampled_from([64, 128]))
    return make_shard("prop", T_q, T_k, D, H, off, real, padded, g, Hkv, kv_off, lq, lk,
                      pos_q=pos_q, pos_k=pos_k, causal=causal, single_sequence=single)


@settings(max_examples=200, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(shards())
def test_schedule_matches_the_mask(sh):
    d = lib_desc(sh)
    kw = oracle_kw(sh)
    # (pieces of one sequence are one segment to the oracle)
    seg_q, seg_k = A.segment_ids(kw["cu_q"], sh.T_q), A.segment_ids(kw["cu_k"], sh.T_k)
    mask = A.allowed_mask(np.arange(sh.T_q), seg_q, seg_k, sh.pos_q, sh.pos_k, sh.causal)
    real = [h for h in range(sh.H_loc) if sh.head_offset + h < sh.num_real_heads]
    for op, kind in ((sp.SP_OP_FWD, "rows"), (sp.SP_OP_BWD, "keys")):
        items = sp.sp_attn_schedule(d, op)
        assert set(int(h) for h in items[:, 5]) <= set(real)
        if sh.T_q > 0 and sh.T_k > 0 and mask.any():
            assert set(int(h) for h in items[:, 5]) == set(real)
        for it in items:
            assert it[6] == sh.kv_of(int(it[5]))
        cov = _coverage_from_schedule(sh, items, kind)
        for h in real:
            got = cov.get(h, np.zeros((sh.T_q, sh.T_k), np.int32))
            assert np.array_equal(got, mask.astype(np.int32)), (op, h)
        # every row (forward) / key (dK/dV) of a real head tiled at most once,
        # and the forward tiles every row once (its O / LSE get written)
        n_ax = sh.T_q if kind == "rows" else sh.T_k
        for h in real:
            cnt = np.zeros(n_ax, np.int32)
            for it in items[items[:, 5] == h]:
                cnt[it[0]:it[1]] += 1
            assert cnt.max(initial=0) <= 1, (op, h)
            if kind == "rows":
                assert np.all(cnt == 1), (op, h)
        a, b, step = (2, 3, 64) if kind == "rows" else (2, 3, 32)
        cost = np.array([-(-(int(it[b]) - (int(it[a]) & ~7)) // step) if it[b] > it[a] else 0
                         for it in items])
        for r in range(8):  # longest first on every XCD (positions 8 apart)
            assert np.all(np.diff(cost[r::8]) <= 0), (op, r, cost[r::8][:20])
        if kind == "keys":  # dealt in list order: longest first along the whole list
            assert np.all(np.diff(cost) <= 0), (op, cost[:20])


def _costs(items, kind):
    a, b, step = (2, 3, 64) if kind == "rows" else (2, 3, 32)
    return np.array([-(-(int(it[b]) - (int(it[a]) & ~7)) // step) if it[b] > it[a] else 0
                     for it in items])


def _check_cost_shares(items, cost, n_front=None):
    """For every cost value: the items of that cost on one XCD (list
    positions p with (n_front + p) % 8 == x) are one contiguous slice of that
    cost's items taken head by head, rows (keys) ascending, and the slices
    follow each other in XCD order (from XCD 0 when n_front is given, else
    from some XCD)."""
    for c in sorted(set(cost.tolist())):
        idx = np.nonzero(cost == c)[0]
        run = [tuple(int(x) for x in items[i]) for i in idx]
        enum = sorted(run, key=lambda it: (it[5], it[0], it[2]))
        slot = {it: k for k, it in enumerate(enum)}
        by_x = {}
        for i, it in zip(idx, run):
            by_x.setdefault(int(i) % 8 if n_front is None else (n_front + int(i)) % 8, []).append(it)
        order = sorted(by_x, key=lambda x: slot[by_x[x][0]])
        tiles = []
        for x in order:
            g = by_x[x]
            k0 = slot[g[0]]
            assert g == enum[k0:k0 + len(g)], (c, x)
            tiles += g
        assert tiles == enum, c
        if n_front is not None:
            assert order == sorted(order), (c, order)
        else:  # a rotation of XCD order
            assert all((order[i + 1] - order[i]) % 8 >= 1 for i in range(len(order) - 1))
            assert sum((order[i + 1] - order[i]) % 8 for i in range(len(order) - 1)) < 8


@settings(max_examples=200, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(shards())
def test_equal_costs_are_cut_per_xcd(sh):
    """Within each cost the items one XCD receives are one contiguous share
    of that cost's items, head by head (whatever the number of fill items in
    front)."""
    d = lib_desc(sh)
    for op, kind in ((sp.SP_OP_FWD, "rows"), (sp.SP_OP_BWD, "keys")):
        items = sp.sp_attn_schedule(d, op)
        _check_cost_shares(items, _costs(items, kind))


def _xcd_shard(T, causal, n_dummy, H=28, sp_n=4):
    real = H - n_dummy
    off = (sp_n - 1) * H  # the last of sp_n ranks (fewer dummies than ranks)
    return make_shard("xcd", T, T, 128, H, off, off + real, sp_n * H, 1, real, off, [T],
                      causal=causal)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n_dummy", [0, 1])
def test_xcd_shares_large(causal, n_dummy):
    """A ring-sized chunk (8192 rows and keys, 28 slots, n_dummy of them
    dummies): with the fill items in front counted, list position p runs on
    XCD (n_front + p) % 8; within each cost, XCD x holds share x of that
    cost's items (head by head); every XCD runs its share longest first."""
    T = 8192
    sh = _xcd_shard(T, causal, n_dummy)
    d = lib_desc(sh)
    # fills in front: one per dummy slot (rows); none for the keys (every
    # KV head here is read by a real head)
    for op, kind, n_front in ((sp.SP_OP_FWD, "rows", n_dummy), (sp.SP_OP_BWD, "keys", 0)):
        items = sp.sp_attn_schedule(d, op)
        cost = _costs(items, kind)
        _check_cost_shares(items, cost, n_front)
        for x in range(8):
            mine = cost[[p for p in range(len(cost)) if (n_front + p) % 8 == x]]
            assert np.all(np.diff(mine) <= 0), (op, x)
    if not causal:  # one cost: XCD x holds heads about x*real/8 .. (x+1)*real/8
        real = 28 - n_dummy
        items = sp.sp_attn_schedule(d, sp.SP_OP_FWD)
        for x in range(8):
            heads = {int(items[p, 5]) for p in range(len(items)) if (n_dummy + p) % 8 == x}
            assert len(heads) <= -(-real // 8) + 1, (x, heads)


@pytest.mark.parametrize("n_dummy", [0, 1])
def test_row_items_dealt_in_groups_of_four(n_dummy):
    """Row work lists (forward, dQ) go to each XCD in groups of four near-equal
    items -- one per shader engine, which an XCD feeds in turn -- rounds of
    eight groups alternating direction: on every XCD each full round's four
    costs are four consecutive costs of the longest-first order, and the
    XCDs' totals differ by less than the longest item.  A plain round-robin
    deal would give one XCD's engine the longest of each round."""
    T = 32768  # a 7B-like rank: 4 query slots on one causal sequence
    if n_dummy:  # rank 1 of 2: slots 4..7 of 8, slot 7 a dummy (MHA)
        sh = make_shard("g4", T, T, 128, 4, 4, 7, 8, 1, 3, 4, [T], causal=True)
    else:  # 4 query heads on one KV head
        sh = make_shard("g4", T, T, 128, 4, 0, 4, 4, 4, 1, 0, [T], causal=True)
    items = sp.sp_attn_schedule(lib_desc(sh), sp.SP_OP_FWD)
    n_front = n_dummy * -(-T // 8192)
    cost = _costs(items, "rows")
    srt = np.sort(cost)[::-1]
    spread4 = max(srt[i] - srt[i + 3] for i in range(len(srt) - 3))
    full_rounds = len(cost) // 32
    assert full_rounds >= 8
    totals = []
    for x in range(8):
        mine = cost[[p for p in range(len(cost)) if (n_front + p) % 8 == x]]
        totals.append(int(mine.sum()))
        for r in range(full_rounds):
            grp = mine[4 * r:4 * r + 4]
            assert grp.max() - grp.min() <= spread4, (x, r, grp)
    assert max(totals) - min(totals) < cost.max(), totals
    # and it matters: under round-robin the first four of an XCD are 8 apart
    plain = srt[0:32:8]
    assert plain.max() - plain.min() > spread4


@settings(max_examples=200, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(shards())
def test_causal_row_tiles_end_at_the_segment_end(sh):
    """Forward row tiles of a causal segment end at its end: every tile has
    the full 256 rows except the segment's first, which holds the remainder
    (its rows see the fewest keys); non-causal tiles start at the segment's
    start."""
    if sh.single_sequence:
        return
    d = lib_desc(sh)
    items = sp.sp_attn_schedule(d, sp.SP_OP_FWD)
    real = [h for h in range(sh.H_loc) if sh.head_offset + h < sh.num_real_heads]
    for h in real:
        mine = items[items[:, 5] == h]
        for s in range(len(sh.cu_q) - 1):
            a, b = int(sh.cu_q[s]), int(sh.cu_q[s + 1])
            tiles = sorted((int(it[0]), int(it[1])) for it in mine if a <= it[0] < b)
            n = b - a
            if n == 0:
                assert tiles == []
                continue
            first = n % 256 if (sh.causal and n % 256) else min(256, n)
            expect, at = [], a
            while at < b:
                end = min(b, at + (first if at == a else 256))
                expect.append((at, end))
                at = end
            assert tiles == expect, (s, tiles[:3], expect[:3])


@pytest.mark.parametrize("causal", [True, False])
def test_row_tiles_of_long_segments(causal):
    """The same property on segments longer than a tile (the drawn shards'
    segments are shorter than one): 300, 700, 256, 1000 and 5 rows."""
    lens = [300, 700, 256, 1000, 5]
    T = sum(lens) + 40
    sh = make_shard("long_segs", T, T, 128, 2, 0, 2, 2, 1, 2, 0, lens, causal=causal)
    items = sp.sp_attn_schedule(lib_desc(sh), sp.SP_OP_FWD)
    starts = np.concatenate([[0], np.cumsum(lens)])
    for h in range(2):
        got = sorted((int(it[0]), int(it[1])) for it in items[items[:, 5] == h])
        want = []
        for a, n in zip(starts[:-1], lens):
            first = n % 256 if causal and n % 256 else 256
            bounds = [0] + list(range(first, n, 256)) + [n]
            want += [(int(a + x), int(a + y)) for x, y in zip(bounds[:-1], bounds[1:])]
        want.append((int(starts[-1]), T))  # the padding rows: one item, rows see no key
        assert got == sorted(want), (h, got, want)
    if causal:  # the partial tiles are the segments' first
        assert (300, 300 + 188) in got and (0, 44) in got
