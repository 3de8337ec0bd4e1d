"""CPU simulation of the persistent item scheduler (no GPU needed).

The kernels hand out work items by rank: GEMM1 items (in the order table's
order) then, in the pipelined launch, GEMM2 items.  Work-group g claims from
list g % L, which hands out the ranks congruent to its index modulo L in
increasing order (L = min(8, grid): one list per XCD).  Split-K parts never
wait for each other: each counts its arrival and the last one to arrive
finishes the tile (a GEMM1 tile then signals its ready counter).  A GEMM2 item
waits for the GEMM1 tiles of its K range; a work-group claims its next item
after the last wait of its current one.  The claim in the design is that
every launch finishes for any grid of at least one work-group, because every
wait targets a lower rank.  This simulates that protocol with random item
durations and checks it, and checks that a rank order putting consumers
before their producers can deadlock.
"""
import random

import pytest


def xcd_grouped(Mb, N, wave):
    """The host's XCD-grouped deal: waves of whole column blocks, cut into 8
    near-square sub-blocks (one per XCD, walked column-first); within a wave,
    rank 8 j + x is the j-th tile of sub-block x, and exhausted sub-blocks
    close up."""
    out = []
    C = max(1, wave // Mb)
    for c0 in range(0, N, C):
        cw = min(C, N - c0)
        r = min((r for r in (1, 2, 4, 8) if r <= Mb), key=lambda r: -(-Mb // r) + -(-cw // (8 // r)))
        rows, cols = -(-Mb // r), -(-cw // (8 // r))
        per = [[] for _ in range(8)]
        for x in range(8):
            rg, cg = x % r, x // r
            for nb in range(c0 + cg * cols, min(c0 + cw, c0 + (cg + 1) * cols)):
                per[x] += [nb * Mb + mb for mb in range(rg * rows, min(Mb, (rg + 1) * rows))]
        for j in range(max(len(p) for p in per)):
            out += [p[j] for p in per if j < len(p)]
    return out


def column_first_tiles(Mb, Nb1, order, seed=12345, S2=1, wave=16):
    if order == "xcd":
        return xcd_grouped(Mb, Nb1, wave)
    if order == "halves":  # column-first over each half of the row blocks (a stress order)
        per = -(-Mb // 2)
        return [nb * Mb + mb for g0 in range(0, Mb, per) for nb in range(Nb1) for mb in range(g0, min(Mb, g0 + per))]
    if order == "row":
        return [nb * Mb + mb for mb in range(Mb) for nb in range(Nb1)]
    if order == "reversed":
        return [nb * Mb + mb for nb in reversed(range(Nb1)) for mb in range(Mb)]
    tiles = [nb * Mb + mb for nb in range(Nb1) for mb in range(Mb)]  # column-first (and "auto")
    if order == "shuffled":
        random.Random(seed).shuffle(tiles)
    return tiles


def items(Mb, Nb1, Nb2, S1, S2, order, consumers_first=False, merged_lag=None):
    """Rank-ordered items: (kind, tile, s, needs) with needs = GEMM1 tiles a GEMM2 part reads.

    merged_lag: place each GEMM2 item right after rank (last producer rank + lag), as the
    pipelined kernel's merged table does, instead of after every GEMM1 item."""
    g1 = [("g1", t, s, []) for t in column_first_tiles(Mb, Nb1, order, S2=S2) for s in range(S1)]
    per = -(-Nb1 // S2)
    g2 = []
    tiles2 = xcd_grouped(Mb, Nb2, 16) if order == "xcd" else range(Mb * Nb2)
    for tile in tiles2:
        mb = tile % Mb
        for s in range(S2):
            kbs = range(s * per, min(Nb1, (s + 1) * per))
            g2.append(("g2", tile, s, [kb * Mb + mb for kb in kbs]))
    if merged_lag is not None:
        last = {}
        for r, it in enumerate(g1):
            last[it[1]] = r
        keyed = [(r, 0, it) for r, it in enumerate(g1)]
        keyed += [(max((last[n] for n in it[3]), default=-1) + merged_lag, 1, it) for it in g2]
        keyed.sort(key=lambda k: (k[0], k[1]))
        return [k[2] for k in keyed]
    return g2 + g1 if consumers_first else g1 + g2


def claim_lists(grid):
    """The host's rule: one list per XCD, fewer when the grid is smaller."""
    return min(8, max(1, grid))


def static_count(item_list, grid):
    """The host's rule: work-groups g below the number of leading ranks that
    never wait (GEMM1 items), and below the grid, take rank g as their first
    item without a ticket."""
    lead = 0
    while lead < len(item_list) and item_list[lead][0] == "g1":
        lead += 1
    return min(grid, lead)


def simulate(item_list, S1, S2, grid, seed, lists=None, max_steps=200000, first_static=0, late_start=0):
    """Returns True if every item completes.

    A work-group takes the ticket for its next item as soon as its current
    item has no wait left (at the start of a GEMM1 item, after the last wait
    of a GEMM2 item): the earliest point the kernels allow (they take it a
    little later, when the item's last stage is loaded).  With `first_static`, work-group g
    takes rank g as its first item without a ticket and the lists' tickets
    continue after those ranks.  `late_start` > 0 makes work-groups become
    resident after random delays of up to that many steps."""
    rng = random.Random(seed)
    lists = lists or claim_lists(grid)
    S = {"g1": S1, "g2": S2}
    arrived = {}  # (kind, tile) -> parts arrived
    signals = set()  # GEMM1 tiles whose last part has finished the tile
    done = 0
    ticket = [0] * lists
    skip = [len(range(l, first_static, lists)) for l in range(lists)]

    def claim(g):
        lst = g % lists
        t = ticket[lst]
        ticket[lst] += 1
        return lst + (t + skip[lst]) * lists

    # work-group state: [item rank or None, remaining time, next rank or None, start step]
    order = list(range(grid))
    rng.shuffle(order)  # first claims in any order
    first = {g: (g if g < first_static else claim(g)) for g in order}
    wgs = [[first[g], rng.randint(1, 5), None, rng.randint(0, late_start)] for g in range(grid)]
    for step in range(max_steps):
        progressed = False
        for g, w in enumerate(wgs):
            p, rem, nxt, start = w
            if p is None:
                continue
            if step < start:
                progressed = True  # not resident yet
                continue
            if p >= len(item_list):
                w[0] = None
                progressed = True
                continue
            kind, tile, s, needs = item_list[p]
            if kind == "g2" and any(n not in signals for n in needs):
                continue  # waiting for producer tiles
            if nxt is None:
                w[2] = nxt = claim(g)  # no wait left in this item: take the next ticket
            if rem > 0:
                w[1] -= 1
                progressed = True
                continue
            key = (kind, tile)
            arrived[key] = arrived.get(key, 0) + 1
            if arrived[key] == S[kind] and kind == "g1":
                signals.add(tile)  # the completing part reduces, stores Z and signals
            done += 1
            w[0], w[1], w[2] = nxt, rng.randint(1, 5), None
            progressed = True
        if done == len(item_list):
            return True
        if not progressed:
            return False
    return False


CASES = [
    # Mb, Nb1, Nb2, S1, S2
    (1, 8, 4, 3, 4),
    (2, 6, 3, 2, 3),
    (3, 5, 2, 1, 4),
    (1, 16, 8, 4, 2),
    (2, 4, 4, 1, 1),
    (1, 6, 2, 12, 9),
]


@pytest.mark.parametrize("order", ["auto", "xcd", "row", "reversed", "shuffled", "halves"])
@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
def test_pipelined_schedule_finishes_for_any_grid(order, Mb, Nb1, Nb2, S1, S2):
    lst = items(Mb, Nb1, Nb2, S1, S2, order)
    for grid in (1, 2, 3, 5, 7, 8, 9, 16, 17, 40):
        for seed in range(4):
            assert simulate(lst, S1, S2, grid, seed), (order, grid, seed)


@pytest.mark.parametrize("order", ["auto", "xcd", "row", "shuffled", "halves"])
@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
def test_merged_rank_table_finishes_for_any_grid(order, Mb, Nb1, Nb2, S1, S2):
    for lag in (0, 1, 5, 40):
        lst = items(Mb, Nb1, Nb2, S1, S2, order, merged_lag=lag)
        rank = {id(it): r for r, it in enumerate(lst)}
        g1_rank = {(it[1]): r for r, it in enumerate(lst) if it[0] == "g1"}
        for it in lst:  # every consumer ranks above each producer tile it reads
            if it[0] == "g2":
                assert all(g1_rank[n] < rank[id(it)] for n in it[3])
        for grid in (1, 2, 3, 8, 9, 17):
            for seed in range(3):
                assert simulate(lst, S1, S2, grid, seed), (order, lag, grid, seed)


@pytest.mark.parametrize("order", ["auto", "row", "shuffled"])
@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
def test_static_first_items_and_late_residency(order, Mb, Nb1, Nb2, S1, S2):
    """Static first items (as many as the host allows) and work-groups that
    become resident late: every launch still finishes."""
    for lag in (0, 5, 40):
        lst = items(Mb, Nb1, Nb2, S1, S2, order, merged_lag=lag)
        for grid in (1, 3, 8, 9, 17):
            fs = static_count(lst, grid)
            assert all(lst[r][0] == "g1" for r in range(fs))
            for seed in range(3):
                assert simulate(lst, S1, S2, grid, seed, first_static=fs, late_start=30), (order, lag, grid, seed, fs)
    for grid in (2, 8, 17):  # the sequential kernels: no item waits
        g1 = [it for it in items(Mb, Nb1, Nb2, S1, S2, order) if it[0] == "g1"]
        assert simulate(g1, S1, S2, grid, 7, first_static=static_count(g1, grid), late_start=30)


def test_host_rule_takes_static_first_items_only_below_the_first_waiting_rank():
    lst = items(1, 4, 2, 1, 2, "auto", consumers_first=True)
    assert static_count(lst, 3) == 0
    merged = items(1, 4, 2, 1, 2, "auto", merged_lag=4)
    n = static_count(merged, 8)
    assert 0 < n < 8 and merged[n][0] == "g2"


@pytest.mark.parametrize("Mb,N,wave", [(16, 112, 512), (16, 32, 512), (3, 10, 17), (5, 7, 8), (1, 9, 4), (40, 3, 64), (8, 64, 64)])
def test_xcd_grouped_deal_is_a_permutation_of_whole_column_waves(Mb, N, wave):
    order = xcd_grouped(Mb, N, wave)
    assert sorted(order) == list(range(Mb * N))
    C = max(1, wave // Mb)
    done = set()
    for r, t in enumerate(order):  # column blocks complete wave by wave
        assert t // Mb < (r // (C * Mb) + 1) * C
        done.add(t)
    if Mb == 16 and N == 112 and wave == 512:  # prefill: XCD x holds an 8 x 8 sub-block of each wave
        for x in range(8):
            tiles = [order[8 * j + x] for j in range(64)]
            assert len({t % Mb for t in tiles}) == 8 and len({t // Mb for t in tiles}) == 8
