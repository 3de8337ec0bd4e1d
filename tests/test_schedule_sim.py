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


def banded(Mb, N, wave, band):
    """The host's row bands: `band` row blocks with all their column blocks,
    band after band, each dealt like xcd_grouped."""
    out = []
    for r0 in range(0, Mb, band):
        rb = min(band, Mb - r0)
        out += [(t // rb) * Mb + r0 + t % rb for t in xcd_grouped(rb, N, wave)]
    return out


def column_first_tiles(Mb, Nb1, order, seed=12345, S2=1, wave=16):
    if order == "xcd":
        return xcd_grouped(Mb, Nb1, wave)
    if order == "banded":
        return banded(Mb, Nb1, wave, max(1, wave // Nb1))
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

    merged_lag: place each GEMM2 item right after rank (last producer rank + lag), or after
    every GEMM1 item in GEMM2 order when lag >= the GEMM1 count, as the
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
        keyed += [(len(g1) if merged_lag >= len(g1) else max((last[n] for n in it[3]), default=-1) + merged_lag, 1, it)
                  for it in g2]
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


@pytest.mark.parametrize("order", ["auto", "xcd", "banded", "row", "shuffled", "halves"])
@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
def test_merged_rank_table_finishes_for_any_grid(order, Mb, Nb1, Nb2, S1, S2):
    for lag in (0, 1, 5, 40, Mb * Nb1 * S1):  # the last: every GEMM2 item after every GEMM1 item
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


def simulate_workqueue(Mb, Nb1, Nb2, S1, S2, grid, seed, k_ranges=None, order="auto", late_start=0):
    """Step simulation of the workqueue mode (Sec. III-A.2-3 scheduling).

    GEMM1 items are claimed by rank through the claim lists (the first
    min(grid, items) ranks taken without tickets, as the host arranges);
    a work-group whose claim runs past them takes the next queue slot and
    waits until a unit is there.  A GEMM2 unit enters the queue when the last
    part of the last GEMM1 tile it reads finishes (its scoreboard reaches its
    producer count).  `k_ranges[s]` lists the Z column blocks part s reads
    (default: even shares); parts of neighbouring ranges may share a block.
    Returns the units in run order with their start step and the step at
    which their producers were all done, or None on deadlock."""
    rng = random.Random(seed)
    lists = claim_lists(grid)
    items1 = [(t, s) for t in column_first_tiles(Mb, Nb1, order) for s in range(S1)]
    per = -(-Nb1 // S2)
    k_ranges = k_ranges or [list(range(s * per, min(Nb1, (s + 1) * per))) for s in range(S2)]
    k_ranges = [r for r in k_ranges if r]  # the host's S2 = ceil(F / kc2): no part reads nothing
    S2 = len(k_ranges)
    units = [(tile, s) for tile in range(Mb * Nb2) for s in range(S2)]
    needs = {u: [kb * Mb + u[0] % Mb for kb in k_ranges[u[1]]] for u in units}
    users = {}
    for u in units:
        for t in needs[u]:
            users.setdefault(t, []).append(u)
    board = {u: 0 for u in units}
    parts = {}
    queue, head = [], [0]
    ready_at, ran = {}, []
    first_static = min(grid, len(items1))
    ticket = [0] * lists
    skip = [len(range(l, first_static, lists)) for l in range(lists)]

    def claim(g):
        l = g % lists
        t = ticket[l]
        ticket[l] += 1
        return l + (t + skip[l]) * lists

    # work-group: [phase, item, remaining, start]; phase "g1", "pop", "g2", "done"
    wgs = []
    for g in range(grid):
        r = g if g < first_static else claim(g)
        wgs.append(["g1", r, rng.randint(1, 6), rng.randint(0, late_start)])
    for step in range(200000):
        if all(w[0] == "done" for w in wgs):
            return ran
        progressed = False
        for g, w in enumerate(wgs):
            phase = w[0]
            if phase == "done" or step < w[3]:
                progressed |= phase != "done"
                continue
            progressed = True
            if phase == "g1":
                if w[1] >= len(items1):
                    w[0], w[1] = "pop", None
                    continue
                if w[2] > 0:
                    w[2] -= 1
                    continue
                tile, s = items1[w[1]]
                parts[tile] = parts.get(tile, 0) + 1
                if parts[tile] == S1:  # the tile is complete: count down its users' scoreboards
                    for u in users.get(tile, []):
                        board[u] += 1
                        if board[u] == len(needs[u]):
                            queue.append(u)
                            ready_at[u] = step
                w[1], w[2] = claim(g), rng.randint(1, 6)
            elif phase == "pop":
                if w[1] is None:
                    w[1] = head[0]
                    head[0] += 1
                if w[1] >= len(units):
                    w[0] = "done"
                elif w[1] < len(queue):  # the slot is filled
                    u = queue[w[1]]
                    ran.append((u, step, ready_at[u]))
                    w[0], w[1], w[2] = "g2", u, rng.randint(1, 6)
                else:
                    progressed = any(x[0] in ("g1", "g2") for x in wgs) or progressed
            elif phase == "g2":
                if w[2] > 0:
                    w[2] -= 1
                else:
                    w[0], w[1] = "pop", None
        if not progressed:
            return None
    return None


@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
@pytest.mark.parametrize("order", ["auto", "xcd", "reversed", "shuffled"])
def test_workqueue_schedule_runs_every_unit_after_its_producers(Mb, Nb1, Nb2, S1, S2, order):
    for grid in (1, 2, 3, 8, 9, 17):
        for seed in range(3):
            ran = simulate_workqueue(Mb, Nb1, Nb2, S1, S2, grid, seed, order=order, late_start=20 if seed else 0)
            assert ran is not None, (grid, seed)
            parts = len({s for _, s in (u for u, _, _ in ran)})
            assert sorted(u for u, _, _ in ran) == sorted((t, s) for t in range(Mb * Nb2) for s in range(parts))
            assert all(start >= ready for _, start, ready in ran)


def test_workqueue_schedule_with_parts_sharing_a_column_block():
    # 1152 columns in blocks of 128 split into parts of 192: block 1 feeds parts 0 and 1, ...
    k_ranges = [sorted({c // 128 for c in range(s * 192, (s + 1) * 192)}) for s in range(6)]
    assert k_ranges[0] == [0, 1] and k_ranges[1] == [1, 2]
    for grid in (1, 4, 9):
        ran = simulate_workqueue(2, 9, 3, 1, 6, grid, seed=grid, k_ranges=k_ranges)
        assert ran is not None and len(ran) == 2 * 3 * 6
        assert all(start >= ready for _, start, ready in ran)


@pytest.mark.parametrize("seed", range(5))
def test_counter_targets_hold_across_any_sequence_of_modes(seed):
    """Counters carry over from run to run without host resets.  Ready counters
    advance once per run in every mode but the sentinel mode (workqueue
    producers signal them too; sentinel producers signal nothing), so a
    pipelined consumer's target is (epoch - s) + 1, s the number of earlier
    sentinel runs, and a counter never reaches the target before its tile
    signals in this run; scoreboards advance only in workqueue runs, so a unit
    with n producers completes at (w + 1) * n, w the number of earlier
    workqueue runs; split-K arrivals count S per run in every mode; sentinel
    runs alternate between two intermediates by the parity of s."""
    rng = random.Random(seed)
    tiles, n_of = list(range(6)), {"u0": 2, "u1": 3, "u2": 1}
    users = {"u0": [0, 1], "u1": [2, 3, 4], "u2": [5]}
    ready = {t: 0 for t in tiles}
    board = {u: 0 for u in n_of}
    arrivals, S = 0, 3
    epoch = wq = sn = 0
    fresh = [True, True]  # each sentinel intermediate holds sentinels before its run
    for _ in range(80):
        mode = rng.choice(["sequential", "pipelined", "workqueue", "sentinel"])
        if mode == "sentinel":
            buf = sn & 1
            assert fresh[buf]
            fresh[buf] = False      # this run writes it ...
            fresh[1 - buf] = True   # ... and refills the other one
        else:
            if mode == "pipelined":  # before this run's signals: not yet ready
                assert all(ready[t] < (epoch - sn) + 1 for t in tiles)
            for t in tiles:  # every GEMM1 tile signals once per run
                ready[t] += 1
            if mode == "pipelined":
                assert all(ready[t] >= (epoch - sn) + 1 for t in tiles)
        if mode == "workqueue":
            for u, ts in users.items():
                for k, t in enumerate(ts):
                    board[u] += 1
                    assert (board[u] == (wq + 1) * n_of[u]) == (k == len(ts) - 1), (u, board[u], wq)
        for s in range(S):  # split-K parts of one tile: the last arrival completes it
            arrivals += 1
            assert (arrivals == (epoch + 1) * S) == (s == S - 1)
        epoch += 1
        wq += mode == "workqueue"
        sn += mode == "sentinel"


MASK = 0xFFFFFFFF


def reached(v, target):
    """The kernels' wrap-safe test of a 32-bit counter against a 32-bit
    target: the difference taken as a signed 32-bit value is >= 0."""
    d = (v - target) & MASK
    return d < 0x80000000


@pytest.mark.parametrize("seed", range(4))
def test_counter_targets_hold_across_the_32_bit_wrap(seed):
    """The same run-to-run protocol with every counter and target a 32-bit
    value, starting a few dozen runs before the epoch wraps, each counter in
    the state those runs leave it in, and each decision taken as the kernels
    take it: a ready counter against its target with the wrap-safe compare
    (not ready before this run's signal, ready after it); a split-K arrival
    or a scoreboard increment by 32-bit equality of its fetch-and-add result
    with the run's target (complete exactly at the last producer)."""
    rng = random.Random(100 + seed)
    tiles, n_of = list(range(6)), {"u0": 2, "u1": 3, "u2": 1}
    users = {"u0": [0, 1], "u1": [2, 3, 4], "u2": [5]}
    S = 3
    epoch, wq, sn = (1 << 32) - 37 - seed, 11 + seed, 5
    ready = {t: (epoch - sn) & MASK for t in tiles}
    board = {u: (wq * n) & MASK for u, n in n_of.items()}
    arrivals = (epoch * S) & MASK
    wrapped = False
    for _ in range(80):
        mode = rng.choice(["sequential", "pipelined", "workqueue", "sentinel"])
        target = (epoch - sn + 1) & MASK
        if mode != "sentinel":
            if mode == "pipelined":
                assert not any(reached(ready[t], target) for t in tiles)
            for t in tiles:
                ready[t] = (ready[t] + 1) & MASK
            if mode == "pipelined":
                assert all(reached(ready[t], target) for t in tiles)
        if mode == "workqueue":
            for u, ts in users.items():
                for k, t in enumerate(ts):
                    old = board[u]
                    board[u] = (old + 1) & MASK
                    assert (((old + 1) & MASK) == ((wq + 1) * n_of[u]) & MASK) == (k == len(ts) - 1)
        for s_ in range(S):
            old = arrivals
            arrivals = (old + 1) & MASK
            assert (old == (((epoch + 1) * S) - 1) & MASK) == (s_ == S - 1)
        epoch = (epoch + 1) & MASK
        wrapped |= epoch == 0
        wq += mode == "workqueue"
        sn += mode == "sentinel"
    assert wrapped


def test_wrap_safe_compare_pins():
    assert reached(5, 5) and reached(6, 5) and not reached(4, 5)
    assert reached(0, MASK) and reached(3, MASK - 2) and not reached(MASK, 0)
    assert not reached(MASK - 2, 3) and reached(0x7FFFFFFF, 0) and not reached(0x80000000, 0)


@pytest.mark.parametrize("Mb,N,wave,band", [(128, 64, 512, 8), (16, 112, 512, 4), (5, 7, 8, 2), (3, 10, 17, 1), (40, 3, 64, 21)])
def test_banded_deal_is_a_permutation_band_by_band(Mb, N, wave, band):
    order = banded(Mb, N, wave, band)
    assert sorted(order) == list(range(Mb * N))
    bands = [(t % Mb) // band for t in order]
    assert bands == sorted(bands)  # every tile of a band before the next band
