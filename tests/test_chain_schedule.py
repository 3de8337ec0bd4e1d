"""The GEMM chain's one-launch rank table and claim protocol, on the CPU.

The table mirrors the host's rule: every layer's tiles (tile = nb * Mb +
mb) in the layer order, the XCD-grouped deal of the two-layer plan's GEMMs
when there are several row blocks (waves of about one grid of tiles, each
cut into 8 sub-blocks, one per XCD, dealt rank by rank), else column blocks
in order; layer 0 in that order, then each later layer merged in layer by
layer, the item of tile (mb, nb) right after rank h + lag of the table
built so far (h = the highest rank among the layer below's tiles of row
block mb, all of which it reads), items of equal key in layer order.

* the layer order is a permutation of the layer's tiles;

* the table is a permutation of every item, and every item ranks above all
  of its producers;
* the claim protocol (8 claim lists over the ranks, the next ticket taken
  only once the current item's waits are over) finishes for any grid size,
  with random item durations and work-groups that become resident late;
* a table that puts consumers first deadlocks a small grid (the simulator
  does detect a stuck launch).
"""
import random

import pytest


def cdiv(a, b):
    return -(-a // b)


def xcd_grouped(Mb, N, wave):
    """Waves of C = wave // Mb whole column blocks; each wave cut into 8
    sub-blocks (r row groups x 8 / r column groups, r the power of two up to
    8 and Mb with the fewest rows + columns per sub-block), one per XCD,
    walked column-first; the j-th group of 8 ranks takes the j-th tile of
    every sub-block that still has one."""
    out = []
    C = max(1, wave // Mb)
    for c0 in range(0, N, C):
        cw = min(C, N - c0)
        best_r, best_cost, r = 1, None, 1
        while r <= 8 and r <= Mb:
            cost = cdiv(Mb, r) + cdiv(cw, 8 // r)
            if best_cost is None or cost < best_cost:
                best_r, best_cost = r, cost
            r *= 2
        rows, cols = cdiv(Mb, best_r), cdiv(cw, 8 // best_r)
        per = []
        for x in range(8):
            rg, cg = x % best_r, x // best_r
            per.append([nb * Mb + mb
                        for nb in range(c0 + cg * cols, min(c0 + cw, c0 + (cg + 1) * cols))
                        for mb in range(rg * rows, min(Mb, (rg + 1) * rows))])
        for j in range(max(len(q) for q in per)):
            out += [q[j] for q in per if j < len(q)]
    return out


def layer_order(Mb, nb, wave):
    return xcd_grouped(Mb, nb, wave) if Mb > 1 else list(range(nb))


def rank_table(Mb, widths, lag, wave=None):
    """widths: column blocks per layer (Nb_0 .. Nb_{L-1}); wave: the grid the
    layer order deals (the host passes the launch grid, as it does for lag).
    Entries (layer, tile)."""
    wave = lag if wave is None else wave
    table = [(0, t) for t in layer_order(Mb, widths[0], wave)]
    for l in range(1, len(widths)):
        row_last = [-1] * Mb
        for r, (lay, t) in enumerate(table):
            if lay == l - 1:
                row_last[t % Mb] = max(row_last[t % Mb], r)
        add = sorted(((min(row_last[t % Mb] + lag, len(table) - 1), t) for t in layer_order(Mb, widths[l], wave)),
                     key=lambda kt: kt[0])  # stable: layer order within a key
        merged, k = [], 0
        for r, e in enumerate(table):
            merged.append(e)
            while k < len(add) and add[k][0] == r:
                merged.append((l, add[k][1]))
                k += 1
        table = merged
    return table


def producers(Mb, widths, layer, tile):
    if layer == 0:
        return []
    mb = tile % Mb
    return [(layer - 1, kb * Mb + mb) for kb in range(widths[layer - 1])]


def simulate(table, Mb, widths, grid, seed, late_start=0, max_steps=100000):
    rng = random.Random(seed)
    lists = min(8, max(1, grid))
    ticket = [0] * lists
    signalled, done = set(), 0

    def claim(g):
        l = g % lists
        t = ticket[l]
        ticket[l] += 1
        return l + t * lists

    order = list(range(grid))
    rng.shuffle(order)
    first = {g: claim(g) for g in order}
    wgs = [[first[g], rng.randint(1, 4), None, rng.randint(0, late_start)] for g in range(grid)]
    for step in range(max_steps):
        progressed = False
        for g, w in enumerate(wgs):
            p, rem, nxt, start = w
            if p is None:
                continue
            if step < start:
                progressed = True
                continue
            if p >= len(table):
                w[0] = None
                progressed = True
                continue
            item = table[p]
            if any(n not in signalled for n in producers(Mb, widths, *item)):
                continue
            if nxt is None:
                w[2] = nxt = claim(g)
            if rem > 0:
                w[1] -= 1
                progressed = True
                continue
            signalled.add(item)
            done += 1
            w[0], w[1], w[2] = nxt, rng.randint(1, 4), None
            progressed = True
        if done == len(table):
            return True
        if not progressed:
            return False
    return False


CASES = [
    # Mb, column blocks per layer
    (1, [2, 3, 2]),
    (2, [4, 1, 3, 2]),
    (3, [2, 2, 2, 2, 2]),
    (4, [8, 2]),
    (1, [1]),
    (5, [12, 7, 3]),
    (16, [32, 32]),
]


@pytest.mark.parametrize("Mb,N", [(2, 1), (3, 5), (5, 12), (8, 64), (16, 32), (9, 7), (64, 3)])
@pytest.mark.parametrize("wave", [1, 7, 24, 256, 512])
def test_layer_order_is_a_permutation_dealt_in_sub_blocks(Mb, N, wave):
    order = xcd_grouped(Mb, N, wave)
    assert sorted(order) == list(range(Mb * N))
    # every wave of whole column blocks comes before the next one
    C = max(1, wave // Mb)
    waves = [t // Mb // C for t in order]
    assert waves == sorted(waves)
    # rank r goes to XCD r % 8: per wave, the distinct row and column blocks
    # each XCD reads (its L2's operand slices) number no more than under the
    # plain column-first deal
    def slices(seq):
        total = 0
        for w in set(t // Mb // C for t in seq):
            for x in range(8):
                mine = [t for r, t in enumerate(seq) if r % 8 == x and t // Mb // C == w]
                total += len({t % Mb for t in mine}) + len({t // Mb for t in mine})
        return total
    assert slices(order) <= slices(list(range(Mb * N)))


@pytest.mark.parametrize("Mb,widths", CASES)
@pytest.mark.parametrize("lag", [1, 3, 16])
def test_table_is_a_permutation_with_every_item_after_its_producers(Mb, widths, lag):
    table = rank_table(Mb, widths, lag)
    every = {(l, t) for l in range(len(widths)) for t in range(Mb * widths[l])}
    assert len(table) == len(every) and set(table) == every
    rank = {e: r for r, e in enumerate(table)}
    for e in table:
        assert all(rank[n] < rank[e] for n in producers(Mb, widths, *e))


@pytest.mark.parametrize("Mb,widths", CASES)
@pytest.mark.parametrize("grid", [1, 2, 3, 5, 8, 13, 64])
def test_claims_finish_for_any_grid(Mb, widths, grid):
    table = rank_table(Mb, widths, grid)
    for seed in range(4):
        assert simulate(table, Mb, widths, grid, seed, late_start=3 * seed)


def test_consumers_first_deadlocks_a_small_grid():
    Mb, widths = 1, [2, 3, 2]
    table = sorted(rank_table(Mb, widths, 1), key=lambda e: -e[0])  # last layer first
    assert not simulate(table, Mb, widths, 1, 0)
