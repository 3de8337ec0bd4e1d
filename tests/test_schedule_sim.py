"""CPU simulation of the persistent ticket scheduler (no GPU needed).

The kernels hand out work items through one ticket counter: GEMM1 items (in
the order table's order) then, in the pipelined launch, GEMM2 items.  A
split-K part waits for its sibling parts; a GEMM2 item waits, K-slice by
K-slice, for the GEMM1 tiles of its row block; a work-group claims its next
ticket after the last wait of its current item.  The claim in the design is
that every launch finishes for any grid of at least max(S1, S2) work-groups,
because the parts of a tile are adjacent tickets.  This simulates that
protocol with random item durations and checks it, and checks that a
split-major numbering of the GEMM2 parts (not adjacent) can deadlock.
"""
import random

import pytest


def column_first_tiles(Mb, Nb1, order, seed=12345):
    if order == "row":
        return [nb * Mb + mb for mb in range(Mb) for nb in range(Nb1)]
    if order == "reversed":
        return [nb * Mb + mb for nb in reversed(range(Nb1)) for mb in range(Mb)]
    tiles = [nb * Mb + mb for nb in range(Nb1) for mb in range(Mb)]
    if order == "shuffled":
        random.Random(seed).shuffle(tiles)
    return tiles


def items(Mb, Nb1, Nb2, S1, S2, kslices_per_part, order, gemm2_split_major=False):
    """Ticket-ordered items: (kind, tile, s, needs) with needs = GEMM1 column blocks a GEMM2 part reads."""
    out = []
    for t in column_first_tiles(Mb, Nb1, order):
        for s in range(S1):
            out.append(("g1", t, s, []))
    tiles2 = Mb * Nb2
    idx = [(tile, s) for tile in range(tiles2) for s in range(S2)]
    if gemm2_split_major:
        idx = [(tile, s) for s in range(S2) for tile in range(tiles2)]
    per = (Nb1 + S2 - 1) // S2
    for tile, s in idx:
        mb = tile % Mb
        kbs = [kb for kb in range(s * per, min(Nb1, (s + 1) * per))]
        out.append(("g2", tile, s, [(kb * Mb + mb) for kb in kbs]))
    return out


def simulate(item_list, S1, S2, grid, seed, max_steps=200000):
    """Returns True if every item completes."""
    rng = random.Random(seed)
    S = {"g1": S1, "g2": S2}
    arrived = {}  # (kind, tile) -> parts arrived
    signals = {}  # GEMM1 tile -> parts signalled
    done = 0
    ticket = [0]

    def claim():
        t = ticket[0]
        ticket[0] += 1
        return t

    # work-group state: [item index or None, phase, remaining time, prefetched ticket]
    wgs = [[claim(), "main", rng.randint(1, 5), None] for _ in range(grid)]
    for step in range(max_steps):
        progressed = False
        for w in wgs:
            p, phase, rem, nxt = w
            if p is None:
                continue
            if p >= len(item_list):
                w[0] = None
                progressed = True
                continue
            kind, tile, s, needs = item_list[p]
            if phase == "main":
                # a GEMM2 part may only run once its Z slices are complete
                if kind == "g2" and any(signals.get(n, 0) < S1 for n in needs):
                    continue
                if rem > 0:
                    w[2] -= 1
                    progressed = True
                    continue
                if S[kind] > 1:
                    arrived[(kind, tile)] = arrived.get((kind, tile), 0) + 1
                    w[1] = "siblings"
                else:
                    w[1] = "epilogue"
                    w[3] = claim()
                progressed = True
            elif phase == "siblings":
                if arrived[(kind, tile)] < S[kind]:
                    continue
                w[1] = "epilogue"
                w[3] = claim()
                progressed = True
            elif phase == "epilogue":
                if kind == "g1":
                    signals[tile] = signals.get(tile, 0) + 1
                done += 1
                w[0], w[1], w[2], w[3] = nxt, "main", rng.randint(1, 5), None
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
]


@pytest.mark.parametrize("order", ["column", "row", "reversed", "shuffled"])
@pytest.mark.parametrize("Mb,Nb1,Nb2,S1,S2", CASES)
def test_pipelined_schedule_finishes_for_any_grid_from_max_s(order, Mb, Nb1, Nb2, S1, S2):
    lst = items(Mb, Nb1, Nb2, S1, S2, 1, order)
    for grid in range(max(S1, S2), max(S1, S2) + 6):
        for seed in range(8):
            assert simulate(lst, S1, S2, grid, seed), (order, grid, seed)


def test_split_major_gemm2_parts_can_deadlock():
    """The numbering the kernels avoid: parts of a GEMM2 tile spread over the ticket range."""
    Mb, Nb1, Nb2, S1, S2 = 1, 4, 4, 1, 3
    lst = items(Mb, Nb1, Nb2, S1, S2, 1, "column", gemm2_split_major=True)
    assert not all(simulate(lst, S1, S2, 3, seed) for seed in range(8))
    lst_ok = items(Mb, Nb1, Nb2, S1, S2, 1, "column")
    assert all(simulate(lst_ok, S1, S2, 3, seed) for seed in range(8))
