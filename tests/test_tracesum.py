"""Decoding of the trace build's per-item records (host logic only).

The record layout is the one the trace-attach entry point documents: word 0
holds the rank (high 32 bits) and the order-table entry (low 32 bits, bit 31
marking a GEMM2 item), word 6 the item's core clock cycles (high 32 bits)
above its ring-wait ticks (low 32 bits).
"""
import numpy as np
import torch

from paper_2607_07862_amd import tracesum as T


def _buffer(G, records):
    """records: {(section, group): [8-word records]} -> the flat int64 buffer the kernels fill."""
    a = np.zeros((2, G, 1 + 8 * T.CAP), dtype=np.uint64)
    for (sec, g), recs in records.items():
        a[sec, g, 0] = len(recs)
        for j, r in enumerate(recs):
            a[sec, g, 1 + 8 * j: 9 + 8 * j] = np.array(r, dtype=np.uint64)
    return torch.from_numpy(a.view(np.int64).reshape(-1).copy())


def test_records_split_rank_entry_kind_cycles_and_ring():
    gemm1 = [(7 << 32) | 42, 1000, 1800, 0, 0, 2000, (190000 << 32) | 35, 0]
    gemm2 = [(9 << 32) | 0x80000000 | 5, 2100, 2900, 0, 0, 3000, (170000 << 32) | 12, 40]
    # a reduction item (a slice of a split-K GEMM2 tile): bits 31 and 30 of the entry
    red = [(11 << 32) | 0xC0000000 | 17, 3100, 3150, 0, 0, 3400, (50000 << 32) | 0, 30]
    buf = _buffer(3, {(0, 1): [gemm1], (1, 2): [gemm2, red]})
    recs = sorted(T._records(buf, 3))
    assert recs[0] == (0, 42, 7, 1000, 1800, 2000, 35, 0, 190000)
    assert recs[1] == (1, 5, 9, 2100, 2900, 3000, 12, 40, 170000)
    assert recs[2] == (2, 17, 11, 3100, 3150, 3400, 0, 30, 50000)


def test_records_beyond_the_capacity_are_counted_not_read():
    r = [(1 << 32) | 3, 10, 20, 0, 0, 30, (3000 << 32) | 1, 0]
    buf = _buffer(1, {(0, 0): [r] * T.CAP})
    a = buf.view(2, 1, 1 + 8 * T.CAP)
    a[0, 0, 0] = T.CAP + 5  # the kernel counts items it could not store
    assert len(T._records(buf, 1)) == T.CAP


def test_clock_by_eighth_is_cycles_over_real_time():
    # items of 1000 ticks (10 us): 19000 cycles -> 1900 MHz in the first half, 14000 -> 1400 MHz after
    recs = []
    for e in range(8):
        start = e * 1000
        cycles = 19000 if e < 4 else 14000
        recs.append((0, e, e, start, start + 900, start + 1000, 0, 0, cycles))
    c = T.clock_by_eighth(recs, 0)
    assert [round(v) for v in c[1:4]] == [1900] * 3
    assert [round(v) for v in c[5:]] == [1400] * 3


def test_dependencies_of_a_grouped_plan_use_the_groups_row_blocks():
    # one launch: 4 row blocks; grouped: the records are a 2-row-block group's
    base = {"row_blocks": 4, "bm": 128, "splitk2": 1, "bn1": 128, "items2": 2, "row_group": 0}
    assert T._dependencies(base, 256) == {0: [0, 4], 1: [1, 5]}
    grouped = dict(base, row_group=256)
    assert T._dependencies(grouped, 256) == {0: [0, 2], 1: [1, 3]}
