"""Every tile configuration compiled into the library runs at least once.

The dispatch table of the kernels source (`kEntries` in mlp2_kernels.hip) is
read here, so a configuration added there is covered without editing this
file.  Each entry is planned on a small shape that every configuration
accepts (two row blocks, the second ragged; H and F multiples of 256), with
the tuning that selects exactly it; the test checks that the plan took that
entry, that every mode gives the sequential mode's bits and that Y matches
the fp64 oracle within the bound.
"""
import os
import re

import pytest

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, both_modes, device_inputs, sentinel_mode, workqueue_mode

pytestmark = pytest.mark.gpu

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_07862_amd", "csrc",
                   "mlp2_kernels.hip")


def entries():
    """(bm, bn1, bn2, nb, ns, hv, waves, bk, weights_nt) of every table entry.
    The macros' defaults: HV 1, four waves, 64-deep stages, cached weight loads."""
    src = open(SRC).read()
    start = src.index("static const Entry kEntries[] = {")
    body = src[start:src.index("};", start)]
    out = []
    for m in re.finditer(r"MLP2_ENTRY(_HV|_W|_WK|_WKN)?\(([^)]*)\)", body):
        a = [x.strip() for x in m.group(2).split(",")]
        v = [int(x) for x in a[:5]]
        hv = int(a[5]) if len(a) > 5 else 1
        waves = int(a[6]) if len(a) > 6 else 4
        bk = int(a[7]) if len(a) > 7 else 64
        nt = len(a) > 8 and a[8] == "true"
        out.append((*v, hv, waves, bk, nt))
    return out


ENTRIES = entries()


def test_the_table_was_read():
    assert len(ENTRIES) >= 40 and len(set(ENTRIES)) == len(ENTRIES)


@pytest.mark.parametrize("e", ENTRIES, ids=[f"bm{e[0]}-n{e[1]}-{e[2]}-nb{e[3]}-s{e[4]}-hv{e[5]}-w{e[6]}-bk{e[7]}-nt{int(e[8])}"
                                            for e in ENTRIES])
def test_every_entry_runs_every_mode(lib, e):
    bm, bn1, bn2, nb, ns, hv, waves, bk, nt = e
    M, H, F = bm + 5, 512, 1024
    act = 2 if nb == 2 else 1
    print(f"\n[entry] {e} M={M} H={H} F={F} act={act}", flush=True)
    tuning = {"bm": bm, "bn1": bn1, "bn2": bn2, "stages": ns, "waves": waves, "bk": bk, "weights_nt": 1 if nt else -1}
    d = I.make_inputs(M, H, F, act, seed=bm + bn1 + bn2 + ns + waves + bk)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, tuning)
    info = plan.info()
    got = (info["bm"], info["bn1"], info["bn2"], info["stages"], info["waves"], info["bk"], info["weights_nt"])
    assert got == (bm, bn1, bn2, ns, waves, bk, int(nt)), info
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    Yq, Zq = workqueue_mode(plan, g)
    Yn = sentinel_mode(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    assert_bit_equal(Ys, Yn, "Y sequential vs sentinel")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "Y")
    plan.close()
