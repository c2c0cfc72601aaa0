"""Host-side invariants of the pass planner (no GPU): every gate is applied
exactly once (absorbed into the product-state init or a member of one forward
op), the reverse sweep holds every gate once, dense ops find their target
bits in the tile, and tiles have min(n, tile) bits."""
import pytest

from paper_2003_02989_amd import tq
from paper_2003_02989_amd import workloads as wl


def check_plan(w, **kw):
    p = tq.Program(w.program_blob(), **kw)
    d = tq.describe(p)
    tile = d["tile"]
    for g in d["groups"]:
        n = g["n"]
        fwd_members = sum(op["members"] for ps in g["fwd"] for op in ps["ops"])
        assert fwd_members + g["absorbed"] == g["gates"]
        assert sum(len(ps["ops"]) for ps in g["rev"]) == g["gates"]
        assert sum(op["ngrad"] for ps in g["rev"] for op in ps["ops"]) == g["n_gslots"]
        for ps in g["fwd"] + g["rev"]:
            t = ps["t"]
            assert t == min(n, tile if ps in g["fwd"] else min(tile, 12))
            assert ps["c"] + ps["h"] == t
            assert all(ps["c"] <= b < n for b in ps["hb"])
            for op in ps["ops"]:
                if op["kind"] in ("M1", "M2"):
                    assert op["l"][0] < t
                if op["kind"] in ("M2", "P2"):
                    assert op["l"][1] < t and op["l"][0] != op["l"][1]
        assert g["fwd"][0]["product_init"] == 1
    return d


@pytest.mark.parametrize("seed", range(6))
def test_random_plans(seed):
    w = wl.random_batch(seed, B=4, n=14, n_gates=80, n_symbols=5, hetero=True)
    check_plan(w)
    check_plan(w, max_tile_qubits=8, low_qubits=3)
    check_plan(w, fuse=False)


def test_config_plans():
    for w in (wl.c1_hea(), wl.c2_qnn(B=4), wl.c3_qaoa(B=2), wl.c5_vqe(B=2), wl.c4_random(n_shots=1)):
        d = check_plan(w)
        assert len(d["groups"]) == 1  # every row shares one structure


def test_structure_dedupe_keeps_per_row_constants():
    # c2 rows differ only in their encoding constants: one group, per-row slots
    d = tq.describe(tq.Program(wl.c2_qnn(B=8).program_blob()))
    assert len(d["groups"]) == 1 and d["groups"][0]["rows"] == 8 and d["groups"][0]["uniform_slots"] == 0
    d = tq.describe(tq.Program(wl.c5_vqe(B=8, n=6, layers=2, n_terms=5).program_blob()))
    assert d["groups"][0]["uniform_slots"] == 1


def test_scheduler_variants():
    # the 30-qubit random circuit: the best of the schedule variants (both
    # tie rules, five or six low bits forced into the tiles) takes 22 forward
    # passes instead of 30, its tiles holding five or six contiguous low bits
    d = check_plan(wl.c4_random(n_shots=1), specialize=True)
    g = d["groups"][0]
    assert len(g["fwd"]) <= 22
    assert all(ps["c"] in (5, 6) for ps in g["fwd"]) and any(ps["c"] == 5 for ps in g["fwd"])
    # the VQE ansatz would save one pass of 15 with five low bits: too little,
    # it keeps six
    d = check_plan(wl.c5_vqe(B=2), specialize=True)
    g = d["groups"][0]
    assert len(g["fwd"]) == 15 and all(ps["c"] == 6 for ps in g["fwd"])
