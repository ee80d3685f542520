"""SLO-constrained EC-aware chunk scheduling (SPEAR section 4.3): the
library's scheduler (libspear.so, include/spear_sched.h) against the exact
rational oracle, plus the oracle's own pins. Host-only; no GPU."""
from __future__ import annotations

import random
from fractions import Fraction

import pytest

from oracle import sched_oracle as SO
from paper_2606_11244_amd import spear as sp


def _model(luts, sel, extra=None):
    return sp.LatencyModel(luts, sel, extra)


# ---------------------------------------------------------------------------
# pins of the oracle against what section 4.3 and arithmetic fix
# ---------------------------------------------------------------------------

def test_oracle_table_reading_by_hand():
    """A two-entry table at hand-worked points: the floor below the first
    entry, exact interpolation, linear continuation, zero tokens free."""
    M, lat = [4, 12], [10.0, 30.0]
    assert SO.table_latency(M, lat, 0) == 0
    assert SO.table_latency(M, lat, 1) == 10
    assert SO.table_latency(M, lat, 4) == 10
    assert SO.table_latency(M, lat, 8) == 20          # halfway
    assert SO.table_latency(M, lat, 6) == 15
    assert SO.table_latency(M, lat, 12) == 30
    assert SO.table_latency(M, lat, 20) == 50         # slope 2.5 continued
    # a dip in a measured table is read as the running maximum
    assert SO.table_latency([1, 2, 3], [5.0, 3.0, 9.0], 2) == 5
    assert SO.table_latency([1, 2, 3], [5.0, 3.0, 9.0], 3) == 9
    assert SO.table_latency([7], [2.5], 100) == Fraction(5, 2)


def test_oracle_iteration_sum_by_hand():
    """Two layers x two module types with the EC on (0, 1) and (1, 0): each
    call contributes its own table's entry."""
    luts = [([1, 3], [1.0, 3.0], [2.0, 6.0]), ([1, 3], [10.0, 30.0], [11.0, 33.0])]
    sel = [[0, 1], [1, 0]]
    # at M = 2: module 0 -> w4 2, ec 4; module 1 -> w4 20, ec 22
    assert SO.iteration_latency(luts, sel, 2, 2, 2) == 2 + 22 + 4 + 20
    assert SO.iteration_latency(luts, sel, 2, 2, 0) == 0
    extra = ([1, 3], [100.0, 300.0])
    assert SO.iteration_latency(luts, sel, 2, 2, 2, extra) == 48 + 2 * 200


def test_oracle_chunk_closed_form():
    """Linear tables through the origin give T(M) = a M: the largest chunk
    is floor((T_SLO - a d) / a), clipped to [c_min, c_max], or 0."""
    luts = [([1, 1000], [3.0, 3000.0], [5.0, 5000.0])]
    sel = [[1], [0], [1]]          # a = 5 + 3 + 5 = 13 per token
    for d, slo, lo, hi in [(4, 500.0, 1, 64), (0, 130.0, 1, 64), (10, 100.0, 1, 64),
                           (2, 1000.0, 8, 40), (1, 13.0 * 20, 16, 64)]:
        exp = int((Fraction(slo) - 13 * d) // 13)
        exp = min(exp, hi)
        exp = exp if exp >= lo else 0
        assert SO.chunk(luts, sel, 3, 1, d, slo, lo, hi) == exp, (d, slo, lo, hi)


def test_oracle_monotone_in_slo_and_d():
    rng = random.Random(5)
    luts = [(sorted(rng.sample(range(1, 300), 5)),
             sorted(rng.uniform(1, 50) for _ in range(5)),
             sorted(rng.uniform(1, 60) for _ in range(5))) for _ in range(3)]
    sel = [[rng.random() < 0.4 for _ in range(3)] for _ in range(4)]
    prev = -1
    for slo in (50.0, 200.0, 400.0, 800.0, 1600.0):
        c = SO.chunk(luts, sel, 4, 3, 8, slo, 1, 256)
        assert c >= prev or c == 0
        prev = max(prev, c)
    cs = [SO.chunk(luts, sel, 4, 3, d, 900.0, 1, 256) for d in (0, 16, 64, 128)]
    assert all(a >= b for a, b in zip(cs, cs[1:]))


# ---------------------------------------------------------------------------
# the library against the oracle
# ---------------------------------------------------------------------------

def _random_case(rng, modules, layers, n):
    luts = []
    for _ in range(modules):
        M = sorted(rng.sample(range(1, 5000), n))
        lw = [rng.uniform(2.0, 300.0) for _ in range(n)]   # unsorted: noisy tables
        le = [v + rng.uniform(0.0, 40.0) for v in lw]
        luts.append((M, lw, le))
    sel = [[int(rng.random() < 0.35) for _ in range(modules)] for _ in range(layers)]
    return luts, sel


@pytest.mark.parametrize("seed", range(6))
def test_library_latency_matches_oracle(seed):
    rng = random.Random(seed)
    luts, sel = _random_case(rng, modules=rng.randint(1, 7), layers=rng.randint(1, 12),
                             n=rng.randint(1, 9))
    extra = ([1, 64, 4096], [5.0, 9.0, 80.0]) if seed % 2 else None
    mdl = _model(luts, sel, extra)
    for m in [0, 1, 2, 3, 7, 31, 100, 999, 4999, 5000, 7000, 20000]:
        want = SO.iteration_latency(luts, sel, len(sel), len(luts), m, extra)
        got = sp.sched_latency(mdl, m)
        assert abs(got - float(want)) <= 1e-9 * max(1.0, float(want)), (m, got, float(want))


@pytest.mark.parametrize("seed", range(6))
def test_library_chunk_matches_brute_force(seed):
    """The binary search returns exactly the oracle's chunk (SLO targets are
    drawn away from the estimate's rounding-level ties)."""
    rng = random.Random(100 + seed)
    luts, sel = _random_case(rng, modules=rng.randint(1, 4), layers=rng.randint(1, 6),
                             n=rng.randint(2, 6))
    mdl = _model(luts, sel)
    L, Mo = len(sel), len(luts)
    for _ in range(12):
        d = rng.randint(0, 64)
        lo = rng.randint(1, 40)
        hi = lo + rng.randint(0, 300)
        base = float(SO.iteration_latency(luts, sel, L, Mo, d))
        slo = base + rng.uniform(0.0, 2.5) * float(SO.iteration_latency(luts, sel, L, Mo, hi))
        want = SO.chunk(luts, sel, L, Mo, d, slo, lo, hi)
        got = sp.sched_chunk(mdl, d, slo, lo, hi)
        if want != got:
            # only a tie within rounding may differ: check the boundary
            t = lambda c: SO.iteration_latency(luts, sel, L, Mo, c)
            edge = max(want, got)
            assert abs(float(SO.iteration_latency(luts, sel, L, Mo, d) + t(edge)) - slo) < 1e-9 * slo
        else:
            assert got == want


def test_library_chunk_exact_ties_on_integer_tables():
    """Integer-valued tables make the estimate exact in binary floating
    point: T(d) + T(c) == T_SLO counts as fitting, as in the oracle."""
    luts = [([1, 100], [2.0, 200.0], [3.0, 300.0]), ([1, 100], [1.0, 100.0], [1.0, 100.0])]
    sel = [[1, 0], [0, 0]]      # T(M) = 3M + M + 2M + M = 7M on the grid M <= 100
    mdl = _model(luts, sel)
    for d in (0, 3, 10):
        for c_star in (1, 5, 40, 90):
            slo = float(7 * d + 7 * c_star)
            assert SO.chunk(luts, sel, 2, 2, d, slo, 1, 100) == c_star
            assert sp.sched_chunk(mdl, d, slo, 1, 100) == c_star
            assert sp.sched_chunk(mdl, d, slo - 0.5, 1, 100) == c_star - 1


def test_library_edge_cases_and_errors():
    luts = [([8, 64], [10.0, 40.0], [12.0, 50.0])]
    mdl = _model(luts, [[1], [0]])
    assert sp.sched_latency(mdl, 0) == 0.0
    assert sp.sched_chunk(mdl, 0, 1.0, 1, 128) == 0            # nothing fits
    assert sp.sched_chunk(mdl, 0, 1e9, 1, 128) == 128          # everything fits
    assert sp.sched_chunk(mdl, 0, 1e9, 5, 5) == 5
    with pytest.raises(sp.SpearError) as e:
        sp.sched_chunk(mdl, 0, 10.0, 0, 5)
    assert e.value.status == -2
    with pytest.raises(sp.SpearError):
        sp.sched_chunk(mdl, -1, 10.0, 1, 5)
    with pytest.raises(sp.SpearError):
        sp.sched_chunk(mdl, 0, 10.0, 9, 5)
    for bad in ([([8, 8], [1.0, 2.0], [1.0, 2.0])], [([0, 8], [1.0, 2.0], [1.0, 2.0])],
                [([8, 9], [1.0, -2.0], [1.0, 2.0])], [([8, 9], [1.0, float("nan")], [1.0, 2.0])]):
        with pytest.raises(sp.SpearError) as e:
            sp.sched_latency(_model(bad, [[0]]), 4)
        assert e.value.status == -2
    import ctypes
    out = ctypes.c_double()
    assert sp.LIB.spear_sched_latency(None, 4, ctypes.byref(out)) == -1
    assert sp.LIB.spear_sched_latency(ctypes.byref(mdl.c), 4, None) == -1
