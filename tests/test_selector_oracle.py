"""Pins for the selector oracle: worked values, closed forms, properties."""
import json
import os
from fractions import Fraction

import pytest

from oracle import selector as sel

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_hand_example():
    """G=10, o_comm=1, o_comp=2, W_comp=30, W_comm=6, L=2, rho=3/2.

    Worked by hand from the equations (P = 2(10-C); A_s = ceil((s+1)30/P);
    q = 1.5 ceil(6/C); F_s = max(A_s, F_{s-1}) + q; Delta = ceil(30/P) P - 30):
      C=1: P=18 A=(2,4) q=9   T=20   Delta=6
      C=2: P=16 A=(2,4) q=4.5 T=11   Delta=2
      C=3: P=14 A=(3,5) q=3   T=9    Delta=12
      C=4: P=12 A=(3,5) q=3   T=9    Delta=6
      C=5: P=10 A=(3,6) q=3   T=9    Delta=0
      C=6: P=8  A=(4,8) q=1.5 T=9.5  Delta=2
    """
    want = {1: (18, [2, 4], Fraction(9), Fraction(20), 6),
            2: (16, [2, 4], Fraction(9, 2), Fraction(11), 2),
            3: (14, [3, 5], Fraction(3), Fraction(9), 12),
            4: (12, [3, 5], Fraction(3), Fraction(9), 6),
            5: (10, [3, 6], Fraction(3), Fraction(9), 0),
            6: (8, [4, 8], Fraction(3, 2), Fraction(19, 2), 2)}
    rho = Fraction(3, 2)
    for C, (P, A, q, T, d) in want.items():
        c = sel.evaluate(C, 30, 6, 2, 10, 1, 2, rho)
        assert (c.P, c.A, c.q, c.T, c.delta) == (P, A, q, T, d)
    best, _ = sel.select_from_work(30, 6, 2, 10, 1, 2, rho, 1, 6)
    assert best.C == 5                       # three-way tie on T, Delta decides
    best4, _ = sel.select_from_work(30, 6, 2, 10, 1, 2, rho, 1, 4)
    assert best4.C == 4


def test_rho_reference_worked_value():
    g = _gold("rho_reference.json")
    rho = (g["comm_time_us"] / g["comm_splits"]) / \
        (g["compute_time_us"] / g["compute_waves"])
    assert abs(rho - g["printed_rho_ref"]) < 0.01


def test_a100_instance_closed_forms():
    g = _gold("a100_instance.json")
    for C in range(g["c_min"], g["c_max"] + 1):
        c = sel.evaluate(C, 1000, 40, 2, g["G"], g["o_comm"], g["o_comp"],
                         Fraction(10))
        assert c.R == C                        # o_comm = 1 => R(C) = C
        assert c.P == 2 * (108 - C)            # P(C) = 2(G - C)
    # rho at the reference configuration equals rho_ref
    r = sel.rho_scaled(Fraction(1005, 100), g["K_ref"], g["K_ref"],
                       g["tile_m_ref"], g["tile_n_ref"], g["tile_m_ref"],
                       g["tile_n_ref"], g["D_ref"], g["D_ref"])
    assert r == Fraction(1005, 100)
    # doubling K halves rho; a 2x larger tile halves it; 2x ranks doubles it
    r2 = sel.rho_scaled(Fraction(10), 704, 352, 128, 256, 128, 128, 8, 4)
    assert r2 == Fraction(10) / 2 / 2 * 2


def test_single_split_closed_form():
    """L = 1: T(C) = ceil(W_comp / P) + rho ceil(W_comm / C)."""
    rho = Fraction(7, 3)
    for W_comp, W_comm in [(1, 1), (100, 7), (4096, 128), (333, 1000)]:
        for C in range(1, 40):
            c = sel.evaluate(C, W_comp, W_comm, 1, 64, 2, 3, rho)
            if c is None:
                assert 3 * (64 - sel.cdiv(C, 2)) <= 0
                continue
            assert c.T == sel.cdiv(W_comp, c.P) + rho * sel.cdiv(W_comm, C)


def test_work_formulas():
    # routed-tile reduction and compute work (g = 1)
    assert sel.routed_m_tiles([0, 1, 128, 129, 256], 128, 5, 514) == 0 + 1 + 1 + 2 + 2
    assert sel.compute_work(6, 2048, 2, 256) == 6 * 4
    assert sel.compute_work(6, 1000, 3, 128) == 6 * 3     # ceil(334/128) = 3
    assert sel.comm_work(16384, 1, 2048, 2, 128, 1024) == 128
    assert sel.comm_work(1000, 4, 2048, 1, 128, 1024) == 2 * 2
    # even-load estimate without host counts
    assert sel.routed_m_tiles(None, 256, 32, 98304) == 32 * 12


def test_structural_properties():
    rho = Fraction(13, 10)
    W_comp, W_comm, L, G = 1600, 128, 2, 256
    prev = None
    for C in range(1, 65):
        c = sel.evaluate(C, W_comp, W_comm, L, G, 1, 1, rho)
        assert c.F[0] >= c.A[0] + c.q
        assert c.T >= L * c.q
        for s in range(1, L):
            assert c.F[s] >= c.F[s - 1] + c.q
            assert c.A[s] >= c.A[s - 1]
        if prev is not None:
            assert c.V_comm <= prev.V_comm      # non-increasing in C
            assert c.P < prev.P                 # capacity shrinks with C
            assert all(a >= b for a, b in zip(c.A, prev.A))
        prev = c


def test_selection_is_the_exhaustive_argmin():
    import random
    rnd = random.Random(0)
    for _ in range(300):
        W_comp, W_comm = rnd.randint(1, 5000), rnd.randint(1, 500)
        L, G = rnd.randint(1, 4), rnd.randint(2, 300)
        o1, o2 = rnd.randint(1, 4), rnd.randint(1, 4)
        rho = Fraction(rnd.randint(1, 400), rnd.randint(1, 40))
        best, cands = sel.select_from_work(W_comp, W_comm, L, G, o1, o2, rho, 1, 64)
        if not cands:
            assert best is None
            continue
        tmin = min(c.T for c in cands)
        assert best.T == tmin
        ties = [c for c in cands if c.T == tmin]
        assert best.delta == min(c.delta for c in ties)
        assert best.C == min(c.C for c in ties if c.delta == best.delta)


def test_no_legal_partition():
    best, cands = sel.select_from_work(10, 10, 1, 2, 1, 1, Fraction(1), 2, 8)
    assert best is None and cands == []


def test_role_switch_candidate_closed_form():
    """C = 0 (an extension, only when c_min = 0): all o_comp G slots compute
    every tile, then serve every consumer task."""
    rho = Fraction(5, 2)
    for W_comp, W_comm, L, G, o in [(1600, 128, 2, 256, 1), (30, 6, 2, 10, 2), (7, 1, 1, 3, 1)]:
        c = sel.evaluate(0, W_comp, W_comm, L, G, 1, o, rho)
        P0 = o * G
        assert c.P == P0 and c.R == 0
        assert c.T == sel.cdiv(L * W_comp, P0) + rho * sel.cdiv(L * W_comm, P0)
    best, cands = sel.select_from_work(30, 6, 2, 10, 1, 2, Fraction(3, 2), 0, 6)
    assert cands[0].C == 0 and cands[0].T == 3 + Fraction(3, 2) * 1
    assert best.C == 0                      # 4.5 beats the paper's best (9)
    best1, _ = sel.select_from_work(30, 6, 2, 10, 1, 2, Fraction(3, 2), 1, 6)
    assert best1.C == 5
