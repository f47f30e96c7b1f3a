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


# ---- the extensions: token-band work counts, the drain term, L as a variable ----

def test_band_work_counts_by_hand():
    """10 routed m-tiles, N = 1024 in 256-wide tiles, T = 1000 tokens in
    64-token x 1024-column consumer tasks, L = 4.
    Column splits: W_comp = 10 * ceil(256/256) = 10, W_comm = ceil(1000/64)
    * ceil(256/1024) = 16.  Token bands: W_comp = ceil(10/4) * 4 = 12,
    W_comm = ceil(16/4) * 1 = 4."""
    assert sel.compute_work(10, 1024, 4, 256) == 10
    assert sel.comm_work(1000, 1, 1024, 4, 64, 1024) == 16
    assert sel.compute_work(10, 1024, 4, 256, split_axis=1) == 12
    assert sel.comm_work(1000, 1, 1024, 4, 64, 1024, split_axis=1) == 4
    # with one split both axes describe the same work
    for m, N, T in ((37, 2048, 16384), (5, 200, 3), (1, 64, 1)):
        assert sel.compute_work(m, N, 1, 256) == sel.compute_work(m, N, 1, 256, split_axis=1)
        assert sel.comm_work(T, 1, N, 1, 64, 1024) == sel.comm_work(T, 1, N, 1, 64, 1024,
                                                                    split_axis=1)


def test_drain_hand_example():
    """G=10, o_comm=o_comp=1, W_comp=30, W_comm=6, L=2, rho=3/2, drain.

    Worked by hand (P = 10 - C; A_s = ceil((s+1) 30 / P); the first split is
    served by the C consumers, q = 1.5 ceil(6/C); the last by all C + P = 10
    slots, 1.5 ceil(6/10) = 1.5):
      C=1: P=9 A=(4,7)  F0=4+9=13     T=max(7,13)+1.5=14.5
      C=2: P=8 A=(4,8)  F0=4+4.5=8.5  T=max(8,8.5)+1.5=10
      C=3: P=7 A=(5,9)  F0=5+3=8      T=max(9,8)+1.5=10.5
      C=4: P=6 A=(5,10) F0=5+3=8      T=10+1.5=11.5
      C=5: P=5 A=(6,12) F0=6+3=9      T=12+1.5=13.5
      C=6: P=4 A=(8,15) F0=8+1.5=9.5  T=15+1.5=16.5
    and without the drain term (the paper's recurrence) the last split also
    takes q: T = 22, 13, 12, 13, 15, 16.5."""
    rho = Fraction(3, 2)
    want = {1: ([4, 7], Fraction(29, 2), Fraction(22)), 2: ([4, 8], Fraction(10), Fraction(13)),
            3: ([5, 9], Fraction(21, 2), Fraction(12)), 4: ([5, 10], Fraction(23, 2), Fraction(13)),
            5: ([6, 12], Fraction(27, 2), Fraction(15)),
            6: ([8, 15], Fraction(33, 2), Fraction(33, 2))}
    for C, (A, T_drain, T_plain) in want.items():
        c = sel.evaluate(C, 30, 6, 2, 10, 1, 1, rho, drain=True)
        assert (c.A, c.T) == (A, T_drain), C
        assert sel.evaluate(C, 30, 6, 2, 10, 1, 1, rho).T == T_plain, C
    best, _ = sel.select_from_work(30, 6, 2, 10, 1, 1, rho, 1, 6, drain=True)
    assert (best.C, best.T) == (2, 10)
    best, _ = sel.select_from_work(30, 6, 2, 10, 1, 1, rho, 1, 6)
    assert (best.C, best.T) == (3, 12)


def test_drain_single_split_closed_form():
    """L = 1: T(C) = ceil(W_comp/P) + rho ceil(W_comm/(C+P)) with drain."""
    for (W, Wc, G, rho) in ((100, 37, 16, Fraction(7, 5)), (1, 1, 2, Fraction(1)),
                            (513, 99, 256, Fraction(141, 100))):
        for C in range(1, G):
            P = G - C
            c = sel.evaluate(C, W, Wc, 1, G, 1, 1, rho, drain=True)
            assert c.T == sel.cdiv(W, P) + rho * sel.cdiv(Wc, C + P)


def test_split_count_as_a_decision_variable_by_hand():
    """Token bands, G=10, o=1, rho=1, 40 routed m-tiles over one 256-wide
    n-tile, T=1280 tokens in 64-token tasks (20 token blocks), one column
    block; candidates C = 1..3.  Per L (W_comp = ceil(40/L), W_comm =
    ceil(20/L)), worked by hand:
      L=1: C=3 best: P=7, A=ceil(40/7)=6, q=ceil(20/3)=7       -> T=13
      L=2: C=3 best: P=7, A=(3,6), q=ceil(10/3)=4, F=(7,11)    -> T=11
      L=3: C=3 best: P=7, A=(2,4,6), q=ceil(7/3)=3, F=(5,8,11) -> T=11
      L=4: C=3 best: P=7, A=(2,3,5,6), q=ceil(5/3)=2,
           F=(4,6,8,10)                                        -> T=10
    so L in 1..4 picks (L=4, C=3, T=10) and L in 1..2 picks (L=2, C=3)."""
    p = sel.SelectParams(tile_m=256, tile_n=256, comm_tile_m=64, comm_tile_n=1024,
                         occ_comp=1, occ_comm=1, num_cus=10, c_min=1, c_max=3,
                         rho_ref=Fraction(1), k_ref=704, tile_m_ref=256, tile_n_ref=256,
                         d_ref=1, split_axis=1)
    counts = [256 * 10] * 4                   # 4 experts x 10 m-tiles = 40
    per_L = {1: (3, Fraction(13)), 2: (3, Fraction(11)), 4: (3, Fraction(10))}
    for L, (C, T) in per_L.items():
        best, _, W_comp, W_comm, rho = sel.select(1280, 256, 704, 4, 8, L, counts, p)
        assert (W_comp, W_comm, rho) == (sel.cdiv(40, L), sel.cdiv(20, L), 1)
        assert (best.C, best.T) == (C, T), L
    L, best = sel.select_splits(1280, 256, 704, 4, 8, counts, p, 1, 4)
    assert (L, best.C, best.T) == (4, 3, Fraction(10))
    L, best = sel.select_splits(1280, 256, 704, 4, 8, counts, p, 1, 2)
    assert (L, best.C, best.T) == (2, 3, Fraction(11))


def test_task_bytes_factor_by_hand():
    """The k/H-aware extension's factor: (2k + 4) / (2k_ref + 4) times the
    task width over the calibration's (a task reads k bf16 rows and writes
    one fp32 output per token and column)."""
    assert sel.task_bytes_factor(6, 6, 1024, 1024) == 1
    assert sel.task_bytes_factor(4, 6, 512, 1024) == Fraction(12, 16) * Fraction(1, 2)
    assert sel.task_bytes_factor(8, 6, 1024, 1024) == Fraction(20, 16)
    # the task width: a split's columns capped at the task tile (column
    # splits), or the full width capped (token bands)
    assert sel.task_width(2048, 2, 1024) == 1024
    assert sel.task_width(1024, 4, 1024) == 256
    assert sel.task_width(200, 5, 1024) == 40
    assert sel.task_width(200, 5, 1024, split_axis=1) == 200
    assert sel.task_width(4096, 1, 1024, split_axis=1) == 1024


def test_rho_kh_changes_the_pick_by_hand():
    """The hand instance (G = 10, o_comm = 1, o_comp = 2, W_comp = 30,
    W_comm = 6, L = 2, rho = 3/2 gives C* = 5) with rho scaled by 1/2:
    T(C = 1..6) = 11, 6.5, 6.5, 6.5, 7.5, 8.75, ties broken by Delta
    (2, 12, 6 for C = 2, 3, 4), so C* = 2."""
    rho = sel.rho_scaled(Fraction(3, 2), 8, 8, 1, 1, 1, 1, 1, 1) * \
        sel.task_bytes_factor(1, 1, 1, 2)
    assert rho == Fraction(3, 4)
    best, cands = sel.select_from_work(30, 6, 2, 10, 1, 2, rho, 1, 6)
    assert [c.T for c in cands] == [11, Fraction(13, 2), Fraction(13, 2), Fraction(13, 2),
                                    Fraction(15, 2), Fraction(35, 4)]
    assert [c.delta for c in cands[1:4]] == [2, 12, 6]
    assert best.C == 2
    best0, _ = sel.select_from_work(30, 6, 2, 10, 1, 2, Fraction(3, 2), 1, 6)
    assert best0.C == 5


def test_per_wave_readiness_by_hand():
    """readiness = 1 on a small instance worked by hand: G = 4, o_comm =
    o_comp = 1, W_comp = 6, W_comm = 3, L = 1, rho = 2.
    C = 1 (P = 3): waves end 3, 6 tiles and release ceil(3/2) = 2, then 1
    task: F = 1 + 2*2 = 5, then max(2, 5) + 2*1 = 7.
    C = 2 (P = 2): three waves release 1 task each: F = 3, 5, 7.
    C = 3 (P = 1): six waves release 1, 0, 1, 0, 1, 0: F = 3, 3, 5, 5, 7, 7.
    All tie at 7 with Delta = 0, so C* = 1; the split-level model of the
    paper gives T = 8, 7, 8 (A_0 = 2, 3, 6 and q = 6, 4, 2) and C* = 2."""
    best, cands = sel.select_from_work(6, 3, 1, 4, 1, 1, Fraction(2), 1, 4, readiness=1)
    assert [c.C for c in cands] == [1, 2, 3]
    assert [c.F for c in cands] == [[5, 7], [3, 5, 7], [3, 3, 5, 5, 7, 7]]
    assert [c.A for c in cands] == [[1, 2], [1, 2, 3], [1, 2, 3, 4, 5, 6]]
    assert [c.delta for c in cands] == [0, 0, 0]
    assert best.C == 1
    best0, cands0 = sel.select_from_work(6, 3, 1, 4, 1, 1, Fraction(2), 1, 4)
    assert [c.T for c in cands0] == [8, 7, 8] and best0.C == 2
    # with the drain the last wave is served by C + P slots: C = 1 (P = 3)
    # then ends at max(2, 5) + 2 * ceil(1 / 4) = 7 as well, C = 3 unchanged
    bd, cd = sel.select_from_work(6, 3, 1, 4, 1, 1, Fraction(2), 1, 4, drain=True,
                                  readiness=1)
    assert [c.T for c in cd] == [7, 7, 7]


def test_per_wave_readiness_releases_every_task_once():
    """The released counts add up to all tasks, each wave's release is what
    its completed tiles cover, and no wave is served before it ends."""
    import random
    rnd = random.Random(3)
    for _ in range(300):
        W_comp, W_comm = rnd.randint(0, 400), rnd.randint(1, 300)
        L, G = rnd.randint(1, 4), rnd.randint(2, 64)
        C = rnd.randint(1, G - 1)
        c = sel.evaluate(C, W_comp, W_comm, L, G, 1, 1, Fraction(rnd.randint(1, 9), 4),
                         readiness=1)
        P = G - C
        if L * W_comp == 0:
            assert len(c.F) == 1
            continue
        assert len(c.A) == -(-L * W_comp // P)
        assert all(f >= a for a, f in zip(c.A, c.F))
        assert all(b >= a for a, b in zip(c.F, c.F[1:]))
        # served at least as the split-level model's single last split
        assert c.T >= Fraction(c.A[-1])


def test_finer_last_split_hand_example():
    """The hand example's workload (G=10, o_comm=1, o_comp=2, W_comp=30,
    W_comm=6, L=2, rho=3/2, 30 tokens in tasks of 5) with the last split's
    tasks cut to 2 tokens: W_last = ceil(30/2) = 15 tasks of
    rho_last = 3/2 * 2/5 = 3/5, a : b = 5 : 2.  By hand:
      C=5: P=10, A=(3,6), F_0 = 3 + 3/2 ceil(6/5) = 6,
           F_1 = max(6, 6) + 3/5 ceil(15/5) = 39/5   (the paper's model: 9);
      C=2: P=16, A=(2,4), F_0 = 2 + 3/2 ceil(6/2) = 13/2,
           F_1 = 13/2 + 3/5 ceil(15/2) = 13/2 + 24/5 = 113/10   (the paper's model: 11);
      C=0: P0=20, A=ceil(60/20)=3, units = 5*1*6 + 2*15 = 60,
           T = 3 + (3/2)/5 ceil(60/20) = 39/10       (the paper's extension: 9/2).
    """
    rho = Fraction(3, 2)
    last = sel.LastSplit(W=15, rho=Fraction(3, 5), a=5, b=2)
    c5 = sel.evaluate(5, 30, 6, 2, 10, 1, 2, rho, last=last)
    assert (c5.P, c5.A, c5.F) == (10, [3, 6], [Fraction(6), Fraction(39, 5)])
    c2 = sel.evaluate(2, 30, 6, 2, 10, 1, 2, rho, last=last)
    assert (c2.A, c2.F) == ([2, 4], [Fraction(13, 2), Fraction(113, 10)])
    c0 = sel.evaluate(0, 30, 6, 2, 10, 1, 2, rho, last=last)
    assert (c0.P, c0.T) == (20, Fraction(39, 10))
    # through select(): one expert of 30 rows, 1-row tiles, two 1-column splits
    p = sel.SelectParams(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                         occ_comm=1, num_cus=10, c_min=0, c_max=6, rho_ref=Fraction(3, 2),
                         k_ref=8, tile_m_ref=1, tile_n_ref=1, d_ref=1, comm_tile_m_last=2)
    best, cands, W_comp, W_comm, r = sel.select(30, 2, 8, 1, 1, 2, [30], p)
    assert (W_comp, W_comm, r) == (30, 6, rho)
    byC = {c.C: c.T for c in cands}
    assert byC[5] == Fraction(39, 5) and byC[2] == Fraction(113, 10) and byC[0] == Fraction(39, 10)
    assert best.C == 0


def test_finer_last_split_reduces_to_the_paper_model():
    """T_M^last = T_M^comm (or 0) is the model without the extension, for
    every candidate, with and without drain."""
    for drain in (False, True):
        for tm_last in (0, 64):
            p = sel.SelectParams(tile_m=256, tile_n=256, comm_tile_m=64, comm_tile_n=1024,
                                 occ_comp=1, occ_comm=1, num_cus=256, c_min=0, c_max=64,
                                 rho_ref=Fraction(148, 100), k_ref=704, tile_m_ref=256,
                                 tile_n_ref=256, d_ref=1, drain=drain, comm_tile_m_last=tm_last)
            counts = [3072 + 97 * (e % 7) for e in range(32)]
            _, cands, W_comp, W_comm, rho = sel.select(16384, 2048, 704, 32, 6, 2, counts, p)
            assert sel.last_split(16384, 1, 2048, 2, p, rho) is None
            for c in cands:
                ref = sel.evaluate(c.C, W_comp, W_comm, 2, 256, 1, 1, rho, drain)
                assert c.T == ref.T and c.F == ref.F


def test_finer_last_split_service_by_brute_force():
    """For C >= 1 the last split's service is rho_last times the number of
    rounds in which C consumers clear W_last tasks, found by simulating the
    rounds one at a time; the splits before it are unchanged."""
    rho = Fraction(7, 3)
    for W_last, C in ((1, 1), (15, 4), (16, 4), (17, 4), (100, 7), (3, 50)):
        last = sel.LastSplit(W=W_last, rho=rho / 2, a=2, b=1)
        c = sel.evaluate(C, 40, 9, 3, 64, 1, 1, rho, last=last)
        ref = sel.evaluate(C, 40, 9, 3, 64, 1, 1, rho)
        left, rounds = W_last, 0
        while left > 0:
            left -= min(C, left)
            rounds += 1
        assert c.F[:2] == ref.F[:2]
        assert c.F[2] - max(Fraction(c.A[2]), c.F[1]) == rho / 2 * rounds


def test_finer_last_split_needs_column_splits():
    p = sel.SelectParams(tile_m=256, tile_n=256, comm_tile_m=64, comm_tile_n=1024, occ_comp=1,
                         occ_comm=1, num_cus=256, c_min=0, c_max=8, rho_ref=Fraction(1),
                         k_ref=704, tile_m_ref=256, tile_n_ref=256, d_ref=1,
                         comm_tile_m_last=32, split_axis=1)
    with pytest.raises(ValueError):
        sel.select(4096, 2048, 704, 8, 2, 2, None, p)


def test_work_conserving_drain_hand_example():
    """The hand example's workload (G=10, o_comm=1, o_comp=2, W_comp=30,
    W_comm=6, L=2, rho=3/2) with drain = 2, worked by hand:
      C=1: P=18, A=(2,4), E=4; split 0 from 2 needs 6 rounds, 2 begin before
           E (at 2 and 3.5): 2 tasks claimed, the last round ends at 5;
           R = 10, T = max(4 + 1.5 ceil(10/19), 5) = 11/2
           (drain = 1: F_0 = 2 + 9 = 11, T = 11 + 1.5 = 25/2);
      C=2: P=16, A=(2,4); 3 rounds needed, 2 begin before E: 4 claimed, the
           last ends at 5; R = 8, T = max(4 + 1.5 ceil(8/18), 5) = 11/2
           (drain = 1: 8);
      C=5: P=10, A=(3,6), E=6; 2 rounds needed, both begin before E: split 0
           ends at 6, R = 6, T = max(6 + 1.5 ceil(6/15), 6) = 15/2
           (= drain 1's 15/2).
    """
    rho = Fraction(3, 2)
    want = {1: ([2, 4], [Fraction(11, 2), Fraction(11, 2)], Fraction(11, 2)),
            2: ([2, 4], [Fraction(11, 2), Fraction(11, 2)], Fraction(11, 2)),
            5: ([3, 6], [Fraction(6), Fraction(15, 2)], Fraction(15, 2))}
    for C, (A, F, T) in want.items():
        c = sel.evaluate(C, 30, 6, 2, 10, 1, 2, rho, drain=2)
        assert (c.A, c.F, c.T) == (A, F, T), C
    assert sel.evaluate(1, 30, 6, 2, 10, 1, 2, rho, drain=1).T == Fraction(25, 2)
    assert sel.evaluate(2, 30, 6, 2, 10, 1, 2, rho, drain=1).T == 8
    assert sel.evaluate(5, 30, 6, 2, 10, 1, 2, rho, drain=1).T == Fraction(15, 2)


def test_idle_slots_and_split_cost_hand_example():
    """drain = 2 on G=10, o=1, W_comp=13, W_comm=12, L=2, rho=1/2, worked by
    hand (the idle compute slots of the last compute wave, and the split
    cost pi):
      C=0: P0=10, 26 tiles in V=3 waves, Idle = 30 - 26 = 4 slots free from
           E - 1 = 2; split 0 is ready (A_0 = ceil(13/10) = 2 <= 2); they
           begin ceil(1/rho) = 2 rounds before E = 3 and take 8 of its 12
           tasks, ending at 2 + 2 rho = 3; R = 24 - 8 = 16,
           T = max(3 + rho ceil(16/10), 3) = 4, against 3 + rho ceil(24/10)
           = 9/2 without the idle slots, and 9/2 for the same work in one
           split (L=1: nothing is ready before E);
      C=0, pi=1/4: E = 3 + 1/4 = 13/4, the idle slots from 9/4 (split 0
           ready) take 8 in 2 rounds ending at 13/4; T = 13/4 + 1 = 17/4;
      C=2: P=8, A=(2,4)=(A_0,E), V=4, Idle=6; the consumers begin 4 rounds
           before E (2, 5/2, 3, 7/2) and claim 8, the last ending at 4; the
           idle slots from 3 take the other 4 (one round, ending at 7/2);
           R = 12, T = max(4 + rho ceil(12/10), 4) = 5;
      C=2, pi=1/4: A = (2, 17/4); the consumers begin 5 rounds before E and
           claim 10 (ending at 9/2), the idle slots from 13/4 the other 2;
           R = 12, T = 17/4 + 1 = 21/4; and the paper's recurrence with the
           same pi: F_0 = 2 + 6 rho = 5, F_1 = max(17/4, 5) + 6 rho = 8."""
    rho = Fraction(1, 2)
    c = sel.evaluate(0, 13, 12, 2, 10, 1, 1, rho, drain=2)
    assert (c.A, c.F, c.T) == ([3], [4], 4)
    assert sel.evaluate(0, 13, 12, 2, 10, 1, 1, rho).T == Fraction(9, 2)
    assert sel.evaluate(0, 26, 24, 1, 10, 1, 1, rho, drain=2).T == Fraction(9, 2)
    c = sel.evaluate(0, 13, 12, 2, 10, 1, 1, rho, drain=2, pi=Fraction(1, 4))
    assert (c.A, c.T) == ([Fraction(13, 4)], Fraction(17, 4))
    c = sel.evaluate(2, 13, 12, 2, 10, 1, 1, rho, drain=2)
    assert (c.A, c.F, c.T) == ([2, 4], [5, 5], 5)
    c = sel.evaluate(2, 13, 12, 2, 10, 1, 1, rho, drain=2, pi=Fraction(1, 4))
    assert (c.A, c.F, c.T) == ([2, Fraction(17, 4)], [Fraction(21, 4)] * 2, Fraction(21, 4))
    c = sel.evaluate(2, 13, 12, 2, 10, 1, 1, rho, pi=Fraction(1, 4))
    assert (c.A, c.F, c.T) == ([2, Fraction(17, 4)], [5, 8], 8)
    # the split cost scales like rho's first two factors
    p = sel.SelectParams(tile_m=128, tile_n=256, comm_tile_m=64, comm_tile_n=1024, occ_comp=1,
                         occ_comm=1, num_cus=256, c_min=0, c_max=8, rho_ref=Fraction(1),
                         k_ref=704, tile_m_ref=256, tile_n_ref=256, d_ref=1,
                         split_cost=Fraction(43, 100))
    assert sel.split_cost(p, 1408) == Fraction(43, 100) * Fraction(1, 2) * 2


def test_work_conserving_drain_properties():
    """drain = 2 never predicts a later end than drain = 1 (the compute slots
    only add service), equals it where the consumers finish every split but
    the last by the time the compute ends (and for L = 1), and matches a
    direct simulation of the consumers' rounds."""
    import random
    rnd = random.Random(7)
    n_equal = 0
    for _ in range(400):
        W_comp, W_comm = rnd.randint(0, 600), rnd.randint(0, 300)
        L, G, o = rnd.randint(1, 5), rnd.randint(2, 40), rnd.randint(1, 2)
        rho = Fraction(rnd.randint(1, 50), rnd.randint(1, 20))
        for C in range(1, min(12, G)):
            c2 = sel.evaluate(C, W_comp, W_comm, L, G, 1, o, rho, drain=2)
            if c2 is None:
                continue
            c1 = sel.evaluate(C, W_comp, W_comm, L, G, 1, o, rho, drain=1)
            assert c2.T <= c1.T
            if L == 1 or c1.F[L - 2] <= c1.A[L - 1]:
                assert c2.T == c1.T
                n_equal += 1
            assert c2.T == _simulate_work_conserving(C, c2.P, c2.A, W_comp, W_comm, L, rho)
        # the role switch: no consumers, the compute slots only
        c0 = sel.evaluate(0, W_comp, W_comm, L, G, 1, o, rho, drain=2)
        A0 = [Fraction(sel.cdiv((s + 1) * W_comp, o * G)) for s in range(L)]
        assert c0.T == _simulate_work_conserving(0, o * G, A0, W_comp, W_comm, L, rho)
        assert c0.T <= sel.evaluate(0, W_comp, W_comm, L, G, 1, o, rho).T
    assert n_equal > 100


def _simulate_work_conserving(C, P, A, W_comp, W_comm, L, rho):
    """The drain = 2 model by direct simulation, one round at a time: the
    consumers' rounds that begin before E each claim up to C tasks of the
    current split; then the compute slots idle in the last compute wave,
    from E - 1, claim up to that many tasks per round of the splits ready by
    then, in rounds that begin before E; every slot serves the rest."""
    E, t, claimed, last = Fraction(A[L - 1]), None, 0, Fraction(0)
    for s in range(L - 1 if C > 0 else 0):
        t = Fraction(A[s]) if t is None else max(Fraction(A[s]), t)
        left = W_comm
        while left > 0 and t < E:
            k = min(C, left)
            left -= k
            claimed += k
            t += rho
            last = t
        if left > 0:
            break
    V = -(-(L * W_comp) // P)
    idle = V * P - L * W_comp
    if V > 0 and idle > 0:
        ready = sum(W_comm for s in range(L - 1) if A[s] <= E - 1)
        left = ready - claimed
        t = E - 1
        while left > 0 and t < E:
            k = min(idle, left)
            left -= k
            claimed += k
            t += rho
            last = max(last, t)
    return max(E + rho * sel.cdiv(L * W_comm - claimed, C + P), last)
