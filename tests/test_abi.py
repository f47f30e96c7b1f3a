"""The C ABI on the CPU: exports, the selector (bit-exact against the Python
oracle) and host-side validation.  Nothing here launches GPU work."""
import ctypes
import math
import os
import random
import re
from fractions import Fraction

import numpy as np
import pytest

from oracle import selector as osel
from paper_2609_07536_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "moe_gemm2.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_\w+)\s*\(", src)))


def test_library_exports_every_declared_function():
    L = B.lib()
    declared = _declared_functions()
    assert len(declared) >= 11
    for name in declared:
        assert hasattr(L, name), name
    assert set(declared) == set(B.EXPORTED)
    assert L.moe_gemm2_abi_version() == 108


def _params(**kw):
    p = B.SelectParams(tile_m=256, tile_n=256, comm_tile_m=128, comm_tile_n=1024,
                       occ_comp=1, occ_comm=1, num_cus=256, c_min=1, c_max=64, groups=1,
                       rho_ref_num=4, rho_ref_den=3, k_ref=704, tile_m_ref=256,
                       tile_n_ref=256, d_ref=1, rho_kh=0, topk_ref=6, comm_tile_n_ref=1024,
                       readiness=0, comm_tile_m_last=0)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _oracle_params(p):
    return osel.SelectParams(
        tile_m=p.tile_m, tile_n=p.tile_n, comm_tile_m=p.comm_tile_m,
        comm_tile_n=p.comm_tile_n, occ_comp=p.occ_comp, occ_comm=p.occ_comm,
        num_cus=p.num_cus, c_min=p.c_min, c_max=p.c_max,
        rho_ref=Fraction(p.rho_ref_num, p.rho_ref_den), k_ref=p.k_ref,
        tile_m_ref=p.tile_m_ref, tile_n_ref=p.tile_n_ref, d_ref=p.d_ref, groups=p.groups,
        split_axis=p.split_axis, drain=int(p.drain), rho_kh=bool(p.rho_kh),
        topk_ref=p.topk_ref, comm_tile_n_ref=p.comm_tile_n_ref, readiness=p.readiness,
        comm_tile_m_last=p.comm_tile_m_last,
        split_cost=(Fraction(p.split_cost_num, p.split_cost_den) if p.split_cost_num > 0
                    else Fraction(0)))


def _time_den(p, rho, I=None):
    """The library's time unit: rho's denominator, times a / gcd(rho's
    numerator, a) when the last split's tasks are cut finer
    (a : b = comm_tile_m : comm_tile_m_last in lowest terms), then the least
    common multiple with the split cost's denominator (K = I)."""
    tm_last = p.comm_tile_m_last or p.comm_tile_m
    a = p.comm_tile_m // math.gcd(p.comm_tile_m, tm_last)
    den = rho.denominator * a // math.gcd(rho.numerator, a)
    if p.split_cost_num > 0:
        pd = osel.split_cost(_oracle_params(p), I).denominator
        den = den * pd // math.gcd(den, pd)
    return den


def test_hand_example_through_the_abi():
    """G=10, o_comm=1, o_comp=2, W_comp=30, W_comm=6, L=2, rho=3/2 (C* = 5)."""
    # one expert with 30 rows, 1-row tiles, 2 columns in 2 splits of 1 column,
    # 30 tokens in comm tiles of 5 tokens: W_comp = 30, W_comm = 6
    p = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                occ_comm=1, num_cus=10, c_max=6, rho_ref_num=3, rho_ref_den=2,
                k_ref=8, tile_m_ref=1, tile_n_ref=1)
    wl, keep = B.make_workload(T=30, H=2, I=8, E=1, topk=1, splits=2, counts=[30])
    r, part = B.select_partition(wl, p)
    assert r == 5 and part.C == 5 and part.P == 10 and part.R == 5
    assert part.W_comp == 30 and part.W_comm == 6
    assert Fraction(part.T_num, part.T_den) == 9 and part.delta_comp == 0
    n, table, den = B.select_evaluate(wl, p)
    want = [20, 11, 9, 9, 9, Fraction(19, 2)]
    assert [Fraction(t, den) for t in table] == want
    p.c_max = 4
    r, part = B.select_partition(wl, p)
    assert r == 4


def test_rho_kh_hand_example_through_the_abi():
    """The same instance with the k/H-aware rho: top-1 against a top-1
    calibration (2k + 4 equal) and a task width of 1 column against 2, so
    rho = 3/2 * 1/2 = 3/4.  By hand: T(C = 1..6) = 11, 6.5, 6.5, 6.5, 7.5,
    8.75; the tie at 6.5 goes to the least Delta (C = 2: 2, C = 3: 12,
    C = 4: 6), so C* = 2 where the printed rho gives C* = 5."""
    p = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                occ_comm=1, num_cus=10, c_max=6, rho_ref_num=3, rho_ref_den=2,
                k_ref=8, tile_m_ref=1, tile_n_ref=1, rho_kh=1, topk_ref=1, comm_tile_n_ref=2)
    wl, keep = B.make_workload(T=30, H=2, I=8, E=1, topk=1, splits=2, counts=[30])
    r, part = B.select_partition(wl, p)
    assert r == 2 and part.delta_comp == 2 and part.T_den == 4
    assert Fraction(part.T_num, part.T_den) == Fraction(13, 2)
    n, table, den = B.select_evaluate(wl, p)
    assert [Fraction(t, den) for t in table] == [11, Fraction(13, 2), Fraction(13, 2),
                                                 Fraction(13, 2), Fraction(15, 2),
                                                 Fraction(35, 4)]
    for bad in (dict(rho_kh=2), dict(topk_ref=0), dict(comm_tile_n_ref=0)):
        q = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                    occ_comm=1, num_cus=10, c_max=6, rho_ref_num=3, rho_ref_den=2,
                    k_ref=8, tile_m_ref=1, tile_n_ref=1, rho_kh=1, topk_ref=1,
                    comm_tile_n_ref=2)
        for k, v in bad.items():
            setattr(q, k, v)
        assert B.select_partition(wl, q)[0] == B.MOE_ERR_INVALID_ARG, bad


def test_finer_last_split_hand_example_through_the_abi():
    """The hand example with the last split's tasks cut to 2 tokens
    (W_last = 15, rho_last = 3/5): T(5) = 39/5, T(2) = 113/10 and the role
    switch T(0) = 39/10, over the time unit 1/(2 * 5 / gcd(3, 5)) = 1/10."""
    p = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                occ_comm=1, num_cus=10, c_min=0, c_max=6, rho_ref_num=3, rho_ref_den=2,
                k_ref=8, tile_m_ref=1, tile_n_ref=1, comm_tile_m_last=2)
    wl, keep = B.make_workload(30, 2, 8, 1, 1, 2, [30])
    n, table, den = B.select_evaluate(wl, p)
    assert den == 10
    assert Fraction(table[0], den) == Fraction(39, 10)
    assert Fraction(table[2], den) == Fraction(113, 10)
    assert Fraction(table[5], den) == Fraction(39, 5)
    r, part = B.select_partition(wl, p)
    assert r == 0 and part.W_comm == 6 and part.T_den == 10
    r, num, rden, A, F = B.select_candidate(wl, p, 5)
    assert (num, rden) == (15, 10) and A == [30, 60] and F == [60, 78]
    # defined for column splits ready a split at a time only; negative is invalid
    for bad in (dict(split_axis=1), dict(readiness=1), dict(comm_tile_m_last=-1)):
        q = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                    occ_comm=1, num_cus=10, c_min=0, c_max=6, rho_ref_num=3, rho_ref_den=2,
                    k_ref=8, tile_m_ref=1, tile_n_ref=1, comm_tile_m_last=2)
        for k, v in bad.items():
            setattr(q, k, v)
        assert B.select_partition(wl, q)[0] == B.MOE_ERR_INVALID_ARG, bad


def test_work_conserving_drain_hand_example_through_the_abi():
    """The hand example with drain = 2: T(1) = T(2) = 11/2, T(5) = 15/2
    (drain = 1: 25/2, 8, 15/2); the split times of C = 5 are (3, 6) and
    (6, 15/2).  drain = 2 with per-wave readiness or a finer last split is
    refused."""
    p = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                occ_comm=1, num_cus=10, c_min=1, c_max=6, rho_ref_num=3, rho_ref_den=2,
                k_ref=8, tile_m_ref=1, tile_n_ref=1, drain=2)
    wl, keep = B.make_workload(30, 2, 8, 1, 1, 2, [30])
    n, table, den = B.select_evaluate(wl, p)
    assert den == 2
    assert [Fraction(t, den) for t in (table[0], table[1], table[4])] == \
        [Fraction(11, 2), Fraction(11, 2), Fraction(15, 2)]
    r, num, rden, A, F = B.select_candidate(wl, p, 5)
    assert (num, rden) == (3, 2) and A == [6, 12] and F == [12, 15]
    for bad in (dict(readiness=1), dict(comm_tile_m_last=2), dict(drain=3)):
        q = _params(tile_m=1, tile_n=1, comm_tile_m=5, comm_tile_n=1, occ_comp=2,
                    occ_comm=1, num_cus=10, c_min=1, c_max=6, rho_ref_num=3, rho_ref_den=2,
                    k_ref=8, tile_m_ref=1, tile_n_ref=1, drain=2)
        for k, v in bad.items():
            setattr(q, k, v)
        assert B.select_partition(wl, q)[0] == B.MOE_ERR_INVALID_ARG, bad


def test_idle_slots_and_split_cost_through_the_abi():
    """The oracle's hand example for the idle compute slots and the split
    cost (G=10, W_comp=13, W_comm=12, L=2, rho=1/2, drain = 2): one expert of
    13 rows in 1x1 tiles over two 1-column splits, 24 tokens in tasks of 2.
    T(0), T(1), T(2) = 4, 4, 5; with pi = 1/4: 17/4, 17/4, 21/4."""
    p = _params(tile_m=1, tile_n=1, comm_tile_m=2, comm_tile_n=1, occ_comp=1, occ_comm=1,
                num_cus=10, c_min=0, c_max=2, rho_ref_num=1, rho_ref_den=2, k_ref=8,
                tile_m_ref=1, tile_n_ref=1, drain=2)
    wl, keep = B.make_workload(T=24, H=2, I=8, E=1, topk=1, splits=2, counts=[13])
    n, table, den = B.select_evaluate(wl, p)
    assert [Fraction(t, den) for t in table] == [4, 4, 5]
    p.split_cost_num, p.split_cost_den = 1, 4
    n, table, den = B.select_evaluate(wl, p)
    assert den == 4 and [Fraction(t, den) for t in table] == \
        [Fraction(17, 4), Fraction(17, 4), Fraction(21, 4)]
    assert B.select_candidate(wl, p, 2) == (2, 2, 4, [8, 17], [21, 21])
    assert B.select_candidate(wl, p, 0) == (1, 2, 4, [13], [17])
    # a split cost needs split readiness; a negative one is invalid
    p.readiness = 1
    p.drain = 0
    assert B.select_partition(wl, p)[0] == B.MOE_ERR_INVALID_ARG
    p.readiness = 0
    p.split_cost_num = -1
    assert B.select_partition(wl, p)[0] == B.MOE_ERR_INVALID_ARG
    p.split_cost_num, p.split_cost_den = 1, 0
    assert B.select_partition(wl, p)[0] == B.MOE_ERR_INVALID_ARG


def _random_case(rnd):
    E = rnd.randint(1, 64)
    topk = rnd.randint(1, min(E, 8))
    T = rnd.randint(0, 40000)
    L = rnd.randint(1, 4)
    H = 8 * L * rnd.randint(1, 512)
    I = 8 * rnd.randint(1, 200)
    counts = None
    if rnd.random() < 0.8:
        w = np.array([rnd.random() ** 3 for _ in range(E)])
        c = np.floor(w / w.sum() * T * topk).astype(np.int64)
        c[0] += T * topk - c.sum()
        counts = [int(v) for v in c]
    p = _params(tile_m=rnd.choice([64, 128, 256]), tile_n=rnd.choice([64, 128, 256]),
                comm_tile_m=rnd.choice([64, 128]), comm_tile_n=rnd.choice([512, 1024]),
                occ_comp=rnd.randint(1, 3), occ_comm=rnd.randint(1, 3),
                num_cus=rnd.choice([8, 64, 108, 256, 304]), c_min=rnd.choice([0, 1, 1, 1]),
                c_max=rnd.randint(1, 80), rho_ref_num=rnd.randint(1, 100000),
                rho_ref_den=rnd.randint(1, 10000), k_ref=rnd.choice([352, 704, 1408]),
                tile_m_ref=rnd.choice([128, 256]), tile_n_ref=rnd.choice([128, 256]),
                d_ref=rnd.choice([1, 4]), split_axis=rnd.choice([0, 0, 1]),
                drain=rnd.choice([0, 0, 1, 2]), rho_kh=rnd.choice([0, 0, 1]),
                topk_ref=rnd.randint(1, 16), comm_tile_n_ref=rnd.choice([256, 512, 1024, 2048]))
    if p.split_axis == 0:
        # per-wave readiness walks every compute wave in the oracle: keep it to
        # workloads of at most 2000 tiles so the suite stays fast
        m_tiles = osel.routed_m_tiles(counts, p.tile_m, E, T * topk)
        tiles = L * osel.compute_work(m_tiles, H, L, p.tile_n, p.groups)
        if tiles <= 2000 and p.drain != 2:
            p.readiness = rnd.choice([0, 1, 1])
        if p.readiness == 0 and p.drain != 2:
            p.comm_tile_m_last = rnd.choice([0, 0, p.comm_tile_m // 2, 16, 48, p.comm_tile_m])
    if p.readiness == 0 and rnd.random() < 0.4:
        p.split_cost_num = rnd.choice([1, 2, 43, 100, 7919])
        p.split_cost_den = rnd.choice([1, 3, 100, 257])
    D = rnd.choice([1, 1, 2, 4])
    return T, H, I, E, topk, L, counts, p, D


def test_selector_bit_exact_against_oracle():
    rnd = random.Random(2024)
    n_checked = 0
    for _ in range(3000):
        T, H, I, E, topk, L, counts, p, D = _random_case(rnd)
        wl, keep = B.make_workload(T, H, I, E, topk, L, counts, ranks=D)
        r, part = B.select_partition(wl, p)
        best, cands, W_comp, W_comm, rho = osel.select(T, H, I, E, topk, L, counts,
                                                        _oracle_params(p), D=D)
        if best is None:
            assert r == B.MOE_ERR_NO_LEGAL_PARTITION
            continue
        assert r == best.C
        assert (part.C, part.R, part.P, part.delta_comp) == (best.C, best.R, best.P, best.delta)
        assert (part.W_comp, part.W_comm) == (W_comp, W_comm)
        assert part.T_den == _time_den(p, rho, I)
        assert Fraction(part.T_num, part.T_den) == best.T
        # whole table
        n, table, den = B.select_evaluate(wl, p)
        assert n == p.c_max - p.c_min + 1
        byC = {c.C: c.T for c in cands}
        for i, tnum in enumerate(table):
            C = p.c_min + i
            if C in byC:
                assert Fraction(tnum, den) == byC[C]
            else:
                assert tnum == -1
        n_checked += 1
    assert n_checked > 2000


def test_candidate_internals_bit_exact_against_oracle():
    """moe_select_candidate (rho and the split arrival and finish times of
    one candidate) against the oracle's candidate on random workloads, at
    random C including the role switch."""
    rnd = random.Random(91)
    n = 0
    for _ in range(600):
        T, H, I, E, topk, L, counts, p, D = _random_case(rnd)
        wl, keep = B.make_workload(T, H, I, E, topk, L, counts, ranks=D)
        C = rnd.randint(p.c_min, p.c_max)
        r, num, den, A, F = B.select_candidate(wl, p, C)
        best, cands, W_comp, W_comm, rho = osel.select(T, H, I, E, topk, L, counts,
                                                        _oracle_params(p), D=D)
        byC = {c.C: c for c in cands}
        if C not in byC:
            assert r == B.MOE_ERR_NO_LEGAL_PARTITION, (r, C)
            continue
        cand = byC[C]
        assert Fraction(num, den) == rho and den == _time_den(p, rho, I)
        assert r == len(cand.A) == len(cand.F)
        if p.readiness == 0:
            assert r == (1 if C == 0 else L)
        assert [Fraction(a, den) for a in A] == [Fraction(a) for a in cand.A]
        assert [Fraction(f, den) for f in F] == list(cand.F)
        n += 1
    assert n > 400
    wl, keep = B.make_workload(100, 256, 64, 4, 2, 2, [50, 50, 50, 50])
    assert B.select_candidate(wl, _params(), -1)[0] == B.MOE_ERR_INVALID_ARG
    L_ = B.lib()
    buf = (ctypes.c_int64 * 1)()
    assert L_.moe_select_candidate(ctypes.byref(wl), ctypes.byref(_params()), 3, None, None,
                                   buf, None, 1) == B.MOE_ERR_INVALID_ARG   # n < L
    assert L_.moe_select_candidate(ctypes.byref(wl), ctypes.byref(_params()), 3, None, None,
                                   None, None, 0) == 2


def test_scaled_time_overflow_boundary():
    """The scaled integer time is int64: one tile, one task, L = 1 on two
    slots, rho = X / 1, so every variant's T(C) is 1 + X compute-wave units
    (C = 1: A = 1, q = X; C = 0: ceil(1/2) = 1 of each; drain and per-wave
    readiness likewise).  X = 2^63 - 2 gives exactly INT64_MAX and matches
    the oracle; X = 2^63 - 1 overflows and is an invalid argument.  The same
    for the arrival term: two tiles on one compute slot at rho = 1 / X make
    A = 2 X."""
    big = 2 ** 63 - 1
    wl, keep = B.make_workload(T=1, H=1, I=8, E=1, topk=1, splits=1, counts=[1])
    variants = [dict(), dict(drain=1), dict(readiness=1), dict(readiness=1, drain=1),
                dict(c_min=0, c_max=0)]
    for v in variants:
        kw = dict(tile_m=1, tile_n=1, comm_tile_m=1, comm_tile_n=1, num_cus=2,
                  c_min=1, c_max=1, k_ref=8, tile_m_ref=1, tile_n_ref=1, rho_ref_den=1)
        kw.update(v)
        p = _params(rho_ref_num=big - 1, **kw)
        r, part = B.select_partition(wl, p)
        assert r == kw["c_min"] and part.T_num == big and part.T_den == 1, (v, r)
        best = osel.select(1, 1, 8, 1, 1, 1, [1], _oracle_params(p))[0]
        assert best.T == big, v
        n, table, den = B.select_evaluate(wl, p)
        assert n == 1 and table == [big], v
        p = _params(rho_ref_num=big, **kw)
        assert B.select_partition(wl, p)[0] == B.MOE_ERR_INVALID_ARG, v
        assert B.select_evaluate(wl, p)[0] == B.MOE_ERR_INVALID_ARG, v
        assert B.select_candidate(wl, p, kw["c_min"])[0] == B.MOE_ERR_INVALID_ARG, v
    wl2, keep2 = B.make_workload(T=1, H=1, I=8, E=1, topk=1, splits=1, counts=[2])
    for v in variants[:4]:
        p = _params(tile_m=1, tile_n=1, comm_tile_m=1, comm_tile_n=1, num_cus=2, c_min=1,
                    c_max=1, k_ref=8, tile_m_ref=1, tile_n_ref=1, rho_ref_num=1,
                    rho_ref_den=big, **v)
        assert B.select_partition(wl2, p)[0] == B.MOE_ERR_INVALID_ARG, v
        # X = 2^62 - 2: A_0 = 2 X < 2^63 - 1, then + rho_num = 1; with per-wave
        # readiness the one task is released by the first of the two waves
        # (F_1 = X + 1), so T = max(2 X, X + 1) + 0 = 2 X
        p.rho_ref_den = big // 2 - 1
        r, part = B.select_partition(wl2, p)
        want = 2 * (big // 2 - 1) + (0 if v.get("readiness") else 1)
        assert r == 1 and part.T_den == big // 2 - 1 and part.T_num == want, v
        best = osel.select(1, 1, 8, 1, 1, 1, [2], _oracle_params(p))[0]
        assert best.T == Fraction(want, big // 2 - 1), v


def test_split_selection_bit_exact_against_oracle():
    """moe_select_partition_splits (L as a decision variable) against the
    oracle's select_splits on random workloads, both split axes, with and
    without the drain term."""
    rnd = random.Random(77)
    n = 0
    for _ in range(400):
        T, H, I, E, topk, L, counts, p, D = _random_case(rnd)
        l_min = rnd.randint(1, 3)
        l_max = l_min + rnd.randint(0, 6)
        wl, keep = B.make_workload(T, H, I, E, topk, L, counts, ranks=D)
        r, Lb, part = B.select_partition_splits(wl, p, l_min, l_max)
        L_o, best = osel.select_splits(T, H, I, E, topk, counts, _oracle_params(p), l_min,
                                       l_max, D=D)
        if best is None:
            assert r == B.MOE_ERR_NO_LEGAL_PARTITION
            continue
        assert (r, Lb) == (best.C, L_o)
        assert Fraction(part.T_num, part.T_den) == best.T
        n += 1
    assert n > 300
    wl, keep = B.make_workload(100, 256, 64, 4, 2, 1, [50, 50, 50, 50])
    assert B.select_partition_splits(wl, _params(), 0, 3)[0] == B.MOE_ERR_INVALID_ARG
    assert B.select_partition_splits(wl, _params(), 3, 2)[0] == B.MOE_ERR_INVALID_ARG
    for field, bad in (("split_axis", 2), ("drain", 3), ("drain", -1), ("readiness", 2)):
        assert B.select_partition(wl, _params(**{field: bad}))[0] == B.MOE_ERR_INVALID_ARG
    # per-wave readiness is defined for column splits only
    assert B.select_partition(wl, _params(split_axis=1, readiness=1))[0] == \
        B.MOE_ERR_INVALID_ARG


def test_selector_argument_errors():
    p = _params()
    wl, keep = B.make_workload(T=100, H=2048, I=704, E=4, topk=2, splits=2,
                               counts=[50, 50, 50, 50])
    assert B.select_partition(wl, p)[0] >= 1
    for field, bad in [("c_min", -1), ("occ_comp", 0), ("num_cus", 0), ("rho_ref_den", 0),
                       ("rho_ref_num", -3), ("tile_m", 0)]:
        q = _params(**{field: bad})
        assert B.select_partition(wl, q)[0] == B.MOE_ERR_INVALID_ARG, field
    q = _params(c_min=10, c_max=5)
    assert B.select_partition(wl, q)[0] == B.MOE_ERR_INVALID_ARG
    bad_wl, k2 = B.make_workload(T=100, H=2048, I=704, E=4, topk=2, splits=2,
                                 counts=[50, -1, 50, 50])
    assert B.select_partition(bad_wl, p)[0] == B.MOE_ERR_INVALID_ARG
    # P(C) <= 0 for every candidate
    q = _params(num_cus=4, c_min=4, c_max=10)
    assert B.select_partition(wl, q)[0] == B.MOE_ERR_NO_LEGAL_PARTITION
    L = B.lib()
    assert L.moe_select_partition(None, None, None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_strerror(-4).decode().startswith("no legal partition")


def test_combine_host_validation_without_gpu():
    """Every check below fails before any HIP call, so it runs on the CPU."""
    import ctypes
    L = B.lib()
    vp = ctypes.c_void_p
    A = 0x100000                       # a 256-aligned fake address, never touched
    wl, keep = B.make_workload(T=256, H=1024, I=512, E=8, topk=2, splits=1)
    need = B.workspace_size(wl)
    assert need > 256 * 2 * 1024 * 2

    def call(x=A, w=A, off=A, tid=A, g=A, out=A, wlp=wl, C=-1, ws=A, wsb=need):
        return L.moe_gemm2_combine(vp(x), vp(w), vp(off), vp(tid), vp(g), vp(out),
                                   ctypes.byref(wlp) if wlp is not None else None, C,
                                   vp(ws), ctypes.c_size_t(wsb), vp(0))

    assert call(wlp=None) == B.MOE_ERR_INVALID_ARG
    assert call(x=0) == B.MOE_ERR_INVALID_ARG
    assert call(out=0) == B.MOE_ERR_INVALID_ARG
    assert call(x=A + 8) == B.MOE_ERR_ALIGNMENT
    assert call(out=A + 4) == B.MOE_ERR_ALIGNMENT
    assert call(tid=A + 2) == B.MOE_ERR_ALIGNMENT
    assert call(ws=A + 128) == B.MOE_ERR_ALIGNMENT
    assert call(ws=0) == B.MOE_ERR_WORKSPACE
    assert call(wsb=need - 1) == B.MOE_ERR_WORKSPACE
    assert call(C=-2) == B.MOE_ERR_INVALID_ARG
    for kw in [dict(H=1020), dict(I=500), dict(E=2000), dict(topk=65), dict(H=1024, splits=3)]:
        args = dict(T=256, H=1024, I=512, E=8, topk=2, splits=1)
        args.update(kw)
        w2, k2 = B.make_workload(**args)
        assert call(wlp=w2) == B.MOE_ERR_UNSUPPORTED, kw
        # column splits need H % (8 splits) == 0; token bands (mode 2) do not,
        # so the workspace size is defined for any split count
        assert (B.workspace_size(w2) == 0) == ("splits" not in kw), kw
    w3, k3 = B.make_workload(T=256, H=1024, I=512, E=8, topk=2, splits=1,
                             counts=[64] * 7 + [63])         # sums to 511 != 512
    assert call(wlp=w3) == B.MOE_ERR_INVALID_ARG
    # the mode entry point: same checks, and only modes 0 and 1

    def call_ex(mode, C=-1, wlp=wl, out=A):
        return L.moe_gemm2_combine_ex(vp(A), vp(A), vp(A), vp(A), vp(A), vp(out),
                                      ctypes.byref(wlp), C, mode, vp(A), ctypes.c_size_t(need),
                                      vp(0), vp(0), ctypes.c_size_t(0))

    for mode in (-1, 3, 7):
        assert call_ex(mode) == B.MOE_ERR_INVALID_ARG, mode
    for mode in (0, 1, 2):
        assert call_ex(mode, out=A + 4) == B.MOE_ERR_ALIGNMENT
        assert call_ex(mode, C=-2) == B.MOE_ERR_INVALID_ARG
    assert L.moe_gemm2_default_params_ex(0, 2, 1, None) == B.MOE_ERR_INVALID_ARG
    p = B.SelectParams()
    assert L.moe_gemm2_launch_params(0, 0, ctypes.byref(wl), None) == B.MOE_ERR_INVALID_ARG
    for mode in (-1, 3):
        assert L.moe_gemm2_launch_params(0, mode, ctypes.byref(wl),
                                         ctypes.byref(p)) == B.MOE_ERR_INVALID_ARG
    bad, kb = B.make_workload(T=256, H=1020, I=512, E=8, topk=2, splits=1)
    assert L.moe_gemm2_launch_params(0, 0, ctypes.byref(bad),
                                     ctypes.byref(p)) == B.MOE_ERR_UNSUPPORTED
    assert L.moe_gemm2_workspace_init(None, 0, None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_gemm2_status(None, None, 0) == B.MOE_ERR_INVALID_ARG

    # the entry point without a workspace argument: the same argument checks,
    # and a workload whose workspace would exceed the library's scratch is
    # refused before any HIP call
    def call_na(mode=0, C=-1, wlp=wl, out=A, x=A):
        return L.moe_gemm2_combine_noalloc(vp(x), vp(A), vp(A), vp(A), vp(A), vp(out),
                                           ctypes.byref(wlp) if wlp is not None else None,
                                           C, mode, vp(0))

    assert call_na(wlp=None) == B.MOE_ERR_INVALID_ARG
    assert call_na(mode=3) == B.MOE_ERR_INVALID_ARG
    assert call_na(C=-2) == B.MOE_ERR_INVALID_ARG
    assert call_na(x=0) == B.MOE_ERR_INVALID_ARG
    assert call_na(out=A + 4) == B.MOE_ERR_ALIGNMENT
    assert call_na(wlp=w3) == B.MOE_ERR_INVALID_ARG
    big, kbig = B.make_workload(T=8192, H=2048, I=704, E=30, topk=4, splits=2)
    assert B.workspace_size(big) > B.NOALLOC_SCRATCH_BYTES
    for mode in (0, 1):
        assert call_na(mode=mode, wlp=big) == B.MOE_ERR_WORKSPACE
    fits, kfits = B.make_workload(T=4096, H=1024, I=256, E=16, topk=8, splits=1)
    assert 0 < B.workspace_size(fits) <= B.NOALLOC_SCRATCH_BYTES


def _task_tokens(T, H, L):
    """The documented owner-write task size: 64 tokens, halved down to 16
    while the launch would have fewer than 512 tasks."""
    cb = -(-(H // L) // min(1024, H // L))
    tm = 64
    while tm > 16 and L * -(-T // tm) * cb < 512:
        tm //= 2
    return tm


@pytest.mark.parametrize("T,H,L,tm", [(16384, 2048, 2, 64), (8192, 2048, 2, 32),
                                      (4096, 1024, 1, 16), (4096, 2048, 2, 16),
                                      (32768, 2048, 2, 64), (256, 1024, 1, 16),
                                      (20000, 1024, 1, 32), (1, 64, 1, 16)])
def test_trace_size_counts_the_adaptive_consumer_tasks(T, H, L, tm):
    """trace_size holds one record per owner-write task, and the task size
    follows the documented rule (checked without a device)."""
    assert _task_tokens(T, H, L) == tm
    E, k, I = 8, 2, 64
    wl, _ = B.make_workload(T=T, H=H, I=I, E=E, topk=k, splits=L)
    rows = T * k
    max_tiles = L * -(-(H // L) // 256) * (-(-rows // 256) + E)
    tm_last = min(tm, max(16, tm // 4))      # the last split's tasks are cut finer
    cb = -(-(H // L) // 1024)
    tasks = (L - 1) * -(-T // tm) * cb + -(-T // tm_last) * cb
    assert B.trace_size(wl) == 8 * (4 * max_tiles + 4 * max(tasks, max_tiles))


def test_32bit_offset_limits():
    """The ring loads address one expert's weight slice (and, in the
    up-projection, hidden) with 32-bit byte offsets, so shapes past 2 GiB
    there are refused on the host, and the largest ones below are taken."""
    over, _ = B.make_workload(T=256, H=16384, I=65536, E=2, topk=1, splits=1)   # 2 I H = 2^31
    assert B.workspace_size(over) == 0
    assert B.layer_workspace_size(over) == 0
    edge, _ = B.make_workload(T=256, H=16384, I=65528, E=2, topk=1, splits=1)   # 2^31 - 2^18
    assert B.workspace_size(edge) > 0
    hid, _ = B.make_workload(T=65536, H=16384, I=64, E=2, topk=1, splits=1)     # 2 T H = 2^31
    assert B.workspace_size(hid) > 0          # the down-projection stage does not read hidden
    assert B.layer_workspace_size(hid) == 0
    w1, _ = B.make_workload(T=256, H=16384, I=32768, E=2, topk=1, splits=1)     # 4 H I = 2^31
    assert B.workspace_size(w1) > 0
    assert B.layer_workspace_size(w1) == 0
    ok, _ = B.make_workload(T=256, H=16384, I=32752, E=2, topk=1, splits=1)
    assert B.layer_workspace_size(ok) > 0


def test_workspace_size_grows_with_rows():
    a, _ = B.make_workload(T=1024, H=2048, I=704, E=32, topk=6, splits=2)
    b, _ = B.make_workload(T=2048, H=2048, I=704, E=32, topk=6, splits=2)
    sa, sb = B.workspace_size(a), B.workspace_size(b)
    assert sa >= 1024 * 6 * 2048 * 2 and sb >= 2048 * 6 * 2048 * 2 and sb > sa
    assert B.trace_size(a) > 0
