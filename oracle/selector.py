"""CPU oracle for the wave-quantized launch-time partition selector
(test infrastructure: only tests and the benchmark use it).

It evaluates the paper's model in exact rational arithmetic
(``fractions.Fraction``), step by step in the order of Algorithm 1
("CPU-side communication-grid selection"):

  routed-tile reduction      eq:routed-tile-reduction   sum_e ceil(M_e / T_M)
  compute work per split     eq:compute-work            W_comp
  communication work         eq:communication-work      W_comm
  reservation                eq:reservation             R(C) = ceil(C / o_comm)
  compute capacity           eq:compute-capacity        P(C) = o_comp (G - R(C))
  split readiness            eq:split-arrival           A_s = ceil((s+1) W_comp / P)
  communication waves        eq:communication-waves     V_comm = ceil(W_comm / C)
  service time               eq:comm-service            q = rho V_comm
  split completion           eq:split-finish            F_s = max(A_s, F_{s-1}) + q
  makespan                   eq:makespan                T(C) = F_{L-1}
  tie-break                  eq:tie-breaker             Delta = V_comp P - W_comp
  rho at run time            eq:rho-scaling             rho_ref (K_ref/K)(tile_ref/tile)(D/D_ref)

Readings where the paper is silent (each listed in the design notes):
  * g (input groups) = 1;
  * when no host counts exist, the routed-tile sum is estimated from the
    total assignments spread evenly over E experts:
    E * ceil(ceil(M k / E) / T_M);
  * a candidate whose P(C) <= 0 is not in the legal set;
  * ties left after Delta go to the smaller C;
  * D = 1 on one GPU, so the token count per rank is M itself.

Extension beyond the paper's legal set (only when c_min = 0): the
role-switch candidate C = 0, where all o_comp * G slots run every compute
tile and then all of them serve the consumer tasks,
T(0) = ceil(L W_comp / P0) + rho ceil(L W_comm / P0) with P0 = o_comp G.

Further extensions, off unless asked for (the paper's model is their
special case split_axis = 0, drain = False, one given L):
  * split_axis = 1, token bands: the L splits cut the routed rows instead
    of the output columns, so a split holds about 1/L of the m-tiles over
    the full width and 1/L of the token blocks:
    W_comp = ceil(g m_tiles / L) ceil(N / T_N),
    W_comm = ceil(ceil(ceil(M/D) / T_M^comm) / L) ceil(N / T_N^comm);
  * drain (1): compute slots join the consumers after their last tile, so
    the last split is served by all C + P slots:
    F_{L-1} = max(A_{L-1}, F_{L-2}) + rho ceil(W_comm / (C + P));
  * work-conserving drain (2; readiness 0, no finer last split): the compute
    slots serve whatever remains of every split once the compute ends at
    E = A_{L-1}.  Until then the C consumers take the splits in order,
    split s from start = max(A_s, the end of split s-1), in rounds of C
    tasks of rho each; the rounds that start before E claim
    min(W_comm, C ceil((E - start)/rho)) tasks of split s, stopping at the
    first split not wholly claimed.  The Idle = V P - L W_comp compute
    slots that hold no tile in the last of the V = ceil(L W_comp / P)
    compute waves are free from E - 1; in the ceil(1/rho) rounds they begin
    before E they take up to Idle ceil(1/rho) of the tasks not yet claimed
    of the splits ready by then (A_s <= E - 1, s < L - 1), ending at
    E - 1 + rho ceil(taken / Idle).  With R the tasks left of all L W_comm
    and e the end of the last claimed round,
    T(C) = max(E + rho ceil(R / (C + P)), e); C = 0 is the same with no
    consumers and P0 slots;
  * split cost pi_ref (readiness 0): each split's publish delays the
    compute of the splits after it by pi = pi_ref (K_ref/K)
    (T_M,ref T_N,ref)/(T_M T_N) compute waves: A_s = ceil((s+1) W_comp / P)
    + s pi, and for C = 0 the compute ends at ceil(L W_comp / P0) + (L-1) pi;
  * L as a decision variable: the (L, C) pair with the least T(C) over a
    range of L, ties to the smaller L;
  * readiness = 1 (column splits): the consumer work is released a compute
    wave at a time rather than a split at a time.  The L W_comp tiles end in
    V = ceil(L W_comp / P) waves; wave v ends t_v = min(v P, L W_comp) of
    them and releases w_v = ceil(t_v L W_comm / (L W_comp)) - (what earlier
    waves released) tasks, served as F_v = max(v, F_{v-1}) + rho ceil(w_v / C)
    (drain: the last wave over C + P slots); T(C) = F_V.  C = 0 is unchanged;
  * rho_kh = 1: rho also scales with the bytes of one consumer task against
    the calibration's, k bf16 rows read and one fp32 output written per
    token and column: rho times (2 k + 4) / (2 k_ref + 4) times w / w_ref,
    with the task width w = min(T_N^comm, ceil(N/L)) for column splits and
    min(T_N^comm, N) for token bands;
  * a finer last split (column splits, readiness 0): the last split's
    consumer tasks hold T_M^last tokens instead of T_M^comm, so it has
    W_last = ceil(ceil(M/D) / T_M^last) ceil(ceil(N/L) / T_N^comm) tasks,
    each served in rho_last = rho T_M^last / T_M^comm (a task's bytes follow
    its tokens): F_{L-1} = max(A_{L-1}, F_{L-2}) + rho_last ceil(W_last / C)
    (drain: C + P slots).  For C = 0 every task is counted in units of rho/a,
    with a : b = T_M^comm : T_M^last in lowest terms (a units for a task of
    the other splits, b for one of the last split), all of them over the P0
    slots: T(0) = ceil(L W_comp / P0) + (rho/a) ceil((a (L-1) W_comm + b W_last) / P0).
    T_M^last = T_M^comm is the model without this extension.
"""
from __future__ import annotations

import dataclasses
import math
from fractions import Fraction
from typing import List, Optional, Sequence


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


@dataclasses.dataclass
class Candidate:
    C: int
    R: int
    P: int
    A: List[int]          # split readiness, compute-wave units
    V_comm: int
    q: Fraction
    F: List[Fraction]
    T: Fraction
    V_comp: int
    delta: int


def routed_m_tiles(counts: Optional[Sequence[int]], tile_m: int, E: int,
                   total_assignments: int) -> int:
    """sum_e ceil(M_e / T_M) from host counts, or the even-load estimate."""
    if counts is not None:
        return sum(cdiv(int(m), tile_m) for m in counts)
    per_expert = cdiv(total_assignments, E)
    return E * cdiv(per_expert, tile_m)


def compute_work(m_tiles: int, N: int, L: int, tile_n: int, g: int = 1,
                 split_axis: int = 0) -> int:
    """Column splits: W_comp = g * (sum_e ceil(M_e/T_M)) * ceil(ceil(N/L) / T_N).
    Token bands: ceil(g * sum_e ceil(M_e/T_M) / L) * ceil(N / T_N)."""
    if split_axis == 0:
        return g * m_tiles * cdiv(cdiv(N, L), tile_n)
    return cdiv(g * m_tiles, L) * cdiv(N, tile_n)


def comm_work(M: int, D: int, N: int, L: int, comm_m: int, comm_n: int,
              split_axis: int = 0) -> int:
    """Column splits: W_comm = ceil(ceil(M/D) / T_M^comm) * ceil(ceil(N/L) / T_N^comm).
    Token bands: ceil(ceil(ceil(M/D) / T_M^comm) / L) * ceil(N / T_N^comm)."""
    if split_axis == 0:
        return cdiv(cdiv(M, D), comm_m) * cdiv(cdiv(N, L), comm_n)
    return cdiv(cdiv(cdiv(M, D), comm_m), L) * cdiv(N, comm_n)


def rho_scaled(rho_ref: Fraction, K: int, K_ref: int, tile_m: int, tile_n: int,
               tile_m_ref: int, tile_n_ref: int, D: int, D_ref: int) -> Fraction:
    """eq:rho-scaling."""
    return (Fraction(rho_ref) * Fraction(K_ref, K)
            * Fraction(tile_m_ref * tile_n_ref, tile_m * tile_n)
            * Fraction(D, D_ref))


def task_bytes_factor(topk: int, topk_ref: int, width: int, width_ref: int) -> Fraction:
    """The k/H-aware extension: a task's bytes per token and column are
    2 k (its k bf16 rows) + 4 (one fp32 output), times the task width."""
    return Fraction(2 * topk + 4, 2 * topk_ref + 4) * Fraction(width, width_ref)


def task_width(H: int, L: int, comm_n: int, split_axis: int = 0) -> int:
    span = cdiv(H, L) if split_axis == 0 else H
    return min(span, comm_n)


@dataclasses.dataclass
class LastSplit:
    """The finer last split: its task count, its rho, and a : b."""
    W: int
    rho: Fraction
    a: int
    b: int


def evaluate(C: int, W_comp: int, W_comm: int, L: int, G: int, o_comm: int,
             o_comp: int, rho: Fraction, drain: int = 0,
             readiness: int = 0, last: Optional[LastSplit] = None,
             pi: Fraction = Fraction(0)) -> Optional[Candidate]:
    """The recurrence for one candidate C; None if P(C) <= 0 (illegal).
    pi: the split cost, compute waves each earlier split's publish adds to
    A_s (0 in the paper's model)."""
    pi = Fraction(pi)
    if pi and readiness != 0:
        raise ValueError("a split cost is defined for split readiness")
    if C == 0:
        P0 = o_comp * G
        A_last = cdiv(L * W_comp, P0) + (L - 1) * pi
        if drain == 2:
            A = [cdiv((s + 1) * W_comp, P0) + s * pi for s in range(L)]
            return _work_conserving(0, 0, P0, A, W_comm, L, rho, cdiv(L * W_comm, P0),
                                    Fraction(0), cdiv(W_comp, P0), W_comp)
        if last is None:
            q = Fraction(rho) * cdiv(L * W_comm, P0)
        else:
            units = last.a * (L - 1) * W_comm + last.b * last.W
            q = Fraction(rho) / last.a * cdiv(units, P0)
        T = A_last + q
        V_comp = cdiv(W_comp, P0)
        return Candidate(C=0, R=0, P=P0, A=[A_last], V_comm=cdiv(L * W_comm, P0), q=q,
                         F=[T], T=T, V_comp=V_comp, delta=V_comp * P0 - W_comp)
    R = cdiv(C, o_comm)
    P = o_comp * (G - R)
    if P <= 0:
        return None
    V_comm = cdiv(W_comm, C)
    q = Fraction(rho) * V_comm
    V_comp = cdiv(W_comp, P)
    if readiness == 1:
        return _per_wave(C, R, P, W_comp, W_comm, L, rho, drain, V_comm, q, V_comp)
    A = [cdiv((s + 1) * W_comp, P) + s * pi for s in range(L)]
    if drain == 2:
        return _work_conserving(C, R, P, A, W_comm, L, rho, V_comm, q, V_comp, W_comp)
    F: List[Fraction] = []
    prev = Fraction(0)
    W_l, rho_l = (W_comm, Fraction(rho)) if last is None else (last.W, last.rho)
    for s in range(L):
        if s == L - 1:
            # the last split: its own tasks, and with drain every slot serves
            # it once its tiles are done
            prev = max(Fraction(A[s]), prev) + rho_l * cdiv(W_l, C + P if drain else C)
        else:
            prev = max(Fraction(A[s]), prev) + q
        F.append(prev)
    return Candidate(C=C, R=R, P=P, A=A, V_comm=V_comm, q=q, F=F, T=F[-1],
                     V_comp=V_comp, delta=V_comp * P - W_comp)


def _work_conserving(C, R, P, A, W_comm, L, rho, V_comm, q, V_comp, W_comp) -> Candidate:
    """The drain = 2 model: the consumers' claims until the compute ends,
    the claims of the compute slots idle in the last compute wave, then
    every slot on what remains.  C = 0: no consumers, P = P0 (one A and one
    F entry: the end of the compute and T)."""
    rho = Fraction(rho)
    end = Fraction(A[L - 1])                # E, the end of the compute
    cur = Fraction(A[0])
    claimed = 0
    last_end = Fraction(0)
    F: List[Fraction] = []
    # the C consumers, split by split in order, rounds begun before E
    for s in range(L - 1 if C > 0 else 0):
        start = max(Fraction(A[s]), cur)
        need = cdiv(W_comm, C)
        started = math.ceil((end - start) / rho) if start < end else 0
        if started >= need:
            claimed += W_comm
            cur = start + need * rho
            if need > 0:
                last_end = cur
            F.append(cur)
        else:
            claimed += C * started
            if started > 0:
                last_end = start + started * rho
            break
    # compute slots with no tile in the last of the V compute waves: free
    # from E - 1, they take unclaimed tasks of the splits ready by then
    V = cdiv(L * W_comp, P)
    idle = V * P - L * W_comp
    if V > 0 and idle > 0:
        t0 = end - 1
        ready = [s for s in range(L - 1) if A[s] <= t0]
        avail = len(ready) * W_comm - claimed
        if avail > 0:
            rounds = math.ceil(1 / rho)         # rounds they begin before E
            take = min(avail, idle * rounds)
            claimed += take
            last_end = max(last_end, t0 + cdiv(take, idle) * rho)
    T = max(end + rho * cdiv(L * W_comm - claimed, C + P), last_end)
    if C == 0:
        return Candidate(C=0, R=0, P=P, A=[end], V_comm=V_comm, q=rho * V_comm, F=[T], T=T,
                         V_comp=V_comp, delta=V_comp * P - W_comp)
    F += [T] * (L - len(F))
    return Candidate(C=C, R=R, P=P, A=A, V_comm=V_comm, q=q, F=F, T=T,
                     V_comp=V_comp, delta=V_comp * P - W_comp)


def _per_wave(C, R, P, W_comp, W_comm, L, rho, drain, V_comm, q, V_comp) -> Candidate:
    """The readiness = 1 recurrence: tasks released as compute waves end."""
    tiles, tasks = L * W_comp, L * W_comm
    delta = V_comp * P - W_comp
    if tiles == 0:
        T = Fraction(rho) * cdiv(tasks, C + P if drain else C)
        return Candidate(C=C, R=R, P=P, A=[0], V_comm=V_comm, q=q, F=[T], T=T,
                         V_comp=V_comp, delta=delta)
    V = cdiv(tiles, P)
    A: List[int] = []
    F: List[Fraction] = []
    released = 0
    prev = Fraction(0)
    for v in range(1, V + 1):
        t = min(v * P, tiles)
        rel = cdiv(t * tasks, tiles)          # tasks whose tiles have all ended
        w = rel - released
        released = rel
        slots = C + P if (drain and v == V) else C
        prev = max(Fraction(v), prev) + Fraction(rho) * cdiv(w, slots)
        A.append(v)
        F.append(prev)
    return Candidate(C=C, R=R, P=P, A=A, V_comm=V_comm, q=q, F=F, T=F[-1],
                     V_comp=V_comp, delta=delta)


def select_from_work(W_comp: int, W_comm: int, L: int, G: int, o_comm: int,
                     o_comp: int, rho: Fraction, c_min: int, c_max: int,
                     drain: int = 0, readiness: int = 0,
                     last: Optional[LastSplit] = None, pi: Fraction = Fraction(0)):
    """Argmin of T(C) over the legal C, then smallest Delta, then smallest C.

    Returns (best Candidate or None, list of all legal candidates)."""
    cands = []
    for C in range(c_min, c_max + 1):
        c = evaluate(C, W_comp, W_comm, L, G, o_comm, o_comp, rho, drain, readiness, last, pi)
        if c is not None:
            cands.append(c)
    if not cands:
        return None, cands
    best = min(cands, key=lambda c: (c.T, c.delta, c.C))
    return best, cands


@dataclasses.dataclass
class SelectParams:
    tile_m: int
    tile_n: int
    comm_tile_m: int
    comm_tile_n: int
    occ_comp: int
    occ_comm: int
    num_cus: int
    c_min: int
    c_max: int
    rho_ref: Fraction
    k_ref: int
    tile_m_ref: int
    tile_n_ref: int
    d_ref: int
    groups: int = 1
    split_axis: int = 0
    drain: int = 0                 # 0, 1 or 2 (see the module notes)
    rho_kh: bool = False
    topk_ref: int = 6
    comm_tile_n_ref: int = 1024
    readiness: int = 0
    comm_tile_m_last: int = 0      # 0: the last split's tasks as the others'
    split_cost: Fraction = Fraction(0)   # pi_ref; 0: no split cost (the paper)


def select(T: int, H: int, I: int, E: int, topk: int, L: int,
           counts: Optional[Sequence[int]], p: SelectParams, D: int = 1):
    """Algorithm 1 on a workload: returns (best, candidates, W_comp, W_comm, rho)."""
    m_tiles = routed_m_tiles(counts, p.tile_m, E, T * topk)
    W_comp = compute_work(m_tiles, H, L, p.tile_n, p.groups, p.split_axis)
    W_comm = comm_work(T, D, H, L, p.comm_tile_m, p.comm_tile_n, p.split_axis)
    rho = rho_scaled(p.rho_ref, I, p.k_ref, p.tile_m, p.tile_n,
                     p.tile_m_ref, p.tile_n_ref, D, p.d_ref)
    if p.rho_kh:
        rho *= task_bytes_factor(topk, p.topk_ref,
                                 task_width(H, L, p.comm_tile_n, p.split_axis),
                                 p.comm_tile_n_ref)
    last = last_split(T, D, H, L, p, rho)
    pi = split_cost(p, I)
    best, cands = select_from_work(W_comp, W_comm, L, p.num_cus, p.occ_comm,
                                   p.occ_comp, rho, p.c_min, p.c_max, int(p.drain),
                                   p.readiness, last, pi)
    return best, cands, W_comp, W_comm, rho


def split_cost(p: SelectParams, K: int) -> Fraction:
    """pi = pi_ref (K_ref/K) (T_M,ref T_N,ref)/(T_M T_N): a publish costs a
    fixed time, a compute wave scales with the tile's work."""
    return (Fraction(p.split_cost) * Fraction(p.k_ref, K)
            * Fraction(p.tile_m_ref * p.tile_n_ref, p.tile_m * p.tile_n))


def last_split(T: int, D: int, H: int, L: int, p: SelectParams,
               rho: Fraction) -> Optional[LastSplit]:
    """The finer last split of the parameters, or None when its tasks are
    the other splits' (then the model is the paper's)."""
    tm, tm_last = p.comm_tile_m, p.comm_tile_m_last or p.comm_tile_m
    if tm_last == tm:
        return None
    if p.split_axis != 0 or p.readiness != 0 or int(p.drain) == 2:
        raise ValueError("a finer last split is defined for column splits ready a split at a time")
    g = math.gcd(tm, tm_last)
    return LastSplit(W=comm_work(T, D, H, L, tm_last, p.comm_tile_n),
                     rho=Fraction(rho) * Fraction(tm_last, tm), a=tm // g, b=tm_last // g)


def select_splits(T: int, H: int, I: int, E: int, topk: int,
                  counts: Optional[Sequence[int]], p: SelectParams,
                  l_min: int, l_max: int, D: int = 1):
    """L as a decision variable: the model for every L in [l_min, l_max];
    returns (L, best Candidate) with the least T, ties to the smaller L, or
    (None, None) when no L has a legal candidate."""
    best_L, best = None, None
    for L in range(l_min, l_max + 1):
        b, _, _, _, _ = select(T, H, I, E, topk, L, counts, p, D)
        if b is not None and (best is None or b.T < best.T):
            best_L, best = L, b
    return best_L, best
