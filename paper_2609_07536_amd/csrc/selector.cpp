// Launch-time partition selector: the wave-quantized makespan model of the
// paper's Method section, evaluated exactly on the host.
//
// Time is kept as an integer count of 1/rho_den compute waves, where
// rho = rho_num / rho_den is the service-time ratio of eq:rho-scaling
// (reduced, unless the last split's tasks are cut finer: see below), so T(C)
// compares exactly and ties (eq:tie-breaker) are real ties.
//
//   W_comp = g * (sum_e ceil(M_e/T_M)) * ceil(ceil(N/L)/T_N)       eq:compute-work
//   W_comm = ceil(ceil(M/D)/T_M^comm) * ceil(ceil(N/L)/T_N^comm)    eq:communication-work
//   R(C)   = ceil(C/o_comm)                                         eq:reservation
//   P(C)   = o_comp (G - R(C))                                      eq:compute-capacity
//   A_s    = ceil((s+1) W_comp / P(C))                              eq:split-arrival
//   q      = rho ceil(W_comm / C)                                   eq:comm-service
//   F_s    = max(A_s, F_{s-1}) + q,  T(C) = F_{L-1}                 eq:split-finish, eq:makespan
//   Delta  = ceil(W_comp/P) P - W_comp                              eq:tie-breaker
//
// Extension beyond the paper's legal set (used only when c_min == 0): the
// role-switch candidate C = 0, where all o_comp G slots compute every tile
// and then all of them serve the consumer tasks:
//   T(0) = ceil(L W_comp / P0) + rho ceil(L W_comm / P0),   P0 = o_comp G.
//
// Further extensions, each off unless its parameter asks for it:
//   split_axis = 1: the L splits cut the routed rows (token bands) instead
//     of the output columns; a band holds about 1/L of the m-tiles over the
//     full width and 1/L of the token blocks:
//       W_comp = ceil(g m_tiles / L) ceil(N / T_N)
//       W_comm = ceil(ceil(ceil(M/D) / T_M^comm) / L) ceil(N / T_N^comm)
//   drain = 1: the compute slots join the consumers after their last tile,
//     so the last split is served by all C + P slots:
//       F_{L-1} = max(A_{L-1}, F_{L-2}) + rho ceil(W_comm / (C + P));
//   drain = 2 (readiness 0, no finer last split): the same, but the compute
//     slots serve whatever remains of every split: the C consumers take the
//     splits in order, split s from start_s = max(A_s, the end of split
//     s-1), in rounds of C tasks of rho each; the rounds that start before
//     the compute ends at E = A_{L-1} claim
//       min(W_comm, C ceil((E - start_s) / rho)) tasks of split s,
//     stopping at the first split not wholly claimed.  The
//     Idle = V P - L W_comp compute slots with no tile in the last compute
//     wave (V = ceil(L W_comp / P)) are free from E - 1 and claim, in their
//     ceil(1/rho) rounds begun before E, up to Idle ceil(1/rho) unclaimed
//     tasks of the splits ready by then (A_s <= E - 1, s < L - 1).  With R
//     the tasks left (of all L W_comm) and e the end of the last claimed
//     round,
//       T(C) = max(E + rho ceil(R / (C + P)), e);
//     C = 0 is the same with no consumers over P0 slots;
//   split_cost = pi_ref > 0 (readiness 0): each split's publish delays the
//     compute after it by pi = pi_ref (K_ref/K) (T_M,ref T_N,ref)/(T_M T_N)
//     compute waves: A_s = ceil((s+1) W_comp / P) + s pi (C = 0: the compute
//     ends at ceil(L W_comp / P0) + (L-1) pi);
//   readiness = 1 (column splits): consumer work is released a compute wave
//     at a time: of V = ceil(L W_comp / P) waves, wave v releases the tasks
//     of the tiles it completes, w_v = ceil(t_v L W_comm / (L W_comp)) -
//     ceil(t_{v-1} ...), t_v = min(v P, L W_comp), and
//       F_v = max(v, F_{v-1}) + rho ceil(w_v / C),   T(C) = F_V
//     (drain: the last wave's tasks over C + P slots);
//   rho_kh = 1: rho also scales with the consumer task's bytes,
//       (2 k + 4) / (2 k_ref + 4) * w / w_ref (w: the task width);
//   comm_tile_m_last = T_M^last (column splits, split readiness): the last
//     split's consumer tasks hold T_M^last tokens, so
//       W_last = ceil(ceil(M/D)/T_M^last) ceil(ceil(N/L)/T_N^comm),
//       rho_last = rho T_M^last / T_M^comm,
//       F_{L-1} = max(A_{L-1}, F_{L-2}) + rho_last ceil(W_last / C)  (drain: C + P),
//     and for C = 0, with a : b = T_M^comm : T_M^last in lowest terms (a task
//     of the other splits is a units of rho/a, one of the last split b units),
//       T(0) = ceil(L W_comp / P0) + (rho/a) ceil((a (L-1) W_comm + b W_last) / P0).
//     Time is then counted in 1/(rho_den a / gcd(rho_num, a)) compute waves.
#include <cstdint>
#include <cstdlib>

#include "moe_gemm2.h"

namespace {

typedef __int128 i128;

const i128 kI64Max = (i128)INT64_MAX;

// the largest split count moe_select_partition_splits searches
constexpr int32_t kMaxSplitsSearched = 1024;
// the most splits, or compute waves with readiness = 1, a candidate's
// recurrence walks
constexpr int64_t kMaxSteps = 1 << 20;

// ceil(a / b) for a >= 0, b > 0; in 32 bits when both fit (a 64-bit
// division costs several times a 32-bit one, and a selection does hundreds)
inline int64_t cdiv64(int64_t a, int64_t b) {
  if (a == 0) return 0;
  if (((uint64_t)a | (uint64_t)b) >> 32 == 0) return (int64_t)(((uint32_t)a - 1u) / (uint32_t)b + 1u);
  return (a - 1) / b + 1;
}

inline i128 gcd128(i128 a, i128 b) {
  if (a <= (i128)INT64_MAX && b <= (i128)INT64_MAX) {
    uint64_t x = (uint64_t)a, y = (uint64_t)b;
    while (y != 0) {
      const uint64_t t = x % y;
      x = y;
      y = t;
    }
    return (i128)x;
  }
  while (b != 0) {
    const i128 t = a % b;
    a = b;
    b = t;
  }
  return a;
}

struct Model {
  int64_t W_comp = 0, W_comm = 0;
  int64_t rho_num = 0, rho_den = 1;   // rho over the time unit (not reduced when the last
                                      // split's tasks are cut finer)
  int64_t W_last = 0;                 // consumer tasks of the last split
  int64_t rho_last = 0;               // rho_last over the same unit
  int64_t a = 1, b = 1;               // T_M^comm : T_M^last in lowest terms
  int64_t rho_unit = 0;               // rho / a over the time unit
  int64_t pi = 0;                     // split_cost over the time unit
  int L = 1;
  int drain = 0;
  int readiness = 0;
};

// Builds the per-split work counts and the scaled rho; returns a status.
int build_model(const moe_workload_t* wl, const moe_select_params_t* p, Model* m) {
  if (!wl || !p) return MOE_ERR_INVALID_ARG;
  if (wl->T < 0 || wl->H <= 0 || wl->I <= 0 || wl->E <= 0 || wl->topk <= 0 ||
      wl->splits <= 0 || wl->ranks <= 0 || wl->rows < 0)
    return MOE_ERR_INVALID_ARG;
  if (p->tile_m <= 0 || p->tile_n <= 0 || p->comm_tile_m <= 0 || p->comm_tile_n <= 0 ||
      p->occ_comp <= 0 || p->occ_comm <= 0 || p->num_cus <= 0 || p->c_min < 0 ||
      p->c_max < p->c_min || p->groups <= 0 || p->rho_ref_num <= 0 || p->rho_ref_den <= 0 ||
      p->k_ref <= 0 || p->tile_m_ref <= 0 || p->tile_n_ref <= 0 || p->d_ref <= 0)
    return MOE_ERR_INVALID_ARG;
  // P(C) <= P(0) = o_comp G is reported as an int32
  if ((int64_t)p->occ_comp * p->num_cus > INT32_MAX) return MOE_ERR_INVALID_ARG;
  // the recurrence walks the splits (and with readiness = 1 the compute
  // waves) of every candidate: bounded so that a selection stays cheap
  if (wl->splits > kMaxSteps) return MOE_ERR_INVALID_ARG;

  // eq:routed-tile-reduction, or the even-load estimate when the counts only
  // live on the device (Method, "System Integration and Correctness").
  int64_t m_tiles = 0;
  if (wl->host_expert_counts) {
    for (int e = 0; e < wl->E; ++e) {
      int64_t me = wl->host_expert_counts[e];
      if (me < 0) return MOE_ERR_INVALID_ARG;
      m_tiles += cdiv64(me, p->tile_m);
    }
  } else {
    int64_t total = wl->rows > 0 ? wl->rows : (int64_t)wl->T * wl->topk;
    m_tiles = (int64_t)wl->E * cdiv64(cdiv64(total, wl->E), p->tile_m);
  }
  if (p->split_axis != 0 && p->split_axis != 1) return MOE_ERR_INVALID_ARG;
  if (p->drain < 0 || p->drain > 2) return MOE_ERR_INVALID_ARG;
  if (p->drain == 2 && p->readiness != 0) return MOE_ERR_INVALID_ARG;
  if (p->readiness != 0 && p->readiness != 1) return MOE_ERR_INVALID_ARG;
  if (p->readiness == 1 && p->split_axis != 0) return MOE_ERR_INVALID_ARG;
  const int64_t token_blocks = cdiv64(cdiv64(wl->T, wl->ranks), p->comm_tile_m);
  if (p->comm_tile_m_last < 0) return MOE_ERR_INVALID_ARG;
  const int64_t tm_last = p->comm_tile_m_last > 0 ? p->comm_tile_m_last : p->comm_tile_m;
  if (tm_last != p->comm_tile_m && (p->split_axis != 0 || p->readiness != 0 || p->drain == 2))
    return MOE_ERR_INVALID_ARG;   // defined for column splits ready a split at a time
  if (p->split_axis == 0) {
    const int64_t n_split = cdiv64(wl->H, wl->splits);
    m->W_comp = (int64_t)p->groups * m_tiles * cdiv64(n_split, p->tile_n);
    m->W_comm = token_blocks * cdiv64(n_split, p->comm_tile_n);
    m->W_last = cdiv64(cdiv64(wl->T, wl->ranks), tm_last) * cdiv64(n_split, p->comm_tile_n);
  } else {
    m->W_comp = cdiv64((int64_t)p->groups * m_tiles, wl->splits) * cdiv64(wl->H, p->tile_n);
    m->W_comm = cdiv64(token_blocks, wl->splits) * cdiv64(wl->H, p->comm_tile_n);
    m->W_last = m->W_comm;
  }
  m->L = wl->splits;
  m->drain = p->drain;
  m->readiness = p->readiness;

  // eq:rho-scaling: rho = rho_ref (K_ref/K) (T_M,ref T_N,ref)/(T_M T_N) (D/D_ref)
  i128 num = (i128)p->rho_ref_num * p->k_ref * p->tile_m_ref * p->tile_n_ref * wl->ranks;
  i128 den = (i128)p->rho_ref_den * wl->I * p->tile_m * p->tile_n * p->d_ref;
  if (p->rho_kh != 0 && p->rho_kh != 1) return MOE_ERR_INVALID_ARG;
  if (p->rho_kh) {
    // extension: the consumer task's bytes relative to the calibration's,
    // (2 k + 4) per token and column (k bf16 rows read, one fp32 written)
    // times the task width
    if (p->topk_ref <= 0 || p->comm_tile_n_ref <= 0) return MOE_ERR_INVALID_ARG;
    const int64_t span = p->split_axis == 0 ? cdiv64(wl->H, wl->splits) : (int64_t)wl->H;
    const int64_t width = span < p->comm_tile_n ? span : p->comm_tile_n;
    num *= (i128)(2 * (int64_t)wl->topk + 4) * width;
    den *= (i128)(2 * (int64_t)p->topk_ref + 4) * p->comm_tile_n_ref;
  }
  // reduce, then require both to fit in 63 bits
  const i128 gd = gcd128(num, den);
  num /= gd;
  den /= gd;
  if (num > kI64Max || den > kI64Max) return MOE_ERR_INVALID_ARG;
  // the last split's rho over a common unit: rho = num/den = (num a/g)/(den a/g)
  // and rho_last = (num b/g)/(den a/g), g = gcd(num, a), integral as gcd(a, b) = 1
  const i128 gab = gcd128(p->comm_tile_m, tm_last);
  const i128 a = p->comm_tile_m / gab, b = tm_last / gab;
  const i128 g = gcd128(num, a);
  const i128 rn = num * (a / g), rd = den * (a / g), rl = num / g * b, ru = num / g;
  if (rn > kI64Max || rd > kI64Max || rl > kI64Max) return MOE_ERR_INVALID_ARG;
  // the split cost pi = pi_ref (K_ref/K) (T_M,ref T_N,ref)/(T_M T_N) waves,
  // pn/pd in lowest terms; the time unit becomes 1/lcm(rd, pd) waves
  i128 pn = 0, pd = 1;
  if (p->split_cost_num < 0) return MOE_ERR_INVALID_ARG;
  if (p->split_cost_num > 0) {
    if (p->split_cost_den <= 0 || p->readiness != 0) return MOE_ERR_INVALID_ARG;
    pn = (i128)p->split_cost_num * p->k_ref * p->tile_m_ref * p->tile_n_ref;
    pd = (i128)p->split_cost_den * wl->I * p->tile_m * p->tile_n;
    const i128 gp = gcd128(pn, pd);
    pn /= gp;
    pd /= gp;
  }
  const i128 u = pd / gcd128(rd, pd);
  const i128 rn2 = rn * u, rd2 = rd * u, rl2 = rl * u, ru2 = ru * u;
  if (rn2 > kI64Max || rd2 > kI64Max || rl2 > kI64Max || pn > kI64Max)
    return MOE_ERR_INVALID_ARG;
  const i128 pi = pn * (rd2 / pd);
  if (pi > kI64Max / (wl->splits > 1 ? wl->splits : 1)) return MOE_ERR_INVALID_ARG;
  m->pi = (int64_t)pi;
  m->rho_num = (int64_t)rn2;
  m->rho_den = (int64_t)rd2;
  m->rho_last = (int64_t)rl2;
  m->rho_unit = (int64_t)ru2;
  m->a = (int64_t)a;
  m->b = (int64_t)b;
  return MOE_OK;
}

// The split arrival time A_s = ceil((s+1) W_comp / P) + s pi over the time
// unit (exact in 128 bits).
inline i128 arrival(const Model& m, int s, int64_t P) {
  return (i128)cdiv64((int64_t)(s + 1) * m.W_comp, P) * m.rho_den + (i128)s * m.pi;
}

// The work-conserving drain (drain = 2) for C >= 0 consumers beside P
// compute slots: the consumers' claims until the compute ends at
// E = A_{L-1}, the claims of the compute slots that hold no tile in the last
// compute wave, then every slot on what remains.  Returns T(C); false on
// overflow.  Records A_s and F_s for s < L when C > 0.
bool work_conserving(const Model& m, int64_t C, int64_t P, i128* T, int64_t* A_rec,
                     int64_t* F_rec) {
  const i128 E = arrival(m, m.L - 1, P);
  i128 cur = arrival(m, 0, P);
  i128 last_end = 0;      // end of the last claimed round
  int64_t claimed = 0;
  int s_stop = C > 0 ? m.L - 1 : 0;   // first split the consumers do not wholly claim
  for (int s = 0; C > 0 && s + 1 < m.L; ++s) {
    const i128 A = arrival(m, s, P);
    if (A_rec) A_rec[s] = (int64_t)A;
    const i128 start = A > cur ? A : cur;
    const int64_t need = cdiv64(m.W_comm, C);
    // rounds that start before E
    const i128 started = start < E ? (E - start + m.rho_num - 1) / m.rho_num : 0;
    if (started >= need) {
      claimed += m.W_comm;
      cur = start + (i128)need * m.rho_num;
      if (need > 0) last_end = cur;
      if (F_rec) F_rec[s] = (int64_t)cur;
    } else {
      claimed += (int64_t)((i128)C * started);
      if (started > 0) last_end = start + started * m.rho_num;
      s_stop = s;
      break;
    }
  }
  // the compute slots with no tile in the last compute wave, free one wave
  // before E, on the unclaimed tasks of the splits ready by then
  const int64_t tiles = (int64_t)m.L * m.W_comp;
  const int64_t V = cdiv64(tiles, P);
  const i128 idle = (i128)V * P - tiles;
  if (V > 0 && idle > 0) {
    const i128 t0 = E - m.rho_den;
    int ready = 0;
    while (ready + 1 < m.L && arrival(m, ready, P) <= t0) ++ready;
    const i128 avail = (i128)ready * m.W_comm - claimed;
    if (avail > 0) {
      const i128 rounds = ((i128)m.rho_den + m.rho_num - 1) / m.rho_num;
      const i128 cap = idle * rounds;
      const i128 take = avail < cap ? avail : cap;
      claimed += (int64_t)take;
      const i128 end = t0 + (take + idle - 1) / idle * m.rho_num;
      if (end > last_end) last_end = end;
    }
  }
  const int64_t R = (int64_t)((i128)m.L * m.W_comm - claimed);
  i128 F = E + (i128)m.rho_num * cdiv64(R, C + P);
  if (last_end > F) F = last_end;
  if (F > kI64Max) return false;
  if (C > 0)
    for (int s = s_stop; s < m.L; ++s) {   // splits finished in the drain end with it
      if (A_rec) A_rec[s] = (int64_t)arrival(m, s, P);
      if (F_rec) F_rec[s] = (int64_t)F;
    }
  *T = F;
  return true;
}

// One candidate; returns false if P(C) <= 0.  Status MOE_ERR_INVALID_ARG on
// overflow of the scaled integer time.  With A_rec / F_rec, also records the
// split arrival and finish times (one entry for C = 0: all tiles, then all
// tasks; else L).
bool eval_candidate(const Model& m, const moe_select_params_t* p, int32_t C, int64_t* T_out,
                    int32_t* R_out, int32_t* P_out, int* status,
                    int64_t* A_rec = nullptr, int64_t* F_rec = nullptr) {
  if (C == 0) {
    const int64_t P0 = (int64_t)p->occ_comp * p->num_cus;
    const i128 A = arrival(m, m.L - 1, P0);
    i128 F;
    if (m.drain == 2) {
      if (!work_conserving(m, 0, P0, &F, nullptr, nullptr)) {
        *status = MOE_ERR_INVALID_ARG;
        return false;
      }
    } else {
      // every task in units of rho/a: a for the other splits' tasks, b for
      // the last split's (a = b = 1 gives rho ceil(L W_comm / P0))
      const i128 units = (i128)m.a * (m.L - 1) * m.W_comm + (i128)m.b * m.W_last;
      if (units > kI64Max) {
        *status = MOE_ERR_INVALID_ARG;
        return false;
      }
      F = A + (i128)m.rho_unit * cdiv64((int64_t)units, P0);
    }
    if (A > kI64Max || F > kI64Max) {
      *status = MOE_ERR_INVALID_ARG;
      return false;
    }
    if (A_rec) A_rec[0] = (int64_t)A;
    if (F_rec) F_rec[0] = (int64_t)F;
    *T_out = (int64_t)F;
    *R_out = 0;
    *P_out = (int32_t)P0;
    return true;
  }
  const int64_t R = cdiv64(C, p->occ_comm);
  const int64_t P = (int64_t)p->occ_comp * ((int64_t)p->num_cus - R);
  if (P <= 0) return false;
  i128 F = 0;
  if (m.readiness == 1) {
    // per compute wave: wave v releases the tasks of the tiles it completes
    const int64_t tiles = (int64_t)m.L * m.W_comp, tasks = (int64_t)m.L * m.W_comm;
    if (tiles == 0) {
      F = (i128)m.rho_num * cdiv64(tasks, m.drain ? (int64_t)C + P : C);
      if (A_rec) A_rec[0] = 0;
      if (F_rec) F_rec[0] = (int64_t)F;
    } else {
      const int64_t V = cdiv64(tiles, P);
      if (V > kMaxSteps) {
        *status = MOE_ERR_INVALID_ARG;
        return false;
      }
      int64_t released = 0;
      for (int64_t v = 1; v <= V; ++v) {
        const int64_t t = v * P < tiles ? v * P : tiles;
        const int64_t rel = (int64_t)(((i128)t * tasks + tiles - 1) / tiles);
        const int64_t w = rel - released;
        released = rel;
        const i128 A = (i128)v * m.rho_den;
        const int64_t slots = m.drain && v == V ? (int64_t)C + P : C;
        F = (A > F ? A : F) + (i128)m.rho_num * cdiv64(w, slots);
        if (F > kI64Max) {
          *status = MOE_ERR_INVALID_ARG;
          return false;
        }
        if (A_rec) A_rec[v - 1] = (int64_t)A;
        if (F_rec) F_rec[v - 1] = (int64_t)F;
      }
    }
  } else if (m.drain == 2) {
    if (!work_conserving(m, C, P, &F, A_rec, F_rec)) {
      *status = MOE_ERR_INVALID_ARG;
      return false;
    }
  } else {
    // 64-bit with overflow checks: F_s >= A_s and F_s >= q, so any term
    // that overflows makes T(C) overflow too, the same error either way
    // q for the splits before the last, q_last for the last (its own task
    // size; with drain = 1 served by all C + P slots)
    int64_t q, q_last, F64 = 0;
    bool ovf = __builtin_mul_overflow(m.rho_num, cdiv64(m.W_comm, C), &q);
    ovf |= __builtin_mul_overflow(m.rho_last, cdiv64(m.W_last, m.drain ? (int64_t)C + P : C),
                                  &q_last);
    for (int s = 0; s < m.L && !ovf; ++s) {
      int64_t A;
      ovf |= __builtin_mul_overflow(cdiv64((int64_t)(s + 1) * m.W_comp, P), m.rho_den, &A);
      ovf |= __builtin_add_overflow(A, (int64_t)s * m.pi, &A);
      ovf |= __builtin_add_overflow(A > F64 ? A : F64, s == m.L - 1 ? q_last : q, &F64);
      if (A_rec) A_rec[s] = A;
      if (F_rec) F_rec[s] = F64;
    }
    if (ovf) {
      *status = MOE_ERR_INVALID_ARG;
      return false;
    }
    F = F64;
  }
  *T_out = (int64_t)F;
  *R_out = (int32_t)R;
  *P_out = (int32_t)P;
  return true;
}

// eq:tie-breaker: empty slots in the last compute wave of a split.
inline int64_t delta_of(const Model& m, int64_t P) { return cdiv64(m.W_comp, P) * P - m.W_comp; }

}  // namespace

extern "C" int moe_select_partition(const moe_workload_t* wl, const moe_select_params_t* p,
                                    moe_partition_t* out) {
  Model m;
  int st = build_model(wl, p, &m);
  if (st != MOE_OK) return st;
  bool found = false;
  int64_t bestT = 0, bestD = -1;   // bestD < 0: not computed yet (Delta is needed only on ties)
  int32_t bestC = 0, bestR = 0, bestP = 0;
  // P(C) does not grow with C, so past the first C >= 1 with P(C) <= 0
  // no candidate is legal (and a huge c_max costs nothing)
  for (int64_t C = p->c_min; C <= p->c_max; ++C) {
    int64_t T;
    int32_t R, P;
    st = MOE_OK;
    if (!eval_candidate(m, p, (int32_t)C, &T, &R, &P, &st)) {
      if (st != MOE_OK) return st;
      if (C >= 1) break;
      continue;
    }
    // lexicographic (T, Delta, C); C ascends, so strict improvement only
    bool better = !found || T < bestT;
    int64_t D = -1;
    if (!better && T == bestT) {
      if (bestD < 0) bestD = delta_of(m, bestP);
      D = delta_of(m, P);
      better = D < bestD;
    }
    if (better) {
      found = true;
      bestT = T;
      bestD = D;
      bestC = (int32_t)C;
      bestR = R;
      bestP = P;
    }
  }
  if (found && bestD < 0) bestD = delta_of(m, bestP);
  if (!found) return MOE_ERR_NO_LEGAL_PARTITION;
  if (out) {
    out->C = bestC;
    out->R = bestR;
    out->P = bestP;
    out->delta_comp = (int32_t)bestD;
    out->T_num = bestT;
    out->T_den = m.rho_den;
    out->W_comp = m.W_comp;
    out->W_comm = m.W_comm;
  }
  return bestC;
}

extern "C" int moe_select_partition_splits(const moe_workload_t* wl, const moe_select_params_t* p,
                                          int32_t l_min, int32_t l_max, moe_partition_t* out,
                                          int32_t* splits_out) {
  if (!wl || !p || l_min < 1 || l_max < l_min || l_max > kMaxSplitsSearched)
    return MOE_ERR_INVALID_ARG;
  bool found = false;
  moe_partition_t best{};
  int32_t bestL = 0;
  for (int32_t L = l_min; L <= l_max; ++L) {
    moe_workload_t w = *wl;
    w.splits = L;
    moe_partition_t cur;
    const int r = moe_select_partition(&w, p, &cur);
    if (r == MOE_ERR_NO_LEGAL_PARTITION) continue;
    if (r < 0) return r;
    // T(C) of different L share the unit (compute waves of the same P(C)),
    // but not the denominator: compare T_num / T_den exactly
    const i128 lhs = (i128)cur.T_num * (found ? best.T_den : 1);
    const i128 rhs = (i128)(found ? best.T_num : 0) * cur.T_den;
    if (!found || lhs < rhs) {   // L ascends: ties keep the smaller L
      found = true;
      best = cur;
      bestL = L;
    }
  }
  if (!found) return MOE_ERR_NO_LEGAL_PARTITION;
  if (out) *out = best;
  if (splits_out) *splits_out = bestL;
  return best.C;
}

extern "C" int moe_select_evaluate(const moe_workload_t* wl, const moe_select_params_t* p,
                                   int64_t* T_num_out, int32_t n, int64_t* T_den_out) {
  Model m;
  int st = build_model(wl, p, &m);
  if (st != MOE_OK) return st;
  const int64_t count = (int64_t)p->c_max - p->c_min + 1;
  if (!T_num_out || n < count) return MOE_ERR_INVALID_ARG;
  bool past = false;   // past the legal candidates (P(C) does not grow with C)
  for (int64_t i = 0; i < count; ++i) {
    int64_t T;
    int32_t R, P;
    st = MOE_OK;
    const int64_t C = p->c_min + i;
    if (!past && eval_candidate(m, p, (int32_t)C, &T, &R, &P, &st)) {
      T_num_out[i] = T;
    } else {
      if (st != MOE_OK) return st;
      if (C >= 1) past = true;
      T_num_out[i] = -1;
    }
  }
  if (T_den_out) *T_den_out = m.rho_den;
  return (int)count;
}

extern "C" int moe_select_candidate(const moe_workload_t* wl, const moe_select_params_t* p,
                                    int32_t C, int64_t* rho_num, int64_t* rho_den,
                                    int64_t* A_out, int64_t* F_out, int32_t n) {
  Model m;
  int st = build_model(wl, p, &m);
  if (st != MOE_OK) return st;
  if (C < 0) return MOE_ERR_INVALID_ARG;
  int64_t entries = C == 0 ? 1 : m.L;
  if (C > 0 && m.readiness == 1) {
    const int64_t R = cdiv64(C, p->occ_comm);
    const int64_t P = (int64_t)p->occ_comp * ((int64_t)p->num_cus - R);
    const int64_t tiles = (int64_t)m.L * m.W_comp;
    entries = P <= 0 ? 1 : tiles == 0 ? 1 : cdiv64(tiles, P);
  }
  if (entries > INT32_MAX || ((A_out || F_out) && n < entries)) return MOE_ERR_INVALID_ARG;
  int64_t T;
  int32_t R, P;
  st = MOE_OK;
  if (!eval_candidate(m, p, C, &T, &R, &P, &st, A_out, F_out))
    return st != MOE_OK ? st : MOE_ERR_NO_LEGAL_PARTITION;
  if (rho_num) *rho_num = m.rho_num;
  if (rho_den) *rho_den = m.rho_den;
  return (int)entries;
}

extern "C" const char* moe_strerror(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_ALIGNMENT: return "misaligned pointer";
    case MOE_ERR_WORKSPACE: return "workspace missing or too small";
    case MOE_ERR_NO_LEGAL_PARTITION: return "no legal partition: every candidate leaves P(C) <= 0";
    case MOE_ERR_HIP: return "HIP runtime error";
    case MOE_ERR_TIMEOUT: return "a consumer wait timed out";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape";
    case MOE_ERR_BAD_ROUTING: return "bad routing data on the device";
    default: return status >= 0 ? "ok" : "unknown error";
  }
}

extern "C" int moe_gemm2_abi_version(void) { return 108; }
