// Host driver for the selector under AddressSanitizer and
// UndefinedBehaviorSanitizer (test infrastructure).  Reads one case per
// line on stdin (workload, parameters, a candidate C and an L range, all
// integers) and prints, per case, what the selector's entry points return:
// moe_select_partition, moe_select_evaluate, moe_select_partition_splits
// and moe_select_candidate.  Built with g++ together with the selector's
// source; the test compares its output with the shared library's.
#include <cstdint>
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "moe_gemm2.h"

int main() {
  std::string line;
  while (std::getline(std::cin, line)) {
    if (line.empty()) continue;
    std::istringstream in(line);
    moe_workload_t wl{};
    long long rows = 0;
    int has_counts = 0;
    in >> wl.T >> wl.H >> wl.I >> wl.E >> wl.topk >> wl.splits >> wl.ranks >> rows >> has_counts;
    wl.rows = rows;
    std::vector<int32_t> counts;
    if (has_counts) {
      counts.resize(wl.E > 0 ? wl.E : 0);
      for (auto& c : counts) in >> c;
      wl.host_expert_counts = counts.data();
    }
    moe_select_params_t p{};
    long long rn = 0, rd = 0, sn = 0, sd = 0;
    in >> p.tile_m >> p.tile_n >> p.comm_tile_m >> p.comm_tile_n >> p.occ_comp >> p.occ_comm >>
        p.num_cus >> p.c_min >> p.c_max >> p.groups >> rn >> rd >> p.k_ref >> p.tile_m_ref >>
        p.tile_n_ref >> p.d_ref >> p.split_axis >> p.drain >> p.rho_kh >> p.topk_ref >>
        p.comm_tile_n_ref >> p.readiness >> p.comm_tile_m_last >> sn >> sd;
    p.rho_ref_num = rn;
    p.rho_ref_den = rd;
    p.split_cost_num = sn;
    p.split_cost_den = sd;
    int Cq = 0, l_min = 1, l_max = 1;
    in >> Cq >> l_min >> l_max;
    if (!in) {
      std::printf("parse error\n");
      return 2;
    }
    moe_partition_t part{};
    const int r = moe_select_partition(&wl, &p, &part);
    std::printf("part %d", r);
    if (r >= 0)
      std::printf(" %d %d %d %d %lld %lld %lld %lld", part.C, part.R, part.P, part.delta_comp,
                  (long long)part.T_num, (long long)part.T_den, (long long)part.W_comp,
                  (long long)part.W_comm);
    const long long span = (long long)p.c_max - p.c_min;
    const int n = span >= 0 && span < 100000 ? (int)span + 1 : 0;
    std::vector<int64_t> table(n > 0 ? n : 1);
    int64_t den = 0;
    const int re = moe_select_evaluate(&wl, &p, table.data(), n, &den);
    std::printf(" | eval %d", re);
    if (re > 0) {
      std::printf(" %lld", (long long)den);
      for (int i = 0; i < re; ++i) std::printf(" %lld", (long long)table[i]);
    }
    moe_partition_t sp{};
    int32_t L = 0;
    const int rs = moe_select_partition_splits(&wl, &p, l_min, l_max, &sp, &L);
    std::printf(" | splits %d", rs);
    if (rs >= 0) std::printf(" %d %lld %lld", L, (long long)sp.T_num, (long long)sp.T_den);
    int64_t cn = 0, cd = 0;
    const int k = moe_select_candidate(&wl, &p, Cq, &cn, &cd, nullptr, nullptr, 0);
    std::printf(" | cand %d", k);
    if (k > 0) {
      std::vector<int64_t> A(k), F(k);
      const int k2 = moe_select_candidate(&wl, &p, Cq, &cn, &cd, A.data(), F.data(), k);
      std::printf(" %d %lld %lld", k2, (long long)cn, (long long)cd);
      for (int i = 0; i < k2; ++i) std::printf(" %lld %lld", (long long)A[i], (long long)F[i]);
    }
    std::printf("\n");
  }
  return 0;
}
