// Placement planner on the host (Sec. 8, Alg. 1; App. D, Alg. 3).
//
// Stage 1 places every expert on one rank from the step's aggregate load
// (machine-level greedy on computation load and cross-machine traffic, then
// LPT over each machine's ranks). Per micro-step, Stages 2-4 of the policy
// update stage rebalance inside each machine: LPT relocation by this
// micro-step's load, replicas of the heaviest expert onto the least-loaded
// ranks, and water-filling of every replicated expert's tokens over its
// copies. All decisions use integer arithmetic with fixed tie rules (lowest
// expert id, rank id or copy index among equals), so the result is exactly
// reproducible.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "common.h"
#include "foremoe.h"

namespace foremoe {
namespace {

// Expert ids sorted by descending load, ties by ascending id.
std::vector<int> desc_order(const std::vector<int64_t>& w, const std::vector<int>& ids) {
  std::vector<int> o(ids);
  std::sort(o.begin(), o.end(), [&](int a, int b) { return w[a] != w[b] ? w[a] > w[b] : a < b; });
  return o;
}

// LPT over ranks [r0, r0 + R) with at most cap experts per rank; writes
// rank_of[e]. Returns false when the experts do not fit.
bool rank_lpt(const std::vector<int64_t>& w, const std::vector<int>& experts, int r0, int R, int cap,
              std::vector<int>& rank_of) {
  std::vector<int64_t> load(R, 0);
  std::vector<int> used(R, 0);
  for (int e : desc_order(w, experts)) {
    int best = -1;
    for (int r = 0; r < R; ++r) {
      if (used[r] >= cap) continue;
      if (best < 0 || load[r] < load[best]) best = r;
    }
    if (best < 0) return false;
    rank_of[e] = r0 + best;
    load[best] += w[e];
    ++used[best];
  }
  return true;
}

bool check_machine(const foremoe_machine* mc, int64_t E) {
  return mc && mc->M >= 1 && mc->R >= 1 && mc->N_b >= 1 && mc->N_r >= 0 && (int64_t)mc->M * mc->R <= 4096 &&
         E >= 1 && E <= FOREMOE_MAX_EXPERTS && E <= (int64_t)mc->M * mc->R * mc->N_b;
}

}  // namespace
}  // namespace foremoe

using namespace foremoe;

#define REQUIRE(cond, ...)                                      \
  do {                                                          \
    if (!(cond)) return set_error(FOREMOE_EINVAL, __VA_ARGS__); \
  } while (0)

extern "C" {

int foremoe_plan_base(const int32_t* w_agg, int32_t E, const foremoe_machine* mc, int64_t c_load, int64_t c_traffic,
                      int32_t* base_rank) {
  REQUIRE(check_machine(mc, E), "plan_base: machine shape or E out of range");
  REQUIRE(w_agg && base_rank, "plan_base: NULL array");
  REQUIRE(c_load >= 0 && c_traffic >= 0 && c_load <= (1 << 20) && c_traffic <= (1 << 20),
          "plan_base: score weights must be in [0, 2^20]");
  const int M = mc->M, R = mc->R, P = M * R, N_b = mc->N_b;
  std::vector<int64_t> we(E, 0);
  for (int s = 0; s < P; ++s)
    for (int e = 0; e < E; ++e) {
      REQUIRE(w_agg[(int64_t)s * E + e] >= 0, "plan_base: negative load");
      we[e] += w_agg[(int64_t)s * E + e];
    }
  std::vector<int> all(E);
  for (int e = 0; e < E; ++e) all[e] = e;
  // machine level: score = c_load (ML + w_e) + c_traffic (MC + Delta_{m,e})
  std::vector<int64_t> ML(M, 0), MC(M, 0);
  std::vector<int> count(M, 0), machine(E, -1);
  for (int e : desc_order(we, all)) {
    int best = -1;
    int64_t best_score = 0, best_delta = 0;
    for (int m = 0; m < M; ++m) {
      if (count[m] >= R * N_b) continue;
      int64_t inside = 0;
      for (int s = m * R; s < (m + 1) * R; ++s) inside += w_agg[(int64_t)s * E + e];
      const int64_t delta = we[e] - inside;  // tokens of e from other machines
      const int64_t score = c_load * (ML[m] + we[e]) + c_traffic * (MC[m] + delta);
      if (best < 0 || score < best_score) {
        best = m;
        best_score = score;
        best_delta = delta;
      }
    }
    machine[e] = best;
    ML[best] += we[e];
    MC[best] += best_delta;
    ++count[best];
  }
  // rank level: LPT inside each machine
  std::vector<int> rank_of(E, -1);
  for (int m = 0; m < M; ++m) {
    std::vector<int> local;
    for (int e = 0; e < E; ++e)
      if (machine[e] == m) local.push_back(e);
    if (!rank_lpt(we, local, m * R, R, N_b, rank_of)) return set_error(FOREMOE_EINVAL, "plan_base: slots overflow");
  }
  for (int e = 0; e < E; ++e) base_rank[e] = rank_of[e];
  return FOREMOE_OK;
}

int foremoe_plan_micro_step(const int32_t* w, int32_t E, const foremoe_machine* mc, const int32_t* base_rank,
                            int32_t C_max, int32_t* copy_rank, int32_t* counts, int64_t* rank_load) {
  REQUIRE(check_machine(mc, E), "plan_micro_step: machine shape or E out of range");
  REQUIRE(w && base_rank && copy_rank && counts, "plan_micro_step: NULL array");
  REQUIRE(C_max >= 1 && C_max <= FOREMOE_MAX_REPLICAS, "plan_micro_step: C_max=%d out of range", C_max);
  const int M = mc->M, R = mc->R, P = M * R, N_b = mc->N_b, N_r = mc->N_r;
  std::vector<int64_t> we(E, 0);
  for (int s = 0; s < P; ++s)
    for (int e = 0; e < E; ++e) {
      REQUIRE(w[(int64_t)s * E + e] >= 0, "plan_micro_step: negative load");
      we[e] += w[(int64_t)s * E + e];
    }
  std::vector<int> main(E);
  for (int e = 0; e < E; ++e) {
    REQUIRE(base_rank[e] >= 0 && base_rank[e] < P, "plan_micro_step: base_rank[%d]=%d out of range", e, base_rank[e]);
    main[e] = base_rank[e];
  }
  std::vector<std::vector<int>> copies(E);
  for (int m = 0; m < M; ++m) {
    std::vector<int> local;
    for (int e = 0; e < E; ++e)
      if (main[e] / R == m) local.push_back(e);
    // Stage 2: LPT relocation inside the machine by this micro-step's load
    if (!rank_lpt(we, local, m * R, R, N_b, main))
      return set_error(FOREMOE_EINVAL, "plan_micro_step: base slots overflow on machine %d", m);
    for (int e : local) copies[e].assign(1, main[e]);
    // Stage 3: R * N_r replicas; the copies of an expert share its load by
    // the contiguous integer split while placing them
    std::vector<int> used(R, 0);
    for (int k = 0; k < R * N_r && !local.empty(); ++k) {
      int heavy = -1;
      for (int e : local)  // ascending ids: the first maximum of w_e / c_e
        if (heavy < 0 || we[e] * (int64_t)copies[heavy].size() > we[heavy] * (int64_t)copies[e].size()) heavy = e;
      std::vector<int64_t> RL(R, 0);
      for (int e : local) {
        const int64_t c = (int64_t)copies[e].size();
        for (int64_t i = 0; i < c; ++i) RL[copies[e][i] - m * R] += we[e] * (i + 1) / c - we[e] * i / c;
      }
      int best = -1;
      for (int r = 0; r < R; ++r) {
        if (used[r] >= N_r) continue;
        if (std::find(copies[heavy].begin(), copies[heavy].end(), m * R + r) != copies[heavy].end()) continue;
        if (best < 0 || RL[r] < RL[best]) best = r;
      }
      if (best < 0) break;
      copies[heavy].push_back(m * R + best);
      ++used[best];
    }
  }
  for (int e = 0; e < E; ++e)
    if ((int)copies[e].size() > C_max)
      return set_error(FOREMOE_EINVAL, "plan_micro_step: expert %d has %d copies > C_max=%d", e,
                       (int)copies[e].size(), C_max);
  std::fill(counts, counts + (int64_t)P * E * C_max, 0);
  // Stage 4: water-filling per machine, each token unit to the least-loaded copy
  std::vector<int64_t> load(P, 0);
  for (int m = 0; m < M; ++m) {
    std::vector<int> reps;
    for (int e = 0; e < E; ++e) {
      if (copies[e][0] / R != m) continue;
      if (copies[e].size() == 1) {
        for (int s = 0; s < P; ++s) counts[((int64_t)s * E + e) * C_max] = w[(int64_t)s * E + e];
        load[copies[e][0]] += we[e];
      } else {
        reps.push_back(e);
      }
    }
    for (int e : desc_order(we, reps)) {
      const std::vector<int>& c = copies[e];
      const int nc = (int)c.size();
      for (int s = 0; s < P; ++s) {
        // The n units of (s, e), each to the copy with the least load
        // (lowest copy index among equals), in closed form: raise every copy
        // below the level lam to lam, where lam is the highest level the n
        // units reach, then give the rest one each to the copies now at lam,
        // in copy order.
        const int64_t n = w[(int64_t)s * E + e];
        if (n == 0) continue;
        int64_t lo = load[c[0]], hi = load[c[0]];
        for (int i = 1; i < nc; ++i) {
          lo = std::min(lo, load[c[i]]);
          hi = std::max(hi, load[c[i]]);
        }
        hi += n;
        while (lo < hi) {  // largest lam with sum max(0, lam - load) <= n
          const int64_t mid = lo + (hi - lo + 1) / 2;
          int64_t need = 0;
          for (int i = 0; i < nc; ++i) need += std::max<int64_t>(0, mid - load[c[i]]);
          if (need <= n) lo = mid;
          else hi = mid - 1;
        }
        int32_t* out = counts + ((int64_t)s * E + e) * C_max;
        int64_t rest = n;
        for (int i = 0; i < nc; ++i) {
          const int64_t add = std::max<int64_t>(0, lo - load[c[i]]);
          out[i] += (int32_t)add;
          load[c[i]] += add;
          rest -= add;
        }
        for (int i = 0; i < nc && rest > 0; ++i)
          if (load[c[i]] == lo) {
            ++out[i];
            ++load[c[i]];
            --rest;
          }
      }
    }
  }
  for (int e = 0; e < E; ++e)
    for (int i = 0; i < C_max; ++i) copy_rank[(int64_t)e * C_max + i] = i < (int)copies[e].size() ? copies[e][i] : -1;
  if (rank_load)
    for (int r = 0; r < P; ++r) rank_load[r] = load[r];
  return FOREMOE_OK;
}

int foremoe_plan_rank_slots(const int32_t* copy_rank, int32_t E, int32_t C_max, int32_t rank, int32_t max_slots,
                            int32_t* slot_expert, int32_t* slot_replica, int32_t* slot_widx, int32_t* expert_nrep,
                            int32_t* local_experts, int32_t* S_out, int32_t* W_out) {
  REQUIRE(copy_rank && slot_expert && slot_replica && slot_widx && expert_nrep && local_experts && S_out && W_out,
          "plan_rank_slots: NULL array");
  REQUIRE(E >= 1 && E <= FOREMOE_MAX_EXPERTS && C_max >= 1 && C_max <= FOREMOE_MAX_REPLICAS && rank >= 0 &&
              max_slots >= 0,
          "plan_rank_slots: sizes out of range");
  int S = 0, W = 0;
  std::vector<int> widx(E, -1);
  auto add = [&](int e, int c) -> bool {
    if (S >= max_slots) return false;
    if (widx[e] < 0) {
      widx[e] = W;
      local_experts[W++] = e;
    }
    slot_expert[S] = e;
    slot_replica[S] = c;
    slot_widx[S] = widx[e];
    ++S;
    return true;
  };
  // main copies first, then replica copies, each in ascending (expert, copy)
  for (int e = 0; e < E; ++e)
    if (copy_rank[(int64_t)e * C_max] == rank && !add(e, 0))
      return set_error(FOREMOE_EINVAL, "plan_rank_slots: more than max_slots=%d slots", max_slots);
  for (int e = 0; e < E; ++e)
    for (int c = 1; c < C_max; ++c)
      if (copy_rank[(int64_t)e * C_max + c] == rank && !add(e, c))
        return set_error(FOREMOE_EINVAL, "plan_rank_slots: more than max_slots=%d slots", max_slots);
  for (int e = 0; e < E; ++e) {
    int n = 0;
    while (n < C_max && copy_rank[(int64_t)e * C_max + n] >= 0) ++n;
    expert_nrep[e] = n > 0 ? n : 1;
  }
  *S_out = S;
  *W_out = W;
  return FOREMOE_OK;
}

}  // extern "C"
