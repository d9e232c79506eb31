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

// Stage 1 score of expert e on every machine at once: the time-model
// weighted sum of the load the machine would hold and the cross-machine
// tokens it would receive after taking e. Machines without a free base slot
// score INT64_MAX. delta[m] = tokens of e from sources outside machine m.
void machine_scores(const int32_t* w_agg, int E, int e, int M, int R, int64_t we_e, const std::vector<int64_t>& ML,
                    const std::vector<int64_t>& MC, const std::vector<int>& hosted, int cap, int64_t c_load,
                    int64_t c_traffic, std::vector<int64_t>& score, std::vector<int64_t>& delta) {
  for (int m = 0; m < M; ++m) {
    int64_t inside = 0;
    for (int s = m * R; s < (m + 1) * R; ++s) inside += w_agg[(int64_t)s * E + e];
    delta[m] = we_e - inside;
    score[m] = hosted[m] < cap ? c_load * (ML[m] + we_e) + c_traffic * (MC[m] + delta[m]) : INT64_MAX;
  }
}

// Index of the smallest value, the lowest index among equals.
int first_argmin(const std::vector<int64_t>& v) {
  return (int)(std::min_element(v.begin(), v.end()) - v.begin());
}

// Load of every rank of a machine (ranks [r0, r0 + R)) with each copy of an
// expert carrying its share of the expert's load under the contiguous
// integer split, copy 0 first.
std::vector<int64_t> copy_loads(const std::vector<int64_t>& we, const std::vector<int>& local,
                                const std::vector<std::vector<int>>& copies, int r0, int R) {
  std::vector<int64_t> RL(R, 0);
  for (int e : local) {
    const int64_t c = (int64_t)copies[e].size();
    for (int64_t i = 0; i < c; ++i) RL[copies[e][i] - r0] += we[e] * (i + 1) / c - we[e] * i / c;
  }
  return RL;
}

// The locally heaviest expert: the largest load per copy w_e / c_e, compared
// exactly as w_e * c_f against w_f * c_e; the lowest id among equals.
int heaviest_expert(const std::vector<int64_t>& we, const std::vector<int>& local,
                    const std::vector<std::vector<int>>& copies) {
  int heavy = -1;
  for (int e : local)  // ascending ids
    if (heavy < 0 || we[e] * (int64_t)copies[heavy].size() > we[heavy] * (int64_t)copies[e].size()) heavy = e;
  return heavy;
}

// Stage 3 (App. D): R * N_r times, a replica of the locally heaviest expert
// onto the machine rank with the least current load among those with a free
// redundant slot and no copy of that expert; stops when no rank qualifies.
void stage3_replicate(const std::vector<int64_t>& we, const std::vector<int>& local,
                      std::vector<std::vector<int>>& copies, int r0, int R, int N_r) {
  std::vector<int> used(R, 0);
  for (int k = 0; k < R * N_r && !local.empty(); ++k) {
    const int heavy = heaviest_expert(we, local, copies);
    const std::vector<int64_t> RL = copy_loads(we, local, copies, r0, R);
    int best = -1;
    for (int r = 0; r < R; ++r) {
      if (used[r] >= N_r) continue;
      if (std::find(copies[heavy].begin(), copies[heavy].end(), r0 + r) != copies[heavy].end()) continue;
      if (best < 0 || RL[r] < RL[best]) best = r;
    }
    if (best < 0) return;
    copies[heavy].push_back(r0 + best);
    ++used[best];
  }
}

// n token units onto copies whose ranks hold `load`, each unit to the copy
// with the least load (lowest copy index among equals), in closed form:
// every copy below the level lam that the n units reach is raised to lam,
// and the rest go one each to the copies now at lam, in copy order. Adds the
// units per copy to out[] and to load[].
void water_fill_units(int64_t n, const std::vector<int>& c, std::vector<int64_t>& load, int32_t* out) {
  const int nc = (int)c.size();
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

// Stage 4 (App. D) on one machine: non-replicated experts keep their tokens
// on their one copy; then the replicated experts in descending load, and
// within one the source ranks in ascending order, are water-filled.
void stage4_water_fill(const int32_t* w, const std::vector<int64_t>& we, int E, int P, int C_max,
                       const std::vector<int>& local, const std::vector<std::vector<int>>& copies,
                       std::vector<int64_t>& load, int32_t* counts) {
  std::vector<int> reps;
  for (int e : local) {
    if (copies[e].size() == 1) {
      for (int s = 0; s < P; ++s) counts[((int64_t)s * E + e) * C_max] = w[(int64_t)s * E + e];
      load[copies[e][0]] += we[e];
    } else {
      reps.push_back(e);
    }
  }
  for (int e : desc_order(we, reps))
    for (int s = 0; s < P; ++s)
      if (w[(int64_t)s * E + e] > 0)
        water_fill_units(w[(int64_t)s * E + e], copies[e], load, counts + ((int64_t)s * E + e) * C_max);
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
  // machine level: each expert, in descending aggregate load, to the machine
  // with the lowest score (Sec. 8 Stage 1)
  std::vector<int64_t> ML(M, 0), MC(M, 0), score(M), delta(M);
  std::vector<int> hosted(M, 0), machine(E, -1);
  for (int e : desc_order(we, all)) {
    machine_scores(w_agg, E, e, M, R, we[e], ML, MC, hosted, R * N_b, c_load, c_traffic, score, delta);
    const int m = first_argmin(score);
    machine[e] = m;
    ML[m] += we[e];
    MC[m] += delta[m];
    ++hosted[m];
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
  std::vector<std::vector<int>> locals(M);
  for (int m = 0; m < M; ++m) {
    std::vector<int>& local = locals[m];
    for (int e = 0; e < E; ++e)
      if (main[e] / R == m) local.push_back(e);
    // Stage 2: LPT relocation inside the machine by this micro-step's load
    if (!rank_lpt(we, local, m * R, R, N_b, main))
      return set_error(FOREMOE_EINVAL, "plan_micro_step: base slots overflow on machine %d", m);
    for (int e : local) copies[e].assign(1, main[e]);
    // Stage 3: replicas into the machine's R * N_r redundant slots
    stage3_replicate(we, local, copies, m * R, R, N_r);
  }
  for (int e = 0; e < E; ++e)
    if ((int)copies[e].size() > C_max)
      return set_error(FOREMOE_EINVAL, "plan_micro_step: expert %d has %d copies > C_max=%d", e,
                       (int)copies[e].size(), C_max);
  std::fill(counts, counts + (int64_t)P * E * C_max, 0);
  // Stage 4: water-filling, machine by machine
  std::vector<int64_t> load(P, 0);
  for (int m = 0; m < M; ++m) stage4_water_fill(w, we, E, P, C_max, locals[m], copies, load, counts);
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
