// Greedy Overlapping Optimization planner (Section 3.4), host only.
//
// The tile's Q partitions are cut into k_Q chunks and its KV partitions into
// k_KV chunks; the chunk collectives are AG-Q-i, AG-KV-j and RS-Q-i, and the
// compute tasks C-i-j need AG-Q-i and AG-KV-j, while RS-Q-i needs every
// C-i-j.  The planner emits one step per collective plus compute-only steps:
//  * the collective of a step is, among every chunk collective that can run
//    (each AG-Q-i and AG-KV-j not yet run, each RS-Q-i not yet run whose
//    compute tasks are all done), the one with the largest (time of the
//    compute it makes ready) / (its own time); ties go to the one that makes
//    more compute ready, then to AG-KV, AG-Q, RS-Q in that order, then to the
//    lower chunk index;
//  * the step also runs compute tasks that were ready when it started, in
//    (Q chunk, KV chunk) order, stopping once their time reaches gamma times
//    the collective's time;
//  * with no collective able to run, a step runs one ready compute task.
// Sums run in ascending chunk order (profits) or in fill order (step totals)
// so that the schedule is reproducible bit for bit on every GPU of a mesh,
// which must issue the same collectives in the same order.

#include "mesh_attn.h"

#include <cmath>
#include <vector>

#include "host_error.h"

namespace {

struct Cand {
  int32_t kind = MA_GOO_NONE;
  int32_t chunk = -1;
  double profit = 0.0, unlocked = 0.0;
  int rank = 0;  // AG-KV 0, AG-Q 1, RS-Q 2
};

bool better(const Cand& a, const Cand& b) {  // a strictly preferred to b
  if (a.profit != b.profit) return a.profit > b.profit;
  if (a.unlocked != b.unlocked) return a.unlocked > b.unlocked;
  if (a.rank != b.rank) return a.rank < b.rank;
  return a.chunk < b.chunk;
}

}  // namespace

extern "C" ma_status_t mesh_attn_goo_plan(int32_t k_q, int32_t k_kv,
                                          double t_ag_q, double t_ag_kv,
                                          double t_rs_q, const double* t_c,
                                          double gamma, ma_goo_step_t* steps,
                                          int32_t max_steps, int32_t* tasks,
                                          int32_t* num_steps) {
  using mesh_attn::host::fail;
  using mesh_attn::host::ok;
  if (k_q < 1 || k_kv < 1 || int64_t{k_q} * k_kv > 4096)
    return fail(MA_ERR_INVALID_ARG,
                "chunk counts k_q %d, k_kv %d: need >= 1 and k_q*k_kv <= 4096",
                k_q, k_kv);
  const double tc[3] = {t_ag_q, t_ag_kv, t_rs_q};
  for (double t : tc)
    if (!(t > 0.0) || !std::isfinite(t))
      return fail(MA_ERR_INVALID_ARG, "collective times must be finite and > 0");
  if (!(gamma > 0.0) || !std::isfinite(gamma))
    return fail(MA_ERR_INVALID_ARG, "gamma must be finite and > 0");
  if (!t_c || !steps || !tasks || !num_steps)
    return fail(MA_ERR_INVALID_ARG, "NULL argument");
  const int32_t n_tasks = k_q * k_kv;
  for (int32_t t = 0; t < n_tasks; ++t)
    if (!(t_c[t] >= 0.0) || !std::isfinite(t_c[t]))
      return fail(MA_ERR_INVALID_ARG, "t_c[%d] must be finite and >= 0", t);

  std::vector<char> gq(k_q, 0), gkv(k_kv, 0), rs(k_q, 0), done(n_tasks, 0);
  int32_t n_gq = 0, n_gkv = 0, n_rs = 0, n_steps = 0, n_out = 0;
  auto cost = [&](int32_t i, int32_t j) { return t_c[i * k_kv + j]; };
  auto is_ready = [&](int32_t i, int32_t j) {
    return gq[i] && gkv[j] && !done[i * k_kv + j];
  };
  auto emit_step = [&](int32_t kind, int32_t chunk) -> bool {
    if (n_steps >= max_steps) return false;
    steps[n_steps] = ma_goo_step_t{kind, chunk, n_out, 0};
    ++n_steps;
    return true;
  };
  auto emit_task = [&](int32_t i, int32_t j) {
    tasks[2 * n_out] = i;
    tasks[2 * n_out + 1] = j;
    ++n_out;
    ++steps[n_steps - 1].num_tasks;
    done[i * k_kv + j] = 1;
  };

  while (n_gq < k_q || n_gkv < k_kv || n_rs < k_q) {
    Cand best;
    bool have = false;
    auto consider = [&](const Cand& c) {
      if (!have || better(c, best)) best = c;
      have = true;
    };
    for (int32_t j = 0; j < k_kv; ++j) {
      if (gkv[j]) continue;
      Cand c;
      c.kind = MA_GOO_AG_KV;
      c.chunk = j;
      for (int32_t i = 0; i < k_q; ++i)
        if (gq[i]) c.unlocked += cost(i, j);
      c.profit = c.unlocked / t_ag_kv;
      c.rank = 0;
      consider(c);
    }
    for (int32_t i = 0; i < k_q; ++i) {
      if (gq[i]) continue;
      Cand c;
      c.kind = MA_GOO_AG_Q;
      c.chunk = i;
      for (int32_t j = 0; j < k_kv; ++j)
        if (gkv[j]) c.unlocked += cost(i, j);
      c.profit = c.unlocked / t_ag_q;
      c.rank = 1;
      consider(c);
    }
    for (int32_t i = 0; i < k_q; ++i) {
      if (rs[i]) continue;
      bool all = true;
      for (int32_t j = 0; j < k_kv && all; ++j) all = done[i * k_kv + j] != 0;
      if (!all) continue;
      Cand c;
      c.kind = MA_GOO_RS_Q;
      c.chunk = i;
      c.rank = 2;
      consider(c);
    }
    if (!have) {
      // Only compute can advance: one ready task, the first in order.
      int32_t fi = -1, fj = -1;
      for (int32_t i = 0; i < k_q && fi < 0; ++i)
        for (int32_t j = 0; j < k_kv; ++j)
          if (is_ready(i, j)) {
            fi = i;
            fj = j;
            break;
          }
      if (fi < 0)
        return fail(MA_ERR_INVALID_ARG, "planner made no progress");
      if (!emit_step(MA_GOO_NONE, -1))
        return fail(MA_ERR_CAPACITY, "more than %d steps", max_steps);
      emit_task(fi, fj);
      continue;
    }
    // Compute tasks ready at the start of the step, (i, j) order, until
    // their time reaches the target.
    std::vector<std::pair<int32_t, int32_t>> ready;
    for (int32_t i = 0; i < k_q; ++i)
      for (int32_t j = 0; j < k_kv; ++j)
        if (is_ready(i, j)) ready.emplace_back(i, j);
    if (!emit_step(best.kind, best.chunk))
      return fail(MA_ERR_CAPACITY, "more than %d steps", max_steps);
    const double target =
        gamma * (best.kind == MA_GOO_AG_Q ? t_ag_q
                 : best.kind == MA_GOO_AG_KV ? t_ag_kv : t_rs_q);
    double total = 0.0;
    for (const auto& t : ready) {
      if (total >= target) break;
      emit_task(t.first, t.second);
      total += cost(t.first, t.second);
    }
    if (best.kind == MA_GOO_AG_Q) {
      gq[best.chunk] = 1;
      ++n_gq;
    } else if (best.kind == MA_GOO_AG_KV) {
      gkv[best.chunk] = 1;
      ++n_gkv;
    } else {
      rs[best.chunk] = 1;
      ++n_rs;
    }
  }
  *num_steps = n_steps;
  return ok();
}
