// Tail-batching round planner; see tail_batch.hpp for the policy.
#include "tail_batch.hpp"

#include <algorithm>
#include <cmath>
#include <deque>
#include <numeric>
#include <stdexcept>

namespace rollpack {

namespace {

// Indices of the k smallest lengths among the first r_spec responses of a
// prompt, lower index first on ties.
std::vector<int32_t> shortest_k(const int32_t* row, int32_t r_spec, int32_t k) {
  std::vector<int32_t> idx(r_spec);
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) { return row[a] < row[b]; });
  idx.resize(std::min<size_t>(idx.size(), static_cast<size_t>(k)));
  return idx;
}

}  // namespace

int32_t spec_count(double eta, int32_t k) {
  const double x = eta * k;
  return static_cast<int32_t>(std::ceil(x - 1e-6 * x));
}

TailBatchPlan plan_tail_batching(int32_t n_prompts, int32_t r_spec, const int32_t* lens,
                                 int32_t P0, int32_t R0, double eta_p, double eta_r) {
  if (n_prompts < 0 || P0 < 1 || R0 < 1 || !(eta_p >= 1.0) || !(eta_r >= 1.0) || std::isinf(eta_p) ||
      std::isinf(eta_r) || eta_p * P0 > 1e9 || eta_r * R0 > 1e9)
    throw std::invalid_argument("tail batching needs n >= 0, P0 >= 1, R0 >= 1 and finite eta_p, eta_r >= 1");
  if (r_spec != spec_count(eta_r, R0)) throw std::invalid_argument("r_spec must equal ceil(eta_r * R0)");
  const int32_t p_spec = spec_count(eta_p, P0);

  TailBatchPlan plan;
  plan.accept_round.assign(n_prompts, -1);
  plan.kept.assign(static_cast<size_t>(n_prompts) * r_spec, 0);

  int32_t next_fresh = 0;
  std::deque<int32_t> queue;
  while (next_fresh < n_prompts || !queue.empty()) {
    PlannedRound rnd;
    const int32_t round_idx = static_cast<int32_t>(plan.rounds.size());
    if (static_cast<int32_t>(queue.size()) >= P0 || (next_fresh >= n_prompts && !queue.empty())) {
      // Long round: the oldest queued prompts, R0 responses each, run to completion.
      rnd.kind = 1;
      while (!queue.empty() && static_cast<int32_t>(rnd.launched.size()) < P0) {
        rnd.launched.push_back(queue.front());
        queue.pop_front();
      }
      std::sort(rnd.launched.begin(), rnd.launched.end());
      rnd.run_steps.assign(rnd.launched.size() * r_spec, 0);
      for (size_t i = 0; i < rnd.launched.size(); ++i) {
        const int32_t p = rnd.launched[i];
        for (int32_t r = 0; r < R0; ++r) {
          const int32_t L = lens[static_cast<size_t>(p) * r_spec + r];
          rnd.run_steps[i * r_spec + r] = L;
          rnd.time = std::max(rnd.time, L);
          plan.kept[static_cast<size_t>(p) * r_spec + r] = 1;
        }
        plan.accept_round[p] = round_idx;
      }
      rnd.accepted = rnd.launched;
    } else {
      // Short round: race to completion among ceil(eta_p*P0) fresh prompts.
      rnd.kind = 0;
      for (int32_t i = 0; i < p_spec && next_fresh < n_prompts; ++i) rnd.launched.push_back(next_fresh++);
      const size_t n = rnd.launched.size();
      std::vector<int32_t> done_at(n);
      for (size_t i = 0; i < n; ++i) {
        const int32_t* row = lens + static_cast<size_t>(rnd.launched[i]) * r_spec;
        std::vector<int32_t> sorted(row, row + r_spec);
        std::sort(sorted.begin(), sorted.end());
        done_at[i] = sorted[R0 - 1];
      }
      std::vector<size_t> order(n);
      std::iota(order.begin(), order.end(), 0);
      std::stable_sort(order.begin(), order.end(),
                       [&](size_t a, size_t b) { return done_at[a] < done_at[b]; });
      const size_t keep_n = std::min<size_t>(n, static_cast<size_t>(P0));
      std::vector<uint8_t> is_acc(n, 0);
      for (size_t j = 0; j < keep_n; ++j) {
        is_acc[order[j]] = 1;
        rnd.time = std::max(rnd.time, done_at[order[j]]);
      }
      rnd.run_steps.assign(n * r_spec, 0);
      for (size_t i = 0; i < n; ++i) {
        const int32_t p = rnd.launched[i];
        const int32_t* row = lens + static_cast<size_t>(p) * r_spec;
        const int32_t stop = is_acc[i] ? done_at[i] : rnd.time;
        for (int32_t r = 0; r < r_spec; ++r) rnd.run_steps[i * r_spec + r] = std::min(row[r], stop);
        if (is_acc[i]) {
          rnd.accepted.push_back(p);
          plan.accept_round[p] = round_idx;
          for (int32_t r : shortest_k(row, r_spec, R0)) plan.kept[static_cast<size_t>(p) * r_spec + r] = 1;
        } else {
          rnd.rejected.push_back(p);
          queue.push_back(p);
        }
      }
    }
    plan.rounds.push_back(std::move(rnd));
  }
  return plan;
}

}  // namespace rollpack
