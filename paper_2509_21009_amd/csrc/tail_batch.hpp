// Tail-batching round planner (paper section 3), host only.
//
// Each rollout step needs P0 prompts with R0 responses each.  A short round
// over-provisions: it launches ceil(eta_p*P0) prompts with ceil(eta_r*R0)
// responses each (section 6.3 varies the two factors separately) and keeps
// the first P0 prompts to complete, each with its first R0 completed
// responses ("race to completion").  Prompts aborted in a
// short round join a FIFO long-prompt queue; when the queue holds P0 prompts
// they run as a long round with speculation disabled, so no prompt is ever
// dropped.  With forced response lengths, "first to complete" is decided by
// the lengths: a response finishes after as many decode steps as its length.
//
// Readings where the paper is silent: ties go to the lower index; the round
// ends when its P0-th prompt completes; a short round with fewer than
// ceil(eta_p*P0) fresh prompts launches what is left and keeps min(P0, n);
// when no fresh prompt is left, queued prompts are flushed in long rounds.
// A product eta*P0 within one part in 10^6 of an integer counts as that
// integer, so that factors such as 1.1 given in single precision round as
// their decimal value does.
#pragma once

#include <cstdint>
#include <vector>

namespace rollpack {

struct PlannedRound {
  int kind = 0;                    // 0 short, 1 long
  int32_t time = 0;                // decode steps until the round ends
  std::vector<int32_t> launched;   // ascending prompt ids
  std::vector<int32_t> run_steps;  // [launched.size() * r_spec]
  std::vector<int32_t> accepted;   // ascending prompt ids
  std::vector<int32_t> rejected;   // ascending prompt ids
};

struct TailBatchPlan {
  std::vector<PlannedRound> rounds;
  std::vector<int32_t> accept_round;  // [n_prompts]
  std::vector<uint8_t> kept;          // [n_prompts * r_spec]
};

// ceil(eta * k) with the tolerance above.
int32_t spec_count(double eta, int32_t k);

// lens: [n_prompts * r_spec] response lengths (>= 0).  Requires P0, R0 >= 1,
// eta_p, eta_r >= 1 and r_spec == spec_count(eta_r, R0).
TailBatchPlan plan_tail_batching(int32_t n_prompts, int32_t r_spec, const int32_t* lens,
                                 int32_t P0, int32_t R0, double eta_p, double eta_r);

}  // namespace rollpack
