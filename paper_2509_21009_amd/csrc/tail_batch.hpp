// Tail-batching round planner (paper section 3), host only.
//
// Each rollout step needs P0 prompts with R0 responses each.  A short round
// over-provisions: it launches ceil(eta*P0) prompts with ceil(eta*R0)
// responses each and keeps the first P0 prompts to complete, each with its
// first R0 completed responses ("race to completion").  Prompts aborted in a
// short round join a FIFO long-prompt queue; when the queue holds P0 prompts
// they run as a long round with speculation disabled, so no prompt is ever
// dropped.  With forced response lengths, "first to complete" is decided by
// the lengths: a response finishes after as many decode steps as its length.
//
// Readings where the paper is silent: ties go to the lower index; the round
// ends when its P0-th prompt completes; a short round with fewer than
// ceil(eta*P0) fresh prompts launches what is left and keeps min(P0, n);
// when no fresh prompt is left, queued prompts are flushed in long rounds.
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

// lens: [n_prompts * r_spec] response lengths (>= 0).  Requires P0, R0 >= 1,
// eta >= 1 and r_spec == ceil(eta * R0).
TailBatchPlan plan_tail_batching(int32_t n_prompts, int32_t r_spec, const int32_t* lens,
                                 int32_t P0, int32_t R0, double eta);

}  // namespace rollpack
