// extern "C" surface of the rollout library (declared in include/rollpack.h).
// Every entry point validates its arguments, converts exceptions into
// rp_status codes and records a thread-local message for rp_last_error().
#include <cmath>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "engine.hpp"
#include "static_ws.hpp"
#include "tail_batch.hpp"

namespace {

thread_local std::string g_last_error;

template <typename F>
rp_status guarded(F&& f) {
  try {
    f();
    g_last_error.clear();
    return RP_OK;
  } catch (const rollpack::RpError& e) {
    g_last_error = e.what();
    return e.status;
  } catch (const std::bad_alloc&) {
    g_last_error = "host allocation failed";
    return RP_ERR_CAPACITY;
  } catch (const std::exception& e) {
    g_last_error = e.what();
    return RP_ERR_INVALID_ARG;
  }
}

rollpack::Engine* live_engine(rp_engine* eng) {
  if (!eng || !eng->impl) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null engine");
  if (eng->impl->broken())
    throw rollpack::RpError(RP_ERR_BAD_STATE, "engine is unusable after an earlier HIP error");
  return eng->impl;
}

// Marks the engine unusable when a HIP error escapes mid-operation.
template <typename F>
rp_status engine_call(rp_engine* eng, F&& f) {
  return guarded([&] {
    rollpack::Engine* e = live_engine(eng);
    try {
      f(e);
    } catch (const rollpack::RpError& err) {
      if (err.status == RP_ERR_HIP) e->mark_broken();
      throw;
    }
  });
}

// Runs one rollout call of the given schedule mode on a fresh engine (the
// one-shot entry points).  Returns the number of rounds.
int32_t run_one_shot(rollpack::Engine& e, int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens,
                     const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed, float temperature,
                     int32_t schedule_mode, const int32_t* round_ids, const rp_tail_params* tail,
                     int32_t* resp_tokens_out, float* resp_logprobs_out, int32_t* resp_len_out, int32_t* kept_out,
                     rp_round_stats* stats_out, int32_t max_stats) {
  using rollpack::RpError;
  if (max_stats < 0) throw RpError(RP_ERR_INVALID_ARG, "max_stats must be >= 0");
  if (n < 1) throw RpError(RP_ERR_INVALID_ARG, "n must be >= 1");
  switch (schedule_mode) {
    case RP_SCHEDULE_NONE:
    case RP_SCHEDULE_ROUNDS: {
      if ((schedule_mode == RP_SCHEDULE_ROUNDS) != (round_ids != nullptr))
        throw RpError(RP_ERR_INVALID_ARG, "round_ids are given exactly under RP_SCHEDULE_ROUNDS");
      if (tail) throw RpError(RP_ERR_INVALID_ARG, "tail parameters belong to RP_SCHEDULE_TAIL_BATCHING");
      const int32_t r = e.rollout(n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                                  round_ids, resp_tokens_out, resp_logprobs_out, resp_len_out, stats_out, max_stats);
      if (kept_out)
        for (int32_t i = 0; i < n; ++i) kept_out[i] = 1;
      return r;
    }
    case RP_SCHEDULE_TAIL_BATCHING: {
      if (!tail || round_ids) throw RpError(RP_ERR_INVALID_ARG, "tail batching needs rp_tail_params and no round_ids");
      if (tail->r_spec < 1 || n % tail->r_spec != 0)
        throw RpError(RP_ERR_INVALID_ARG, "tail batching: n must be a multiple of r_spec >= 1");
      const int32_t n_prompts = n / tail->r_spec;
      std::vector<int32_t> accept(static_cast<size_t>(n_prompts)), kept;
      if (!kept_out) kept.resize(static_cast<size_t>(n));
      return e.rollout_tail_batched(n_prompts, tail->r_spec, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens,
                                    seed, temperature, tail->P0, tail->R0, tail->eta_p, tail->eta_r, resp_tokens_out,
                                    resp_logprobs_out, resp_len_out, accept.data(), kept_out ? kept_out : kept.data(),
                                    stats_out, max_stats);
    }
    default:
      throw RpError(RP_ERR_INVALID_ARG, "unknown schedule mode");
  }
}

}  // namespace

extern "C" {

rp_status rp_kv_bytes_per_token(const rp_model_config* cfg, size_t* bytes) {
  return guarded([&] {
    if (!cfg || !bytes) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null argument");
    rollpack::validate_config(*cfg);
    const size_t esz = cfg->dtype == RP_DTYPE_BF16 ? 2 : 4;
    *bytes = static_cast<size_t>(cfg->n_layers) * 2 * cfg->n_kv_heads * cfg->head_dim * esz;
  });
}

rp_status rp_workspace_size(const rp_model_config* cfg, const rp_engine_limits* limits, size_t* kv_bytes,
                            size_t* scratch_bytes) {
  return guarded([&] {
    if (!cfg || !limits || !kv_bytes || !scratch_bytes) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null argument");
    rollpack::validate_config(*cfg);
    rollpack::validate_limits(*limits);
    *kv_bytes = rollpack::kv_pool_bytes(*cfg, limits->kv_pages);
    *scratch_bytes = rollpack::plan_scratch(*cfg, *limits).total;
  });
}

rp_status rp_engine_create(const rp_model_config* cfg, const rp_weights* weights, const rp_engine_limits* limits,
                           void* kv_ws, size_t kv_bytes, void* scratch_ws, size_t scratch_bytes, void* hip_stream,
                           rp_engine** out) {
  return guarded([&] {
    if (!cfg || !weights || !limits || !out) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null argument");
    *out = nullptr;
    rollpack::validate_config(*cfg);
    rollpack::validate_limits(*limits);
    auto* impl = new rollpack::Engine(*cfg, *weights, *limits, kv_ws, kv_bytes, scratch_ws, scratch_bytes,
                                      static_cast<hipStream_t>(hip_stream));
    *out = new rp_engine{impl};
  });
}

void rp_engine_destroy(rp_engine* eng) {
  if (!eng) return;
  delete eng->impl;
  delete eng;
}

rp_status rp_packed_weights_bytes(const rp_model_config* cfg, size_t* bytes) {
  return guarded([&] {
    if (!cfg || !bytes) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null argument");
    rollpack::validate_config(*cfg);
    *bytes = rollpack::packed_weights_bytes(*cfg);
  });
}

rp_status rp_engine_set_packed_weights(rp_engine* eng, void* packed_ws, size_t bytes) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->set_packed_weights(packed_ws, bytes); });
}

rp_status rp_prefill(rp_engine* eng, int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens,
                     const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed, float temperature,
                     float* logits_out, int32_t* first_tokens_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    e->prefill(n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature, logits_out,
               first_tokens_out);
  });
}

rp_status rp_decode_step(rp_engine* eng, const int32_t* forced_tokens, float* logits_out, int64_t* row_ids_out,
                         int32_t* n_active_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    const int32_t b = e->decode_step(forced_tokens, logits_out, row_ids_out);
    if (n_active_out) *n_active_out = b;
  });
}

rp_status rp_free_finished(rp_engine* eng, int64_t* finished_ids_out, int32_t cap, int32_t* n_finished_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    if (cap < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "cap must be >= 0");
    const int32_t k = e->free_finished(finished_ids_out, cap);
    if (n_finished_out) *n_finished_out = k;
  });
}

rp_status rp_abort(rp_engine* eng, int32_t n, const int64_t* seq_ids) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->abort(n, seq_ids); });
}

rp_status rp_get_tokens(rp_engine* eng, int64_t seq_id, int32_t* out, int32_t cap, int32_t* len_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    if (cap < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "cap must be >= 0");
    const int32_t k = e->get_tokens(seq_id, out, cap);
    if (len_out) *len_out = k;
  });
}

rp_status rp_rollout_generate(rp_engine* eng, int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens,
                              const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed,
                              float temperature, const int32_t* round_ids, int32_t* resp_tokens_out,
                              float* resp_logprobs_out, int32_t* resp_len_out, rp_round_stats* stats_out,
                              int32_t max_stats, int32_t* n_rounds_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    if (max_stats < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "max_stats must be >= 0");
    const int32_t r = e->rollout(n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                                 round_ids, resp_tokens_out, resp_logprobs_out, resp_len_out, stats_out, max_stats);
    if (n_rounds_out) *n_rounds_out = r;
  });
}

rp_status rp_generate(const rp_model_config* cfg, const rp_weights* weights, const rp_engine_limits* limits,
                      void* kv_ws, size_t kv_bytes, void* scratch_ws, size_t scratch_bytes, void* hip_stream,
                      int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens, const int64_t* prompt_offsets,
                      const int32_t* max_new_tokens, uint64_t seed, float temperature, int32_t schedule_mode,
                      const int32_t* round_ids, const rp_tail_params* tail, int32_t* resp_tokens_out,
                      float* resp_logprobs_out, int32_t* resp_len_out, int32_t* kept_out, rp_round_stats* stats_out,
                      int32_t max_stats, int32_t* n_rounds_out) {
  return guarded([&] {
    if (!cfg || !weights || !limits) throw rollpack::RpError(RP_ERR_INVALID_ARG, "null argument");
    rollpack::validate_config(*cfg);
    rollpack::validate_limits(*limits);
    std::unique_ptr<rollpack::Engine> e(new rollpack::Engine(*cfg, *weights, *limits, kv_ws, kv_bytes, scratch_ws,
                                                             scratch_bytes, static_cast<hipStream_t>(hip_stream)));
    const int32_t r = run_one_shot(*e, n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                                   schedule_mode, round_ids, tail, resp_tokens_out, resp_logprobs_out, resp_len_out,
                                   kept_out, stats_out, max_stats);
    if (n_rounds_out) *n_rounds_out = r;
  });
}

rp_status rp_generate_static(const rp_model_config* cfg, const rp_weights* weights, const rp_engine_limits* limits,
                             void* hip_stream, int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens,
                             const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed,
                             float temperature, int32_t schedule_mode, const int32_t* round_ids,
                             const rp_tail_params* tail, int32_t* resp_tokens_out, float* resp_logprobs_out,
                             int32_t* resp_len_out, int32_t* kept_out, rp_round_stats* stats_out, int32_t max_stats,
                             int32_t* n_rounds_out) {
  return guarded([&] {
    using rollpack::RpError;
    if (!cfg || !weights || !limits) throw RpError(RP_ERR_INVALID_ARG, "null argument");
    rollpack::validate_config(*cfg);
    rollpack::validate_limits(*limits);
    const size_t kv = rollpack::kv_pool_bytes(*cfg, limits->kv_pages);  // a multiple of 256
    const size_t sc = rollpack::plan_scratch(*cfg, *limits).total;
    if (kv + sc > rollpack::kStaticWorkspaceBytes)
      throw RpError(RP_ERR_CAPACITY, "rp_generate_static: these limits need " + std::to_string(kv + sc) +
                                         " bytes of KV pool and scratch; the library's static workspace holds " +
                                         std::to_string(rollpack::kStaticWorkspaceBytes));
    auto check = [](hipError_t e, const char* what) {
      if (e != hipSuccess) throw RpError(RP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
    };
    int dev = -1;
    check(hipGetDevice(&dev), "hipGetDevice");
    const hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    if (stream) {
      hipDevice_t sdev = -1;
      check(hipStreamGetDevice(stream, &sdev), "hipStreamGetDevice");
      if (sdev != dev) throw RpError(RP_ERR_INVALID_ARG, "rp_generate_static: the stream belongs to another device");
    }
    std::lock_guard<std::mutex> hold(rollpack::static_workspace_lock());
    void* base = nullptr;
    check(rollpack::static_workspace(dev, &base), "hipGetSymbolAddress");
    char* b = static_cast<char*>(base);
    rollpack::Engine e(*cfg, *weights, *limits, b, kv, b + kv, sc, stream, /*no_alloc=*/true);
    const int32_t r = run_one_shot(e, n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed, temperature,
                                   schedule_mode, round_ids, tail, resp_tokens_out, resp_logprobs_out, resp_len_out,
                                   kept_out, stats_out, max_stats);
    if (n_rounds_out) *n_rounds_out = r;
  });
}

rp_status rp_rollout_tail_batched(rp_engine* eng, int32_t n_prompts, int32_t r_spec, const int64_t* seq_ids,
                                  const int32_t* prompt_tokens, const int64_t* prompt_offsets,
                                  const int32_t* max_new_tokens, uint64_t seed, float temperature, int32_t P0,
                                  int32_t R0, float eta_p, float eta_r, int32_t* resp_tokens_out,
                                  float* resp_logprobs_out, int32_t* resp_len_out, int32_t* accept_round_out,
                                  int32_t* kept_out, rp_round_stats* stats_out, int32_t max_stats,
                                  int32_t* n_rounds_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    if (max_stats < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "max_stats must be >= 0");
    const int32_t r = e->rollout_tail_batched(n_prompts, r_spec, seq_ids, prompt_tokens, prompt_offsets,
                                              max_new_tokens, seed, temperature, P0, R0, eta_p, eta_r,
                                              resp_tokens_out, resp_logprobs_out, resp_len_out, accept_round_out,
                                              kept_out, stats_out, max_stats);
    if (n_rounds_out) *n_rounds_out = r;
  });
}

rp_status rp_get_logprobs(rp_engine* eng, int64_t seq_id, float* out, int32_t cap, int32_t* len_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    if (cap < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "cap must be >= 0");
    const int32_t k = e->get_logprobs(seq_id, out, cap);
    if (len_out) *len_out = k;
  });
}

rp_status rp_set_eos(rp_engine* eng, int32_t eos_token) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->set_eos(eos_token); });
}

rp_status rp_plan_tail_batching(int32_t n_prompts, int32_t r_spec, const int32_t* lens, int32_t P0, int32_t R0,
                                float eta_p, float eta_r, int32_t max_rounds, int32_t cap_launch, int32_t* round_kind_out,
                                int32_t* round_time_out, int32_t* launch_off_out, int32_t* launch_prompt_out,
                                int32_t* run_steps_out, int32_t* accept_round_out, int32_t* kept_out,
                                int32_t* n_rounds_out) {
  return guarded([&] {
    if (n_prompts < 0 || r_spec < 1 || (n_prompts > 0 && !lens) || !n_rounds_out || max_rounds < 0 ||
        cap_launch < 0)
      throw rollpack::RpError(RP_ERR_INVALID_ARG, "tail batching: bad arguments");
    for (int64_t i = 0; i < static_cast<int64_t>(n_prompts) * r_spec; ++i)
      if (lens[i] < 0) throw rollpack::RpError(RP_ERR_INVALID_ARG, "tail batching: negative length");
    const rollpack::TailBatchPlan plan = rollpack::plan_tail_batching(n_prompts, r_spec, lens, P0, R0, eta_p, eta_r);
    const int32_t nr = static_cast<int32_t>(plan.rounds.size());
    size_t launches = 0;
    for (const auto& r : plan.rounds) launches += r.launched.size();
    if (nr > max_rounds || launches > static_cast<size_t>(cap_launch))
      throw rollpack::RpError(RP_ERR_CAPACITY, "tail batching: output arrays too small");
    if (!round_kind_out || !round_time_out || !launch_off_out || !launch_prompt_out || !run_steps_out ||
        !accept_round_out || !kept_out)
      throw rollpack::RpError(RP_ERR_INVALID_ARG, "tail batching: null output array");
    size_t pos = 0;
    launch_off_out[0] = 0;
    for (int32_t k = 0; k < nr; ++k) {
      const auto& r = plan.rounds[k];
      round_kind_out[k] = r.kind;
      round_time_out[k] = r.time;
      for (size_t j = 0; j < r.launched.size(); ++j, ++pos) {
        launch_prompt_out[pos] = r.launched[j];
        for (int32_t q = 0; q < r_spec; ++q) run_steps_out[pos * r_spec + q] = r.run_steps[j * r_spec + q];
      }
      launch_off_out[k + 1] = static_cast<int32_t>(pos);
    }
    for (int32_t p = 0; p < n_prompts; ++p) accept_round_out[p] = plan.accept_round[p];
    for (size_t i = 0; i < plan.kept.size(); ++i) kept_out[i] = plan.kept[i];
    *n_rounds_out = nr;
  });
}

rp_status rp_set_kv_policy(rp_engine* eng, int32_t policy) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->set_kv_policy(policy); });
}

rp_status rp_kv_status(rp_engine* eng, int64_t* free_pages, int32_t* running, int32_t* waiting, int64_t* preemptions,
                       int64_t* recomputed_tokens) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    e->kv_status(free_pages, running, waiting, preemptions, recomputed_tokens);
  });
}

rp_status rp_step_trace_enable(rp_engine* eng, int32_t cap) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->step_trace_enable(cap); });
}

rp_status rp_step_trace_read(rp_engine* eng, rp_step_record* out, int32_t cap, int32_t* n_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    const int32_t n = e->step_trace_read(out, cap);
    if (n_out) *n_out = n;
  });
}

rp_status rp_profile_enable(rp_engine* eng, uint32_t class_mask) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->profile_enable(class_mask); });
}

rp_status rp_profile_every(rp_engine* eng, int32_t every) {
  return engine_call(eng, [&](rollpack::Engine* e) { e->profile_every(every); });
}

rp_status rp_profile_read(rp_engine* eng, rp_kernel_stats* out, int32_t cap, int32_t* n_out) {
  return engine_call(eng, [&](rollpack::Engine* e) {
    const int32_t n = e->profile_read(out, cap);
    if (n_out) *n_out = n;
  });
}

rp_status rp_stream_read_gbs(const void* dev_buf, size_t bytes, int32_t reps, void* hip_stream, double* gbs_out) {
  return guarded([&] {
    if (!dev_buf || bytes < (size_t{1} << 20) || reinterpret_cast<uintptr_t>(dev_buf) % 16 || reps < 1 || !gbs_out)
      throw rollpack::RpError(RP_ERR_INVALID_ARG, "stream read: need a 16-byte aligned buffer of >= 1 MiB, reps >= 1");
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    auto check = [](hipError_t e, const char* what) {
      if (e != hipSuccess) throw rollpack::RpError(RP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
    };
    hipEvent_t e0, e1;
    check(hipEventCreate(&e0), "hipEventCreate");
    check(hipEventCreate(&e1), "hipEventCreate");
    float best = 0.f;
    hipError_t err = rollpack::launch_stream_read(dev_buf, bytes, s);  // warm-up
    for (int32_t r = 0; r < reps && err == hipSuccess; ++r) {
      err = hipEventRecord(e0, s);
      if (err == hipSuccess) err = rollpack::launch_stream_read(dev_buf, bytes, s);
      if (err == hipSuccess) err = hipEventRecord(e1, s);
      if (err == hipSuccess) err = hipEventSynchronize(e1);
      float ms = 0.f;
      if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
      if (err == hipSuccess && (best == 0.f || ms < best)) best = ms;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    check(err, "stream read");
    *gbs_out = static_cast<double>(bytes / 16 * 16) / (best * 1e-3) / 1e9;
  });
}

const char* rp_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
