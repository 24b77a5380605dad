// Rollout engine: host-side state and step loop of the C ABI in rollpack.h.
#pragma once

#include <hip/hip_runtime.h>

#include <array>
#include <cstdint>
#include <deque>
#include <stdexcept>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/rollpack.h"
#include "kernels.hpp"
#include "kv_pool.hpp"

namespace rollpack {

struct RpError : std::runtime_error {
  rp_status status;
  RpError(rp_status s, const std::string& m) : std::runtime_error(m), status(s) {}
};

// Byte offsets of every buffer carved from the caller's scratch workspace.
struct ScratchPlan {
  size_t x, h, part, q, attn, act, hsel, logits, att_o, att_ml, rope_cos, rope_sin, page_table,
      tokens_cur, hist, logp, resp, resp_logp, slot_seed, slot_id, slot_temp, meta, cand_val, cand_idx, cand_m,
      cand_s;
  size_t total;
  size_t part_elems;
  int32_t split_cap;   // decode attention work-item capacity (splits)
  int32_t max_pages;   // page-table row width
  int32_t meta_ints;
};

ScratchPlan plan_scratch(const rp_model_config& c, const rp_engine_limits& l);
// Bytes of the packed copy of the decode-GEMM weights (every projection and
// the LM head), each tensor 256-byte aligned; 0 for the fp32 model.
size_t packed_weights_bytes(const rp_model_config& c);
size_t kv_pool_bytes(const rp_model_config& c, int64_t pages);
void validate_config(const rp_model_config& c);
void validate_limits(const rp_engine_limits& l);

struct Seq {
  int64_t id = -1;
  int32_t prompt_len = 0;
  int32_t max_new = 0;
  int32_t n_gen = 0;     // tokens sampled so far
  uint64_t seed = 0;
  float temp = 0.f;
  bool live = false;
  bool finished = false;
  int64_t arrival = 0;   // admission order of the sequence's first prefill
  bool stopped = false;  // ended by the end-of-sequence token
  int64_t last_step = -1;  // sample step that produced its latest token
  std::vector<int32_t> pages;
  std::vector<int32_t> prompt;  // kept under on-demand pages, for a recompute after preemption
};

// A sequence preempted under KV pressure: its pages and slot are gone, its
// tokens wait on the host until it is recomputed.
struct Waiting {
  int64_t id;
  int32_t prompt_len, max_new, n_gen;
  uint64_t seed;
  float temp;
  int64_t arrival;
  std::vector<int32_t> tokens;  // prompt followed by the n_gen generated tokens
  std::vector<float> logp;      // log-probabilities of the n_gen generated tokens
};

// One sequence to (re)admit: prefill `ntok` tokens at positions 0..ntok-1 and
// sample the token at position ntok into history entry n_gen0.
struct AdmitSeq {
  int64_t id;
  const int32_t* toks;
  int32_t ntok, prompt_len, max_new, n_gen0;
  uint64_t seed;
  float temp;
  int64_t arrival;
};

// A contiguous run of one sequence's tokens inside a prefill chunk.
struct PrefillPiece {
  int32_t slot;
  const int32_t* toks;
  int32_t pos0, ntok, hist0;
  int32_t seq;  // index of the sequence in its admit call; -1 unless the piece ends it
};

// Per-sequence inputs of one rollout call (prompt CSR per sequence).
struct SeqArrays {
  float* logp_out;          // host, nullable: log-probabilities laid out like the tokens
  const int64_t* ids;
  const int32_t* toks;
  const int64_t* offs;
  const int32_t* max_new;
  const int64_t* resp_off;  // [n + 1] token offsets into the response buffer
  uint64_t seed;
  float temp;
};

// Race-to-completion state of a short round (section 3): members are the
// responses of n_prompts prompts; the first `keep` prompts with R0 finished
// responses are accepted, each keeping its first R0 finished responses.
struct Race {
  std::vector<int32_t> prompt;     // [members] prompt (0..n_prompts-1) of each member
  int32_t n_prompts = 0, R0 = 1, keep = 1;
  std::vector<uint8_t> accepted;   // [n_prompts] out
  std::vector<uint8_t> kept;       // [members] out
};

class Engine {
 public:
  // no_alloc: the engine then makes no allocating HIP call (no pinned host
  // memory, no events): staging buffers are ordinary host memory, waits on a
  // copy or a step become stream synchronisations, and the round statistics
  // are timed with the host clock after the stream has drained.  End-of-
  // sequence checks, the step trace and profiling are refused in that mode.
  Engine(const rp_model_config& cfg, const rp_weights& w, const rp_engine_limits& lim, void* kv_ws,
         size_t kv_bytes, void* scratch_ws, size_t scratch_bytes, hipStream_t stream, bool no_alloc = false);
  ~Engine();

  void prefill(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
               const int32_t* max_new, uint64_t seed, float temp, float* logits_out, int32_t* first_out);
  int32_t decode_step(const int32_t* forced, float* logits_out, int64_t* row_ids_out);
  int32_t free_finished(int64_t* ids_out, int32_t cap);
  void abort(int32_t n, const int64_t* ids);
  int32_t get_tokens(int64_t id, int32_t* out, int32_t cap);
  int32_t get_logprobs(int64_t id, float* out, int32_t cap);
  void set_eos(int32_t token);
  int32_t rollout(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
                  const int32_t* max_new, uint64_t seed, float temp, const int32_t* round_ids,
                  int32_t* resp_out, float* logp_out, int32_t* len_out, rp_round_stats* stats,
                  int32_t max_stats);
  int32_t rollout_tail_batched(int32_t n_prompts, int32_t r_spec, const int64_t* ids, const int32_t* ptoks,
                               const int64_t* poffs, const int32_t* max_new, uint64_t seed, float temp,
                               int32_t P0, int32_t R0, float eta_p, float eta_r, int32_t* resp_out,
                               float* logp_out, int32_t* gen_out,
                               int32_t* accept_round_out, int32_t* kept_out, rp_round_stats* stats,
                               int32_t max_stats);

  // Packs every projection and the LM head into the caller's workspace (on the
  // engine's stream) and points the decode GEMMs at the packed copy from then
  // on; nullptr goes back to the row-major weights.
  void set_packed_weights(void* ws, size_t bytes);
  void profile_enable(uint32_t mask);
  void profile_every(int32_t every);
  int32_t profile_read(rp_kernel_stats* out, int32_t cap);
  void set_kv_policy(int32_t policy);
  void step_trace_enable(int32_t cap);
  int32_t step_trace_read(rp_step_record* out, int32_t cap);
  void kv_status(int64_t* free_pages, int32_t* running, int32_t* waiting, int64_t* preemptions,
                 int64_t* recomputed_tokens) const;

  bool broken() const { return broken_; }
  void mark_broken() { broken_ = true; }
  int32_t live_count() const { return static_cast<int32_t>(order_.size() + waiting_.size()); }

 private:
  struct Staging {
    void* host = nullptr;
    hipEvent_t ev = nullptr;
    bool pending = false;
  };
  // Host buffer of `bytes` for staging copies: pinned normally, ordinary
  // memory (owned by host_store_) without allocations.
  void* host_buffer(size_t bytes);
  // Stream-ordered completion points: a HIP event, or (ev == nullptr, the
  // no-allocation mode) a stream synchronisation when waited on.
  void fence_record(hipEvent_t ev);
  void fence_wait(hipEvent_t ev);
  // Time marks of run_round: mark k is recorded in stream order; mark_ms(a, b)
  // is the time between two recorded marks.
  void mark(size_t k);
  double mark_ms(size_t a, size_t b);

  void forward(int M, bool is_prefill, int n_seq_prefill, int total_items, int total_splits, int tps);
  int32_t* stage_meta(size_t ints);
  void upload_meta(const int32_t* host, size_t ints);
  void upload_slot_tables();
  void check_admission(int32_t n, const int64_t* ids, const int64_t* offs, const int32_t* toks,
                       const int32_t* max_new, float temp) const;
  // Pages a sequence takes at admission: its whole length when reserving,
  // else the tokens to prefill (on demand).
  int64_t admit_pages(int64_t prompt_len, int64_t max_new, int64_t ntok) const;
  std::vector<int32_t> admit_seqs(const std::vector<AdmitSeq>& a, const std::vector<const Waiting*>& restore,
                                  float* logits_out);
  void run_prefill_chunk(const std::vector<PrefillPiece>& pcs, float* logits_out);
  // On-demand pages: resume waiting sequences that fit, then give every
  // running row a page for its next position, preempting the latest arrivals
  // when the pool runs dry.  Returns the slots resumed (they advanced already).
  std::vector<int32_t> schedule_pages();
  void preempt(const std::vector<int32_t>& victims);
  // End-of-sequence checks: after each sampler launch the sampled tokens are
  // copied to pinned memory; they are read two sample steps later (or when
  // the caller needs final state), so the host never waits on the step it
  // just launched.  A sequence that sampled the token is cut after it.
  void note_samples(const std::vector<std::array<int64_t, 3>>& rows);  // (slot, id, history index)
  void apply_eos(int64_t upto);
  void drain_eos() { apply_eos(sample_step_ - 1); }
  bool settled(const Seq& q) const { return eos_token_ < 0 || q.last_step <= eos_applied_; }
  bool known_id(int64_t id) const;
  Waiting* find_waiting(int64_t id);
  void release(int32_t slot);
  void validate_seqs(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
                     const int32_t* max_new, float temp, std::vector<int64_t>& resp_off) const;
  hipEvent_t event_at(size_t k);
  // Runs one round over `members` (indices into a) to its end: admits them
  // (in waves when the pool is short, all at once for a race), decodes, and
  // copies each departing sequence's tokens to resp_out.  With a race the
  // round ends when race->keep prompts are accepted and the rest are aborted.
  void run_round(const std::vector<int32_t>& members, const SeqArrays& a, int32_t* resp_out, int32_t* gen_out,
                 Race* race, rp_round_stats* st);
  template <typename T> T* sp(size_t off) const { return reinterpret_cast<T*>(scratch_ + off); }

  rp_model_config cfg_;
  rp_engine_limits lim_;
  std::vector<rp_layer_weights> layers_;
  rp_weights w_;
  std::vector<rp_layer_weights> packed_layers_;  // empty: no packed copy
  const void* packed_lm_ = nullptr;
  hipStream_t stream_;
  bool bf16_;
  size_t esz_;
  int nqkv_;
  ScratchPlan plan_;
  char* kv_;
  char* scratch_;
  size_t layer_kv_bytes_;  // bytes of one layer's K (or V) pool
  PagePool pool_;
  std::vector<Seq> slots_;
  std::vector<int32_t> free_slots_;
  std::vector<int32_t> order_;  // live slots in admission order
  std::vector<Waiting> waiting_;  // preempted sequences, by arrival
  int32_t kv_policy_ = RP_KV_RESERVE;
  int64_t arrival_next_ = 0;
  int64_t n_preempt_ = 0, n_recompute_tok_ = 0;
  struct EosCheck {
    int64_t step;
    hipEvent_t ev;
    int32_t* host;  // pinned copy of tokens_cur
    std::vector<std::array<int64_t, 3>> rows;
  };
  // per-step trace (rp_step_trace_*)
  struct TraceRec {
    rp_step_record rec;
    hipEvent_t e0, e1;
    hipEvent_t round_start;  // recorded at its round's start (nullptr outside a rollout call)
  };
  hipEvent_t trace_event();
  hipEvent_t cur_round_ev_ = nullptr;          // round-start event of the running round (trace on)
  std::vector<hipEvent_t> trace_round_evs_;    // round-start events referenced by trace_
  std::vector<TraceRec> trace_;
  std::vector<hipEvent_t> trace_pool_;
  int32_t trace_cap_ = 0;
  int32_t cur_round_ = -1;
  TraceRec* trace_begin(int kind, int rows, int64_t sum_ctx);
  void trace_end(TraceRec* t);
  int32_t eos_token_ = -1;
  int64_t sample_step_ = 0;   // sampler launches so far
  int64_t eos_applied_ = -1;  // every sample step up to this one has been checked
  std::deque<EosCheck> eos_pending_;
  std::vector<EosCheck> eos_free_;
  std::unordered_map<int64_t, int32_t> id2slot_;
  // pinned host mirrors
  int32_t* h_page_table_ = nullptr;
  uint64_t* h_slot_seed_ = nullptr;
  uint64_t* h_slot_id_ = nullptr;
  float* h_slot_temp_ = nullptr;
  hipEvent_t ev_tables_ = nullptr;
  bool tables_pending_ = false;
  std::vector<Staging> ring_;
  size_t ring_next_ = 0;
  size_t ring_bytes_ = 0;
  bool broken_ = false;
  bool no_alloc_ = false;
  std::vector<std::vector<char>> host_store_;  // host buffers of the no-allocation mode
  std::vector<double> host_marks_;             // mark times (ms, host clock) of the no-allocation mode
  // device metadata views (set by the last stage/upload)
  const int32_t* d_meta_ = nullptr;
  // metadata pointers used by forward()
  const int32_t *m_in_tok_ = nullptr, *m_slot_ = nullptr, *m_pos_ = nullptr, *m_hist_ = nullptr,
                *m_ctx_ = nullptr, *m_split_off_ = nullptr, *m_seq_slot_ = nullptr,
                *m_seq_row0_ = nullptr, *m_seq_pos0_ = nullptr, *m_seq_ntok_ = nullptr,
                *m_item_off_ = nullptr, *m_last_row_ = nullptr, *m_gen_pos_ = nullptr,
                *m_gen_hist_ = nullptr, *m_gen_slot_ = nullptr, *m_split_desc_ = nullptr;
  std::vector<int32_t> ctx_scratch_;  // decode_step: per-row context lengths
  int max_row_splits_ = 0;            // decode_step: most attention splits of any row
  std::vector<hipEvent_t> events_;

  // per-kernel-class profiling (rp_profile_*)
  struct ProfRec {
    int cls, phase;
    hipEvent_t e0, e1;
    double bytes, flops;
  };
  struct ProfAcc {
    int64_t launches = 0;
    double ms = 0, bytes = 0, flops = 0;
  };
  template <typename F> void launch_timed(int cls, double bytes, double flops, F&& launch);
  void prof_harvest();
  uint32_t prof_mask_ = 0;
  int32_t prof_every_ = 1;                   // time one launch in prof_every_ per class and phase
  int64_t prof_seen_[RP_K_COUNT][2] = {};    // selected launches since rp_profile_every
  int phase_ = 0;             // 0 prefill, 1 decode
  double sum_ctx_ = 0;        // attended KV tokens of the current forward (decode)
  double sum_ctx_sq_ = 0;     // sum of squared prompt lengths (prefill attention)
  std::vector<ProfRec> prof_pending_;
  std::vector<hipEvent_t> prof_pool_;
  ProfAcc prof_acc_[RP_K_COUNT][2];
};

}  // namespace rollpack

struct rp_engine {
  rollpack::Engine* impl;
};
