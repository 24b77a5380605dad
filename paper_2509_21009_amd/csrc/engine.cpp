// Rollout engine: admission with paged KV reservation, chunked prefill, the
// decode step loop and round-by-round rollout with per-round measurements.
//
// Rollout (paper section 2.1) generates R0 responses for each of P0 prompts;
// the batch shrinks as responses finish (section 2.2), so finished
// sequences give their KV pages back and later steps run with fewer rows.
// All device work is enqueued on one stream; per-step metadata is O(rows)
// integers copied from pinned staging buffers.
#include "engine.hpp"
#include "tail_batch.hpp"

#include <algorithm>
#include <chrono>
#include <array>
#include <cmath>
#include <cstring>
#include <deque>
#include <map>
#include <numeric>

namespace rollpack {

namespace {

constexpr int kMaxGemmSplits = 16;

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) throw RpError(RP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}
#define HIP_TRY(expr) hip_check((expr), #expr)

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

int decode_split_target(const rp_model_config& c) { return std::max(1, 2048 / c.n_kv_heads); }

}  // namespace

void validate_config(const rp_model_config& c) {
  auto bad = [](const std::string& m) { throw RpError(RP_ERR_INVALID_ARG, m); };
  if (c.n_layers < 1 || c.hidden < 1 || c.n_q_heads < 1 || c.n_kv_heads < 1 || c.intermediate < 1 ||
      c.vocab < 2)
    bad("model config: sizes must be positive");
  if (c.n_q_heads % c.n_kv_heads != 0) bad("model config: n_q_heads must be a multiple of n_kv_heads");
  if (c.head_dim != 64 && c.head_dim != 128) bad("model config: head_dim must be 64 or 128");
  if (c.dtype != RP_DTYPE_F32 && c.dtype != RP_DTYPE_BF16) bad("model config: unknown dtype");
  if (!(c.rms_eps > 0.f) || !(c.rope_theta > 1.f)) bad("model config: rms_eps > 0 and rope_theta > 1 required");
  if (c.dtype == RP_DTYPE_BF16) {
    const int nqkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
    if (c.n_q_heads / c.n_kv_heads > 16) bad("bf16 path: at most 16 query heads per KV head");
    if (c.hidden % 128 || c.intermediate % 128 || (c.n_q_heads * c.head_dim) % 128 || nqkv % 128 ||
        c.vocab % 128)
      bad("bf16 path: hidden, intermediate, n_q*head_dim, qkv width and vocab must be multiples of 128");
  }
}

void validate_limits(const rp_engine_limits& l) {
  if (l.page_tokens != kPageTokens) throw RpError(RP_ERR_INVALID_ARG, "limits: page_tokens must be 64");
  if (l.max_seqs < 1 || l.max_prefill_tokens < 1 || l.max_context < 2 || l.max_context > 65536 ||
      l.kv_pages < 1 || l.kv_pages > (int64_t{1} << 24) || l.max_seqs > (1 << 20) || l.max_prefill_tokens > (1 << 22))
    throw RpError(RP_ERR_INVALID_ARG,
                  "limits: 1 <= max_seqs <= 2^20, 1 <= max_prefill_tokens <= 2^22, 1 <= kv_pages <= 2^24, "
                  "2 <= max_context <= 65536");
}

size_t packed_weights_bytes(const rp_model_config& c) {
  if (c.dtype != RP_DTYPE_BF16) return 0;
  const size_t H = c.hidden, I = c.intermediate, hd = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads;
  const size_t layer = align256(nq * hd * H * 2) + 2 * align256(nkv * hd * H * 2) + align256(H * nq * hd * 2) +
                       2 * align256(I * H * 2) + align256(H * I * 2);
  return layer * c.n_layers + align256(static_cast<size_t>(c.vocab) * H * 2);
}

size_t kv_pool_bytes(const rp_model_config& c, int64_t pages) {
  const size_t esz = c.dtype == RP_DTYPE_BF16 ? 2 : 4;
  return align256(static_cast<size_t>(pages) * c.n_layers * 2 * c.n_kv_heads * kPageTokens * c.head_dim * esz);
}

ScratchPlan plan_scratch(const rp_model_config& c, const rp_engine_limits& l) {
  ScratchPlan p{};
  const size_t esz = c.dtype == RP_DTYPE_BF16 ? 2 : 4;
  const size_t H = c.hidden, I = c.intermediate, V = c.vocab, hd = c.head_dim;
  const size_t nq = c.n_q_heads, nkv = c.n_kv_heads;
  const size_t nqkv = (nq + 2 * nkv) * hd;
  const size_t mmax = std::max<size_t>(l.max_prefill_tokens, l.max_seqs);
  const size_t nmax = std::max(nqkv, H);
  p.max_pages = static_cast<int32_t>((l.max_context + kPageTokens - 1) / kPageTokens);
  p.split_cap = c.dtype == RP_DTYPE_BF16 ? decode_split_target(c) + l.max_seqs : 0;
  p.part_elems = std::max(static_cast<size_t>(l.max_prefill_tokens) * nmax,
                          static_cast<size_t>(kMaxGemmSplits) * l.max_seqs * nmax);
  const size_t T = l.max_prefill_tokens, S = l.max_seqs;
  // decode: 7 ints per row + 1, padded to 16 bytes, then 4 per split; prefill: 3 per token + 8 per row + 1
  p.meta_ints = static_cast<int32_t>(std::max(7 * S + 4 + 4 * static_cast<size_t>(p.split_cap), 3 * T + 8 * S + 1));
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  p.x = take(mmax * H * 4);
  p.h = take(mmax * H * esz);
  p.part = take(p.part_elems * 4);
  p.q = take(mmax * nq * hd * esz);
  p.attn = take(mmax * nq * hd * esz);
  p.act = take(mmax * I * esz);
  p.hsel = take(S * H * esz);
  p.logits = take(S * V * 4);
  p.att_o = take(static_cast<size_t>(p.split_cap) * nkv * 16 * hd * 4);
  p.att_ml = take(static_cast<size_t>(p.split_cap) * nkv * 32 * 4);
  p.rope_cos = take(static_cast<size_t>(l.max_context) * (hd / 2) * 4);
  p.rope_sin = take(static_cast<size_t>(l.max_context) * (hd / 2) * 4);
  p.page_table = take(S * p.max_pages * 4);
  p.tokens_cur = take(S * 4);
  p.hist = take(S * static_cast<size_t>(l.max_context) * 4);
  p.logp = take(S * static_cast<size_t>(l.max_context) * 4);
  p.resp = take(S * static_cast<size_t>(l.max_context) * 4);
  p.resp_logp = take(S * static_cast<size_t>(l.max_context) * 4);
  p.slot_seed = take(S * 8);
  p.slot_id = take(S * 8);
  p.slot_temp = take(S * 4);
  p.meta = take(static_cast<size_t>(p.meta_ints) * 4);
  p.cand_val = take(S * static_cast<size_t>(sample_chunks(c.vocab)) * 4);
  p.cand_idx = take(S * static_cast<size_t>(sample_chunks(c.vocab)) * 4);
  p.cand_m = take(S * static_cast<size_t>(sample_chunks(c.vocab)) * 4);
  p.cand_s = take(S * static_cast<size_t>(sample_chunks(c.vocab)) * 4);
  p.total = off;
  return p;
}

Engine::Engine(const rp_model_config& cfg, const rp_weights& w, const rp_engine_limits& lim, void* kv_ws,
               size_t kv_bytes, void* scratch_ws, size_t scratch_bytes, hipStream_t stream, bool no_alloc)
    : cfg_(cfg), lim_(lim), stream_(stream), pool_(lim.kv_pages) {
  no_alloc_ = no_alloc;
  validate_config(cfg);
  validate_limits(lim);
  bf16_ = cfg.dtype == RP_DTYPE_BF16;
  esz_ = bf16_ ? 2 : 4;
  nqkv_ = (cfg.n_q_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  plan_ = plan_scratch(cfg, lim);
  if (!kv_ws || !scratch_ws || (reinterpret_cast<uintptr_t>(kv_ws) & 255) ||
      (reinterpret_cast<uintptr_t>(scratch_ws) & 255))
    throw RpError(RP_ERR_INVALID_ARG, "workspaces must be non-null and 256-byte aligned");
  if (kv_bytes < kv_pool_bytes(cfg, lim.kv_pages) || scratch_bytes < plan_.total)
    throw RpError(RP_ERR_INVALID_ARG, "workspace smaller than rp_workspace_size");
  if (!w.embed || !w.final_norm || !w.layers || (!cfg.tied_embeddings && !w.lm_head))
    throw RpError(RP_ERR_INVALID_ARG, "weights: embed, final_norm, layers (and lm_head unless tied) required");
  layers_.assign(w.layers, w.layers + cfg.n_layers);
  for (const auto& L : layers_) {
    if (!L.attn_norm || !L.wq || !L.bq || !L.wk || !L.bk || !L.wv || !L.bv || !L.wo || !L.mlp_norm ||
        !L.w_gate || !L.w_up || !L.w_down)
      throw RpError(RP_ERR_INVALID_ARG, "weights: a layer tensor pointer is null");
  }
  w_ = w;
  w_.layers = layers_.data();
  if (cfg.tied_embeddings) w_.lm_head = w.embed;
  kv_ = static_cast<char*>(kv_ws);
  scratch_ = static_cast<char*>(scratch_ws);
  layer_kv_bytes_ = static_cast<size_t>(lim.kv_pages) * cfg.n_kv_heads * kPageTokens * cfg.head_dim * esz_;

  slots_.resize(lim.max_seqs);
  for (int32_t s = lim.max_seqs - 1; s >= 0; --s) free_slots_.push_back(s);

  const size_t pt_bytes = static_cast<size_t>(lim.max_seqs) * plan_.max_pages * 4;
  h_page_table_ = static_cast<int32_t*>(host_buffer(pt_bytes));
  h_slot_seed_ = static_cast<uint64_t*>(host_buffer(lim.max_seqs * 8));
  h_slot_id_ = static_cast<uint64_t*>(host_buffer(lim.max_seqs * 8));
  h_slot_temp_ = static_cast<float*>(host_buffer(lim.max_seqs * 4));
  std::memset(h_page_table_, 0, pt_bytes);
  std::memset(h_slot_seed_, 0, lim.max_seqs * 8);
  std::memset(h_slot_id_, 0, lim.max_seqs * 8);
  std::memset(h_slot_temp_, 0, lim.max_seqs * 4);
  if (!no_alloc_) HIP_TRY(hipEventCreateWithFlags(&ev_tables_, hipEventDisableTiming));
  ring_bytes_ = static_cast<size_t>(plan_.meta_ints) * 4;
  ring_.resize(8);
  for (auto& r : ring_) {
    r.host = host_buffer(ring_bytes_);
    if (!no_alloc_) HIP_TRY(hipEventCreateWithFlags(&r.ev, hipEventDisableTiming));
  }

  // RoPE table: angle = pos * theta^(-2d/hd), computed in double, stored fp32.
  const int half = cfg.head_dim / 2;
  std::vector<float> cs(static_cast<size_t>(lim.max_context) * half), sn(cs.size());
  for (int pos = 0; pos < lim.max_context; ++pos)
    for (int d = 0; d < half; ++d) {
      const double inv = std::pow(static_cast<double>(cfg.rope_theta), -2.0 * d / cfg.head_dim);
      const double ang = static_cast<double>(pos) * inv;
      cs[static_cast<size_t>(pos) * half + d] = static_cast<float>(std::cos(ang));
      sn[static_cast<size_t>(pos) * half + d] = static_cast<float>(std::sin(ang));
    }
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, stream_));
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, stream_));
  // Zero the KV pool once: masked-out tail tokens of a page are multiplied by
  // zero probabilities, which must not meet NaN bit patterns.
  HIP_TRY(hipMemsetAsync(kv_, 0, kv_pool_bytes(cfg, lim.kv_pages), stream_));
  HIP_TRY(hipMemsetAsync(scratch_ + plan_.page_table, 0, pt_bytes, stream_));
  HIP_TRY(hipMemsetAsync(scratch_ + plan_.tokens_cur, 0, lim.max_seqs * 4, stream_));
  HIP_TRY(hipStreamSynchronize(stream_));
}

Engine::~Engine() {
  (void)hipStreamSynchronize(stream_);
  for (auto& r : ring_) {
    if (r.host && !no_alloc_) (void)hipHostFree(r.host);
    if (r.ev) (void)hipEventDestroy(r.ev);
  }
  for (auto e : events_) (void)hipEventDestroy(e);
  if (ev_tables_) (void)hipEventDestroy(ev_tables_);
  if (!no_alloc_) {
    if (h_page_table_) (void)hipHostFree(h_page_table_);
    if (h_slot_seed_) (void)hipHostFree(h_slot_seed_);
    if (h_slot_id_) (void)hipHostFree(h_slot_id_);
    if (h_slot_temp_) (void)hipHostFree(h_slot_temp_);
  }
  for (auto& c : eos_free_) {
    (void)hipHostFree(c.host);
    (void)hipEventDestroy(c.ev);
  }
  for (auto& c : eos_pending_) {
    (void)hipHostFree(c.host);
    (void)hipEventDestroy(c.ev);
  }
  for (auto& t : trace_) {
    (void)hipEventDestroy(t.e0);
    (void)hipEventDestroy(t.e1);
  }
  for (auto e : trace_round_evs_) (void)hipEventDestroy(e);
  for (auto e : trace_pool_) (void)hipEventDestroy(e);
}

void* Engine::host_buffer(size_t bytes) {
  if (no_alloc_) {
    host_store_.emplace_back(std::max<size_t>(bytes, 16));
    return host_store_.back().data();
  }
  void* p = nullptr;
  HIP_TRY(hipHostMalloc(&p, bytes, hipHostMallocDefault));
  return p;
}

void Engine::fence_record(hipEvent_t ev) {
  if (ev) HIP_TRY(hipEventRecord(ev, stream_));
}

void Engine::fence_wait(hipEvent_t ev) {
  if (ev)
    HIP_TRY(hipEventSynchronize(ev));
  else
    HIP_TRY(hipStreamSynchronize(stream_));
}

void Engine::mark(size_t k) {
  if (!no_alloc_) {
    HIP_TRY(hipEventRecord(event_at(k), stream_));
    return;
  }
  HIP_TRY(hipStreamSynchronize(stream_));
  if (host_marks_.size() <= k) host_marks_.resize(k + 1);
  host_marks_[k] = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

double Engine::mark_ms(size_t a, size_t b) {
  if (no_alloc_) return host_marks_[b] - host_marks_[a];
  float ms = 0.f;
  HIP_TRY(hipEventElapsedTime(&ms, events_[a], events_[b]));
  return ms;
}

hipEvent_t Engine::trace_event() {
  hipEvent_t e;
  if (!trace_pool_.empty()) {
    e = trace_pool_.back();
    trace_pool_.pop_back();
  } else {
    HIP_TRY(hipEventCreate(&e));
  }
  return e;
}

Engine::TraceRec* Engine::trace_begin(int kind, int rows, int64_t sum_ctx) {
  if (static_cast<int32_t>(trace_.size()) >= trace_cap_) return nullptr;
  TraceRec t{rp_step_record{kind, cur_round_, rows, 0, sum_ctx, 0.0, -1.0}, trace_event(), trace_event(),
             cur_round_ev_};
  HIP_TRY(hipEventRecord(t.e0, stream_));
  trace_.push_back(t);
  return &trace_.back();
}

void Engine::trace_end(TraceRec* t) {
  if (t) HIP_TRY(hipEventRecord(t->e1, stream_));
}

void Engine::step_trace_enable(int32_t cap) {
  if (cap < 0) throw RpError(RP_ERR_INVALID_ARG, "trace capacity must be >= 0");
  if (no_alloc_ && cap > 0) throw RpError(RP_ERR_BAD_STATE, "no step trace without allocations");
  HIP_TRY(hipStreamSynchronize(stream_));
  for (auto& t : trace_) {
    trace_pool_.push_back(t.e0);
    trace_pool_.push_back(t.e1);
  }
  trace_.clear();
  for (auto e : trace_round_evs_) trace_pool_.push_back(e);
  trace_round_evs_.clear();
  trace_.reserve(static_cast<size_t>(cap));  // pointers handed out by trace_begin stay valid
  trace_cap_ = cap;
}

int32_t Engine::step_trace_read(rp_step_record* out, int32_t cap) {
  if (cap < 0 || (cap > 0 && !out)) throw RpError(RP_ERR_INVALID_ARG, "step_trace_read: bad output");
  HIP_TRY(hipStreamSynchronize(stream_));
  const int32_t n = std::min<int32_t>(cap, static_cast<int32_t>(trace_.size()));
  for (int32_t i = 0; i < n; ++i) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, trace_[i].e0, trace_[i].e1));
    out[i] = trace_[i].rec;
    out[i].ms = ms;
    if (trace_[i].round_start) {
      HIP_TRY(hipEventElapsedTime(&ms, trace_[i].round_start, trace_[i].e1));
      out[i].end_ms = ms;
    }
  }
  for (auto& t : trace_) {
    trace_pool_.push_back(t.e0);
    trace_pool_.push_back(t.e1);
  }
  trace_.clear();
  // a running round keeps its start event for the steps still to come
  for (auto e : trace_round_evs_)
    if (e != cur_round_ev_) trace_pool_.push_back(e);
  trace_round_evs_.clear();
  if (cur_round_ev_) trace_round_evs_.push_back(cur_round_ev_);
  return n;
}

void Engine::set_eos(int32_t token) {
  if (token < -1 || token >= cfg_.vocab) throw RpError(RP_ERR_INVALID_ARG, "end-of-sequence token out of range");
  if (live_count() != 0) throw RpError(RP_ERR_BAD_STATE, "the end-of-sequence token changes only with no live sequences");
  if (no_alloc_ && token >= 0) throw RpError(RP_ERR_BAD_STATE, "no end-of-sequence checks without allocations");
  eos_token_ = token;
}

void Engine::note_samples(const std::vector<std::array<int64_t, 3>>& rows) {
  const int64_t step = sample_step_++;
  for (const auto& r : rows) slots_[r[0]].last_step = step;
  if (eos_token_ < 0 || rows.empty()) return;
  EosCheck c;
  if (!eos_free_.empty()) {
    c = std::move(eos_free_.back());
    eos_free_.pop_back();
  } else {
    HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&c.host), static_cast<size_t>(lim_.max_seqs) * 4,
                          hipHostMallocDefault));
    HIP_TRY(hipEventCreateWithFlags(&c.ev, hipEventDisableTiming));
  }
  c.step = step;
  c.rows = rows;
  HIP_TRY(hipMemcpyAsync(c.host, scratch_ + plan_.tokens_cur, static_cast<size_t>(lim_.max_seqs) * 4,
                         hipMemcpyDeviceToHost, stream_));
  HIP_TRY(hipEventRecord(c.ev, stream_));
  eos_pending_.push_back(std::move(c));
}

void Engine::apply_eos(int64_t upto) {
  while (!eos_pending_.empty() && eos_pending_.front().step <= upto) {
    EosCheck& c = eos_pending_.front();
    HIP_TRY(hipEventSynchronize(c.ev));
    for (const auto& r : c.rows) {
      const int32_t slot = static_cast<int32_t>(r[0]);
      Seq& q = slots_[slot];
      if (!q.live || q.id != r[1] || q.stopped || c.host[slot] != eos_token_) continue;
      q.stopped = true;
      q.finished = true;
      q.n_gen = std::min<int32_t>(q.n_gen, static_cast<int32_t>(r[2]) + 1);
    }
    eos_applied_ = c.step;
    eos_free_.push_back(std::move(c));
    eos_pending_.pop_front();
  }
  if (eos_pending_.empty()) eos_applied_ = sample_step_ - 1;
}

int32_t* Engine::stage_meta(size_t ints) {
  if (ints * 4 > ring_bytes_) throw RpError(RP_ERR_CAPACITY, "step metadata exceeds the staging capacity");
  Staging& st = ring_[ring_next_];
  if (st.pending) {
    fence_wait(st.ev);
    st.pending = false;
  }
  return static_cast<int32_t*>(st.host);
}

void Engine::upload_meta(const int32_t* host, size_t ints) {
  Staging& st = ring_[ring_next_];
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.meta, host, ints * 4, hipMemcpyHostToDevice, stream_));
  fence_record(st.ev);
  st.pending = true;
  ring_next_ = (ring_next_ + 1) % ring_.size();
  d_meta_ = sp<int32_t>(plan_.meta);
}

void Engine::upload_slot_tables() {
  const size_t pt_bytes = static_cast<size_t>(lim_.max_seqs) * plan_.max_pages * 4;
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.page_table, h_page_table_, pt_bytes, hipMemcpyHostToDevice, stream_));
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.slot_seed, h_slot_seed_, lim_.max_seqs * 8, hipMemcpyHostToDevice, stream_));
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.slot_id, h_slot_id_, lim_.max_seqs * 8, hipMemcpyHostToDevice, stream_));
  HIP_TRY(hipMemcpyAsync(scratch_ + plan_.slot_temp, h_slot_temp_, lim_.max_seqs * 4, hipMemcpyHostToDevice, stream_));
  fence_record(ev_tables_);
  tables_pending_ = true;
}

void Engine::check_admission(int32_t n, const int64_t* ids, const int64_t* offs, const int32_t* toks,
                             const int32_t* max_new, float temp) const {
  if (n < 1 || !ids || !offs || !toks || !max_new) throw RpError(RP_ERR_INVALID_ARG, "prefill: null array or n < 1");
  if (!(temp >= 0.f) || std::isinf(temp)) throw RpError(RP_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  if (offs[0] != 0) throw RpError(RP_ERR_INVALID_ARG, "prompt_offsets[0] must be 0");
  if (n > static_cast<int32_t>(free_slots_.size()))
    throw RpError(RP_ERR_CAPACITY, "more sequences than free slots (max_seqs)");
  std::unordered_map<int64_t, int> seen;
  int64_t pages = 0;
  for (int32_t i = 0; i < n; ++i) {
    const int64_t p = offs[i + 1] - offs[i];
    if (p < 1) throw RpError(RP_ERR_INVALID_ARG, "every prompt needs at least one token");
    if (max_new[i] < 1) throw RpError(RP_ERR_INVALID_ARG, "max_new_tokens must be >= 1");
    if (p + max_new[i] - 1 > lim_.max_context) throw RpError(RP_ERR_CAPACITY, "prompt + max_new_tokens - 1 exceeds max_context");
    if (known_id(ids[i]) || seen.count(ids[i])) throw RpError(RP_ERR_DUPLICATE_ID, "sequence id already live");
    seen[ids[i]] = 1;
    for (int64_t t = offs[i]; t < offs[i + 1]; ++t)
      if (toks[t] < 0 || toks[t] >= cfg_.vocab) throw RpError(RP_ERR_INVALID_ARG, "prompt token id out of range");
    if (PagePool::pages_for(p + max_new[i] - 1, kPageTokens) > pool_.capacity())
      throw RpError(RP_ERR_OUT_OF_PAGES, "a sequence needs more pages than the pool holds");
    pages += admit_pages(p, max_new[i], p);
  }
  if (!pool_.can_take(pages)) throw RpError(RP_ERR_OUT_OF_PAGES, "KV pool cannot hold the admitted sequences");
}

int64_t Engine::admit_pages(int64_t prompt_len, int64_t max_new, int64_t ntok) const {
  return kv_policy_ == RP_KV_RESERVE ? PagePool::pages_for(prompt_len + max_new - 1, kPageTokens)
                                     : PagePool::pages_for(ntok, kPageTokens);
}

bool Engine::known_id(int64_t id) const {
  if (id2slot_.count(id)) return true;
  for (const Waiting& w : waiting_)
    if (w.id == id) return true;
  return false;
}

Waiting* Engine::find_waiting(int64_t id) {
  for (Waiting& w : waiting_)
    if (w.id == id) return &w;
  return nullptr;
}

template <typename F>
void Engine::launch_timed(int cls, double bytes, double flops, F&& launch) {
  if (!(prof_mask_ & (1u << cls)) || prof_seen_[cls][phase_]++ % prof_every_ != 0) {
    HIP_TRY(launch());
    return;
  }
  auto take = [&]() {
    if (prof_pool_.empty()) {
      hipEvent_t e;
      HIP_TRY(hipEventCreate(&e));
      return e;
    }
    hipEvent_t e = prof_pool_.back();
    prof_pool_.pop_back();
    return e;
  };
  // The kernels stamp the events from their own dispatch: no marker packets
  // between kernels, so profiling does not slow the step it measures.
  hipEvent_t e0 = take(), e1 = take();
  LaunchEvents& ev = launch_events();
  ev = LaunchEvents{e0, e1};
  const hipError_t err = launch();
  const bool launched = ev.start == nullptr;
  ev = LaunchEvents{};
  HIP_TRY(err);
  if (!launched) {  // nothing to do (an empty batch): no kernel, no stamps
    prof_pool_.push_back(e0);
    prof_pool_.push_back(e1);
    return;
  }
  prof_pending_.push_back({cls, phase_, e0, e1, bytes, flops});
  if (prof_pending_.size() >= 4096) prof_harvest();
}

void Engine::prof_harvest() {
  if (prof_pending_.empty()) return;
  HIP_TRY(hipEventSynchronize(prof_pending_.back().e1));
  for (auto& r : prof_pending_) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.e0, r.e1));
    ProfAcc& a = prof_acc_[r.cls][r.phase];
    a.launches += 1;
    a.ms += ms;
    a.bytes += r.bytes;
    a.flops += r.flops;
    prof_pool_.push_back(r.e0);
    prof_pool_.push_back(r.e1);
  }
  prof_pending_.clear();
}

void Engine::forward(int M, bool pre, int n_seq, int total_items, int total_splits, int tps) {
  const int H = cfg_.hidden, I = cfg_.intermediate, V = cfg_.vocab, hd = cfg_.head_dim;
  const int nq = cfg_.n_q_heads, nkv = cfg_.n_kv_heads;
  const float eps = cfg_.rms_eps;
  const double e = static_cast<double>(esz_);
  hipStream_t s = stream_;
  phase_ = pre ? 0 : 1;
  float* x = sp<float>(plan_.x);
  void* h = scratch_ + plan_.h;
  float* part = sp<float>(plan_.part);
  void* q = scratch_ + plan_.q;
  void* attn = scratch_ + plan_.attn;
  void* act = scratch_ + plan_.act;
  int32_t* tokens_cur = sp<int32_t>(plan_.tokens_cur);
  const int32_t* pt = sp<int32_t>(plan_.page_table);

  auto splits_for = [&](int N, int K) {
    const size_t cap = plan_.part_elems / (static_cast<size_t>(M) * N);
    const int lim = static_cast<int>(std::min<size_t>(std::max<size_t>(cap, 1), kMaxGemmSplits));
    return gemm_pick_splits(bf16_, M, N, K, false, lim);
  };
  // Algorithmic traffic of C[M,N] = A[M,K] W[N,K]^T: weights and activations
  // read once, the fp32 (or storage-type) result written once.
  auto gemm_bytes = [&](double m, double n, double k, double out_esz) { return (n * k + m * k) * e + m * n * out_esz; };
  const double Md = M;

  EmbedArgs ea{w_.embed, layers_[0].attn_norm, m_in_tok_, m_slot_, tokens_cur, M, H, eps, x, h};
  launch_timed(RP_K_EMBED_NORM, Md * H * (2 * e + 4), 0, [&] { return launch_embed_norm(bf16_, ea, s); });

  const int s_qkv = splits_for(nqkv_, H);
  const int s_o = splits_for(H, nq * hd);
  const int s_d = splits_for(H, I);
  const double kv_tok_bytes = 2.0 * nkv * hd * e;  // one layer's K and V of one token
  double attn_bytes, attn_flops;
  if (pre) {
    attn_bytes = Md * kv_tok_bytes + 2.0 * Md * nq * hd * e;
    attn_flops = 2.0 * nq * hd * sum_ctx_sq_;
  } else {
    attn_bytes = sum_ctx_ * kv_tok_bytes + 2.0 * Md * nq * hd * e;
    attn_flops = 4.0 * nq * hd * sum_ctx_;
  }
  for (int l = 0; l < cfg_.n_layers; ++l) {
    const rp_layer_weights& L = layers_[l];
    char* kpool = kv_ + static_cast<size_t>(l) * layer_kv_bytes_;
    char* vpool = kv_ + static_cast<size_t>(cfg_.n_layers + l) * layer_kv_bytes_;

    const rp_layer_weights* P = packed_layers_.empty() ? nullptr : &packed_layers_[l];
    GemmArgs g{};
    g.A = h; g.lda = H; g.M = M; g.N = nqkv_; g.K = H;
    g.W = WSeg{{L.wq, L.wk, L.wv}, {nq * hd, nkv * hd, nkv * hd}, 3};
    if (P) g.Wp = WSeg{{P->wq, P->wk, P->wv}, {nq * hd, nkv * hd, nkv * hd}, 3};
    g.epi = kEpiPartial; g.splits = s_qkv; g.part = part;
    launch_timed(RP_K_GEMM_QKV, gemm_bytes(Md, nqkv_, H, 4), 2.0 * Md * nqkv_ * H,
                 [&] { return launch_gemm(bf16_, g, s); });

    RopeArgs ra{part, s_qkv, M, L.bq, L.bk, L.bv, nq, nkv, hd, m_pos_, m_slot_, pt, plan_.max_pages,
                sp<float>(plan_.rope_cos), sp<float>(plan_.rope_sin), q, kpool, vpool};
    launch_timed(RP_K_ROPE_APPEND, Md * nqkv_ * (4.0 + e), 0, [&] { return launch_rope_append(bf16_, ra, s); });

    AttnArgs aa{};
    aa.q = q; aa.k_pool = kpool; aa.v_pool = vpool; aa.page_table = pt; aa.pt_stride = plan_.max_pages;
    aa.n_q = nq; aa.n_kv = nkv; aa.hd = hd; aa.scale = 1.0f / std::sqrt(static_cast<float>(hd));
    aa.n_rows = M; aa.tok_slot = m_slot_; aa.tok_pos = m_pos_;
    aa.out = attn;
    if (pre) {
      aa.n_seq = n_seq; aa.seq_slot = m_seq_slot_; aa.seq_row0 = m_seq_row0_; aa.seq_pos0 = m_seq_pos0_;
      aa.seq_ntok = m_seq_ntok_; aa.item_off = m_item_off_; aa.total_items = total_items;
      launch_timed(RP_K_ATTN, attn_bytes, attn_flops, [&] { return launch_attn_prefill(bf16_, aa, s); });
    } else {
      aa.B = M; aa.row_slot = m_slot_; aa.row_ctx = m_ctx_; aa.split_off = m_split_off_;
      aa.total_splits = total_splits; aa.tokens_per_split = tps; aa.split_desc = m_split_desc_;
      aa.max_row_splits = max_row_splits_;
      aa.part_o = sp<float>(plan_.att_o); aa.part_ml = sp<float>(plan_.att_ml);
      launch_timed(RP_K_ATTN, attn_bytes, attn_flops, [&] { return launch_attn_decode(bf16_, aa, s); });
      if (bf16_) {
        const double pbytes = static_cast<double>(total_splits) * nkv * (nq / nkv) * (hd + 2.0) * 4;
        launch_timed(RP_K_ATTN_MERGE, pbytes + Md * nq * hd * e, 0, [&] { return launch_attn_merge(aa, s); });
      }
    }

    g = GemmArgs{};
    g.A = attn; g.lda = nq * hd; g.M = M; g.N = H; g.K = nq * hd;
    g.W = WSeg{{L.wo, nullptr, nullptr}, {H, 0, 0}, 1};
    if (P) g.Wp = WSeg{{P->wo, nullptr, nullptr}, {H, 0, 0}, 1};
    g.epi = kEpiPartial; g.splits = s_o; g.part = part;
    launch_timed(RP_K_GEMM_O, gemm_bytes(Md, H, nq * hd, 4), 2.0 * Md * H * nq * hd,
                 [&] { return launch_gemm(bf16_, g, s); });

    AddNormArgs an{x, part, s_o, L.mlp_norm, M, H, eps, h};
    launch_timed(RP_K_ADD_NORM, Md * H * (4.0 * 3 + e), 0, [&] { return launch_add_rmsnorm(bf16_, an, s); });

    g = GemmArgs{};
    g.A = h; g.lda = H; g.M = M; g.N = I; g.K = H;
    g.W = WSeg{{L.w_gate, L.w_up, nullptr}, {I, I, 0}, 2};
    if (P) g.Wp = WSeg{{P->w_gate, P->w_up, nullptr}, {I, I, 0}, 2};
    g.epi = kEpiSiluMul; g.splits = 1; g.act_out = act;
    launch_timed(RP_K_GEMM_GATE_UP, gemm_bytes(Md, 2.0 * I, H, 0) + Md * I * e, 4.0 * Md * I * H,
                 [&] { return launch_gemm(bf16_, g, s); });

    g = GemmArgs{};
    g.A = act; g.lda = I; g.M = M; g.N = H; g.K = I;
    g.W = WSeg{{L.w_down, nullptr, nullptr}, {H, 0, 0}, 1};
    if (P) g.Wp = WSeg{{P->w_down, nullptr, nullptr}, {H, 0, 0}, 1};
    g.epi = kEpiPartial; g.splits = s_d; g.part = part;
    launch_timed(RP_K_GEMM_DOWN, gemm_bytes(Md, H, I, 4), 2.0 * Md * H * I, [&] { return launch_gemm(bf16_, g, s); });

    const void* next_norm = (l + 1 < cfg_.n_layers) ? layers_[l + 1].attn_norm : w_.final_norm;
    AddNormArgs an2{x, part, s_d, next_norm, M, H, eps, h};
    launch_timed(RP_K_ADD_NORM, Md * H * (4.0 * 3 + e), 0, [&] { return launch_add_rmsnorm(bf16_, an2, s); });
  }

  const void* lm_in = h;
  int m_lm = M;
  if (pre) {
    HIP_TRY(launch_gather_rows(h, m_last_row_, n_seq, H, static_cast<int>(esz_), scratch_ + plan_.hsel, s));
    lm_in = scratch_ + plan_.hsel;
    m_lm = n_seq;
  }
  GemmArgs g{};
  g.A = lm_in; g.lda = H; g.M = m_lm; g.N = V; g.K = H;
  g.W = WSeg{{w_.lm_head, nullptr, nullptr}, {V, 0, 0}, 1};
  if (packed_lm_) g.Wp = WSeg{{packed_lm_, nullptr, nullptr}, {V, 0, 0}, 1};
  g.epi = kEpiPartial; g.splits = 1; g.part = sp<float>(plan_.logits);
  launch_timed(RP_K_GEMM_LM_HEAD, gemm_bytes(m_lm, V, H, 4), 2.0 * m_lm * V * H,
               [&] { return launch_gemm(bf16_, g, s); });

  SampleArgs sa{sp<float>(plan_.logits), m_lm, V, m_gen_slot_, m_gen_pos_, m_gen_hist_,
                sp<uint64_t>(plan_.slot_seed), sp<uint64_t>(plan_.slot_id), sp<float>(plan_.slot_temp),
                tokens_cur, sp<int32_t>(plan_.hist), lim_.max_context, sp<float>(plan_.logp),
                sp<float>(plan_.cand_val), sp<int32_t>(plan_.cand_idx), sp<float>(plan_.cand_m),
                sp<float>(plan_.cand_s)};
  launch_timed(RP_K_SAMPLE, static_cast<double>(m_lm) * V * 4, 0, [&] { return launch_sample(sa, s); });
}

void Engine::run_prefill_chunk(const std::vector<PrefillPiece>& pcs, float* logits_out) {
  const int n = static_cast<int>(pcs.size());
  int T = 0;
  for (const PrefillPiece& pc : pcs) T += pc.ntok;
  const size_t ints = 3 * static_cast<size_t>(T) + 8 * static_cast<size_t>(n) + 1;
  int32_t* m = stage_meta(ints);
  int32_t* in_tok = m;
  int32_t* slot = in_tok + T;
  int32_t* pos = slot + T;
  int32_t* seq_slot = pos + T;
  int32_t* seq_row0 = seq_slot + n;
  int32_t* seq_pos0 = seq_row0 + n;
  int32_t* seq_ntok = seq_pos0 + n;
  int32_t* item_off = seq_ntok + n;
  int32_t* last_row = item_off + n + 1;
  int32_t* gen_pos = last_row + n;
  int32_t* gen_hist = gen_pos + n;
  const int tpi = attn_prefill_tokens_per_item(bf16_, cfg_.n_q_heads / cfg_.n_kv_heads);
  int row = 0, items = 0;
  sum_ctx_sq_ = 0;
  for (int j = 0; j < n; ++j) {
    const PrefillPiece& pc = pcs[j];
    for (int t = 0; t < pc.ntok; ++t) {
      in_tok[row + t] = pc.toks[t];
      slot[row + t] = pc.slot;
      pos[row + t] = pc.pos0 + t;
    }
    seq_slot[j] = pc.slot;
    seq_row0[j] = row;
    seq_pos0[j] = pc.pos0;
    seq_ntok[j] = pc.ntok;
    // attended keys summed over the piece's queries, x2 (the causal-attention flop count)
    sum_ctx_sq_ += 2.0 * pc.ntok * pc.pos0 + static_cast<double>(pc.ntok) * (pc.ntok + 1);
    item_off[j] = items;
    items += (pc.ntok + tpi - 1) / tpi;
    last_row[j] = row + pc.ntok - 1;
    // A piece that does not end its sequence samples into the same history
    // entry the final piece overwrites later.
    gen_pos[j] = pc.pos0 + pc.ntok;
    gen_hist[j] = pc.hist0;
    row += pc.ntok;
  }
  item_off[n] = items;
  upload_meta(m, ints);
  const int32_t* d = d_meta_;
  m_in_tok_ = d; m_slot_ = d + T; m_pos_ = d + 2 * T;
  m_seq_slot_ = d + 3 * T; m_seq_row0_ = m_seq_slot_ + n; m_seq_pos0_ = m_seq_row0_ + n;
  m_seq_ntok_ = m_seq_pos0_ + n; m_item_off_ = m_seq_ntok_ + n; m_last_row_ = m_item_off_ + n + 1;
  m_gen_pos_ = m_last_row_ + n; m_gen_hist_ = m_gen_pos_ + n; m_gen_slot_ = m_seq_slot_;
  TraceRec* tr = trace_cap_ ? trace_begin(1, T, static_cast<int64_t>(sum_ctx_sq_ / 2)) : nullptr;
  forward(T, true, n, items, 0, 0);
  trace_end(tr);
  std::vector<std::array<int64_t, 3>> sampled;  // pieces that end their sequence sampled its next token
  for (const PrefillPiece& pc : pcs)
    if (pc.seq >= 0) sampled.push_back({pc.slot, slots_[pc.slot].id, pc.hist0});
  note_samples(sampled);
  if (logits_out) {
    // logits rows of the pieces that end a sequence, in runs of consecutive sequences
    int j = 0;
    while (j < n) {
      if (pcs[j].seq < 0) { ++j; continue; }
      int k = j + 1;
      while (k < n && pcs[k].seq == pcs[k - 1].seq + 1) ++k;
      HIP_TRY(hipMemcpyAsync(logits_out + static_cast<size_t>(pcs[j].seq) * cfg_.vocab,
                             sp<float>(plan_.logits) + static_cast<size_t>(j) * cfg_.vocab,
                             static_cast<size_t>(k - j) * cfg_.vocab * 4, hipMemcpyDeviceToDevice, stream_));
      j = k;
    }
  }
}

std::vector<int32_t> Engine::admit_seqs(const std::vector<AdmitSeq>& a, const std::vector<const Waiting*>& restore,
                                        float* logits_out) {
  const int32_t n = static_cast<int32_t>(a.size());
  if (tables_pending_) {
    fence_wait(ev_tables_);
    tables_pending_ = false;
  }
  std::vector<int32_t> new_slots(n);
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = free_slots_.back();
    free_slots_.pop_back();
    Seq& q = slots_[s];
    q = Seq{};
    q.id = a[i].id;
    q.prompt_len = a[i].prompt_len;
    q.max_new = a[i].max_new;
    q.n_gen = a[i].n_gen0;
    q.seed = a[i].seed;
    q.temp = a[i].temp;
    q.live = true;
    q.arrival = a[i].arrival;
    if (kv_policy_ == RP_KV_ON_DEMAND) q.prompt.assign(a[i].toks, a[i].toks + a[i].prompt_len);
    pool_.take(admit_pages(a[i].prompt_len, a[i].max_new, a[i].ntok), s, q.pages);
    int32_t* row = h_page_table_ + static_cast<size_t>(s) * plan_.max_pages;
    std::fill(row, row + plan_.max_pages, 0);
    std::copy(q.pages.begin(), q.pages.end(), row);
    h_slot_seed_[s] = a[i].seed;
    h_slot_id_[s] = static_cast<uint64_t>(a[i].id);
    h_slot_temp_[s] = a[i].temp;
    id2slot_[q.id] = s;
    order_.push_back(s);
    new_slots[i] = s;
  }
  upload_slot_tables();
  // Tokens (and their log-probabilities) a resumed sequence generated before
  // its preemption go back into its history rows.
  bool restored = false;
  for (int32_t i = 0; i < n; ++i)
    if (a[i].n_gen0 > 0 && restore[i]) {
      const size_t at = static_cast<size_t>(new_slots[i]) * lim_.max_context;
      HIP_TRY(hipMemcpyAsync(sp<int32_t>(plan_.hist) + at, restore[i]->tokens.data() + restore[i]->prompt_len,
                             static_cast<size_t>(a[i].n_gen0) * 4, hipMemcpyHostToDevice, stream_));
      HIP_TRY(hipMemcpyAsync(sp<float>(plan_.logp) + at, restore[i]->logp.data(),
                             static_cast<size_t>(a[i].n_gen0) * 4, hipMemcpyHostToDevice, stream_));
      restored = true;
    }
  if (restored) HIP_TRY(hipStreamSynchronize(stream_));
  // Chunks of at most max_prefill_tokens tokens.  A sequence that fits is
  // never split; a longer one is cut into pieces that continue at their
  // position (the attention of a piece reads the earlier keys from its pages).
  const int32_t budget = lim_.max_prefill_tokens;
  std::vector<PrefillPiece> chunk;
  int32_t tok = 0;
  auto flush = [&]() {
    if (!chunk.empty()) run_prefill_chunk(chunk, logits_out);
    chunk.clear();
    tok = 0;
  };
  for (int32_t i = 0; i < n; ++i) {
    const int32_t len = a[i].ntok;
    if (len <= budget) {
      if (tok + len > budget) flush();
      chunk.push_back({new_slots[i], a[i].toks, 0, len, a[i].n_gen0, i});
      tok += len;
      continue;
    }
    flush();
    for (int32_t o = 0; o < len; o += budget) {
      const int32_t take = std::min(budget, len - o);
      chunk.push_back({new_slots[i], a[i].toks + o, o, take, a[i].n_gen0, o + take == len ? i : -1});
      tok += take;
      if (o + take < len) flush();
    }
  }
  flush();
  for (int32_t s : new_slots) {
    slots_[s].n_gen += 1;
    if (slots_[s].n_gen >= slots_[s].max_new) slots_[s].finished = true;
  }
  return new_slots;
}

void Engine::prefill(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
                     const int32_t* max_new, uint64_t seed, float temp, float* logits_out, int32_t* first_out) {
  check_admission(n, ids, offs, toks, max_new, temp);
  std::vector<AdmitSeq> a(n);
  for (int32_t i = 0; i < n; ++i) {
    const int32_t p = static_cast<int32_t>(offs[i + 1] - offs[i]);
    a[i] = AdmitSeq{ids[i], toks + offs[i], p, p, max_new[i], 0, seed, temp, arrival_next_++};
  }
  const std::vector<int32_t> new_slots = admit_seqs(a, std::vector<const Waiting*>(n, nullptr), logits_out);
  if (first_out) {
    HIP_TRY(hipStreamSynchronize(stream_));
    std::vector<int32_t> cur(lim_.max_seqs);
    HIP_TRY(hipMemcpy(cur.data(), scratch_ + plan_.tokens_cur, cur.size() * 4, hipMemcpyDeviceToHost));
    for (int32_t k = 0; k < n; ++k) first_out[k] = cur[new_slots[k]];
  }
}

int32_t Engine::decode_step(const int32_t* forced, float* logits_out, int64_t* row_ids_out) {
  if (forced && kv_policy_ == RP_KV_ON_DEMAND)
    throw RpError(RP_ERR_INVALID_ARG, "teacher forcing needs the reserving KV policy");
  if (eos_token_ >= 0) apply_eos(sample_step_ - 2);  // the step before last has finished by now
  std::vector<int32_t> resumed;
  if (kv_policy_ == RP_KV_ON_DEMAND) resumed = schedule_pages();
  std::vector<int32_t> rows;
  rows.reserve(order_.size());
  for (int32_t s : order_)
    if (!slots_[s].finished && std::find(resumed.begin(), resumed.end(), s) == resumed.end()) rows.push_back(s);
  const int B = static_cast<int>(rows.size());
  if (B == 0) return 0;
  if (forced) {
    for (int i = 0; i < B; ++i)
      if (forced[i] < 0 || forced[i] >= cfg_.vocab) throw RpError(RP_ERR_INVALID_ARG, "forced token out of range");
  }
  // Per-row context first: the split plan sizes the metadata.
  std::vector<int32_t>& ctx_h = ctx_scratch_;
  ctx_h.resize(B);
  int64_t total_pages = 0;
  sum_ctx_ = 0;
  for (int i = 0; i < B; ++i) {
    const Seq& q = slots_[rows[i]];
    ctx_h[i] = q.prompt_len + q.n_gen;
    total_pages += PagePool::pages_for(ctx_h[i], kPageTokens);
    sum_ctx_ += ctx_h[i];
  }
  int tps = 0, total_splits = 0;
  if (bf16_) {
    const int64_t target = decode_split_target(cfg_);
    const int64_t pps = std::max<int64_t>(1, (total_pages + target - 1) / target);
    tps = static_cast<int>(pps * kPageTokens);
    max_row_splits_ = 0;
    for (int i = 0; i < B; ++i) {
      const int n = (ctx_h[i] + tps - 1) / tps;
      total_splits += n;
      max_row_splits_ = std::max(max_row_splits_, n);
    }
    if (total_splits > plan_.split_cap) throw RpError(RP_ERR_CAPACITY, "decode split capacity exceeded");
  }
  const size_t desc_at = (7 * static_cast<size_t>(B) + 1 + 3) & ~static_cast<size_t>(3);
  const size_t ints = desc_at + 4 * static_cast<size_t>(total_splits);
  int32_t* m = stage_meta(ints);
  int32_t* in_tok = m;
  int32_t* slot = in_tok + B;
  int32_t* pos = slot + B;
  int32_t* ctx = pos + B;
  int32_t* split_off = ctx + B;
  int32_t* gen_pos = split_off + B + 1;
  int32_t* gen_hist = gen_pos + B;
  int32_t* desc = m + desc_at;
  int32_t sx = 0;
  for (int i = 0; i < B; ++i) {
    const Seq& q = slots_[rows[i]];
    in_tok[i] = forced ? forced[i] : -1;
    slot[i] = rows[i];
    pos[i] = q.prompt_len + q.n_gen - 1;
    ctx[i] = pos[i] + 1;
    gen_pos[i] = pos[i] + 1;
    gen_hist[i] = q.n_gen;
    split_off[i] = sx;
    if (bf16_) {
      // one descriptor per split: row (+ 2^30 when it is the row's only split), key range, slot
      const int n = (ctx[i] + tps - 1) / tps;
      for (int j = 0; j < n; ++j, ++sx) {
        desc[4 * sx + 0] = i | (n == 1 ? (1 << 30) : 0);
        desc[4 * sx + 1] = j * tps;
        desc[4 * sx + 2] = std::min(j * tps + tps, ctx[i]);
        desc[4 * sx + 3] = rows[i];
      }
    }
  }
  split_off[B] = total_splits;
  upload_meta(m, ints);
  const int32_t* d = d_meta_;
  m_in_tok_ = d; m_slot_ = d + B; m_pos_ = d + 2 * B; m_ctx_ = d + 3 * B; m_split_off_ = d + 4 * B;
  m_gen_pos_ = d + 5 * B + 1; m_gen_hist_ = d + 6 * B + 1; m_gen_slot_ = m_slot_;
  m_split_desc_ = d + desc_at;
  TraceRec* tr = trace_cap_ ? trace_begin(0, B, sum_ctx_) : nullptr;
  forward(B, false, 0, 0, total_splits, tps);
  trace_end(tr);
  if (logits_out) {
    HIP_TRY(hipMemcpyAsync(logits_out, scratch_ + plan_.logits, static_cast<size_t>(B) * cfg_.vocab * 4,
                           hipMemcpyDeviceToDevice, stream_));
  }
  std::vector<std::array<int64_t, 3>> sampled(B);
  for (int i = 0; i < B; ++i) sampled[i] = {rows[i], slots_[rows[i]].id, slots_[rows[i]].n_gen};
  note_samples(sampled);
  for (int i = 0; i < B; ++i) {
    Seq& q = slots_[rows[i]];
    if (row_ids_out) row_ids_out[i] = q.id;
    q.n_gen += 1;
    if (q.n_gen >= q.max_new) q.finished = true;
  }
  return B;
}

void Engine::set_packed_weights(void* ws, size_t bytes) {
  if (!ws) {
    HIP_TRY(hipStreamSynchronize(stream_));  // launches already queued may still read the packed copy
    packed_layers_.clear();
    packed_lm_ = nullptr;
    return;
  }
  if (!bf16_) throw RpError(RP_ERR_INVALID_ARG, "packed weights apply to bf16 models only");
  if (reinterpret_cast<uintptr_t>(ws) & 255) throw RpError(RP_ERR_INVALID_ARG, "packed workspace must be 256-byte aligned");
  if (bytes < packed_weights_bytes(cfg_)) throw RpError(RP_ERR_INVALID_ARG, "packed workspace smaller than rp_packed_weights_bytes");
  const int H = cfg_.hidden, I = cfg_.intermediate, qd = cfg_.n_q_heads * cfg_.head_dim,
            kvd = cfg_.n_kv_heads * cfg_.head_dim;
  char* p = static_cast<char*>(ws);
  auto pack = [&](const void* w, int rows, int K) {
    void* dst = p;
    HIP_TRY(launch_pack_weights(w, dst, rows, K, stream_));
    p += align256(static_cast<size_t>(rows) * K * 2);
    return static_cast<const void*>(dst);
  };
  std::vector<rp_layer_weights> pl(layers_.size());
  for (size_t l = 0; l < layers_.size(); ++l) {
    const rp_layer_weights& L = layers_[l];
    pl[l] = L;  // norms and biases stay the caller's
    pl[l].wq = pack(L.wq, qd, H);
    pl[l].wk = pack(L.wk, kvd, H);
    pl[l].wv = pack(L.wv, kvd, H);
    pl[l].wo = pack(L.wo, H, qd);
    pl[l].w_gate = pack(L.w_gate, I, H);
    pl[l].w_up = pack(L.w_up, I, H);
    pl[l].w_down = pack(L.w_down, H, I);
  }
  packed_lm_ = pack(w_.lm_head, cfg_.vocab, H);
  packed_layers_ = std::move(pl);
}

void Engine::profile_every(int32_t every) {
  if (every < 1) throw RpError(RP_ERR_INVALID_ARG, "profile sampling: every must be >= 1");
  prof_every_ = every;
  for (auto& c : prof_seen_) c[0] = c[1] = 0;
}

void Engine::profile_enable(uint32_t mask) {
  if (mask >> RP_K_COUNT) throw RpError(RP_ERR_INVALID_ARG, "profile mask names an unknown kernel class");
  if (no_alloc_ && mask) throw RpError(RP_ERR_BAD_STATE, "no profiling without allocations");
  prof_mask_ = mask;
}

int32_t Engine::profile_read(rp_kernel_stats* out, int32_t cap) {
  if (cap < 0 || (cap > 0 && !out)) throw RpError(RP_ERR_INVALID_ARG, "profile_read: bad output");
  HIP_TRY(hipStreamSynchronize(stream_));
  prof_harvest();
  int32_t n = 0;
  for (int c = 0; c < RP_K_COUNT; ++c)
    for (int ph = 0; ph < 2; ++ph) {
      ProfAcc& a = prof_acc_[c][ph];
      if (a.launches == 0) continue;
      if (n < cap) out[n] = rp_kernel_stats{c, ph, a.launches, a.ms, a.bytes, a.flops};
      ++n;
      a = ProfAcc{};
    }
  return std::min(n, cap);
}

void Engine::release(int32_t slot) {
  Seq& q = slots_[slot];
  pool_.give_back(q.pages, slot);
  id2slot_.erase(q.id);
  order_.erase(std::find(order_.begin(), order_.end(), slot));
  free_slots_.push_back(slot);
  q = Seq{};
}

int32_t Engine::free_finished(int64_t* ids_out, int32_t cap) {
  drain_eos();
  std::vector<int32_t> fin;
  for (int32_t s : order_)
    if (slots_[s].finished && static_cast<int32_t>(fin.size()) < cap) fin.push_back(s);
  for (size_t k = 0; k < fin.size(); ++k) {
    if (ids_out) ids_out[k] = slots_[fin[k]].id;
    release(fin[k]);
  }
  return static_cast<int32_t>(fin.size());
}

void Engine::abort(int32_t n, const int64_t* ids) {
  if (n < 0 || (n > 0 && !ids)) throw RpError(RP_ERR_INVALID_ARG, "abort: bad arguments");
  std::unordered_map<int64_t, int> seen;
  for (int32_t i = 0; i < n; ++i) {
    if (!known_id(ids[i])) throw RpError(RP_ERR_UNKNOWN_ID, "abort: unknown sequence id");
    if (seen.count(ids[i])) throw RpError(RP_ERR_INVALID_ARG, "abort: duplicate id");
    seen[ids[i]] = 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    auto it = id2slot_.find(ids[i]);
    if (it != id2slot_.end()) {
      release(it->second);
    } else {
      waiting_.erase(std::find_if(waiting_.begin(), waiting_.end(), [&](const Waiting& w) { return w.id == ids[i]; }));
    }
  }
}

void Engine::set_kv_policy(int32_t policy) {
  if (policy != RP_KV_RESERVE && policy != RP_KV_ON_DEMAND) throw RpError(RP_ERR_INVALID_ARG, "unknown KV policy");
  if (live_count() != 0) throw RpError(RP_ERR_BAD_STATE, "the KV policy changes only with no live sequences");
  kv_policy_ = policy;
}

void Engine::kv_status(int64_t* free_pages, int32_t* running, int32_t* waiting, int64_t* preemptions,
                       int64_t* recomputed_tokens) const {
  if (free_pages) *free_pages = pool_.free_pages();
  if (running) *running = static_cast<int32_t>(order_.size());
  if (waiting) *waiting = static_cast<int32_t>(waiting_.size());
  if (preemptions) *preemptions = n_preempt_;
  if (recomputed_tokens) *recomputed_tokens = n_recompute_tok_;
}

void Engine::preempt(const std::vector<int32_t>& victims) {
  if (victims.empty()) return;
  HIP_TRY(hipStreamSynchronize(stream_));  // the history rows hold the last sampled tokens
  for (int32_t s : victims) {
    const Seq& q = slots_[s];
    Waiting w{q.id, q.prompt_len, q.max_new, q.n_gen, q.seed, q.temp, q.arrival, q.prompt, {}};
    w.tokens.resize(static_cast<size_t>(q.prompt_len) + q.n_gen);
    w.logp.resize(static_cast<size_t>(q.n_gen));
    HIP_TRY(hipMemcpy(w.tokens.data() + q.prompt_len, sp<int32_t>(plan_.hist) + static_cast<size_t>(s) * lim_.max_context,
                      static_cast<size_t>(q.n_gen) * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(w.logp.data(), sp<float>(plan_.logp) + static_cast<size_t>(s) * lim_.max_context,
                      static_cast<size_t>(q.n_gen) * 4, hipMemcpyDeviceToHost));
    release(s);
    waiting_.insert(std::upper_bound(waiting_.begin(), waiting_.end(), w.arrival,
                                     [](int64_t a, const Waiting& x) { return a < x.arrival; }),
                    std::move(w));
    ++n_preempt_;
  }
}

std::vector<int32_t> Engine::schedule_pages() {
  // Pages the running rows need for the position each one writes next.
  std::vector<int32_t> rows;
  int64_t need = 0;
  auto extra = [&](int32_t s) {
    const Seq& q = slots_[s];
    return std::max<int64_t>(0, PagePool::pages_for(q.prompt_len + q.n_gen, kPageTokens) -
                                    static_cast<int64_t>(q.pages.size()));
  };
  for (int32_t s : order_)
    if (!slots_[s].finished) {
      rows.push_back(s);
      need += extra(s);
    }
  // Resume preempted sequences, oldest arrival first, while the pool has
  // room for them beyond what the running rows need this step.
  std::vector<AdmitSeq> adm;
  std::vector<const Waiting*> restore;
  std::vector<Waiting> taken;
  int64_t reserve = need;
  size_t k = 0;
  while (k < waiting_.size() && adm.size() < free_slots_.size()) {
    const Waiting& w = waiting_[k];
    const int64_t ntok = static_cast<int64_t>(w.prompt_len) + w.n_gen;
    const int64_t pages = PagePool::pages_for(std::min<int64_t>(ntok + 1, w.prompt_len + w.max_new - 1), kPageTokens);
    if (reserve + pages > pool_.free_pages()) break;
    reserve += pages;
    ++k;
  }
  if (k > 0) {
    taken.assign(std::make_move_iterator(waiting_.begin()), std::make_move_iterator(waiting_.begin() + k));
    waiting_.erase(waiting_.begin(), waiting_.begin() + k);
    for (const Waiting& w : taken) {
      const int32_t ntok = w.prompt_len + w.n_gen;
      adm.push_back(AdmitSeq{w.id, w.tokens.data(), ntok, w.prompt_len, w.max_new, w.n_gen, w.seed, w.temp,
                             w.arrival});
      restore.push_back(&w);
      n_recompute_tok_ += ntok;
    }
  }
  std::vector<int32_t> resumed;
  if (!adm.empty()) resumed = admit_seqs(adm, restore, nullptr);
  // Preempt the latest arrivals until the remaining rows fit (after reading
  // every pending end-of-sequence check, so that no stopped row is chosen).
  if (need > pool_.free_pages() && eos_token_ >= 0) {
    drain_eos();
    need = 0;
    rows.erase(std::remove_if(rows.begin(), rows.end(), [&](int32_t s) { return slots_[s].finished; }), rows.end());
    for (int32_t s : rows) need += extra(s);
  }
  std::vector<int32_t> victims;
  while (need > pool_.free_pages()) {
    if (rows.empty()) throw RpError(RP_ERR_OUT_OF_PAGES, "KV pool held by finished sequences; free them first");
    auto v = std::max_element(rows.begin(), rows.end(),
                              [&](int32_t a, int32_t b) { return slots_[a].arrival < slots_[b].arrival; });
    need -= extra(*v);
    victims.push_back(*v);
    rows.erase(v);
  }
  preempt(victims);
  bool grew = false;
  for (int32_t s : rows) {
    const int64_t e = extra(s);
    if (e == 0) continue;
    if (!grew && tables_pending_) {
      fence_wait(ev_tables_);
      tables_pending_ = false;
    }
    Seq& q = slots_[s];
    const size_t old = q.pages.size();
    pool_.take(e, s, q.pages);
    int32_t* row = h_page_table_ + static_cast<size_t>(s) * plan_.max_pages;
    std::copy(q.pages.begin() + old, q.pages.end(), row + old);
    grew = true;
  }
  if (grew) upload_slot_tables();
  return resumed;
}

int32_t Engine::get_tokens(int64_t id, int32_t* out, int32_t cap) {
  if (const Waiting* w = find_waiting(id)) {
    const int32_t k = std::min(cap, w->n_gen);
    if (k > 0) {
      if (!out) throw RpError(RP_ERR_INVALID_ARG, "get_tokens: null output");
      std::copy(w->tokens.begin() + w->prompt_len, w->tokens.begin() + w->prompt_len + k, out);
    }
    return w->n_gen;
  }
  auto it = id2slot_.find(id);
  if (it == id2slot_.end()) throw RpError(RP_ERR_UNKNOWN_ID, "get_tokens: unknown sequence id");
  HIP_TRY(hipStreamSynchronize(stream_));
  drain_eos();
  const Seq& q = slots_[it->second];
  const int32_t k = std::min(cap, q.n_gen);
  if (k > 0) {
    if (!out) throw RpError(RP_ERR_INVALID_ARG, "get_tokens: null output");
    HIP_TRY(hipMemcpy(out, sp<int32_t>(plan_.hist) + static_cast<size_t>(it->second) * lim_.max_context, k * 4,
                      hipMemcpyDeviceToHost));
  }
  return q.n_gen;
}

int32_t Engine::get_logprobs(int64_t id, float* out, int32_t cap) {
  if (const Waiting* w = find_waiting(id)) {
    const int32_t k = std::min(cap, w->n_gen);
    if (k > 0) {
      if (!out) throw RpError(RP_ERR_INVALID_ARG, "get_logprobs: null output");
      std::copy(w->logp.begin(), w->logp.begin() + k, out);
    }
    return w->n_gen;
  }
  auto it = id2slot_.find(id);
  if (it == id2slot_.end()) throw RpError(RP_ERR_UNKNOWN_ID, "get_logprobs: unknown sequence id");
  HIP_TRY(hipStreamSynchronize(stream_));
  drain_eos();
  const Seq& q = slots_[it->second];
  const int32_t k = std::min(cap, q.n_gen);
  if (k > 0) {
    if (!out) throw RpError(RP_ERR_INVALID_ARG, "get_logprobs: null output");
    HIP_TRY(hipMemcpy(out, sp<float>(plan_.logp) + static_cast<size_t>(it->second) * lim_.max_context, k * 4,
                      hipMemcpyDeviceToHost));
  }
  return q.n_gen;
}

void Engine::validate_seqs(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
                           const int32_t* max_new, float temp, std::vector<int64_t>& resp_off) const {
  if (!(temp >= 0.f) || std::isinf(temp)) throw RpError(RP_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  if (offs[0] != 0) throw RpError(RP_ERR_INVALID_ARG, "prompt_offsets[0] must be 0");
  std::unordered_map<int64_t, int> seen;
  resp_off.assign(static_cast<size_t>(n) + 1, 0);
  for (int32_t i = 0; i < n; ++i) {
    const int64_t p = offs[i + 1] - offs[i];
    if (p < 1 || max_new[i] < 1) throw RpError(RP_ERR_INVALID_ARG, "prompts and max_new_tokens must be >= 1");
    if (p + max_new[i] - 1 > lim_.max_context)
      throw RpError(RP_ERR_CAPACITY, "a sequence exceeds max_context");
    if (PagePool::pages_for(p + max_new[i] - 1, kPageTokens) > pool_.capacity())
      throw RpError(RP_ERR_OUT_OF_PAGES, "a sequence needs more pages than the pool holds");
    if (seen.count(ids[i])) throw RpError(RP_ERR_DUPLICATE_ID, "duplicate sequence id");
    seen[ids[i]] = 1;
    for (int64_t t = offs[i]; t < offs[i + 1]; ++t)
      if (toks[t] < 0 || toks[t] >= cfg_.vocab) throw RpError(RP_ERR_INVALID_ARG, "prompt token id out of range");
    resp_off[i + 1] = resp_off[i] + max_new[i];
  }
}

hipEvent_t Engine::event_at(size_t k) {
  while (events_.size() <= k) {
    hipEvent_t e;
    HIP_TRY(hipEventCreate(&e));
    events_.push_back(e);
  }
  return events_[k];
}

void Engine::run_round(const std::vector<int32_t>& members, const SeqArrays& a, int32_t* resp_out,
                       int32_t* gen_out, Race* race, rp_round_stats* st) {
  const size_t resp_cap = static_cast<size_t>(lim_.max_seqs) * lim_.max_context;
  int32_t* resp_dev = sp<int32_t>(plan_.resp);
  float* resp_logp_dev = sp<float>(plan_.resp_logp);
  const int32_t* hist = sp<int32_t>(plan_.hist);
  const float* logp_hist = sp<float>(plan_.logp);
  size_t next = 0;
  // time marks: 0 round start, 1 end of the first admission, 2 round end, then one per step with departures
  const size_t ev_start = 0, ev_pre = 1, ev_end = 2;
  size_t n_ev = 3;
  std::vector<std::pair<size_t, int32_t>> left_ev;     // (mark index, member position) per departure
  std::vector<std::array<int64_t, 3>> pending_copies;  // dev offset, host offset, length
  size_t resp_cursor = 0;
  std::unordered_map<int64_t, int32_t> id_member;      // sequence id -> position in members
  pool_.reset_peak();
  int32_t steps = 0;
  int64_t prompt_tokens = 0, gen_tokens = 0;
  const int64_t preempt0 = n_preempt_, recompute0 = n_recompute_tok_;
  // On demand, fresh sequences are admitted only while no preempted one waits
  // and a watermark of 1% of the pool stays free (none for a race round,
  // which starts everything at once).
  const bool on_demand = kv_policy_ == RP_KV_ON_DEMAND;
  const int64_t watermark = on_demand && !race ? std::max<int64_t>(1, pool_.capacity() / 100) : 0;

  // Race bookkeeping: finished members per prompt in completion order, and
  // whether each prompt has been decided (accepted, or lost the race).
  std::vector<std::vector<int32_t>> done;
  std::vector<uint8_t> decided;
  int32_t n_acc = 0;
  if (race) {
    done.resize(race->n_prompts);
    decided.assign(race->n_prompts, 0);
    race->accepted.assign(race->n_prompts, 0);
    race->kept.assign(members.size(), 0);
  }

  auto flush = [&]() {
    if (pending_copies.empty()) return;
    HIP_TRY(hipStreamSynchronize(stream_));
    for (auto& c : pending_copies) {
      HIP_TRY(hipMemcpy(resp_out + c[1], resp_dev + c[0], static_cast<size_t>(c[2]) * 4, hipMemcpyDeviceToHost));
      if (a.logp_out)
        HIP_TRY(hipMemcpy(a.logp_out + c[1], resp_logp_dev + c[0], static_cast<size_t>(c[2]) * 4,
                          hipMemcpyDeviceToHost));
    }
    pending_copies.clear();
    resp_cursor = 0;
  };
  auto admit = [&]() {
    if (!waiting_.empty()) return;
    std::vector<int64_t> b_ids, b_offs{0};
    std::vector<int32_t> b_toks, b_new, b_mem;
    int64_t pages = 0;
    while (next < members.size() && b_ids.size() < free_slots_.size()) {
      const int32_t i = members[next];
      const int64_t p = a.offs[i + 1] - a.offs[i];
      const int64_t need = admit_pages(p, a.max_new[i], p);
      if (!pool_.can_take(pages + need + watermark)) break;
      pages += need;
      b_ids.push_back(a.ids[i]);
      b_toks.insert(b_toks.end(), a.toks + a.offs[i], a.toks + a.offs[i + 1]);
      b_offs.push_back(static_cast<int64_t>(b_toks.size()));
      b_new.push_back(a.max_new[i]);
      b_mem.push_back(static_cast<int32_t>(next));
      prompt_tokens += p;
      ++next;
    }
    if (b_ids.empty()) return;
    prefill(static_cast<int32_t>(b_ids.size()), b_ids.data(), b_toks.data(), b_offs.data(), b_new.data(), a.seed,
            a.temp, nullptr, nullptr);
    for (size_t k = 0; k < b_mem.size(); ++k) id_member[b_ids[k]] = b_mem[k];
  };
  // Copies a departing sequence's tokens out, then frees its slot and pages.
  auto retire = [&](int32_t s) {
    const int32_t k = id_member.at(slots_[s].id);
    const int32_t i = members[k];
    const int64_t len = slots_[s].n_gen;
    if (resp_cursor + len > resp_cap) flush();
    HIP_TRY(hipMemcpyAsync(resp_dev + resp_cursor, hist + static_cast<size_t>(s) * lim_.max_context, len * 4,
                           hipMemcpyDeviceToDevice, stream_));
    if (a.logp_out)
      HIP_TRY(hipMemcpyAsync(resp_logp_dev + resp_cursor, logp_hist + static_cast<size_t>(s) * lim_.max_context,
                             len * 4, hipMemcpyDeviceToDevice, stream_));
    pending_copies.push_back({static_cast<int64_t>(resp_cursor), a.resp_off[i], len});
    resp_cursor += len;
    if (gen_out) gen_out[i] = static_cast<int32_t>(len);
    left_ev.push_back({n_ev, k});
    gen_tokens += len;
    id_member.erase(slots_[s].id);
    release(s);
  };
  // The same for a preempted member: its tokens are on the host already.
  auto retire_waiting = [&](const Waiting& w) {
    const int32_t k = id_member.at(w.id);
    const int32_t i = members[k];
    std::copy(w.tokens.begin() + w.prompt_len, w.tokens.end(), resp_out + a.resp_off[i]);
    if (a.logp_out) std::copy(w.logp.begin(), w.logp.end(), a.logp_out + a.resp_off[i]);
    if (gen_out) gen_out[i] = w.n_gen;
    left_ev.push_back({n_ev, k});
    gen_tokens += w.n_gen;
    id_member.erase(w.id);
  };
  auto collect = [&]() {
    std::vector<int32_t> leaving;
    std::vector<uint8_t> abort_prompt;
    bool stop = false;
    if (race) {
      // Completions of this step, in member order (responses of a prompt by index).
      std::vector<std::pair<int32_t, int32_t>> fin;  // (member, prompt)
      for (int32_t s : order_)
        if (slots_[s].finished && settled(slots_[s])) {
          const int32_t k = id_member.at(slots_[s].id);
          fin.push_back({k, race->prompt[k]});
        }
      std::sort(fin.begin(), fin.end());
      std::vector<int32_t> fresh;
      for (auto& f : fin) {
        const int32_t p = f.second;
        if (decided[p]) continue;
        done[p].push_back(f.first);
        if (static_cast<int32_t>(done[p].size()) == race->R0) fresh.push_back(p);
      }
      std::sort(fresh.begin(), fresh.end());
      abort_prompt.assign(race->n_prompts, 0);
      for (int32_t p : fresh) {
        decided[p] = 1;
        if (n_acc < race->keep) {
          ++n_acc;
          race->accepted[p] = 1;
          for (int32_t j = 0; j < race->R0; ++j) race->kept[done[p][j]] = 1;
          abort_prompt[p] = 1;  // its other responses can no longer be kept
        }
      }
      stop = n_acc >= race->keep;
    }
    // Sequences about to be aborted take their pending end-of-sequence checks first.
    if (race && eos_token_ >= 0 && (stop || std::find(abort_prompt.begin(), abort_prompt.end(), 1) != abort_prompt.end()))
      drain_eos();
    auto goes = [&](int64_t id) { return stop || (race && abort_prompt[race->prompt[id_member.at(id)]]); };
    for (int32_t s : order_)
      if ((slots_[s].finished && settled(slots_[s])) || goes(slots_[s].id)) leaving.push_back(s);
    std::vector<int64_t> leaving_waiting;
    if (race)
      for (const Waiting& w : waiting_)
        if (id_member.count(w.id) && goes(w.id)) leaving_waiting.push_back(w.id);
    if (leaving.empty() && leaving_waiting.empty()) return;
    // Departure time: the end of the step that finished them, before their tokens are copied out.
    mark(n_ev);
    for (int32_t s : leaving) retire(s);
    for (int64_t id : leaving_waiting) {
      auto it = std::find_if(waiting_.begin(), waiting_.end(), [&](const Waiting& w) { return w.id == id; });
      retire_waiting(*it);
      waiting_.erase(it);
    }
    ++n_ev;
  };

  mark(ev_start);
  if (trace_cap_ > 0) {  // the trace's own copy of the round start, kept until the trace is read
    cur_round_ev_ = trace_event();
    HIP_TRY(hipEventRecord(cur_round_ev_, stream_));
    trace_round_evs_.push_back(cur_round_ev_);
  }
  admit();
  if (race && next < members.size())
    throw RpError(RP_ERR_CAPACITY, "a race round must start all of its responses together");
  mark(ev_pre);
  collect();
  while (true) {
    if (next < members.size()) {
      admit();
      collect();
    }
    if (order_.empty() && waiting_.empty() && next >= members.size()) break;
    if (order_.empty() && waiting_.empty()) throw RpError(RP_ERR_OUT_OF_PAGES, "rollout: a sequence cannot be admitted");
    if (decode_step(nullptr, nullptr, nullptr) > 0)
      ++steps;
    else
      drain_eos();  // only finished sequences are left: settle their end-of-sequence checks
    collect();
  }
  mark(ev_end);
  cur_round_ev_ = nullptr;
  flush();
  HIP_TRY(hipStreamSynchronize(stream_));

  if (!st) return;
  const int32_t round_id = st->round_id, kind = st->kind;
  *st = rp_round_stats{};
  st->round_id = round_id;
  st->kind = kind;
  st->n_seqs = static_cast<int32_t>(members.size());
  st->decode_steps = steps;
  st->prompt_tokens = prompt_tokens;
  st->generated_tokens = gen_tokens;
  st->peak_pages = pool_.peak_used();
  st->preemptions = n_preempt_ - preempt0;
  st->recomputed_tokens = n_recompute_tok_ - recompute0;
  st->makespan_ms = mark_ms(ev_start, ev_end);
  st->prefill_ms = mark_ms(ev_start, ev_pre);
  st->decode_ms = st->makespan_ms - st->prefill_ms;
  double idle = 0.0;
  for (auto& le : left_ev) idle += std::max(0.0, mark_ms(le.first, ev_end)) * 1e-3;
  st->idle_slot_s = idle;
  const double denom = static_cast<double>(members.size()) * st->makespan_ms * 1e-3;
  st->slot_idle = denom > 0 ? idle / denom : 0.0;
}

int32_t Engine::rollout(int32_t n, const int64_t* ids, const int32_t* toks, const int64_t* offs,
                        const int32_t* max_new, uint64_t seed, float temp, const int32_t* round_ids,
                        int32_t* resp_out, float* logp_out, int32_t* len_out, rp_round_stats* stats,
                        int32_t max_stats) {
  if (live_count() != 0) throw RpError(RP_ERR_BAD_STATE, "rollout needs an engine without live sequences");
  if (n < 1 || !ids || !toks || !offs || !max_new || !resp_out)
    throw RpError(RP_ERR_INVALID_ARG, "rollout: null array or n < 1");
  std::vector<int64_t> resp_off;
  validate_seqs(n, ids, toks, offs, max_new, temp, resp_off);
  std::map<int32_t, std::vector<int32_t>> rounds;
  for (int32_t i = 0; i < n; ++i) rounds[round_ids ? round_ids[i] : 0].push_back(i);
  const SeqArrays arr{logp_out, ids, toks, offs, max_new, resp_off.data(), seed, temp};
  int32_t r_idx = 0;
  for (auto& kv : rounds) {
    rp_round_stats st{};
    st.round_id = kv.first;
    cur_round_ = kv.first;
    run_round(kv.second, arr, resp_out, len_out, nullptr, &st);
    cur_round_ = -1;
    if (stats && r_idx < max_stats) stats[r_idx] = st;
    ++r_idx;
  }
  return r_idx;
}

int32_t Engine::rollout_tail_batched(int32_t n_prompts, int32_t r_spec, const int64_t* ids, const int32_t* ptoks,
                                     const int64_t* poffs, const int32_t* max_new, uint64_t seed, float temp,
                                     int32_t P0, int32_t R0, float eta_p, float eta_r, int32_t* resp_out,
                                     float* logp_out, int32_t* gen_out,
                                     int32_t* accept_round_out, int32_t* kept_out, rp_round_stats* stats,
                                     int32_t max_stats) {
  if (live_count() != 0) throw RpError(RP_ERR_BAD_STATE, "rollout needs an engine without live sequences");
  if (n_prompts < 1 || r_spec < 1 || !ids || !ptoks || !poffs || !max_new || !resp_out || !gen_out ||
      !accept_round_out || !kept_out)
    throw RpError(RP_ERR_INVALID_ARG, "tail-batched rollout: null array or n_prompts < 1");
  if (P0 < 1 || R0 < 1 || !(eta_p >= 1.f) || !(eta_r >= 1.f) || std::isinf(eta_p) || std::isinf(eta_r) ||
      static_cast<double>(eta_p) * P0 > 1e9)
    throw RpError(RP_ERR_INVALID_ARG, "tail-batched rollout needs P0 >= 1, R0 >= 1 and finite eta_p, eta_r >= 1");
  if (r_spec != spec_count(eta_r, R0)) throw RpError(RP_ERR_INVALID_ARG, "r_spec must equal ceil(eta_r * R0)");
  if (static_cast<int64_t>(n_prompts) * r_spec > (int64_t{1} << 30))
    throw RpError(RP_ERR_INVALID_ARG, "too many responses");
  if (poffs[0] != 0) throw RpError(RP_ERR_INVALID_ARG, "prompt_offsets[0] must be 0");
  for (int32_t p = 0; p < n_prompts; ++p)
    if (poffs[p + 1] < poffs[p]) throw RpError(RP_ERR_INVALID_ARG, "prompt_offsets must be non-decreasing");

  // One sequence per (prompt, response), each with its own copy of the prompt.
  const int32_t n = n_prompts * r_spec;
  std::vector<int64_t> offs(static_cast<size_t>(n) + 1, 0);
  std::vector<int32_t> toks;
  toks.reserve(static_cast<size_t>(poffs[n_prompts]) * r_spec);
  for (int32_t p = 0; p < n_prompts; ++p)
    for (int32_t r = 0; r < r_spec; ++r) {
      toks.insert(toks.end(), ptoks + poffs[p], ptoks + poffs[p + 1]);
      offs[static_cast<size_t>(p) * r_spec + r + 1] = static_cast<int64_t>(toks.size());
    }
  std::vector<int64_t> resp_off;
  validate_seqs(n, ids, toks.data(), offs.data(), max_new, temp, resp_off);

  // A short round starts every launched response at once: check that each
  // one fits before anything runs.
  const int32_t p_spec = spec_count(eta_p, P0);
  for (int32_t p0 = 0; p0 < n_prompts; p0 += p_spec) {
    int64_t pages = 0, seqs = 0;
    for (int32_t p = p0; p < std::min(n_prompts, p0 + p_spec); ++p)
      for (int32_t r = 0; r < r_spec; ++r) {
        const size_t i = static_cast<size_t>(p) * r_spec + r;
        pages += admit_pages(offs[i + 1] - offs[i], max_new[i], offs[i + 1] - offs[i]);
        ++seqs;
      }
    if (seqs > lim_.max_seqs || pages > pool_.capacity())
      throw RpError(RP_ERR_CAPACITY, "a short round's responses do not fit max_seqs or the KV pool together");
  }

  const SeqArrays arr{logp_out, ids, toks.data(), offs.data(), max_new, resp_off.data(), seed, temp};
  for (int32_t p = 0; p < n_prompts; ++p) accept_round_out[p] = -1;
  for (int32_t i = 0; i < n; ++i) kept_out[i] = 0, gen_out[i] = 0;
  std::deque<int32_t> queue;  // prompts aborted by short rounds, oldest first
  int32_t next_fresh = 0, k = 0;
  while (next_fresh < n_prompts || !queue.empty()) {
    rp_round_stats st{};
    st.round_id = k;
    cur_round_ = k;
    std::vector<int32_t> launched, members;
    if (static_cast<int32_t>(queue.size()) >= P0 || (next_fresh >= n_prompts && !queue.empty())) {
      // Long round: the oldest queued prompts, R0 responses each, no speculation.
      st.kind = 1;
      while (!queue.empty() && static_cast<int32_t>(launched.size()) < P0) {
        launched.push_back(queue.front());
        queue.pop_front();
      }
      std::sort(launched.begin(), launched.end());
      for (int32_t p : launched)
        for (int32_t r = 0; r < R0; ++r) members.push_back(p * r_spec + r);
      run_round(members, arr, resp_out, gen_out, nullptr, &st);
      for (int32_t p : launched) {
        accept_round_out[p] = k;
        for (int32_t r = 0; r < R0; ++r) kept_out[p * r_spec + r] = 1;
      }
    } else {
      // Short round: race to completion among the next ceil(eta_p * P0) fresh prompts.
      st.kind = 0;
      for (int32_t j = 0; j < p_spec && next_fresh < n_prompts; ++j) launched.push_back(next_fresh++);
      Race race;
      race.n_prompts = static_cast<int32_t>(launched.size());
      race.R0 = R0;
      race.keep = std::min(P0, race.n_prompts);
      for (int32_t j = 0; j < race.n_prompts; ++j)
        for (int32_t r = 0; r < r_spec; ++r) {
          members.push_back(launched[j] * r_spec + r);
          race.prompt.push_back(j);
        }
      run_round(members, arr, resp_out, gen_out, &race, &st);
      for (int32_t j = 0; j < race.n_prompts; ++j) {
        const int32_t p = launched[j];
        if (race.accepted[j]) {
          accept_round_out[p] = k;
          for (int32_t r = 0; r < r_spec; ++r) kept_out[p * r_spec + r] = race.kept[j * r_spec + r];
        } else {
          queue.push_back(p);
        }
      }
    }
    cur_round_ = -1;
    if (stats && k < max_stats) stats[k] = st;
    ++k;
  }
  return k;
}

}  // namespace rollpack
