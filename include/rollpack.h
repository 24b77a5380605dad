/*
 * rollpack.h -- C ABI of the MI355X rollout library.
 *
 * Rollout is the generation stage of synchronous RL post-training (paper
 * section 2.1): the actor model receives P0 prompts and produces R0
 * responses for each, and the stage must finish before training starts.
 * Response lengths are long-tailed (section 2.2), so a batch shrinks as short
 * responses finish while the longest keep the GPU busy; tail batching
 * (section 3) groups prompts into balanced short rounds and consolidated long
 * rounds.  This library generates responses for a batch of sequences with a
 * Qwen2.5-style decoder on one gfx950 GPU and plans tail-batched rounds.
 *
 * Conventions for every call:
 *  - Device pointers are HIP device addresses; host pointers are ordinary
 *    process memory.  Each argument says which it is.
 *  - The caller owns every buffer (weights, KV pool, scratch workspace,
 *    outputs).  Device buffers passed to rp_engine_create must stay valid
 *    until rp_engine_destroy.  Host arrays are read only during the call.
 *    The engine never allocates device memory.
 *  - Every call returns rp_status.  On failure a message is available from
 *    rp_last_error() (thread-local) and the engine state is unchanged,
 *    except after RP_ERR_HIP, which leaves the engine unusable.
 *  - All device work is ordered on the stream given at creation.  A call
 *    returns once its host-visible outputs are ready; device outputs are
 *    ready in stream order.  An engine is not thread-safe.
 *  - Sequences are identified by caller-chosen 64-bit ids, unique among the
 *    engine's live sequences.  The id keys the sampling noise, so a
 *    sequence's tokens do not depend on batching or scheduling.
 */
#ifndef ROLLPACK_H
#define ROLLPACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rp_status {
  RP_OK = 0,
  RP_ERR_INVALID_ARG = 1,   /* a size, pointer or value is out of range */
  RP_ERR_OUT_OF_PAGES = 2,  /* the KV pool cannot hold the admitted sequences */
  RP_ERR_DUPLICATE_ID = 3,  /* a sequence id is already live */
  RP_ERR_UNKNOWN_ID = 4,    /* a sequence id is not live */
  RP_ERR_BAD_STATE = 5,     /* the call does not fit the engine's state */
  RP_ERR_HIP = 6,           /* a HIP runtime call failed */
  RP_ERR_CAPACITY = 7       /* more sequences, tokens or context than the limits allow */
} rp_status;

typedef enum rp_dtype {
  RP_DTYPE_F32 = 0,   /* weights, GEMM inputs and KV in fp32 */
  RP_DTYPE_BF16 = 1   /* weights, GEMM inputs and KV in bf16; fp32 accumulation,
                         residual stream, norms, softmax and logits */
} rp_dtype;

/* Qwen2.5 decoder shape (the paper's models, section 6).  q/k/v carry a
 * bias, o/gate/up/down do not; RMSNorm with eps; rotate-half RoPE with base
 * rope_theta; query head h reads KV head h / (n_q_heads / n_kv_heads). */
typedef struct rp_model_config {
  int32_t n_layers;
  int32_t hidden;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;          /* 64 or 128 */
  int32_t intermediate;
  int32_t vocab;
  float rms_eps;
  float rope_theta;
  int32_t tied_embeddings;   /* 1: the LM head is the embedding matrix */
  int32_t dtype;             /* rp_dtype */
} rp_model_config;

/* Device pointers to one layer's tensors, element type = config dtype,
 * [out, in] row-major: wq [n_q*hd, H], wk/wv [n_kv*hd, H], wo [H, n_q*hd],
 * w_gate/w_up [I, H], w_down [H, I]; bq [n_q*hd], bk/bv [n_kv*hd];
 * attn_norm/mlp_norm [H]. */
typedef struct rp_layer_weights {
  const void* attn_norm;
  const void* wq;
  const void* bq;
  const void* wk;
  const void* bk;
  const void* wv;
  const void* bv;
  const void* wo;
  const void* mlp_norm;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
} rp_layer_weights;

typedef struct rp_weights {
  const void* embed;                /* device [V, H] */
  const void* final_norm;           /* device [H] */
  const void* lm_head;              /* device [V, H]; NULL when tied */
  const rp_layer_weights* layers;   /* HOST array [n_layers], copied at create */
} rp_weights;

typedef struct rp_engine_limits {
  int32_t max_seqs;            /* sequences live at once (KV slots), >= 1 */
  int32_t max_prefill_tokens;  /* tokens per prefill chunk; a longer prompt is prefilled in
                                  pieces that continue at their positions */
  int32_t max_context;         /* longest prompt + response, <= 65536 */
  int32_t page_tokens;         /* tokens per KV page; must be 64 */
  int64_t kv_pages;            /* pages in the KV pool */
} rp_engine_limits;

typedef struct rp_engine rp_engine;

/* Per-round measurements of rp_rollout_generate.  Times come from HIP events
 * on the engine's stream.  slot_idle is the fraction of sequence-slot time
 * spent after a sequence finished while its round was still running: the
 * bubble of section 2.2 counted per sequence slot. */
typedef struct rp_round_stats {
  int32_t round_id;
  int32_t n_seqs;
  int32_t decode_steps;
  int32_t kind;            /* 0: plain or short (speculative) round, 1: long round */
  int64_t prompt_tokens;
  int64_t generated_tokens;
  int64_t peak_pages;
  double makespan_ms;      /* first prefill kernel to the last token of the round */
  double prefill_ms;
  double decode_ms;
  double slot_idle;        /* in [0, 1] */
  double idle_slot_s;      /* sum over sequences of (round end - own finish), seconds */
  int64_t preemptions;     /* sequences preempted during the round (RP_KV_ON_DEMAND) */
  int64_t recomputed_tokens; /* tokens re-prefilled to resume them */
} rp_round_stats;

/* Bytes of the caller-provided KV pool and scratch workspace for this model
 * and these limits.  Paper: the KV cache is the memory that long responses
 * fill and whose shortage causes preemptions (section 4.2); the pool is sized
 * here by the caller, in 64-token pages.  kv_bytes covers limits->kv_pages pages; both are
 * multiples of 256. */
rp_status rp_workspace_size(const rp_model_config* cfg, const rp_engine_limits* limits,
                            size_t* kv_bytes, size_t* scratch_bytes);

/* Bytes of KV cache one token occupies (all layers, K and V); the unit of the
 * KV footprint projected per request (section 4.4). */
rp_status rp_kv_bytes_per_token(const rp_model_config* cfg, size_t* bytes);

/* Create an engine over caller-owned device memory: one rollout instance
 * holding the actor model's weights (section 2.1) that requests are added to
 * and aborted from (section 5, add_request / abort_request).  kv_ws/scratch_ws must
 * be at least the sizes rp_workspace_size returns and 256-byte aligned;
 * hip_stream is a hipStream_t (NULL = default stream).  The weights are not
 * copied; their device memory must outlive the engine. */
rp_status rp_engine_create(const rp_model_config* cfg, const rp_weights* weights,
                           const rp_engine_limits* limits, void* kv_ws, size_t kv_bytes,
                           void* scratch_ws, size_t scratch_bytes, void* hip_stream,
                           rp_engine** out);

void rp_engine_destroy(rp_engine* eng);

/* Bytes of the packed copy of a bf16 model's decode weights (every q/k/v, o,
 * gate, up and down projection and the LM head, each 256-byte aligned), the
 * stream every memory-bound decode step reads (section 2.2); 0 for an fp32
 * model. */
rp_status rp_packed_weights_bytes(const rp_model_config* cfg, size_t* bytes);

/* Give the engine a caller-owned device workspace of at least
 * rp_packed_weights_bytes bytes (256-byte aligned) for a packed copy of its
 * weights.  Decoding is memory-bound (section 2.2): each decode step streams
 * every weight once, and the copy lays each 16-row by 64-column block of a
 * weight matrix out as the two contiguous 1 KB runs that one wave's loads
 * read, so the decode GEMMs (16-64 live rows) stream it with non-temporal
 * 1 KB loads; the products are bit-identical to those of the row-major
 * weights.  The packing runs on the engine's stream (one read of the
 * weights); the workspace must stay valid until the engine is destroyed or
 * this call is made again.  packed_ws NULL goes back to the row-major
 * weights.  Prefill and batches above 64 rows keep reading the caller's
 * row-major weights.  Errors: RP_ERR_INVALID_ARG for an fp32 model, a small
 * or misaligned workspace. */
rp_status rp_engine_set_packed_weights(rp_engine* eng, void* packed_ws, size_t bytes);

/* Admit n sequences and run their prompts through the model (prefill), then
 * sample each sequence's first response token.  Paper: the actor is given
 * prompts and generates responses for them (section 2.1); admitting a request
 * is section 5's add_request.
 *   seq_ids         host [n], new unique ids
 *   prompt_tokens   host, all prompts concatenated (CSR), ids in [0, V)
 *   prompt_offsets  host [n+1], prompt i is tokens [off[i], off[i+1]), length >= 1
 *   max_new_tokens  host [n], >= 1: every generated token counts, the one
 *                   sampled here included; generation stops there (forced
 *                   lengths, no end-of-sequence token)
 *   seed, temperature: the sampling key and temperature of these sequences;
 *                   temperature 0 is greedy
 *   logits_out      DEVICE [n, V] fp32 or NULL: logits of each prompt's last position
 *   first_tokens_out HOST [n] or NULL: the sampled first tokens (synchronises)
 * Under RP_KV_RESERVE, KV pages for prompt + max_new_tokens - 1 positions
 * are reserved at admission; under RP_KV_ON_DEMAND only the prompt's pages
 * are taken.  RP_ERR_OUT_OF_PAGES if the pool cannot hold them. */
rp_status rp_prefill(rp_engine* eng, int32_t n, const int64_t* seq_ids,
                     const int32_t* prompt_tokens, const int64_t* prompt_offsets,
                     const int32_t* max_new_tokens, uint64_t seed, float temperature,
                     float* logits_out, int32_t* first_tokens_out);

/* One decode step for every live, unfinished sequence ("row"), rows in
 * admission order: the autoregressive generation step of rollout (section
 * 2.1), memory-bound at these batch sizes (section 2.2).  Each row feeds its last sampled token (or
 * forced_tokens[row], teacher forcing: the input changes, the sampled history
 * does not), appends its K/V, and samples its next token.
 *   forced_tokens   HOST [n_active] or NULL
 *   logits_out      DEVICE [n_active, V] fp32 or NULL
 *   row_ids_out     HOST [max_seqs] or NULL: the sequence id of each row
 *   n_active_out    HOST, the number of rows in this step (0: nothing to do)
 * A sequence that reaches its max_new_tokens becomes finished and keeps its
 * pages until rp_free_finished.
 * Under RP_KV_ON_DEMAND the step first resumes preempted sequences that fit
 * (oldest arrival first; each is recomputed by a prefill of its prompt and
 * generated tokens, which samples its next token, so it is not among this
 * step's rows), then gives each row a page for its next position, preempting
 * the latest-arrived rows while the pool is short.  forced_tokens must be
 * NULL under that policy. */
rp_status rp_decode_step(rp_engine* eng, const int32_t* forced_tokens, float* logits_out,
                         int64_t* row_ids_out, int32_t* n_active_out);

/* Release the KV pages and slots of finished sequences and report their ids
 * (host [cap]).  Paper: finished requests leave the running set, so the
 * batch shrinks as short responses complete (section 2.2; Algorithm 1's
 * generate returns the finished requests).  The tokens of a released sequence are no longer available. */
rp_status rp_free_finished(rp_engine* eng, int64_t* finished_ids_out, int32_t cap,
                           int32_t* n_finished_out);

/* Stop live (or preempted) sequences now and release them: the speculative
 * abort of tail batching (section 3), section 5's abort_request. */
rp_status rp_abort(rp_engine* eng, int32_t n, const int64_t* seq_ids);

/* Copy the generated tokens of a live (or preempted) sequence to host out
 * [cap] (the responses rollout hands to the reward stage, section 2.1); len_out gets the number generated so far.  Synchronises the stream. */
rp_status rp_get_tokens(rp_engine* eng, int64_t seq_id, int32_t* out, int32_t cap,
                        int32_t* len_out);

/* The same for the log-probability of each generated token under the
 * distribution it was sampled from (the training stage of section 2.1
 * updates the actor from its responses), log softmax(logits / T)[token]
 * (T = 1 for greedy sequences), as RL training needs for its importance
 * ratios; fp32, from the logits the step computed. */
rp_status rp_get_logprobs(rp_engine* eng, int64_t seq_id, float* out, int32_t cap,
                          int32_t* len_out);

/* End-of-sequence token (-1, the default: none); response lengths are what
 * the model decides, long-tailed (section 2.2).  A sequence that samples it
 * stops there, the token included, before max_new_tokens.  The engine reads
 * each step's sampled tokens two steps later, so that it never waits on the
 * step just launched: a stopped sequence may take part in one more step,
 * whose token is discarded, and is reported finished by rp_free_finished
 * (which reads every pending check first).  Responses equal the forced-length
 * ones cut after their first end-of-sequence token, since tokens are keyed by
 * position.  The engine must have no live sequences (RP_ERR_BAD_STATE). */
rp_status rp_set_eos(rp_engine* eng, int32_t eos_token);

/* Whole-batch rollout on an engine: the rollout stage of section 2.1 (P0
 * prompts x R0 responses, one sequence each) run as the rounds of section 3
 * when round_ids are given.  Generate max_new_tokens[i] tokens for each of n
 * sequences, round by round (rounds in increasing round_ids order; NULL =
 * one round).  Within a round all sequences are admitted together (prefill
 * in chunks), then decoded until the last one finishes, freeing KV pages as
 * sequences finish so the batch shrinks.
 *   seq_ids, prompt_tokens, prompt_offsets, max_new_tokens: as rp_prefill
 *   round_ids       host [n] or NULL
 *   resp_tokens_out host [sum max_new_tokens]: sequence i's tokens at
 *                   offset sum_{j<i} max_new_tokens[j]
 *   resp_logprobs_out host [sum max_new_tokens] or NULL: the log-probability
 *                   of each token, laid out like the tokens (rp_get_logprobs)
 *   resp_len_out    host [n] or NULL: tokens generated, max_new_tokens[i]
 *                   unless the sequence stopped at the end-of-sequence token
 *                   (rp_set_eos); entries past it are left untouched
 *   stats_out       host [max_stats] or NULL: one record per round, in order
 *   n_rounds_out    host or NULL
 * The engine must have no live sequences. */
rp_status rp_rollout_generate(rp_engine* eng, int32_t n, const int64_t* seq_ids,
                              const int32_t* prompt_tokens, const int64_t* prompt_offsets,
                              const int32_t* max_new_tokens, uint64_t seed, float temperature,
                              const int32_t* round_ids, int32_t* resp_tokens_out,
                              float* resp_logprobs_out, int32_t* resp_len_out,
                              rp_round_stats* stats_out, int32_t max_stats,
                              int32_t* n_rounds_out);

/* How rp_generate groups its sequences into rounds. */
typedef enum rp_schedule_mode {
  RP_SCHEDULE_NONE = 0,           /* every sequence in one batch (round_ids must be NULL) */
  RP_SCHEDULE_ROUNDS = 1,         /* the caller's rounds, round_ids[i] per sequence */
  RP_SCHEDULE_TAIL_BATCHING = 2   /* tail batching run online (section 3), with rp_tail_params */
} rp_schedule_mode;

/* Tail-batching parameters (section 3; eta_p and eta_r vary separately in
 * section 6.3).  r_spec = ceil(eta_r * R0) candidate responses per prompt. */
typedef struct rp_tail_params {
  int32_t P0;       /* prompts kept per short round */
  int32_t R0;       /* responses kept per prompt */
  int32_t r_spec;   /* responses launched per prompt */
  float eta_p;      /* prompt speculation factor, >= 1 */
  float eta_r;      /* response speculation factor, >= 1 */
} rp_tail_params;

/* One-shot rollout in the form of the problem statement (section 2.1: the
 * actor is given P0 prompts and produces R0 responses for each; Algorithm 1's
 * LLM.generate returns the finished requests): create an engine over the
 * caller's workspaces, generate every response, destroy the engine.
 *   cfg, weights, limits, kv_ws, kv_bytes, scratch_ws, scratch_bytes,
 *   hip_stream      as rp_engine_create (the workspaces are free again when
 *                   the call returns)
 *   n, seq_ids, prompt_tokens, prompt_offsets, max_new_tokens, seed,
 *   temperature     as rp_rollout_generate; under RP_SCHEDULE_TAIL_BATCHING
 *                   as rp_rollout_tail_batched: n = n_prompts * tail->r_spec,
 *                   prompt_offsets has n_prompts + 1 entries (CSR over prompts)
 *   schedule_mode   rp_schedule_mode
 *   round_ids       host [n] under RP_SCHEDULE_ROUNDS, else NULL
 *   tail            host, under RP_SCHEDULE_TAIL_BATCHING, else NULL
 *   resp_tokens_out, resp_logprobs_out (nullable), resp_len_out (nullable,
 *                   except under RP_SCHEDULE_TAIL_BATCHING), stats_out
 *                   (nullable), max_stats, n_rounds_out (nullable): as the
 *                   engine call of the mode
 *   kept_out        host [n] or NULL: 1 for the responses tail batching keeps
 *                   (every response under the other modes)
 * Errors: those of rp_engine_create and of the engine call; no device memory
 * is allocated and nothing is left behind on failure. */
rp_status rp_generate(const rp_model_config* cfg, const rp_weights* weights, const rp_engine_limits* limits,
                      void* kv_ws, size_t kv_bytes, void* scratch_ws, size_t scratch_bytes, void* hip_stream,
                      int32_t n, const int64_t* seq_ids, const int32_t* prompt_tokens,
                      const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed,
                      float temperature, int32_t schedule_mode, const int32_t* round_ids,
                      const rp_tail_params* tail, int32_t* resp_tokens_out, float* resp_logprobs_out,
                      int32_t* resp_len_out, int32_t* kept_out, rp_round_stats* stats_out, int32_t max_stats,
                      int32_t* n_rounds_out);

/* rp_generate for callers that cannot allocate: code that runs where
 * hipMalloc, pinned host allocations or event creation are not allowed, tight
 * serving loops, harnesses that forbid allocation.  The arguments and outputs
 * are rp_generate's without the two workspaces: the KV pool and the scratch
 * workspace come from one device array that the library holds, 64 MiB
 * (67,108,864 bytes) per GPU until the process ends, on the current device
 * (hip_stream, when not NULL, must belong to it).  The call makes no
 * allocating HIP call: staging goes through ordinary host memory and waits
 * are stream synchronisations, so it is slower per step than rp_generate,
 * and the round times in stats_out come from the host clock.
 *   Limits: kv_bytes + scratch_bytes of rp_workspace_size for these limits
 *   must not exceed the array (RP_ERR_CAPACITY otherwise, with the sizes in
 *   the message); about the tiny model or a few 0.5B-shape sequences of a
 *   few hundred tokens.
 *   Sharing: every call on a GPU uses that GPU's one array, which keeps the
 *   last call's contents; the engine clears what must start at zero (the KV
 *   pool, the page table, the current tokens).  Calls in one process are
 *   serialised by a lock; overlapping calls on one GPU from code that
 *   bypassed it would race on the array. */
rp_status rp_generate_static(const rp_model_config* cfg, const rp_weights* weights,
                             const rp_engine_limits* limits, void* hip_stream, int32_t n,
                             const int64_t* seq_ids, const int32_t* prompt_tokens,
                             const int64_t* prompt_offsets, const int32_t* max_new_tokens, uint64_t seed,
                             float temperature, int32_t schedule_mode, const int32_t* round_ids,
                             const rp_tail_params* tail, int32_t* resp_tokens_out,
                             float* resp_logprobs_out, int32_t* resp_len_out, int32_t* kept_out,
                             rp_round_stats* stats_out, int32_t max_stats, int32_t* n_rounds_out);

/* Tail batching run online on the engine (section 3).  n_prompts prompts,
 * submitted in order, each with r_spec = ceil(eta_r * R0) candidate responses;
 * response r of prompt p is sequence seq_ids[p * r_spec + r] with forced
 * length max_new_tokens[p * r_spec + r] and its own copy of prompt p.
 * Rounds follow the policy of rp_plan_tail_batching, but completion is
 * observed on the engine step by step:
 *   short round  the next ceil(eta_p * P0) fresh prompts start all their
 *                responses together (all must fit max_seqs and the KV pool at
 *                once, checked for every short round before anything runs:
 *                RP_ERR_CAPACITY).  When a prompt has R0 finished responses
 *                and fewer than P0 prompts are accepted, it is accepted with
 *                those R0 responses (lower response index first on a tie) and
 *                its other responses are aborted at once.  The round ends
 *                when P0 prompts are accepted (prompts completing in the same
 *                step: lower index first); every response still running is
 *                aborted, its pages freed, and its prompt queued.
 *   long round   when P0 prompts are queued, or no fresh prompt is left,
 *                up to P0 of the oldest queued prompts run responses
 *                0..R0-1 to completion, with no speculation.  They start from
 *                the prompt again: tokens are keyed by (seed, seq_id,
 *                position), so the tokens an aborted response had produced
 *                are produced again.
 *   seq_ids         host [n_prompts * r_spec], unique
 *   prompt_tokens   host, CSR over prompts with prompt_offsets [n_prompts + 1]
 *   resp_tokens_out host [sum max_new_tokens]: response i's tokens at offset
 *                   sum_{j<i} max_new_tokens[j]; only its first resp_len_out[i]
 *                   entries are written
 *   resp_logprobs_out host [sum max_new_tokens] or NULL: their log-probabilities
 *   resp_len_out    host [n_prompts * r_spec]: tokens the response generated in
 *                   the last round it ran in (0 if never launched)
 *   accept_round_out host [n_prompts]: round that accepted the prompt
 *   kept_out        host [n_prompts * r_spec]: 1 for the R0 responses kept per prompt
 *   stats_out       host [max_stats] or NULL: one record per round, round_id =
 *                   round index, kind 0 short / 1 long; idle time counts each
 *                   response from the moment it finished or was aborted
 *   n_rounds_out    host or NULL
 * The engine must have no live sequences.  Other errors as rp_rollout_generate. */
rp_status rp_rollout_tail_batched(rp_engine* eng, int32_t n_prompts, int32_t r_spec,
                                  const int64_t* seq_ids, const int32_t* prompt_tokens,
                                  const int64_t* prompt_offsets, const int32_t* max_new_tokens,
                                  uint64_t seed, float temperature, int32_t P0, int32_t R0,
                                  float eta_p, float eta_r,
                                  int32_t* resp_tokens_out, float* resp_logprobs_out,
                                  int32_t* resp_len_out,
                                  int32_t* accept_round_out, int32_t* kept_out,
                                  rp_round_stats* stats_out, int32_t max_stats,
                                  int32_t* n_rounds_out);

/* Tail-batching plan (section 3), host only.  n_prompts prompts, submitted
 * in order, each with r_spec = ceil(eta_r * R0) candidate responses of known
 * lengths lens[p * r_spec + r], counted in generation steps of one token
 * each (the first token is the prefill's sample).  eta_p and eta_r are the
 * speculation factors for prompts and responses (section 6.3 varies them
 * separately; a product within one part in 10^6 of an integer counts as that
 * integer).  A short round launches the next ceil(eta_p * P0) fresh prompts
 * and keeps the first P0 to have R0 finished responses (ties: lower index), each with its R0 shortest
 * responses; the round ends when its P0-th prompt completes and the other
 * prompts join a FIFO long-prompt queue.  When the queue holds P0 prompts,
 * or no fresh prompt is left, a long round runs up to P0 queued prompts with
 * R0 responses each and no speculation.
 *   round_kind_out  host [max_rounds]: 0 short, 1 long
 *   round_time_out  host [max_rounds]: round length in generation steps (an
 *                   engine runs it in round_time - 1 decode steps)
 *   launch_off_out  host [max_rounds + 1]: CSR offsets into launch_prompt_out
 *   launch_prompt_out host [cap_launch]: prompts launched per round, ascending
 *   run_steps_out   host [cap_launch * r_spec]: tokens each launched response generated
 *                   (responses r >= R0 of a long round run 0 steps)
 *   accept_round_out host [n_prompts]: round that accepted each prompt
 *   kept_out        host [n_prompts * r_spec]: 1 if the response is kept
 *   n_rounds_out    host */
rp_status rp_plan_tail_batching(int32_t n_prompts, int32_t r_spec, const int32_t* lens,
                                int32_t P0, int32_t R0, float eta_p, float eta_r, int32_t max_rounds,
                                int32_t cap_launch, int32_t* round_kind_out,
                                int32_t* round_time_out, int32_t* launch_off_out,
                                int32_t* launch_prompt_out, int32_t* run_steps_out,
                                int32_t* accept_round_out, int32_t* kept_out,
                                int32_t* n_rounds_out);

/* KV page policy of an engine (section 4.2: KV memory pressure causes
 * preemptions, and their count is the pressure signal). */
typedef enum rp_kv_policy {
  RP_KV_RESERVE = 0,    /* reserve every page a sequence will need at admission (default) */
  RP_KV_ON_DEMAND = 1   /* take a page when a sequence's context crosses into it; when
                           none is free, preempt the latest-arrived running sequence and
                           later resume it by recomputing its KV from its tokens */
} rp_kv_policy;

/* Set the KV page policy (rp_kv_policy): reservation, or pages on demand with
 * preemption under KV pressure (section 4.2) and resume by recomputation
 * (the recomputation-based migration of section 5).  The engine must have no live or
 * preempted sequences (RP_ERR_BAD_STATE). */
rp_status rp_set_kv_policy(rp_engine* eng, int32_t policy);

/* Pool and scheduler state (the preemption count is section 4.2's
 * KV-pressure signal); every output is nullable.  Counters accumulate
 * over the engine's life. */
rp_status rp_kv_status(rp_engine* eng, int64_t* free_pages, int32_t* running,
                       int32_t* waiting, int64_t* preemptions, int64_t* recomputed_tokens);

/* Kernel classes of the rollout step, for rp_profile_* (bit i of a mask = class i). */
typedef enum rp_kernel_class {
  RP_K_EMBED_NORM = 0,   /* embedding gather + first RMSNorm */
  RP_K_ADD_NORM = 1,     /* residual add of split-K partials + RMSNorm */
  RP_K_GEMM_QKV = 2,
  RP_K_ROPE_APPEND = 3,  /* q/k/v bias + RoPE + paged KV append */
  RP_K_ATTN = 4,         /* prefill or decode attention */
  RP_K_ATTN_MERGE = 5,   /* decode split merge */
  RP_K_GEMM_O = 6,
  RP_K_GEMM_GATE_UP = 7, /* with the SiLU * up epilogue */
  RP_K_GEMM_DOWN = 8,
  RP_K_GEMM_LM_HEAD = 9,
  RP_K_SAMPLE = 10,
  RP_K_COUNT = 11
} rp_kernel_class;

/* Accumulated measurements of one kernel class in one phase.  bytes and
 * flops are the algorithmic amounts the launches had to move / compute
 * (weights, activations, KV actually attended, outputs; split-K partials are
 * counted once), not hardware counters. */
typedef struct rp_kernel_stats {
  int32_t kernel_class;  /* rp_kernel_class */
  int32_t phase;         /* 0 prefill, 1 decode */
  int64_t launches;
  double total_ms;       /* sum of per-launch HIP event intervals on the engine stream */
  double bytes;
  double flops;
} rp_kernel_stats;

/* Per-kernel timing, the measurement side of the paper's offline profiling
 * phase (section 4.1: prefill and decode throughput against batch size and
 * sequence length).  class_mask selects the classes whose launches are timed
 * from now on (0 stops): the launch's own dispatch stamps a pair of HIP
 * events with its first kernel's start and its last kernel's end.  Timing
 * adds a little host work per selected launch, and the stamped dispatches
 * cost the GPU a few microseconds each; unselected launches are untouched.
 * Every class starts timing all of its launches (see rp_profile_every). */
rp_status rp_profile_enable(rp_engine* eng, uint32_t class_mask);

/* Time only one launch in `every` (>= 1) of each selected class (the
 * profiling of section 4.1, sampled): the first,
 * then every `every`-th, counted per class and phase from this call.  The
 * statistics then cover the timed launches only (launches, total_ms, bytes
 * and flops alike), so averages stay unbiased when the sampled launches
 * spread over the workload.  RP_ERR_INVALID_ARG for every < 1. */
rp_status rp_profile_every(rp_engine* eng, int32_t every);

/* Synchronise, then report and reset the accumulated measurements of the
 * section 4.1 profiling: one
 * record per (class, phase) with launches > 0, into host out [cap]. */
rp_status rp_profile_read(rp_engine* eng, rp_kernel_stats* out, int32_t cap, int32_t* n_out);

/* The practical HBM read ceiling that measurement reports next to the nominal
 * peak (the roofline of the memory-bound decode kernels, section 2.2): streams the
 * caller's device buffer dev_buf (bytes >= 1 MiB, 16-byte aligned; its
 * contents are read, never written) reps times with a read-only kernel in
 * which each of 2048 waves walks its own contiguous share with 8 one-KB
 * non-temporal loads in flight, on hip_stream, and returns
 * the fastest pass in GB/s (1e9 bytes/s) through gbs_out.  Blocks the calling
 * thread; needs no engine and allocates no device memory.  A buffer larger
 * than the 256 MB last-level cache measures HBM.  Errors: RP_ERR_INVALID_ARG
 * on bad arguments, RP_ERR_HIP if a launch or event call fails. */
rp_status rp_stream_read_gbs(const void* dev_buf, size_t bytes, int32_t reps, void* hip_stream, double* gbs_out);

/* One step of the engine: a decode step over `rows` sequences with
 * `sum_ctx` context tokens in total, or one prefill chunk of `rows` tokens
 * (sum_ctx then counts the keys its queries attend to).  ms is the HIP-event
 * time from the step's first launch to its sampler's end on the engine's
 * stream; round_id is the round of rp_rollout_generate /
 * rp_rollout_tail_batched that ran it (-1 outside a rollout call). */
typedef struct rp_step_record {
  int32_t kind;      /* 0 decode step, 1 prefill chunk */
  int32_t round_id;
  int32_t rows;
  int32_t reserved;
  int64_t sum_ctx;
  double ms;
  double end_ms;     /* from the start of its round (the round's makespan origin) to the end of
                        this step; -1 outside a rollout call.  A sequence's finish time in the
                        round statistics is end_ms of the step that produced its last token. */
} rp_step_record;

/* Per-step trace, the measurement behind the paper's step-time profiles
 * (section 4.1) and the round metrics: from now on record up to `cap` steps
 * (0 stops and discards the trace).  Two HIP events bracket each step. */
rp_status rp_step_trace_enable(rp_engine* eng, int32_t cap);

/* Synchronise, then copy the recorded steps (section 4.1's step-time
 * profile) to host out [cap] in order and clear the trace; n_out gets the number copied (steps beyond the enabled
 * capacity are not recorded). */
rp_status rp_step_trace_read(rp_engine* eng, rp_step_record* out, int32_t cap, int32_t* n_out);

/* Message of the last failed call on this thread ("" if none). */
const char* rp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ROLLPACK_H */
