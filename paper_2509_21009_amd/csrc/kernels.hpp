// Kernel launchers of the rollout path (host-callable, gfx950 device code).
//
// Data layout in HBM (all row-major):
//   x      fp32 [M, H]               residual stream
//   h      T    [M, H]               normalised GEMM input (T = float or bf16)
//   part   fp32 [S, M, N]            split-K partial GEMM outputs, summed by the consumer
//   q      T    [M, n_q, hd]         rotated queries
//   K pool fp32 [layer][page][n_kv][64 tokens][hd]
//          bf16 [layer][page][n_kv][64 x hd in MFMA operand order, k_page_offset]
//   V pool T    [layer][page][n_kv][2 halves][hd][32 tokens]   (transposed per half page)
//   page table int32 [slot][max_pages_per_seq]
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rollpack {

// Events that the next kernel launches of this thread stamp from their own
// dispatch (hipExtLaunchKernelGGL), for timing without marker packets
// between kernels: the first launch after they are set stamps `start` (and
// clears it), every launch stamps `stop`, so a launcher of several kernels is
// timed from the first one's start to the last one's end.  With `stop` null,
// launches are plain.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();  // this thread's

template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  LaunchEvents& ev = launch_events();
  if (ev.stop) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev.start, ev.stop, 0, args...);
    ev.start = nullptr;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
}

constexpr int kPageTokens = 64;

// Element offset of (token tok of the page, dimension d) inside one
// (page, KV head) block of the bf16 K cache.  The block is stored in the
// order the attention kernels feed it to v_mfma_f32_16x16x32_bf16 as the
// 16-row operand: [half page h][tile tt][k-step ks][row c][lane group g][8],
// where row c of tile tt of half h is token 32h + 8(c >> 2) + 4tt + (c & 3)
// and k-step ks, group g hold dimensions 32ks + 8g .. 32ks + 8g + 7.  One
// (h, tt, ks) triple is then one contiguous 1 KB run that a wave's single
// 16-byte-per-lane load covers in whole 128-byte lines.
__host__ __device__ __forceinline__ int k_page_offset(int tok, int d, int hd) {
  const int h = tok >> 5, r = tok & 31;
  const int tt = (r >> 2) & 1, c = ((r >> 3) << 2) | (r & 3);
  const int ks = d >> 5, g = (d >> 3) & 3, e = d & 7;
  return ((((h * 2 + tt) * (hd / 32) + ks) * 16 + c) * 4 + g) * 8 + e;
}

// Weight rows split over up to three tensors (q/k/v, or gate/up).  Each
// segment holds `rows` rows of K elements; rows are multiples of 16.
struct WSeg {
  const void* ptr[3];
  int32_t rows[3];
  int32_t n_seg;
};

enum GemmEpilogue { kEpiPartial = 0, kEpiSiluMul = 1 };

struct GemmArgs {
  const void* A;     // [M, lda] activations (dtype T)
  int64_t lda;
  int M, N, K;       // N: output columns (for kEpiSiluMul: I, with W = {gate, up})
  WSeg W;
  WSeg Wp;           // the same segments in the packed layout of launch_pack_weights (n_seg 0: none);
                     // the decode-regime deep kernel reads them when present
  int epi;
  int splits;        // S >= 1; kEpiSiluMul requires 1
  float* part;       // [S, M, N] (kEpiPartial)
  void* act_out;     // [M, N] dtype T (kEpiSiluMul)
  int variant;       // 0: automatic; 1 stream, 2/3 skinny (16/32 rows per wave), 4 tiled, 6 deep
};

// Packed weight layout for the decode GEMM (bf16, rows % 16 == 0, K % 64 == 0):
// 16-byte piece [t][u][j][l] = W[16t + (l & 15)][64u + 16(l >> 4) + 8j .. + 8],
// for row tile t, 64-wide K unit u, half j and lane l.  A (tile, unit) pair is
// one contiguous 2 KB run, and each half of it is the 1 KB that one wave
// instruction loads: lane l gets exactly the MFMA operand it reads from the
// row-major matrix, so the products are unchanged.  Tile t starts at byte
// 32 t K, where row 16t starts in the row-major matrix.
hipError_t launch_pack_weights(const void* w, void* packed, int rows, int K, hipStream_t s);

// Picks the kernel from dtype, M, N and K.  Returns hipSuccess or a launch error.
hipError_t launch_gemm(int dtype_bf16, const GemmArgs& a, hipStream_t s);
// K-split count the launcher plans for this shape (1 = none, never an empty split).
int gemm_pick_splits(int dtype_bf16, int M, int N, int K, bool silu, int max_splits);

struct EmbedArgs {
  const void* embed; const void* norm_g;
  const int32_t* in_tok;     // [M]; < 0: take tokens_cur[row_slot[i]]
  const int32_t* row_slot;   // [M] (only read when in_tok < 0)
  const int32_t* tokens_cur; // [slots]
  int M, H; float eps;
  float* x; void* h;
};
hipError_t launch_embed_norm(int bf16, const EmbedArgs& a, hipStream_t s);

struct AddNormArgs {
  float* x; const float* part; int splits;   // x += sum_s part[s] (part may be null)
  const void* norm_g; int M, H; float eps;
  void* h;
};
hipError_t launch_add_rmsnorm(int bf16, const AddNormArgs& a, hipStream_t s);

struct RopeArgs {
  const float* part; int splits; int M;          // part [S, M, Nqkv]
  const void* bq; const void* bk; const void* bv;
  int n_q, n_kv, hd;
  const int32_t* pos; const int32_t* slot;       // [M]
  const int32_t* page_table; int32_t pt_stride;
  const float* rope_cos; const float* rope_sin;  // [max_ctx, hd/2]
  void* q_out;                                   // [M, n_q, hd]
  void* k_pool; void* v_pool;                    // this layer's pools
};
hipError_t launch_rope_append(int bf16, const RopeArgs& a, hipStream_t s);

struct AttnArgs {
  const void* q;                  // [rows, n_q, hd]
  const void* k_pool; const void* v_pool;
  const int32_t* page_table; int32_t pt_stride;
  int n_q, n_kv, hd;
  float scale;                    // 1 / sqrt(hd)
  // fp32 model: one query row per (token, head), keys 0..tok_pos[row]
  int n_rows; const int32_t* tok_slot; const int32_t* tok_pos;
  // decode (one query token per sequence, split over the context):
  int B; const int32_t* row_slot; const int32_t* row_ctx; const int32_t* split_off;
  int total_splits; int tokens_per_split;
  int max_row_splits;             // most splits of any row (0: unknown); picks the merge kernel
  const int32_t* split_desc;      // [total_splits, 4]: row (+ 2^30 if its only split), first key, end key, slot
  float* part_o; float* part_ml;  // [total_splits * n_kv, 16, hd], [.., 2, 16]
  // prefill (causal over packed prompt chunks):
  int n_seq; const int32_t* seq_slot; const int32_t* seq_row0; const int32_t* seq_pos0;
  const int32_t* seq_ntok; const int32_t* item_off; int total_items;
  // output [rows, n_q * hd]
  void* out;
};
hipError_t launch_attn_decode(int bf16, const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_prefill(int bf16, const AttnArgs& a, hipStream_t s);
// Combine decode splits into out (bf16 model only).
hipError_t launch_attn_merge(const AttnArgs& a, hipStream_t s);
// Query tokens per prefill work item for a GQA group size.
int attn_prefill_tokens_per_item(int bf16, int group);

struct SampleArgs {
  const float* logits; int B; int V;
  const int32_t* row_slot;        // [B]
  const int32_t* row_pos;         // [B] absolute position of the token being sampled
  const int32_t* row_hist;        // [B] index into the slot's token history
  const uint64_t* slot_seed; const uint64_t* slot_id; const float* slot_temp;
  int32_t* tokens_cur; int32_t* hist; int64_t hist_stride;
  float* logp_hist;                     // [slots, hist_stride] log-probability of each sampled token
  float* cand_val; int32_t* cand_idx;   // [B, sample_chunks(V)] per-chunk winners
  float* cand_m; float* cand_s;         // [B, sample_chunks(V)] per-chunk max and sum of exp(s - max)
};
hipError_t launch_sample(const SampleArgs& a, hipStream_t s);
int sample_chunks(int V);

// out[i, :] = src[rows[i], :] for i < n (element size esize bytes, H elements)
// Reads bytes / 16 x 16 bytes of buf (16-byte aligned) once, with nothing written.
hipError_t launch_stream_read(const void* buf, size_t bytes, hipStream_t s);
hipError_t launch_gather_rows(const void* src, const int32_t* rows, int n, int H, int esize,
                              void* out, hipStream_t s);

}  // namespace rollpack
