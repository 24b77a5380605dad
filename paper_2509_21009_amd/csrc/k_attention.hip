// Causal GQA attention over the paged KV cache.
//
// Decode: one 64-lane wave owns a work item: the G query heads of a token
// (up to 16 query rows that share one KV head) and a range of KV tokens.  Per 32-token half page it computes
// S^T = K Q^T as two 16x16 MFMA tiles, runs an online softmax in the log2
// domain, and accumulates O^T = V^T P^T with MFMA.  Both operands are read
// as 16-byte pieces straight from HBM, each load instruction one contiguous
// 1 KB run: a K page is stored in MFMA operand order (k_page_offset; the
// queries use the same dimension order, so every dot product is unchanged),
// and a V page as two 32-token halves, each transposed ([hd][32 tokens]).
// The tokens are assigned to MFMA rows so that each lane's softmax outputs
// are exactly the P^T operand it must supply, with no data exchange between
// lanes.
//
// Prefill stages each K/V page in LDS once per block of query tokens
// (k_attn_prefill_lds below); its waves run the same page step from LDS.
//
// Decode splits each sequence's context into chunks (one work item each, with
// a host-built descriptor) so that small batches with long contexts still
// spread over all CUs; the half pages of an item stream through a ring of
// register stages.  A merge kernel combines the chunk maxima, sums and
// partial outputs.
#include "device_common.hpp"
#include "kernels.hpp"
#include "lds_dma.hpp"

namespace rollpack {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// Token (within a 64-token page) that MFMA row i of S^T tile t stands for.
__device__ __forceinline__ int tile_token(int t, int i) {
  return 32 * (t >> 1) + 8 * (i >> 2) + 4 * (t & 1) + (i & 3);
}

struct SoftmaxState {
  float m, l;
};


// A 16-byte load marked non-temporal, for the KV cache that a decode step
// streams exactly once: the caches then do not keep it at the expense of
// reused lines.  Measured against plain loads, decode attention streams
// 5.7-5.8 TB/s instead of 5.1-5.2 at 16-64 rows.
typedef unsigned u32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t load_bf16x8_nt(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8_t, __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p)));
}

template <int HD>
__global__ __launch_bounds__(64) void k_attn_decode_bf16(AttnArgs a) {
  constexpr int KS = HD / 32, NB = HD / 16, D = 2;
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  const int x = blockIdx.x, kh = blockIdx.y;
  const int4 dsc = reinterpret_cast<const int4*>(a.split_desc)[x];
  const int b = dsc.x & 0x3fffffff;
  const bool single = (dsc.x >> 30) & 1;
  const int t0 = dsc.y, t1 = dsc.z, slot = dsc.w;
  const int G = a.n_q / a.n_kv;

  bf16x8_t qf[KS];
  if (c < G) {  // k-step ks, lane group g: dimensions 32ks + 8g .. +7, the K cache's order
    const bf16_t* qrow = static_cast<const bf16_t*>(a.q) + (static_cast<size_t>(b) * a.n_q + kh * G + c) * HD + g * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = load_bf16x8(qrow + ks * 32);
  } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
  }
  // Lane i holds the page of the item's i-th page (the first 64 pages; later
  // ones, for items longer than 4096 tokens, are read from the table).
  const int* pt = a.page_table + static_cast<size_t>(slot) * a.pt_stride;
  const int p0 = t0 / kPageTokens;
  const int npg = (t1 + kPageTokens - 1) / kPageTokens - p0;
  const int ptv = lane < npg ? pt[p0 + lane] : 0;
  const int u0 = t0 >> 5;
  const int nu = ((t1 + 31) >> 5) - u0;  // half pages of the item
  const bf16_t* kpool = static_cast<const bf16_t*>(a.k_pool);
  const bf16_t* vpool = static_cast<const bf16_t*>(a.v_pool);
  const float scale_log2 = a.scale * kLog2e;

  bf16x8_t kf[D][2][KS], vf[D][NB];
  auto load = [&](int sl, int i) {
    const int u = u0 + min(i, nu - 1);  // prologue stages past the item re-read its last half page
    const int pi = (u >> 1) - p0;
    const int pg = pi < 64 ? __builtin_amdgcn_readlane(ptv, pi) : pt[p0 + pi];
    const int h = u & 1;
    const size_t pb = (static_cast<size_t>(pg) * a.n_kv + kh) * kPageTokens * HD;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      // MFMA row c of S^T tile (2h + tt) of the page is token 32h + 8(c >> 2) + 4tt + (c & 3);
      // its k-step ks is the contiguous 1 KB run ((2h + tt) * KS + ks) of the page's K block
      const bf16_t* krow = kpool + pb + (((2 * h + tt) * KS) * 16 + c) * 32 + g * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[sl][tt][ks] = load_bf16x8_nt(krow + ks * 512);
    }
    const bf16_t* vh = vpool + pb + h * HD * 32;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) vf[sl][blk] = load_bf16x8_nt(vh + (blk * 16 + c) * 32 + 8 * g);
  };

  f32x4_t o[NB];
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) o[blk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  auto compute = [&](int sl, int i) {
    const int u = u0 + i;
    f32x4_t sacc[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      sacc[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sacc[tt] = mfma16x16x32(kf[sl][tt][ks], qf[ks], sacc[tt]);
    }
    float sv[8];
    float pmax = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int tok = 32 * u + 8 * g + 4 * tt + e;
        float v = sacc[tt][e] * scale_log2;
        if (tok < t0 || tok >= t1) v = -INFINITY;
        sv[tt * 4 + e] = v;
        pmax = fmaxf(pmax, v);
      }
    pmax = fmaxf(pmax, __shfl_xor(pmax, 16, 64));
    pmax = fmaxf(pmax, __shfl_xor(pmax, 32, 64));
    const float m_new = fmaxf(m_run, pmax);
    const float shift = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - shift);
    float psum = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      sv[k] = exp2f(sv[k] - shift);
      psum += sv[k];
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    uint4 w;
    w.x = static_cast<uint32_t>(f32_to_bf16(sv[0])) | (static_cast<uint32_t>(f32_to_bf16(sv[1])) << 16);
    w.y = static_cast<uint32_t>(f32_to_bf16(sv[2])) | (static_cast<uint32_t>(f32_to_bf16(sv[3])) << 16);
    w.z = static_cast<uint32_t>(f32_to_bf16(sv[4])) | (static_cast<uint32_t>(f32_to_bf16(sv[5])) << 16);
    w.w = static_cast<uint32_t>(f32_to_bf16(sv[6])) | (static_cast<uint32_t>(f32_to_bf16(sv[7])) << 16);
    const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, w);
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) o[blk] = mfma16x16x32(vf[sl][blk], pf, o[blk] * alpha);
  };

  if (nu > 0) {
    // Unconditional prologue and scheduling barriers: every path into the
    // main loop has the same loads in flight, so its wait counts are exact.
#pragma unroll
    for (int sl = 0; sl < D; ++sl) {
      load(sl, sl);
      __builtin_amdgcn_sched_barrier(0);
    }
    int i = 0;
    for (; i + 2 * D <= nu; i += D) {
#pragma unroll
      for (int sl = 0; sl < D; ++sl) {
        compute(sl, i + sl);
        __builtin_amdgcn_sched_barrier(0);
        load(sl, i + sl + D);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int j = 0; j < 2 * D; ++j) {
      if (i + j < nu) {
        compute(j % D, i + j);
        __builtin_amdgcn_sched_barrier(0);
        if (i + j + D < nu) load(j % D, i + j + D);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  if (c >= G) return;
  if (single) {  // the row's only split: normalise and write the output directly
    const float inv = 1.f / l_run;
    bf16_t* orow = static_cast<bf16_t*>(a.out) + (static_cast<size_t>(b) * a.n_q + kh * G + c) * HD;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      uint2 pk;
      pk.x = static_cast<uint32_t>(f32_to_bf16(o[blk][0] * inv)) | (static_cast<uint32_t>(f32_to_bf16(o[blk][1] * inv)) << 16);
      pk.y = static_cast<uint32_t>(f32_to_bf16(o[blk][2] * inv)) | (static_cast<uint32_t>(f32_to_bf16(o[blk][3] * inv)) << 16);
      *reinterpret_cast<uint2*>(orow + blk * 16 + 4 * g) = pk;
    }
    return;
  }
  const size_t item = static_cast<size_t>(x) * a.n_kv + kh;
  float* po = a.part_o + (item * 16 + c) * HD;
#pragma unroll
  for (int blk = 0; blk < NB; ++blk)
    *reinterpret_cast<float4*>(po + blk * 16 + 4 * g) = make_float4(o[blk][0], o[blk][1], o[blk][2], o[blk][3]);
  if (g == 0) {
    a.part_ml[item * 32 + c] = m_run;
    a.part_ml[item * 32 + 16 + c] = l_run;
  }
}

// One block per (row, query head) with HD x 8 threads (rows with more than
// one split): the splits' maxima
// and sums are staged in LDS, each of 8 thread groups accumulates every 8th
// split for all HD output elements, and the groups are summed in LDS.  Long
// contexts at small batch have hundreds of splits, which a single serial
// loop per element would walk one memory latency at a time.
constexpr int kMergeCache = 512;
constexpr int kMergeGroups = 8;

template <int HD>
__global__ __launch_bounds__(HD * kMergeGroups) void k_attn_merge(AttnArgs a) {
  __shared__ float sm[kMergeCache], sl[kMergeCache];
  __shared__ float part_num[kMergeGroups][HD];
  __shared__ float part_den[kMergeGroups];
  __shared__ float wmax[HD * kMergeGroups / 64];
  const int b = blockIdx.x, h = blockIdx.y;
  const int d = threadIdx.x % HD, q = threadIdx.x / HD;
  const int G = a.n_q / a.n_kv;
  const int kh = h / G, c = h % G;
  const int s0 = a.split_off[b], n = a.split_off[b + 1] - s0;
  if (n <= 1) return;  // single-split rows were written by the decode kernel
  const int nc = min(n, kMergeCache);
  auto m_of = [&](int t) { return a.part_ml[(static_cast<size_t>(s0 + t) * a.n_kv + kh) * 32 + c]; };
  auto l_of = [&](int t) { return a.part_ml[(static_cast<size_t>(s0 + t) * a.n_kv + kh) * 32 + 16 + c]; };
  float mx = -INFINITY;
  for (int t = threadIdx.x; t < n; t += blockDim.x) {
    const float mv = m_of(t);
    if (t < nc) { sm[t] = mv; sl[t] = l_of(t); }
    mx = fmaxf(mx, mv);
  }
  mx = wave_max(mx);
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = -INFINITY;
  for (int i = 0; i < HD * kMergeGroups / 64; ++i) mx = fmaxf(mx, wmax[i]);
  // Split weights into LDS first, so that the loop below issues nothing but
  // independent partial-output loads (unrolled 16 deep: a 256-split row takes
  // two memory round trips per thread instead of one per few splits).
  for (int t = threadIdx.x; t < nc; t += blockDim.x) sm[t] = (sm[t] == -INFINITY) ? 0.f : exp2f(sm[t] - mx);
  __syncthreads();
  const float* po = a.part_o + (static_cast<size_t>(s0) * a.n_kv + kh) * 16 * HD + c * HD + d;
  const size_t po_stride = static_cast<size_t>(a.n_kv) * 16 * HD;  // one split
  float num = 0.f, den = 0.f;
#pragma unroll 16
  for (int t = q; t < nc; t += kMergeGroups) num += sm[t] * po[t * po_stride];
  if (d == 0)
    for (int t = q; t < nc; t += kMergeGroups) den += sm[t] * sl[t];
  for (int t = nc + q; t < n; t += kMergeGroups) {  // splits beyond the LDS cache
    const float ms = m_of(t);
    const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
    num += w * po[t * po_stride];
    if (d == 0) den += w * l_of(t);
  }
  part_num[q][d] = num;
  if (d == 0) part_den[q] = den;
  __syncthreads();
  if (q == 0) {
    float tn = 0.f, td = 0.f;
#pragma unroll
    for (int i = 0; i < kMergeGroups; ++i) { tn += part_num[i][d]; td += part_den[i]; }
    static_cast<bf16_t*>(a.out)[(static_cast<size_t>(b) * a.n_q + h) * HD + d] = f32_to_bf16(tn / td);
  }
}

// The same combination for steps whose rows have at most NMAX (<= 64)
// splits: one wave per (row, query head), lane t holding split t's max and
// sum, and every partial output the lane needs loaded before the split
// weights are known (one memory round trip; splits past the row's count
// re-read its last one and are not added).  Lane j owns dimensions j,
// j + 64, ...  The arithmetic is k_attn_merge's in the same order (per-group
// sums over splits t = q, q + kMergeGroups, ..., then the groups in order),
// so both kernels give identical outputs.
constexpr int kMergeFew = 64;

template <int HD, int NMAX>
__global__ __launch_bounds__(64) void k_attn_merge_few(AttnArgs a) {
  static_assert(NMAX <= 64, "one split per lane");
  constexpr int NPL = HD / 64;
  const int b = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int G = a.n_q / a.n_kv;
  const int kh = h / G, c = h % G;
  const int s0 = a.split_off[b], n = a.split_off[b + 1] - s0;
  if (n <= 1) return;  // single-split rows were written by the decode kernel
  const size_t mi = (static_cast<size_t>(s0 + min(lane, n - 1)) * a.n_kv + kh) * 32 + c;
  const float m_ld = a.part_ml[mi], l_ld = a.part_ml[mi + 16];
  const float* po = a.part_o + (static_cast<size_t>(s0) * a.n_kv + kh) * 16 * HD + c * HD + lane;
  const size_t po_stride = static_cast<size_t>(a.n_kv) * 16 * HD;  // one split
  float pv[NMAX][NPL];
#pragma unroll
  for (int t = 0; t < NMAX; ++t)
#pragma unroll
    for (int k = 0; k < NPL; ++k) pv[t][k] = po[min(t, n - 1) * po_stride + 64 * k];
  const float mv = lane < n ? m_ld : -INFINITY;
  const float mx = wave_max(mv);
  const float wv = (mv == -INFINITY) ? 0.f : exp2f(mv - mx);
  float tn[NPL], td = 0.f;
#pragma unroll
  for (int k = 0; k < NPL; ++k) tn[k] = 0.f;
#pragma unroll
  for (int q = 0; q < kMergeGroups; ++q) {
    float num[NPL], den = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) num[k] = 0.f;
#pragma unroll
    for (int t = q; t < NMAX; t += kMergeGroups) {
      const bool in = t < n;
      const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wv), t));
      const float l = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l_ld), t));
#pragma unroll
      for (int k = 0; k < NPL; ++k) num[k] = in ? num[k] + w * pv[t][k] : num[k];
      den = in ? den + w * l : den;
    }
#pragma unroll
    for (int k = 0; k < NPL; ++k) tn[k] += num[k];
    td += den;
  }
  bf16_t* out = static_cast<bf16_t*>(a.out) + (static_cast<size_t>(b) * a.n_q + h) * HD + lane;
#pragma unroll
  for (int k = 0; k < NPL; ++k) out[64 * k] = f32_to_bf16(tn[k] / td);
}

// Prefill attention with K/V pages staged in LDS and shared by a block.
//
// A block of 8 waves owns one KV head and kPrefillWaveGroups * 8 query groups
// of one sequence piece; a query group is the G query heads of tpi = 16 / G
// consecutive tokens (one 16-column MFMA operand), and each wave holds
// kPrefillWaveGroups of them.  The block walks the causal prefix one 64-token
// page at a time: the page's K and V blocks (copied unchanged from the cache,
// with each 1 KB run reordered so that a wave's read of it is 64 consecutive
// 16-byte pieces) pass through a two-stage LDS ring filled by LDS-DMA
// copies one page ahead, and every wave runs the decode kernel's page step (S^T = K Q^T, online
// softmax in the log2 domain, O^T += V^T P^T) on them for its groups, each K
// and V fragment read once for all of its groups.  The global K/V traffic of
// a prefix is then paid once per block instead of once per group.  Two blocks
// share a CU (under 128 registers per lane and 72 KB of LDS each), so one
// block's barriers and the dependent S -> softmax -> PV chain of its waves
// overlap with the other's MFMAs: measured on the 7B short round's prefill,
// 0.16 of the dense bf16 peak against 0.12 with two groups per wave and one
// block per CU, and 0.14 with 16 waves per block.
constexpr int kPrefillWaveGroups = 1;
constexpr int kPrefillWaves = 8;
constexpr int kMaxContextPages = 65536 / kPageTokens;  // the engine's context limit

typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float f32x2_hw __attribute__((ext_vector_type(2)));

// Two fp32 values to packed bf16, round to nearest even (gfx950's v_cvt_pk_bf16_f32; for the
// finite values here the same result as f32_to_bf16).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_hw{lo, hi}, bf16x2_hw));
}

// One page step of the prefill kernel for a wave's NG query groups.  MASKED: whether any key
// of the page may lie past some column's own position (the diagonal pages); the others are
// compiled without the mask.  The maximum is taken over the raw scores and the softmax scale
// folded into the exponent's fused multiply-add, which leaves the VALU about 115 instructions
// per page against 32 MFMAs (185 with the mask and a separate scaling pass).
// Exponents go through the bare v_exp_f32: their arguments are <= 0, and results below 2^-126,
// which it flushes, are far below what bf16 probabilities resolve.
template <int HD, int NG, bool MASKED>
__device__ __forceinline__ void attend_page_lds(const bf16_t* kb, const bf16_t* vb, int page_tok0,
                                                const bf16x8_t (&qf)[NG][HD / 32], const int (&row_lim)[NG],
                                                float scale_log2, SoftmaxState (&st)[NG],
                                                f32x4_t (&o)[NG][HD / 16]) {
  constexpr int KS = HD / 32;
  const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
  // LDS holds each 1 KB run of the page lane-ordered (the page copies of k_attn_prefill_lds): lane l
  // reads piece l of a run.
  const bf16x8_t* kr = reinterpret_cast<const bf16x8_t*>(kb) + lane;
  const bf16x8_t* vr = reinterpret_cast<const bf16x8_t*>(vb) + lane;
  f32x4_t sacc[NG][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    bf16x8_t kf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = kr[(t * KS + ks) * 64];
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      sacc[q][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sacc[q][t] = mfma16x16x32(kf[ks], qf[q][ks], sacc[q][t]);
    }
  }
  bf16x8_t pf[NG][2];
  float alpha[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    float sv[16];
    float pmax = -INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = sacc[q][t][e];
        if (MASKED && page_tok0 + 32 * (t >> 1) + 8 * g + 4 * (t & 1) + e > row_lim[q]) v = -INFINITY;
        sv[t * 4 + e] = v;
        pmax = fmaxf(pmax, v);
      }
    pmax = fmaxf(pmax, __shfl_xor(pmax, 16, 64));
    pmax = fmaxf(pmax, __shfl_xor(pmax, 32, 64));
    // the scale is positive, so the largest scaled score is the largest score, scaled
    const float m_new = fmaxf(st[q].m, pmax * scale_log2);
    const float shift = (m_new == -INFINITY) ? 0.f : m_new;
    alpha[q] = __builtin_amdgcn_exp2f(st[q].m - shift);
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      sv[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i], scale_log2, -shift));
      psum += sv[i];
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    st[q].l = st[q].l * alpha[q] + psum;
    st[q].m = m_new;
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      uint4 w;
      w.x = pack_bf16x2(sv[pp * 8 + 0], sv[pp * 8 + 1]);
      w.y = pack_bf16x2(sv[pp * 8 + 2], sv[pp * 8 + 3]);
      w.z = pack_bf16x2(sv[pp * 8 + 4], sv[pp * 8 + 5]);
      w.w = pack_bf16x2(sv[pp * 8 + 6], sv[pp * 8 + 7]);
      pf[q][pp] = __builtin_bit_cast(bf16x8_t, w);
    }
  }
#pragma unroll
  for (int q = 0; q < NG; ++q)
#pragma unroll
    for (int blk = 0; blk < HD / 16; ++blk) o[q][blk] = o[q][blk] * alpha[q];
#pragma unroll
  for (int blk = 0; blk < HD / 16; ++blk) {
    bf16x8_t vf[2];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) vf[pp] = vr[(pp * HD / 16 + blk) * 64];
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) o[q][blk] = mfma16x16x32(vf[pp], pf[q][pp], o[q][blk]);
  }
}

template <int HD>
__global__ __launch_bounds__(64 * kPrefillWaves, 2) void k_attn_prefill_lds(AttnArgs a, int tpi) {
  constexpr int KS = HD / 32, NG = kPrefillWaveGroups;
  constexpr int PAGE_EL = kPageTokens * HD;                 // elements of one (page, head) K or V block
  constexpr int RUNS = 2 * PAGE_EL * 2 / 1024;              // 1 KB runs of a page's K and V blocks
  constexpr int DPW = RUNS / kPrefillWaves;                 // runs each wave copies per page
  constexpr int NST = 2, AHEAD = NST - 1;                   // LDS stages; pages in flight
  static_assert(RUNS % kPrefillWaves == 0, "page staging");
  constexpr int NT = 64 * kPrefillWaves;
  __shared__ __attribute__((aligned(1024))) bf16_t kv[NST][2 * PAGE_EL];  // [stage][K block, V block]
  __shared__ int s_off[NT];                                           // item offsets of the chunk's pieces
  __shared__ int s_pt[kMaxContextPages];                              // the piece's page-table row
  const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
  const int wave = threadIdx.x >> 6;
  const int x = blockIdx.x, kh = blockIdx.y;
  // Which piece the block serves: one cooperative load of the item offsets into LDS, then a
  // search there (a global binary search would chain its loads' latencies).
  const int n_cached = min(a.n_seq + 1, NT);
  if (static_cast<int>(threadIdx.x) < n_cached) s_off[threadIdx.x] = a.item_off[threadIdx.x];
  __syncthreads();
  int lo = 0, hi = a.n_seq;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((mid < n_cached ? s_off[mid] : a.item_off[mid]) <= x) lo = mid; else hi = mid;
  }
  const int j = lo;
  // the piece's blocks in reverse: later query tokens attend to more pages, so they start first
  const int n_blk = (j + 1 < n_cached ? s_off[j + 1] : a.item_off[j + 1]) - (j < n_cached ? s_off[j] : a.item_off[j]);
  const int qb = n_blk - 1 - (x - (j < n_cached ? s_off[j] : a.item_off[j]));
  const int ntok = a.seq_ntok[j];
  const int G = a.n_q / a.n_kv;
  const int pos0 = a.seq_pos0[j];
  const int block_tok = kPrefillWaves * NG * tpi;
  const int last_tok = min(qb * block_tok + block_tok, ntok) - 1;
  const int t_end = pos0 + last_tok + 1;  // keys the block needs: [0, t_end)

  // this lane's query column in each of the wave's groups
  bf16x8_t qf[NG][KS];
  int row_lim[NG], tq[NG], head = kh * G + c % G;
  bool valid[NG];
  int wave_lim = -1;
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    tq[q] = qb * block_tok + (wave * NG + q) * tpi + c / G;
    valid[q] = c < tpi * G && tq[q] < ntok;
    row_lim[q] = valid[q] ? pos0 + tq[q] : -1;
    wave_lim = max(wave_lim, row_lim[q]);
    if (valid[q]) {
      const bf16_t* qrow = static_cast<const bf16_t*>(a.q) +
                           ((static_cast<size_t>(a.seq_row0[j] + tq[q])) * a.n_q + head) * HD + g * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[q][ks] = load_bf16x8(qrow + ks * 32);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[q][ks] = __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1)  // the wave's last query position
    wave_lim = max(wave_lim, __shfl_xor(wave_lim, m, 64));
  wave_lim = __builtin_amdgcn_readfirstlane(wave_lim);  // wave-uniform: the page branch below is scalar
  f32x4_t o[NG][HD / 16];
  SoftmaxState st[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    st[q] = SoftmaxState{-INFINITY, 0.f};
#pragma unroll
    for (int blk = 0; blk < HD / 16; ++blk) o[q][blk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const bf16_t* kpool = static_cast<const bf16_t*>(a.k_pool);
  const bf16_t* vpool = static_cast<const bf16_t*>(a.v_pool);
  const float scale_log2 = a.scale * kLog2e;
  const int npages =  // <= kMaxContextPages (max_context <= 65536)
      __builtin_amdgcn_readfirstlane((t_end + kPageTokens - 1) / kPageTokens);
  {
    const int* ptg = a.page_table + static_cast<size_t>(a.seq_slot[j]) * a.pt_stride;
    for (int i = threadIdx.x; i < npages; i += NT) s_pt[i] = ptg[i];
  }
  __syncthreads();
  const int* pt = s_pt;

  // Pages go from the cache straight into LDS (buffer_load ... lds, no register staging), AHEAD
  // pages ahead of the one being computed; wave w copies runs w, w + 8, ... of each page.  Within
  // a run, LDS piece 16g + c receives the cache's piece 4c + g, the one lane 16g + c reads, so a
  // wave's 64 lanes read 64 consecutive LDS pieces, free of bank conflicts.  Past the last page the
  // copies repeat it, so that every iteration waits for the same number of loads (the extra
  // copies land in stages nobody reads again).
  typedef const __attribute__((address_space(3))) char lds_char;
  const uint32_t lds_kv = static_cast<uint32_t>((uintptr_t)(lds_char*)(&kv[0][0]));  // LDS byte address
  const int lane_src = 16 * (((lane & 15) << 2) | (lane >> 4));
  auto issue = [&](int page, int stage) {
    const int pg = __builtin_amdgcn_readfirstlane(pt[page]);
    const size_t pb = (static_cast<size_t>(pg) * a.n_kv + kh) * PAGE_EL;
    const u32x4_raw kres = raw_rsrc(kpool + pb, PAGE_EL * 2), vres = raw_rsrc(vpool + pb, PAGE_EL * 2);
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const int run = wave + kPrefillWaves * i;  // runs below RUNS / 2 are K, the rest V
      const uint32_t dst = __builtin_amdgcn_readfirstlane(lds_kv + static_cast<uint32_t>(stage * PAGE_EL * 4 + run * 1024));
      if (run < RUNS / 2)
        dma16(kres, dst, run * 1024 + lane_src);
      else
        dma16(vres, dst, (run - RUNS / 2) * 1024 + lane_src);
    }
  };
#pragma unroll
  for (int s0 = 0; s0 < AHEAD; ++s0) issue(min(s0, npages - 1), s0);
  // Pages [0, n_open) are visible in full to every column of the block (its first token sees
  // them all) and run without the mask; the rest (the diagonal, one or two pages) run masked.
  const int n_open = __builtin_amdgcn_readfirstlane(min(npages, (pos0 + qb * block_tok + 1) / kPageTokens));
  for (int p = 0; p < n_open; ++p) {
    wait_vmcnt<(AHEAD - 1) * DPW>();  // this wave's copies of page p have landed
    __syncthreads();                  // every wave's have; every wave is done with page p - 1
    issue(min(p + AHEAD, npages - 1), (p + AHEAD) % NST);  // into the stage that held page p - 1
    attend_page_lds<HD, NG, false>(kv[p % NST], kv[p % NST] + PAGE_EL, p * kPageTokens, qf, row_lim, scale_log2, st,
                                   o);
  }
  for (int p = n_open; p < npages; ++p) {
    wait_vmcnt<(AHEAD - 1) * DPW>();
    __syncthreads();
    issue(min(p + AHEAD, npages - 1), (p + AHEAD) % NST);
    if (p * kPageTokens <= wave_lim)
      attend_page_lds<HD, NG, true>(kv[p % NST], kv[p % NST] + PAGE_EL, p * kPageTokens, qf, row_lim, scale_log2,
                                    st, o);
  }

#pragma unroll
  for (int q = 0; q < NG; ++q) {
    if (!valid[q]) continue;
    const float inv = 1.0f / st[q].l;
    bf16_t* out = static_cast<bf16_t*>(a.out) + ((static_cast<size_t>(a.seq_row0[j] + tq[q])) * a.n_q + head) * HD;
#pragma unroll
    for (int blk = 0; blk < HD / 16; ++blk) {
      uint2 pk;
      pk.x = static_cast<uint32_t>(f32_to_bf16(o[q][blk][0] * inv)) | (static_cast<uint32_t>(f32_to_bf16(o[q][blk][1] * inv)) << 16);
      pk.y = static_cast<uint32_t>(f32_to_bf16(o[q][blk][2] * inv)) | (static_cast<uint32_t>(f32_to_bf16(o[q][blk][3] * inv)) << 16);
      *reinterpret_cast<uint2*>(out + blk * 16 + 4 * g) = pk;
    }
  }
}


// fp32 model: one wave per (row, query head), one key at a time.
__global__ __launch_bounds__(64) void k_attn_f32(AttnArgs a) {
  const int i = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int HD = a.hd;
  const int G = a.n_q / a.n_kv, kh = h / G;
  const int slot = a.tok_slot[i], pos = a.tok_pos[i];
  const float* q = static_cast<const float*>(a.q) + (static_cast<size_t>(i) * a.n_q + h) * HD;
  const float* kpool = static_cast<const float*>(a.k_pool);
  const float* vpool = static_cast<const float*>(a.v_pool);
  const int* pt = a.page_table + static_cast<size_t>(slot) * a.pt_stride;
  float qv[2] = {lane < HD ? q[lane] : 0.f, lane + 64 < HD ? q[lane + 64] : 0.f};
  float acc[2] = {0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  for (int t = 0; t <= pos; ++t) {
    const size_t pb = (static_cast<size_t>(pt[t / kPageTokens]) * a.n_kv + kh) * kPageTokens * HD;
    const int off = t % kPageTokens;
    const float* k = kpool + pb + static_cast<size_t>(off) * HD;
    float part = (lane < HD ? qv[0] * k[lane] : 0.f) + (lane + 64 < HD ? qv[1] * k[lane + 64] : 0.f);
    const float s = wave_sum(part) * a.scale;
    const float m_new = fmaxf(m, s);
    const float alpha = expf(m - m_new);
    const float p = expf(s - m_new);
    l = l * alpha + p;
    m = m_new;
    const float* v = vpool + pb;
    const float* vh = v + (off >> 5) * HD * 32 + (off & 31);
    if (lane < HD) acc[0] = acc[0] * alpha + p * vh[static_cast<size_t>(lane) * 32];
    if (lane + 64 < HD) acc[1] = acc[1] * alpha + p * vh[static_cast<size_t>(lane + 64) * 32];
  }
  float* out = static_cast<float*>(a.out) + (static_cast<size_t>(i) * a.n_q + h) * HD;
  if (lane < HD) out[lane] = acc[0] / l;
  if (lane + 64 < HD) out[lane + 64] = acc[1] / l;
}

}  // namespace

// Query tokens of one 16-column MFMA group: the G heads of each token side by side.
static int prefill_group_tokens(int group) {
  const int t = 16 / group;
  return t < 1 ? 1 : t;
}

int attn_prefill_tokens_per_item(int bf16, int group) {
  if (!bf16) return 1;
  return kPrefillWaves * kPrefillWaveGroups * prefill_group_tokens(group);
}

hipError_t launch_attn_decode(int bf16, const AttnArgs& a, hipStream_t s) {
  if (!bf16) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.hd > 128) return hipErrorInvalidValue;
    launch_kernel(k_attn_f32, dim3(a.n_rows, a.n_q), dim3(64), 0, s, a);
    return hipGetLastError();
  }
  if (a.B <= 0 || a.total_splits <= 0) return hipSuccess;
  if (a.n_q / a.n_kv > 16 || a.tokens_per_split % kPageTokens != 0 || !a.split_desc) return hipErrorInvalidValue;
  dim3 grid(a.total_splits, a.n_kv);
  if (a.hd == 128) launch_kernel(k_attn_decode_bf16<128>, grid, dim3(64), 0, s, a);
  else if (a.hd == 64) launch_kernel(k_attn_decode_bf16<64>, grid, dim3(64), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  dim3 grid(a.B, a.n_q);
  // One wave per (row, head) pays off once there are many rows: at 64 rows of 8 splits it takes
  // 4.0 us against 9.6 us; at a single row the 1024-thread blocks are 0.3-1.3 us faster.
  if (a.B >= 8 && a.max_row_splits >= 1 && a.max_row_splits <= kMergeFew) {
    if (a.hd != 128 && a.hd != 64) return hipErrorInvalidValue;
#define RP_MERGE_FEW(NMAX)                                                                    \
    if (a.max_row_splits <= NMAX) {                                                           \
      if (a.hd == 128) launch_kernel(k_attn_merge_few<128, NMAX>, grid, dim3(64), 0, s, a);   \
      else launch_kernel(k_attn_merge_few<64, NMAX>, grid, dim3(64), 0, s, a);                \
      return hipGetLastError();                                                               \
    }
    RP_MERGE_FEW(8) RP_MERGE_FEW(16) RP_MERGE_FEW(32) RP_MERGE_FEW(64)
#undef RP_MERGE_FEW
  }
  if (a.hd == 128) launch_kernel(k_attn_merge<128>, grid, dim3(128 * kMergeGroups), 0, s, a);
  else if (a.hd == 64) launch_kernel(k_attn_merge<64>, grid, dim3(64 * kMergeGroups), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_prefill(int bf16, const AttnArgs& a, hipStream_t s) {
  if (!bf16) {
    if (a.n_rows <= 0) return hipSuccess;
    if (a.hd > 128) return hipErrorInvalidValue;
    launch_kernel(k_attn_f32, dim3(a.n_rows, a.n_q), dim3(64), 0, s, a);
    return hipGetLastError();
  }
  if (a.total_items <= 0) return hipSuccess;
  const int G = a.n_q / a.n_kv;
  if (G > 16) return hipErrorInvalidValue;
  const int tpi = prefill_group_tokens(G);
  dim3 grid(a.total_items, a.n_kv);
  if (a.hd == 128) launch_kernel(k_attn_prefill_lds<128>, grid, dim3(64 * kPrefillWaves), 0, s, a, tpi);
  else if (a.hd == 64) launch_kernel(k_attn_prefill_lds<64>, grid, dim3(64 * kPrefillWaves), 0, s, a, tpi);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace rollpack
