// Row-wise kernels of the decoder step: embedding + RMSNorm, residual add +
// RMSNorm, q/k/v bias + RoPE + paged KV append, and Gumbel-max sampling with
// a Philox4x64-10 counter-based generator.  They move little data, so they
// are written for latency: every load of a thread is issued before the first
// use, and small batches are spread over several blocks per row.
#include "device_common.hpp"
#include "kernels.hpp"

namespace rollpack {

LaunchEvents& launch_events() {
  thread_local LaunchEvents ev;
  return ev;
}

namespace {

// Rows are processed by one block of up to 1024 threads, each owning two
// 4-element chunks, so every load of a row is in flight at once.
constexpr int kRowChunks = 2;

template <typename T> struct Vec4;
template <> struct Vec4<float> {
  static __device__ __forceinline__ float4 load(const float* p, size_t i) { return *reinterpret_cast<const float4*>(p + i); }
  static __device__ __forceinline__ void store(float* p, size_t i, float4 v) { *reinterpret_cast<float4*>(p + i) = v; }
};
template <> struct Vec4<bf16_t> {
  static __device__ __forceinline__ float4 load(const bf16_t* p, size_t i) {
    const uint2 u = *reinterpret_cast<const uint2*>(p + i);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
  }
  static __device__ __forceinline__ void store(bf16_t* p, size_t i, float4 v) {
    uint2 u;
    u.x = static_cast<uint32_t>(f32_to_bf16(v.x)) | (static_cast<uint32_t>(f32_to_bf16(v.y)) << 16);
    u.y = static_cast<uint32_t>(f32_to_bf16(v.z)) | (static_cast<uint32_t>(f32_to_bf16(v.w)) << 16);
    *reinterpret_cast<uint2*>(p + i) = u;
  }
};

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// x holds the row (kRowChunks float4 per thread); writes h = x * rsqrt(mean(x^2)+eps) * g.
template <typename T>
__device__ __forceinline__ void norm_store(const float4 (&xv)[kRowChunks], int H, float eps, const T* g, T* h,
                                           float* red) {
  const int nc = H / 4;
  float ss = 0.f;
#pragma unroll
  for (int v = 0; v < kRowChunks; ++v) {
    const int c = threadIdx.x + v * blockDim.x;
    if (c < nc) ss += xv[v].x * xv[v].x + xv[v].y * xv[v].y + xv[v].z * xv[v].z + xv[v].w * xv[v].w;
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / H + eps);
#pragma unroll
  for (int v = 0; v < kRowChunks; ++v) {
    const int c = threadIdx.x + v * blockDim.x;
    if (c < nc) {
      const float4 gv = Vec4<T>::load(g, 4 * c);
      Vec4<T>::store(h, 4 * static_cast<size_t>(c),
                     make_float4(xv[v].x * inv * gv.x, xv[v].y * inv * gv.y, xv[v].z * inv * gv.z, xv[v].w * inv * gv.w));
    }
  }
}

template <typename T>
__global__ __launch_bounds__(1024) void k_embed_norm(EmbedArgs a) {
  __shared__ float red[16];
  const int i = blockIdx.x;
  int tok = a.in_tok[i];
  if (tok < 0) tok = a.tokens_cur[a.row_slot[i]];
  const T* e = static_cast<const T*>(a.embed) + static_cast<size_t>(tok) * a.H;
  float* x = a.x + static_cast<size_t>(i) * a.H;
  const int nc = a.H / 4;
  float4 xv[kRowChunks];
#pragma unroll
  for (int v = 0; v < kRowChunks; ++v) {
    const int c = threadIdx.x + v * blockDim.x;
    if (c < nc) {
      xv[v] = Vec4<T>::load(e, 4 * c);
      *reinterpret_cast<float4*>(x + 4 * c) = xv[v];
    }
  }
  norm_store<T>(xv, a.H, a.eps, static_cast<const T*>(a.norm_g), static_cast<T*>(a.h) + static_cast<size_t>(i) * a.H,
                red);
}

template <typename T, int S>
__global__ __launch_bounds__(1024) void k_add_rmsnorm(AddNormArgs a) {
  __shared__ float red[16];
  const int i = blockIdx.x;
  float* x = a.x + static_cast<size_t>(i) * a.H;
  const int nc = a.H / 4;
  const size_t plane = static_cast<size_t>(a.M) * a.H;
  float4 xv[kRowChunks];
  float4 pv[S > 0 ? S : 1][kRowChunks];
#pragma unroll
  for (int v = 0; v < kRowChunks; ++v) {
    const int c = threadIdx.x + v * blockDim.x;
    if (c < nc) {
      xv[v] = *reinterpret_cast<const float4*>(x + 4 * c);
#pragma unroll
      for (int s = 0; s < S; ++s)
        pv[s][v] = *reinterpret_cast<const float4*>(a.part + s * plane + static_cast<size_t>(i) * a.H + 4 * c);
    }
  }
  if (S > 0) {
#pragma unroll
    for (int v = 0; v < kRowChunks; ++v) {
      const int c = threadIdx.x + v * blockDim.x;
      if (c < nc) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          xv[v].x += pv[s][v].x; xv[v].y += pv[s][v].y; xv[v].z += pv[s][v].z; xv[v].w += pv[s][v].w;
        }
        *reinterpret_cast<float4*>(x + 4 * c) = xv[v];
      }
    }
  }
  norm_store<T>(xv, a.H, a.eps, static_cast<const T*>(a.norm_g), static_cast<T*>(a.h) + static_cast<size_t>(i) * a.H,
                red);
}

// One thread per rotated (q or k) pair or per v element; blockIdx.y strides
// the row's items so small batches still fill the GPU.
template <typename T, int S>
__global__ __launch_bounds__(256) void k_rope_append(RopeArgs a) {
  const int i = blockIdx.x;
  const int hd = a.hd, half = hd / 2;
  const int nq_el = a.n_q * hd, nk_el = a.n_kv * hd;
  const int nqkv = nq_el + 2 * nk_el;
  const int n_pairs = (a.n_q + a.n_kv) * half;
  const int t = blockIdx.y * blockDim.x + threadIdx.x;
  if (t >= n_pairs + nk_el) return;
  const size_t plane = static_cast<size_t>(a.M) * nqkv;
  const float* __restrict__ prow = a.part + static_cast<size_t>(i) * nqkv;
  const int pos = a.pos[i];
  const int slot = a.slot[i];
  const int page = a.page_table[static_cast<size_t>(slot) * a.pt_stride + pos / kPageTokens];
  const int off = pos % kPageTokens;
  if (t < n_pairs) {
    const int head = t / half, d = t % half;
    const int n1 = head * hd + d, n2 = n1 + half;
    float u1 = 0.f, u2 = 0.f;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      u1 += prow[s * plane + n1];
      u2 += prow[s * plane + n2];
    }
    const bool isq = head < a.n_q;
    const T* b = isq ? static_cast<const T*>(a.bq) : static_cast<const T*>(a.bk);
    const int bi = isq ? n1 : n1 - nq_el;
    u1 += Elem<T>::load(b, bi);
    u2 += Elem<T>::load(b, bi + half);
    const float c = a.rope_cos[static_cast<size_t>(pos) * half + d];
    const float sn = a.rope_sin[static_cast<size_t>(pos) * half + d];
    const float r1 = u1 * c - u2 * sn;
    const float r2 = u2 * c + u1 * sn;
    if (head < a.n_q) {
      T* q = static_cast<T*>(a.q_out) + static_cast<size_t>(i) * nq_el;
      Elem<T>::store(q, n1, r1);
      Elem<T>::store(q, n2, r2);
    } else {
      const int kh = head - a.n_q;
      const size_t blk = (static_cast<size_t>(page) * a.n_kv + kh) * kPageTokens * hd;
      if (sizeof(T) == 2) {  // bf16 cache: MFMA operand order
        Elem<T>::store(static_cast<T*>(a.k_pool), blk + k_page_offset(off, d, hd), r1);
        Elem<T>::store(static_cast<T*>(a.k_pool), blk + k_page_offset(off, d + half, hd), r2);
      } else {
        Elem<T>::store(static_cast<T*>(a.k_pool), blk + static_cast<size_t>(off) * hd + d, r1);
        Elem<T>::store(static_cast<T*>(a.k_pool), blk + static_cast<size_t>(off) * hd + d + half, r2);
      }
    }
  } else {
    const int e = t - n_pairs;
    const int kh = e / hd, d = e % hd;
    const int n = nq_el + nk_el + e;
    float v = 0.f;
#pragma unroll
    for (int s = 0; s < S; ++s) v += prow[s * plane + n];
    v += Elem<T>::load(static_cast<const T*>(a.bv), e);
    // V page: two 32-token halves, each [hd][32 tokens]
    const size_t idx = (static_cast<size_t>(page) * a.n_kv + kh) * hd * kPageTokens + (off >> 5) * hd * 32 + d * 32 + (off & 31);
    Elem<T>::store(static_cast<T*>(a.v_pool), idx, v);
  }
}

// ---- sampling -------------------------------------------------------------

constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;

// Philox4x64, 10 rounds (Salmon et al., SC'11).
__device__ __forceinline__ void philox4x64_10(uint64_t& x0, uint64_t& x1, uint64_t& x2, uint64_t& x3,
                                              uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hi0 = __umul64hi(kPhiloxM0, x0), lo0 = kPhiloxM0 * x0;
    const uint64_t hi1 = __umul64hi(kPhiloxM1, x2), lo1 = kPhiloxM1 * x2;
    const uint64_t n0 = hi1 ^ x1 ^ k0, n2 = hi0 ^ x3 ^ k1;
    x0 = n0; x1 = lo1; x2 = n2; x3 = lo0;
    k0 += kPhiloxW0;
    k1 += kPhiloxW1;
  }
}

// Top 23 bits of a 32-bit word -> (m + 0.5) * 2^-23, exact in fp32, in (0, 1).
__device__ __forceinline__ float word_to_gumbel(uint32_t w) {
  const float u = (static_cast<float>(w >> 9) + 0.5f) * 1.1920928955078125e-07f;
  return -logf(-logf(u));
}

__device__ __forceinline__ void take_best(float& bv, int& bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
}

// Running log-sum-exp state (max m, sum of exp(x - m)); combining two states
// rescales the smaller-max sum.
__device__ __forceinline__ void lse_add(float& m, float& s, float x) {
  if (x > m) { s = s * expf(m - x) + 1.f; m = x; } else { s += expf(x - m); }
}
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  if (m2 == -INFINITY) return;
  if (m2 > m) { s = s * expf(m - m2) + s2; m = m2; } else { s += s2 * expf(m2 - m); }
}

// Pass 1: block (row, chunk) scores kSampleChunk vocabulary entries and
// writes its best (score, index) and the log-sum-exp state of logits / T
// over the chunk.  Pass 2: one wave per row reduces the chunk winners (ties
// -> lowest index), records the token and its log-probability
// logits[token] / T - logsumexp(logits / T) (T = 1 for greedy rows).
constexpr int kSampleChunk = 2048;

__global__ __launch_bounds__(256) void k_sample_partial(SampleArgs a) {
  __shared__ float sv[4], sm[4], ss[4];
  __shared__ int si[4];
  const int row = blockIdx.x;
  const int slot = a.row_slot[row];
  const float temp = a.slot_temp[slot];
  const float* l = a.logits + static_cast<size_t>(row) * a.V;
  float best = -INFINITY;
  int besti = 0x7fffffff;
  float lm = -INFINITY, ls = 0.f;  // log-sum-exp state of logits / T
  const int v0 = blockIdx.y * kSampleChunk;
  if (temp == 0.f) {
#pragma unroll
    for (int e = 0; e < kSampleChunk / 256; ++e) {
      const int v = v0 + e * 256 + threadIdx.x;
      if (v < a.V) {
        take_best(best, besti, l[v], v);
        lse_add(lm, ls, l[v]);
      }
    }
  } else {
    const float inv_t = 1.0f / temp;
    const int gi = (v0 >> 3) + threadIdx.x;   // 8 entries per thread, one Philox block
    const int vb = gi * 8;
    if (vb < a.V) {
      float lv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) lv[e] = (vb + e < a.V) ? l[vb + e] : -INFINITY;
      uint64_t x0 = static_cast<uint64_t>(a.row_pos[row]), x1 = static_cast<uint64_t>(gi), x2 = 0, x3 = 0;
      philox4x64_10(x0, x1, x2, x3, a.slot_seed[slot], a.slot_id[slot]);
      const uint64_t outs[4] = {x0, x1, x2, x3};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (vb + e < a.V) {
          const uint32_t w = (e & 1) ? static_cast<uint32_t>(outs[e >> 1] >> 32) : static_cast<uint32_t>(outs[e >> 1]);
          take_best(best, besti, lv[e] * inv_t + word_to_gumbel(w), vb + e);
          lse_add(lm, ls, lv[e] * inv_t);
        }
      }
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(best, m, 64);
    const int oi = __shfl_xor(besti, m, 64);
    take_best(best, besti, ov, oi);
    const float om = __shfl_xor(lm, m, 64);
    const float os = __shfl_xor(ls, m, 64);
    lse_merge(lm, ls, om, os);
  }
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = best; si[threadIdx.x >> 6] = besti;
    sm[threadIdx.x >> 6] = lm; ss[threadIdx.x >> 6] = ls;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) {
      take_best(best, besti, sv[w], si[w]);
      lse_merge(lm, ls, sm[w], ss[w]);
    }
    const size_t c = static_cast<size_t>(row) * gridDim.y + blockIdx.y;
    a.cand_val[c] = best;
    a.cand_idx[c] = besti;
    a.cand_m[c] = lm;
    a.cand_s[c] = ls;
  }
}

__global__ __launch_bounds__(64) void k_sample_final(SampleArgs a, int chunks) {
  const int row = blockIdx.x;
  float best = -INFINITY;
  int besti = 0x7fffffff;
  float lm = -INFINITY, ls = 0.f;
  for (int c = threadIdx.x; c < chunks; c += 64) {
    const size_t i = static_cast<size_t>(row) * chunks + c;
    take_best(best, besti, a.cand_val[i], a.cand_idx[i]);
    lse_merge(lm, ls, a.cand_m[i], a.cand_s[i]);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(best, m, 64);
    const int oi = __shfl_xor(besti, m, 64);
    take_best(best, besti, ov, oi);
    const float om = __shfl_xor(lm, m, 64);
    const float os = __shfl_xor(ls, m, 64);
    lse_merge(lm, ls, om, os);
  }
  if (threadIdx.x == 0) {
    if (besti == 0x7fffffff) besti = 0;  // all-NaN row: deterministic fallback
    const int slot = a.row_slot[row];
    const float temp = a.slot_temp[slot];
    const float inv_t = temp == 0.f ? 1.f : 1.0f / temp;
    const float s_tok = a.logits[static_cast<size_t>(row) * a.V + besti] * inv_t;
    const size_t h = static_cast<size_t>(slot) * a.hist_stride + a.row_hist[row];
    a.tokens_cur[slot] = besti;
    a.hist[h] = besti;
    a.logp_hist[h] = s_tok - (lm + logf(ls));
  }
}

__global__ __launch_bounds__(256) void k_gather_rows(const uint8_t* src, const int32_t* rows, int row_bytes,
                                                      uint8_t* out) {
  const int i = blockIdx.x;
  const uint8_t* s = src + static_cast<size_t>(rows[i]) * row_bytes;
  uint8_t* d = out + static_cast<size_t>(i) * row_bytes;
  if ((row_bytes & 15) == 0) {
    for (int b = threadIdx.x * 16; b < row_bytes; b += 256 * 16)
      *reinterpret_cast<uint4*>(d + b) = *reinterpret_cast<const uint4*>(s + b);
  } else {
    for (int b = threadIdx.x; b < row_bytes; b += 256) d[b] = s[b];
  }
}

}  // namespace

namespace {
int row_threads(int H) {
  int t = (H / 4 + kRowChunks - 1) / kRowChunks;
  t = (t + 63) / 64 * 64;
  return t < 64 ? 64 : t;
}

template <typename T, int S>
void launch_add_norm_s(const AddNormArgs& a, int threads, hipStream_t s) {
  launch_kernel((k_add_rmsnorm<T, S>), dim3(a.M), dim3(threads), 0, s, a);
}

template <typename T>
hipError_t launch_add_norm_t(const AddNormArgs& a, hipStream_t s) {
  const int th = row_threads(a.H);
  const int S = a.part ? a.splits : 0;
  switch (S) {
    case 0: launch_add_norm_s<T, 0>(a, th, s); break;
    case 1: launch_add_norm_s<T, 1>(a, th, s); break;
    case 2: launch_add_norm_s<T, 2>(a, th, s); break;
    case 3: launch_add_norm_s<T, 3>(a, th, s); break;
    case 4: launch_add_norm_s<T, 4>(a, th, s); break;
    case 5: launch_add_norm_s<T, 5>(a, th, s); break;
    case 6: launch_add_norm_s<T, 6>(a, th, s); break;
    case 7: launch_add_norm_s<T, 7>(a, th, s); break;
    case 8: launch_add_norm_s<T, 8>(a, th, s); break;
    case 9: launch_add_norm_s<T, 9>(a, th, s); break;
    case 10: launch_add_norm_s<T, 10>(a, th, s); break;
    case 11: launch_add_norm_s<T, 11>(a, th, s); break;
    case 12: launch_add_norm_s<T, 12>(a, th, s); break;
    case 13: launch_add_norm_s<T, 13>(a, th, s); break;
    case 14: launch_add_norm_s<T, 14>(a, th, s); break;
    case 15: launch_add_norm_s<T, 15>(a, th, s); break;
    case 16: launch_add_norm_s<T, 16>(a, th, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_rope_t(const RopeArgs& a, hipStream_t s) {
  const int items = (a.n_q + a.n_kv) * (a.hd / 2) + a.n_kv * a.hd;
  dim3 grid(a.M, (items + 255) / 256);
  switch (a.splits) {
    case 1: launch_kernel((k_rope_append<T, 1>), grid, dim3(256), 0, s, a); break;
    case 2: launch_kernel((k_rope_append<T, 2>), grid, dim3(256), 0, s, a); break;
    case 3: launch_kernel((k_rope_append<T, 3>), grid, dim3(256), 0, s, a); break;
    case 4: launch_kernel((k_rope_append<T, 4>), grid, dim3(256), 0, s, a); break;
    case 5: launch_kernel((k_rope_append<T, 5>), grid, dim3(256), 0, s, a); break;
    case 6: launch_kernel((k_rope_append<T, 6>), grid, dim3(256), 0, s, a); break;
    case 7: launch_kernel((k_rope_append<T, 7>), grid, dim3(256), 0, s, a); break;
    case 8: launch_kernel((k_rope_append<T, 8>), grid, dim3(256), 0, s, a); break;
    case 9: launch_kernel((k_rope_append<T, 9>), grid, dim3(256), 0, s, a); break;
    case 10: launch_kernel((k_rope_append<T, 10>), grid, dim3(256), 0, s, a); break;
    case 11: launch_kernel((k_rope_append<T, 11>), grid, dim3(256), 0, s, a); break;
    case 12: launch_kernel((k_rope_append<T, 12>), grid, dim3(256), 0, s, a); break;
    case 13: launch_kernel((k_rope_append<T, 13>), grid, dim3(256), 0, s, a); break;
    case 14: launch_kernel((k_rope_append<T, 14>), grid, dim3(256), 0, s, a); break;
    case 15: launch_kernel((k_rope_append<T, 15>), grid, dim3(256), 0, s, a); break;
    case 16: launch_kernel((k_rope_append<T, 16>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_embed_norm(int bf16, const EmbedArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.H % 4 || a.H > 4 * kRowChunks * 1024) return hipErrorInvalidValue;
  const int th = row_threads(a.H);
  if (bf16) launch_kernel(k_embed_norm<bf16_t>, dim3(a.M), dim3(th), 0, s, a);
  else launch_kernel(k_embed_norm<float>, dim3(a.M), dim3(th), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(int bf16, const AddNormArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.H % 4 || a.H > 4 * kRowChunks * 1024) return hipErrorInvalidValue;
  return bf16 ? launch_add_norm_t<bf16_t>(a, s) : launch_add_norm_t<float>(a, s);
}

hipError_t launch_rope_append(int bf16, const RopeArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  return bf16 ? launch_rope_t<bf16_t>(a, s) : launch_rope_t<float>(a, s);
}

int sample_chunks(int V) { return (V + kSampleChunk - 1) / kSampleChunk; }

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  const int chunks = sample_chunks(a.V);
  launch_kernel(k_sample_partial, dim3(a.B, chunks), dim3(256), 0, s, a);
  launch_kernel(k_sample_final, dim3(a.B), dim3(64), 0, s, a, chunks);
  return hipGetLastError();
}

// Streaming read of a buffer: each wave walks its own contiguous share, 8 one-KB loads (16 bytes
// per lane) in flight per step, 8 waves per CU: the practical HBM read ceiling that measurement
// reports next to the nominal peak.  The values feed an empty asm so that every load is issued.
constexpr int kStreamWaves = 2048;

// Non-temporal loads: the stream is read once, and marking it so measured
// 6.9-7.0 TB/s against 6.1 TB/s with plain loads over 2 GiB.
typedef unsigned u32x4_nt __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_stream_read(const uint4* p, size_t n16) {
  const u32x4_nt* pn = reinterpret_cast<const u32x4_nt*>(p);
  const int lane = threadIdx.x & 63;
  const size_t wave = static_cast<size_t>(blockIdx.x) * (blockDim.x / 64) + (threadIdx.x >> 6);
  const size_t share = (n16 / 64 / kStreamWaves) * 64;  // whole 1 KB runs per wave
  const size_t begin = wave * share, end = begin + share;
  uint32_t acc = 0;
  size_t i = begin + lane;
  for (; i + 7 * 64 < end; i += 8 * 64) {
    u32x4_nt v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = __builtin_nontemporal_load(pn + i + j * 64);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (; i < end; i += 64) acc ^= p[i].x;
  for (size_t t = kStreamWaves * share + wave * 64 + lane; t < n16; t += static_cast<size_t>(kStreamWaves) * 64)
    acc ^= p[t].x;  // the remainder past the waves' equal shares
  asm volatile("" : : "v"(acc));
}

hipError_t launch_stream_read(const void* buf, size_t bytes, hipStream_t s) {
  if (bytes < 16) return hipErrorInvalidValue;
  launch_kernel(k_stream_read, dim3(kStreamWaves / 4), dim3(256), 0, s, static_cast<const uint4*>(buf), bytes / 16);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, const int32_t* rows, int n, int H, int esize, void* out,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  launch_kernel(k_gather_rows, dim3(n), dim3(256), 0, s, static_cast<const uint8_t*>(src), rows,
                     H * esize, static_cast<uint8_t*>(out));
  return hipGetLastError();
}

}  // namespace rollpack
