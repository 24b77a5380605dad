// Row-wise kernels of the decoder step: embedding + RMSNorm, residual add +
// RMSNorm, q/k/v bias + RoPE + paged KV append, and Gumbel-max sampling with
// a Philox4x64-10 counter-based generator.  All are bandwidth-light: one
// 256-thread block per token row.
#include "device_common.hpp"
#include "kernels.hpp"

namespace rollpack {

namespace {

template <typename T>
__global__ __launch_bounds__(256) void k_embed_norm(EmbedArgs a) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  int tok = a.in_tok[i];
  if (tok < 0) tok = a.tokens_cur[a.row_slot[i]];
  const T* e = static_cast<const T*>(a.embed) + static_cast<size_t>(tok) * a.H;
  float* x = a.x + static_cast<size_t>(i) * a.H;
  float ss = 0.f;
  for (int d = threadIdx.x; d < a.H; d += 256) {
    const float v = Elem<T>::load(e, d);
    x[d] = v;
    ss += v * v;
  }
  ss = block256_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / a.H + a.eps);
  const T* g = static_cast<const T*>(a.norm_g);
  T* h = static_cast<T*>(a.h) + static_cast<size_t>(i) * a.H;
  for (int d = threadIdx.x; d < a.H; d += 256) Elem<T>::store(h, d, x[d] * inv * Elem<T>::load(g, d));
}

template <typename T>
__global__ __launch_bounds__(256) void k_add_rmsnorm(AddNormArgs a) {
  __shared__ float red[4];
  const int i = blockIdx.x;
  float* x = a.x + static_cast<size_t>(i) * a.H;
  const size_t plane = static_cast<size_t>(a.M) * a.H;
  float ss = 0.f;
  for (int d = threadIdx.x; d < a.H; d += 256) {
    float v = x[d];
    if (a.part) {
      const float* p = a.part + static_cast<size_t>(i) * a.H + d;
      for (int s = 0; s < a.splits; ++s) v += p[s * plane];
      x[d] = v;
    }
    ss += v * v;
  }
  ss = block256_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / a.H + a.eps);
  const T* g = static_cast<const T*>(a.norm_g);
  T* h = static_cast<T*>(a.h) + static_cast<size_t>(i) * a.H;
  for (int d = threadIdx.x; d < a.H; d += 256) Elem<T>::store(h, d, x[d] * inv * Elem<T>::load(g, d));
}

template <typename T>
__global__ __launch_bounds__(256) void k_rope_append(RopeArgs a) {
  const int i = blockIdx.x;
  const int hd = a.hd, half = hd / 2;
  const int nq_el = a.n_q * hd, nk_el = a.n_kv * hd;
  const int nqkv = nq_el + 2 * nk_el;
  const size_t plane = static_cast<size_t>(a.M) * nqkv;
  const float* prow = a.part + static_cast<size_t>(i) * nqkv;
  const int pos = a.pos[i];
  const int slot = a.slot[i];
  const int page = a.page_table[static_cast<size_t>(slot) * a.pt_stride + pos / kPageTokens];
  const int off = pos % kPageTokens;
  const T* bq = static_cast<const T*>(a.bq);
  const T* bk = static_cast<const T*>(a.bk);
  const T* bv = static_cast<const T*>(a.bv);
  auto value = [&](int n) {
    float v = 0.f;
    for (int s = 0; s < a.splits; ++s) v += prow[s * plane + n];
    if (n < nq_el) return v + Elem<T>::load(bq, n);
    if (n < nq_el + nk_el) return v + Elem<T>::load(bk, n - nq_el);
    return v + Elem<T>::load(bv, n - nq_el - nk_el);
  };
  const float* cs = a.rope_cos + static_cast<size_t>(pos) * half;
  const float* sn = a.rope_sin + static_cast<size_t>(pos) * half;
  T* q = static_cast<T*>(a.q_out) + static_cast<size_t>(i) * nq_el;
  T* kp = static_cast<T*>(a.k_pool);
  T* vp = static_cast<T*>(a.v_pool);
  // Rotate-half RoPE on q and k heads (k heads follow q heads in the qkv row).
  for (int t = threadIdx.x; t < (a.n_q + a.n_kv) * half; t += 256) {
    const int head = t / half, d = t % half;
    const int n1 = head * hd + d;
    const float u1 = value(n1), u2 = value(n1 + half);
    const float c = cs[d], s = sn[d];
    const float r1 = u1 * c - u2 * s;
    const float r2 = u2 * c + u1 * s;
    if (head < a.n_q) {
      Elem<T>::store(q, n1, r1);
      Elem<T>::store(q, n1 + half, r2);
    } else {
      const int kh = head - a.n_q;
      const size_t base = ((static_cast<size_t>(page) * a.n_kv + kh) * kPageTokens + off) * hd;
      Elem<T>::store(kp, base + d, r1);
      Elem<T>::store(kp, base + d + half, r2);
    }
  }
  for (int t = threadIdx.x; t < nk_el; t += 256) {
    const int kh = t / hd, d = t % hd;
    const float v = value(nq_el + nk_el + t);
    const size_t idx = ((static_cast<size_t>(page) * a.n_kv + kh) * hd + d) * kPageTokens + off;
    Elem<T>::store(vp, idx, v);
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

__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int row = blockIdx.x;
  const int slot = a.row_slot[row];
  const float temp = a.slot_temp[slot];
  const float* l = a.logits + static_cast<size_t>(row) * a.V;
  float best = -INFINITY;
  int besti = 0x7fffffff;
  if (temp == 0.f) {
    for (int v = threadIdx.x; v < a.V; v += 256) take_best(best, besti, l[v], v);
  } else {
    const float inv_t = 1.0f / temp;
    const uint64_t key0 = a.slot_seed[slot], key1 = a.slot_id[slot];
    const uint64_t pos = static_cast<uint64_t>(a.row_pos[row]);
    const int groups = (a.V + 7) / 8;
    for (int gi = threadIdx.x; gi < groups; gi += 256) {
      uint64_t x0 = pos, x1 = static_cast<uint64_t>(gi), x2 = 0, x3 = 0;
      philox4x64_10(x0, x1, x2, x3, key0, key1);
      const uint64_t outs[4] = {x0, x1, x2, x3};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int v = gi * 8 + e;
        if (v < a.V) {
          const uint32_t w = (e & 1) ? static_cast<uint32_t>(outs[e >> 1] >> 32)
                                     : static_cast<uint32_t>(outs[e >> 1]);
          take_best(best, besti, l[v] * inv_t + word_to_gumbel(w), v);
        }
      }
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(best, m, 64);
    const int oi = __shfl_xor(besti, m, 64);
    take_best(best, besti, ov, oi);
  }
  if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = best; si[threadIdx.x >> 6] = besti; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) take_best(best, besti, sv[w], si[w]);
    if (besti == 0x7fffffff) besti = 0;  // all-NaN row: deterministic fallback
    a.tokens_cur[slot] = besti;
    a.hist[static_cast<size_t>(slot) * a.hist_stride + a.row_hist[row]] = besti;
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

hipError_t launch_embed_norm(int bf16, const EmbedArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (bf16) hipLaunchKernelGGL(k_embed_norm<bf16_t>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_embed_norm<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(int bf16, const AddNormArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (bf16) hipLaunchKernelGGL(k_add_rmsnorm<bf16_t>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_add_rmsnorm<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rope_append(int bf16, const RopeArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (bf16) hipLaunchKernelGGL(k_rope_append<bf16_t>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_rope_append<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_sample, dim3(a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, const int32_t* rows, int n, int H, int esize, void* out,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows, dim3(n), dim3(256), 0, s, static_cast<const uint8_t*>(src), rows,
                     H * esize, static_cast<uint8_t*>(out));
  return hipGetLastError();
}

}  // namespace rollpack
