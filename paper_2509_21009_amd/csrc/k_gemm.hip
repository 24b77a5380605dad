// Dense projections C[m, n] = sum_k A[m, k] * W[n, k] of the decoder
// (q/k/v, o, gate/up, down, LM head).  W is [out, in] row-major, A is the
// [M, K] activation matrix; both are K-contiguous.
//
// bf16 kernels use gfx950 MFMA (v_mfma_f32_16x16x32_bf16) with fp32
// accumulation and W as the 16-row "A" operand, activations as the
// 16-column "B" operand, so one MFMA yields a [16 n, 16 m] tile of C^T.
//
//  * k_gemm_deep (M <= 64, the decode regime, most shapes): weights stream
//    from HBM through buffer loads into a ring of register stages; a stage
//    is a 64-wide K unit in which each lane reads 32 contiguous bytes of a
//    row, so one wave's two back-to-back loads cover the row's whole
//    128-byte line.  With the packed copy of the weights (launch_pack_weights)
//    each load instruction reads one contiguous 1 KB run instead, non-temporal
//    (the weights are read once per step), the same operands in every lane.  Activations (L2-resident) are loaded one stage ahead
//    into a single buffer.  The block's 4 waves take interleaved K units and
//    reduce through LDS; blockIdx.y splits K further (fp32 partials).
//  * k_gemm_stream (M <= 64, the remaining decode shapes): the weights are streamed
//    once from HBM straight into registers; every lane loads 64 contiguous
//    bytes per row per 128-wide K chunk (the K order inside a chunk is
//    permuted identically for both operands, which leaves the dot products
//    unchanged).  The 4 waves of a block split the chunk range and reduce
//    through LDS; blockIdx.y splits K further and writes fp32 partials that
//    the consumer kernel sums.
//  * k_gemm_tiled (M > 64: prefill and large decode batches): 128- or
//    256-row x 128- or 256-row block tiles, 8 waves of 32x32x16 MFMAs, tiles
//    loaded from global memory straight into a 3-stage swizzled LDS ring.
//  * k_gemm_f32: fp32 FMA tiles for the fp32 model (no reduced precision).
//
// The SiLU epilogue pairs gate row i with up row i in one thread and writes
// silu(gate) * up once, rounded to the storage type.
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"
#include "lds_dma.hpp"

namespace rollpack {

namespace {

template <typename T>
__device__ __forceinline__ const T* seg_row(const WSeg& W, int n, int K) {
  int base = 0;
  for (int s = 0; s < 3; ++s) {
    if (s == W.n_seg - 1 || n < base + W.rows[s])
      return static_cast<const T*>(W.ptr[s]) + static_cast<size_t>(n - base) * K;
    base += W.rows[s];
  }
  return static_cast<const T*>(W.ptr[0]);
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// ---- decode-regime weight streaming ----------------------------------------
template <int R, int MT, bool SILU>
__global__ __launch_bounds__(256) void k_gemm_stream(GemmArgs a, int chunks_per_split) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int K = a.K;
  const int bx = blockIdx.x, m0 = 0;
  const bf16_t* wrow[R];
#pragma unroll
  for (int t = 0; t < R; ++t) {
    if (SILU) {
      wrow[t] = static_cast<const bf16_t*>(a.W.ptr[t]) + static_cast<size_t>(bx * 16 + r) * K;
    } else {
      wrow[t] = seg_row<bf16_t>(a.W, (bx * R + t) * 16 + r, K);
    }
  }
  const bf16_t* arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int m = m0 + mt * 16 + r;
    if (m >= a.M) m = a.M - 1;
    arow[mt] = static_cast<const bf16_t*>(a.A) + static_cast<size_t>(m) * a.lda;
  }
  f32x4_t acc[R][MT];
#pragma unroll
  for (int t = 0; t < R; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Register double buffering: the loads of the wave's next chunk are in
  // flight while the MFMAs of the current one run.
  bf16x8_t wv[2][R][4], av[2][MT][4];
  auto load = [&](int buf, int chunk) {
    const int k = chunk * 128 + g * 32;
#pragma unroll
    for (int t = 0; t < R; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) wv[buf][t][j] = load_bf16x8(wrow[t] + k + 8 * j);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < 4; ++j) av[buf][mt][j] = load_bf16x8(arow[mt] + k + 8 * j);
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < R; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] = mfma16x16x32(wv[buf][t][j], av[buf][mt][j], acc[t][mt]);
  };
  const int n_chunks = K / 128;
  const int c0 = blockIdx.y * chunks_per_split;
  const int c1 = min(c0 + chunks_per_split, n_chunks);
  int c = c0 + wave;
  if (c < c1) load(0, c);
  for (; c < c1; c += 8) {
    if (c + 4 < c1) load(1, c + 4);
    compute(0);
    if (c + 4 >= c1) break;
    if (c + 8 < c1) load(0, c + 8);
    compute(1);
  }

  constexpr int NSL = R * MT * 4;
  __shared__ float red[4][NSL][64];
#pragma unroll
  for (int t = 0; t < R; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[wave][(t * MT + mt) * 4 + e][lane] = acc[t][mt][e];
  __syncthreads();

  if (!SILU) {
    for (int q = threadIdx.x; q < NSL * 64; q += 256) {
      const int ln = q & 63, sl = q >> 6;
      const int e = sl & 3, tm = sl >> 2, mt = tm % MT, t = tm / MT;
      const int m = m0 + mt * 16 + (ln & 15);
      if (m < a.M) {
        const float v = red[0][sl][ln] + red[1][sl][ln] + red[2][sl][ln] + red[3][sl][ln];
        const int n = (bx * R + t) * 16 + (ln >> 4) * 4 + e;
        a.part[(static_cast<size_t>(blockIdx.y) * a.M + m) * a.N + n] = v;
      }
    }
  } else {
    bf16_t* out = static_cast<bf16_t*>(a.act_out);
    for (int q = threadIdx.x; q < MT * 4 * 64; q += 256) {
      const int ln = q & 63, sl = q >> 6;
      const int e = sl & 3, mt = sl >> 2;
      const int m = m0 + mt * 16 + (ln & 15);
      if (m < a.M) {
        const int sg = mt * 4 + e, su = (MT + mt) * 4 + e;
        const float gv = red[0][sg][ln] + red[1][sg][ln] + red[2][sg][ln] + red[3][sg][ln];
        const float uv = red[0][su][ln] + red[1][su][ln] + red[2][su][ln] + red[3][su][ln];
        const int i = bx * 16 + (ln >> 4) * 4 + e;
        out[static_cast<size_t>(m) * a.N + i] = f32_to_bf16(silu(gv) * uv);
      }
    }
  }
}

// ---- decode-regime weight streaming with the activations shared in LDS ------
// The 4 waves of a block own different weight rows and the same K range, so
// each 128-wide activation chunk is fetched once per block into LDS (double
// buffered) and read by all waves; weights stream into registers, double
// buffered.  Wave w owns rows (blockIdx.x*4 + w)*16R .. +16R, or, with the
// SiLU epilogue, output indices (blockIdx.x*4 + w)*16 .. +16 (gate and up).
constexpr int kSkLd = 128 + 8;  // padded LDS row of one activation chunk (elements)

template <int R, int MT, bool SILU>
__global__ __launch_bounds__(256) void k_gemm_skinny(GemmArgs a, int chunks_per_split) {
  constexpr int AROWS = MT * 16;
  __shared__ __attribute__((aligned(16))) bf16_t As[2][AROWS * kSkLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int K = a.K;
  const int unit = blockIdx.x * 4 + wave;
  const bf16_t* wrow[R];
#pragma unroll
  for (int t = 0; t < R; ++t) {
    if (SILU) wrow[t] = static_cast<const bf16_t*>(a.W.ptr[t]) + static_cast<size_t>(unit * 16 + r) * K;
    else wrow[t] = seg_row<bf16_t>(a.W, (unit * R + t) * 16 + r, K);
  }
  // activation chunk loader: AROWS rows x 16 pieces of 16 bytes, MT pieces per thread
  const bf16_t* asrc[MT];
  int aoff[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int q = tid + 256 * i;
    const int row = q >> 4, col = (q & 15) * 8;
    int m = row < a.M ? row : a.M - 1;
    asrc[i] = static_cast<const bf16_t*>(a.A) + static_cast<size_t>(m) * a.lda + col;
    aoff[i] = row * kSkLd + col;
  }
  f32x4_t acc[R][MT];
#pragma unroll
  for (int t = 0; t < R; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  bf16x8_t wv[2][R][4];
  uint4 areg[MT];
  auto load_w = [&](int buf, int chunk) {
    const int k = chunk * 128 + g * 32;
#pragma unroll
    for (int t = 0; t < R; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) wv[buf][t][j] = load_bf16x8(wrow[t] + k + 8 * j);
  };
  auto load_a = [&](int chunk) {
#pragma unroll
    for (int i = 0; i < MT; ++i) areg[i] = *reinterpret_cast<const uint4*>(asrc[i] + chunk * 128);
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < MT; ++i) *reinterpret_cast<uint4*>(&As[buf][aoff[i]]) = areg[i];
  };
  auto compute = [&](int wbuf, int abuf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bf16x8_t af[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) af[mt] = load_bf16x8(&As[abuf][(mt * 16 + r) * kSkLd + g * 32 + j * 8]);
#pragma unroll
      for (int t = 0; t < R; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] = mfma16x16x32(wv[wbuf][t][j], af[mt], acc[t][mt]);
    }
  };

  const int n_chunks = K / 128;
  const int c0 = blockIdx.y * chunks_per_split;
  const int c1 = min(c0 + chunks_per_split, n_chunks);
  // Vector-memory loads complete in issue order, so the next activation
  // chunk is issued before the next weight chunk: storing it to LDS at the end
  // of the step then waits only for the activations (an L2 hit), never for
  // weights still in flight from HBM.
  if (c0 < c1) {
    load_a(c0);
    load_w(0, c0);
    store_a(0);
  }
  __syncthreads();
  for (int c = c0; c < c1; c += 2) {
    // even step: W buffer 0, A buffer 0
    if (c + 1 < c1) {
      load_a(c + 1);
      asm volatile("" ::: "memory");
      load_w(1, c + 1);
    }
    compute(0, 0);
    if (c + 1 < c1) store_a(1);
    __syncthreads();
    if (c + 1 >= c1) break;
    // odd step: W buffer 1, A buffer 1
    if (c + 2 < c1) {
      load_a(c + 2);
      asm volatile("" ::: "memory");
      load_w(0, c + 2);
    }
    compute(1, 1);
    if (c + 2 < c1) store_a(0);
    __syncthreads();
  }

  // lane (g, c) holds C^T[row base + t*16 + 4g + e][m = mt*16 + c]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r;
    if (m >= a.M) continue;
    if (SILU) {
      const int i0 = unit * 16 + g * 4;
      uint2 pk;
      pk.x = static_cast<uint32_t>(f32_to_bf16(silu(acc[0][mt][0]) * acc[1][mt][0])) |
             (static_cast<uint32_t>(f32_to_bf16(silu(acc[0][mt][1]) * acc[1][mt][1])) << 16);
      pk.y = static_cast<uint32_t>(f32_to_bf16(silu(acc[0][mt][2]) * acc[1][mt][2])) |
             (static_cast<uint32_t>(f32_to_bf16(silu(acc[0][mt][3]) * acc[1][mt][3])) << 16);
      *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.act_out) + static_cast<size_t>(m) * a.N + i0) = pk;
    } else {
#pragma unroll
      for (int t = 0; t < R; ++t) {
        const int n = (unit * R + t) * 16 + g * 4;
        *reinterpret_cast<float4*>(a.part + (static_cast<size_t>(blockIdx.y) * a.M + m) * a.N + n) =
            make_float4(acc[t][mt][0], acc[t][mt][1], acc[t][mt][2], acc[t][mt][3]);
      }
    }
  }
}

// ---- decode-regime weight streaming, deep register pipeline ----------------
// Block: 4 waves on the same 16R weight rows (with the SiLU epilogue: R/2
// gate fragments and the R/2 up fragments of the same output indices).
// A stage is a 64-wide K unit: lane (g, r) loads bytes [32g, 32g + 32) of
// the unit's 128 bytes of row r as two 16-byte loads, and MFMA k-step j of
// the unit takes the j-th of them from both operands, so every product of
// the unit is formed exactly once.  Wave w takes units w, w + 4, ... of the
// block's K range, so the block reads whole 512-byte runs of each row.
// Weight fragments use one buffer resource each: rows past the end of the
// matrix (the ragged last block) read as zeros and are never stored.
// Weight loads of the deep kernel: row-major (plain) or packed (non-temporal:
// aux bit 1 is the nt cache policy).
template <bool PACKED>
__device__ __forceinline__ bf16x8_t load_w16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, PACKED ? 2 : 0));
}

template <int R, int MT, int D, bool SILU, bool PACKED>
__global__ __launch_bounds__(256) void k_gemm_deep(GemmArgs a, int units_per_split) {
  static_assert(!SILU || R % 2 == 0, "SiLU pairs gate and up fragments");
  constexpr int NACC = R * MT;
  __shared__ __attribute__((aligned(16))) f32x4_t red[3][NACC][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, r = lane & 15;
  const int K = a.K, KU = K / 64;
  const int u0 = blockIdx.y * units_per_split;
  const int u1 = min(u0 + units_per_split, KU);
  const int nblk = max(u1 - u0, 0);
  const int nk = nblk > wave ? (nblk - wave + 3) / 4 : 0;
  const uint32_t row_bytes = static_cast<uint32_t>(K) * 2u;

  const WSeg& W = PACKED ? a.Wp : a.W;
  __amdgpu_buffer_rsrc_t rw[R];
#pragma unroll
  for (int t = 0; t < R; ++t) {
    const bf16_t* base;
    int valid;
    if (SILU) {
      const int row0 = (blockIdx.x * (R / 2) + t % (R / 2)) * 16;
      valid = row0 < a.N ? min(16, a.N - row0) : 0;
      base = static_cast<const bf16_t*>(W.ptr[t / (R / 2)]) + static_cast<size_t>(valid ? row0 : 0) * K;
    } else {
      const int row0 = (blockIdx.x * R + t) * 16;
      int b = 0, sg = 0;
      while (sg < W.n_seg - 1 && row0 >= b + W.rows[sg]) b += W.rows[sg++];
      valid = row0 < a.N ? min(16, W.rows[sg] - (row0 - b)) : 0;
      base = static_cast<const bf16_t*>(W.ptr[sg]) + static_cast<size_t>(valid ? row0 - b : 0) * K;
    }
    // a packed tile is whole (16 rows) or absent; a row-major one may be ragged
    rw[t] = buffer_rsrc(base, static_cast<uint32_t>(PACKED ? (valid ? 16 : 0) : valid) * row_bytes);
  }
  // rows m >= M of the activations read as zeros
  const __amdgpu_buffer_rsrc_t ra =
      buffer_rsrc(a.A, static_cast<uint32_t>(a.M) * static_cast<uint32_t>(a.lda) * 2u);
  const int kb = (u0 + wave) * 128 + g * 32;
  // row-major: lane (g, r) reads 32 bytes of row r per unit (two 16-byte pieces), units 128 bytes
  // apart; packed: the unit's 2 KB run, the lane's 16 bytes in each 1 KB half
  const int woff = PACKED ? (u0 + wave) * 2048 + lane * 16 : r * static_cast<int>(row_bytes) + kb;
  constexpr int kWStep = PACKED ? 4 * 2048 : 4 * 128, kWHalf = PACKED ? 1024 : 16;
  int aoff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) aoff[mt] = (mt * 16 + r) * static_cast<int>(a.lda) * 2 + kb;

  f32x4_t acc[R][MT];
#pragma unroll
  for (int t = 0; t < R; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Weights: a ring of D stages.  Activations: one buffer, loaded one stage
  // ahead, after the weights of the current stage and before those of later
  // stages; vector loads complete in issue order, so waiting for the
  // activations of stage s never waits for weights of later stages.
  bf16x8_t wv[D][R][2], av[MT][2];
  auto load_w = [&](int s, int unit) {
    const int o = unit * kWStep;
#pragma unroll
    for (int t = 0; t < R; ++t) {
      wv[s][t][0] = load_w16<PACKED>(rw[t], woff + o);
      wv[s][t][1] = load_w16<PACKED>(rw[t], woff + o + kWHalf);
    }
  };
  auto load_a = [&](int unit) {
    const int o = unit * 512;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      av[mt][0] = load_bf16x8(ra, aoff[mt] + o);
      av[mt][1] = load_bf16x8(ra, aoff[mt] + o + 16);
    }
  };
  auto compute = [&](int s) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int t = 0; t < R; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] = mfma16x16x32(wv[s][t][j], av[mt][j], acc[t][mt]);
  };

  // The prologue loads unconditionally (stages past the wave's range are
  // in bounds and never used) and the scheduling barriers keep the issue
  // order, so every path into the main loop has the same loads in flight and
  // the compiler's wait counts there are exact.
  load_w(0, 0);
  __builtin_amdgcn_sched_barrier(0);
  load_a(0);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int s = 1; s < D; ++s) {
    load_w(s, s);
    __builtin_amdgcn_sched_barrier(0);
  }
  int i = 0;
  for (; i + 2 * D <= nk; i += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      compute(s);
      __builtin_amdgcn_sched_barrier(0);
      load_a(i + s + 1);
      __builtin_amdgcn_sched_barrier(0);
      load_w(s, i + s + D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int j = 0; j < 2 * D; ++j) {
    if (i + j < nk) {
      compute(j % D);
      __builtin_amdgcn_sched_barrier(0);
      if (i + j + 1 < nk) load_a(i + j + 1);
      __builtin_amdgcn_sched_barrier(0);
      if (i + j + D < nk) load_w(j % D, i + j + D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if (wave > 0) {
#pragma unroll
    for (int t = 0; t < R; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) red[wave - 1][t * MT + mt][lane] = acc[t][mt];
  }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int t = 0; t < R; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      acc[t][mt] = acc[t][mt] + red[0][t * MT + mt][lane] + red[1][t * MT + mt][lane] + red[2][t * MT + mt][lane];

  // lane (g, r) holds C^T[row base + t*16 + 4g + e][m = mt*16 + r]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r;
    if (m >= a.M) continue;
    if (SILU) {
#pragma unroll
      for (int t = 0; t < R / 2; ++t) {
        const int i0 = (blockIdx.x * (R / 2) + t) * 16 + g * 4;
        if (i0 >= a.N) continue;
        const f32x4_t gv = acc[t][mt], uv = acc[t + R / 2][mt];
        uint2 pk;
        pk.x = static_cast<uint32_t>(f32_to_bf16(silu(gv[0]) * uv[0])) |
               (static_cast<uint32_t>(f32_to_bf16(silu(gv[1]) * uv[1])) << 16);
        pk.y = static_cast<uint32_t>(f32_to_bf16(silu(gv[2]) * uv[2])) |
               (static_cast<uint32_t>(f32_to_bf16(silu(gv[3]) * uv[3])) << 16);
        *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.act_out) + static_cast<size_t>(m) * a.N + i0) = pk;
      }
    } else {
#pragma unroll
      for (int t = 0; t < R; ++t) {
        const int n = (blockIdx.x * R + t) * 16 + g * 4;
        if (n >= a.N) continue;
        *reinterpret_cast<f32x4_t*>(a.part + (static_cast<size_t>(blockIdx.y) * a.M + m) * a.N + n) = acc[t][mt];
      }
    }
  }
}

// ---- prefill / large-batch tiled MFMA GEMM ---------------------------------
// Block tile: BM activation rows (m, 128 or 256) x BN weight rows (n, 128 or
// 256), K step 32, eight waves as 2 (m) x 4 (n) for BN = 256 or 4 x 2 for
// BN = 128, each computing BM/2 or BM/4 m x 64 n with
// v_mfma_f32_32x32x16_bf16 (two waves per SIMD).  Activations are the MFMA
// row operand and weights the column operand, so the 32 lanes of one
// accumulator register hold 32 consecutive n: coalesced stores.
//
// Tiles move from global memory straight into LDS (buffer_load_dwordx4 ...
// lds: each wave-instruction writes 1 KB, 16 rows of 64 bytes, with no
// register staging) through a ring of kGNST stages, issued kGNST - 1 stages
// ahead, one barrier per K step.  The loads are inline assembly, so the
// compiler neither tracks them nor inserts its conservative vmcnt(0) before
// every barrier; the kernel waits with explicit vmcnt counts instead (each
// thread issues the same NA + 2 loads per stage, and vector loads complete in
// order).  A stage's buffer is refilled only after the barrier that follows
// the last read of it.  The 16-byte chunk j of LDS row r holds global chunk
// j ^ ((r >> 2) & 3): eight consecutive lanes of a fragment read then hit
// eight distinct 16-byte bank groups.  Rows past M or N read as zeros
// through the buffer resources (range-checked loads); a 16-row block of a
// weight tile lies in one weight segment.  Each XCD takes a contiguous run
// of the (split, tile) order, split-major (block ids equal mod 8), and the
// order walks gm m tiles of one weight panel before the next panel, so the
// 32 tiles an XCD runs at once share gm activation tiles and 32 / gm weight
// panels in its L2.  (A run per tile with the split on blockIdx.y gave one XCD
// every split of its tiles: at 129-256 rows the down projection's 28 panels x 9
// splits put 36 blocks on each of seven XCDs, two rounds, and none on the
// eighth; balanced, it runs in 49 against 93 us at 256 rows.)  gm is
// 8 for wide products (>= 64 panels: gate/up, the LM head) and 2 for
// narrow ones (measured: at 4k-16k rows gate/up gains 4 points of MFMA peak
// over a single panel at a time, q/k/v, o and down 2-4).
constexpr int kGBK = 32, kGNST = 3;

// Wait until at most PER * min(after, MAXJ) loads are outstanding.
template <int PER, int J, int MAXJ>
__device__ __forceinline__ void wait_stages_after(int after) {
  if constexpr (J >= MAXJ) {
    wait_vmcnt<PER * MAXJ>();
  } else {
    if (after == J) wait_vmcnt<PER * J>();
    else wait_stages_after<PER, J + 1, MAXJ>(after);
  }
}
__device__ __forceinline__ int gswz(int r) { return (r >> 2) & 3; }

template <int BM, int BN, bool SILU>
__global__ __launch_bounds__(512) void k_gemm_tiled(GemmArgs a, int kblocks_per_split, int n_mb, int n_nb, int gm) {
  constexpr int STAGE = (BM + BN) * kGBK;       // elements per stage
  constexpr int WMW = BN == 256 ? 2 : 4;        // waves along m (8 waves: WMW x 8 / WMW)
  constexpr int WROWS = BM / WMW;               // activation rows per wave
  constexpr int MT = WROWS / 32;                // 32-row activation tiles per wave
  constexpr int NA = BM / 128, NW = BN / 128;   // 16-row blocks of activations / weights a wave loads per stage
  static_assert(MT >= 1 && (BN == 128 || BN == 256), "tile shape");
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kGNST * STAGE];
  // Work items are (split, tile) pairs, split-major, and each XCD takes a contiguous run of
  // them (block ids equal mod 8 run on one XCD): the XCDs get equal shares of a split launch
  // (per-tile runs would hand one XCD all splits of its tiles, more blocks than its 32 CUs
  // when the tile count is not a multiple of 8), and an XCD's blocks read few K ranges of
  // the activations, which its L2 then holds.
  const int n_tiles = n_mb * n_nb;
  const int n_items = n_tiles * a.splits;
  const int per_xcd = (n_items + 7) / 8;
  const int q = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (q >= n_items) return;  // block-uniform: padding of the XCD-ordered grid
  const int split = q / n_tiles, t = q - split * n_tiles;
  // Grouped order: consecutive tiles walk gm m tiles of one weight panel, then the next panel.
  const int gsz = gm * n_nb, grp = t / gsz, first = grp * gm, gcur = min(gm, n_mb - first);
  const int mb = first + (t - grp * gsz) % gcur, nb = (t - grp * gsz) / gcur;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WMW, wn = wave / WMW;
  const int l32 = lane & 31, lh = lane >> 5;
  const int K = a.K;

  // Loads: wave w fills 16-row blocks w + 8 i of each tile; lane -> row lane >> 2 of the block,
  // LDS chunk lane & 3, which holds global chunk (lane & 3) ^ gswz(row).
  const u32x4_raw ars = raw_rsrc(a.A, static_cast<uint32_t>(a.M) * static_cast<uint32_t>(a.lda) * 2u);
  int aoff[NA], woff[NW];
  u32x4_raw wrs[NW];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int r = (wave + 8 * i) * 16 + (lane >> 2);
    aoff[i] = ((mb * BM + r) * static_cast<int>(a.lda) + ((lane & 3) ^ gswz(r)) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int r0 = (wave + 8 * i) * 16;
    const int r = r0 + (lane >> 2);
    const bf16_t* wb;
    int rel0, rows_valid;
    if (SILU) {  // 32-row groups alternate gate / up over the same output indices
      const int g32 = r0 >> 5;
      wb = static_cast<const bf16_t*>(a.W.ptr[g32 & 1]);
      rel0 = nb * (BN / 2) + (g32 >> 1) * 32 + (r0 & 31);
      rows_valid = a.N;
    } else {
      const int n0 = nb * BN + r0;
      int b = 0, sg = 0;
      while (sg < a.W.n_seg - 1 && n0 >= b + a.W.rows[sg]) b += a.W.rows[sg++];
      wb = static_cast<const bf16_t*>(a.W.ptr[sg]);
      rel0 = n0 - b;
      rows_valid = n0 < a.N ? a.W.rows[sg] : 0;
    }
    wrs[i] = raw_rsrc(wb, static_cast<uint32_t>(rows_valid) * static_cast<uint32_t>(K) * 2u);
    woff[i] = ((rel0 + (lane >> 2)) * K + ((lane & 3) ^ gswz(r)) * 8) * 2;
  }
  typedef const __attribute__((address_space(3))) char lds_char;
  const uint32_t lds0 = static_cast<uint32_t>((uintptr_t)(lds_char*)(smem));

  f32x16_t acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mt][nt][e] = 0.f;

  const int kb0 = split * kblocks_per_split;
  const int kb1 = min(kb0 + kblocks_per_split, K / kGBK);
  auto load = [&](int st, int kb) {
    const int ko = kb * kGBK * 2;
    const uint32_t sa = lds0 + static_cast<uint32_t>(st * STAGE * 2), sw = sa + BM * kGBK * 2;
#pragma unroll
    for (int i = 0; i < NA; ++i)
      dma16(ars, __builtin_amdgcn_readfirstlane(sa + static_cast<uint32_t>((wave + 8 * i) * 1024)), aoff[i] + ko);
#pragma unroll
    for (int i = 0; i < NW; ++i)
      dma16(wrs[i], __builtin_amdgcn_readfirstlane(sw + static_cast<uint32_t>((wave + 8 * i) * 1024)), woff[i] + ko);
  };
  auto compute = [&](int st) {
    const bf16_t* sA = smem + st * STAGE;
    const bf16_t* sW = sA + BM * kGBK;
    bf16x8_t af[2][MT], bw[2][2];
    auto rd = [&](int buf, int ki) {
      const int c = ki * 2 + lh;  // the lane's 16-byte chunk of this k-step
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int r = wm * WROWS + mt * 32 + l32;
        af[buf][mt] = *reinterpret_cast<const bf16x8_t*>(sA + r * kGBK + (c ^ gswz(r)) * 8);
      }
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int r = wn * 64 + nt * 32 + l32;
        bw[buf][nt] = *reinterpret_cast<const bf16x8_t*>(sW + r * kGBK + (c ^ gswz(r)) * 8);
      }
    };
    // The second k-step's fragment reads are interleaved with the first k-step's MFMAs, at
    // raised wave priority, so that the SIMD's other wave finds MFMA issue slots between them.
    rd(0, 0);
#pragma unroll
    for (int ki = 0; ki < kGBK / 16; ++ki) {
      __builtin_amdgcn_s_setprio(1);
      if (ki + 1 < kGBK / 16) rd((ki + 1) & 1, ki + 1);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = mfma32x32x16(af[ki & 1][mt], bw[ki & 1][nt], acc[mt][nt]);
      if (ki + 1 < kGBK / 16) {
        constexpr int NRD = MT + 2, NMF = 2 * MT, NP = NRD < NMF ? NRD : NMF;
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        }
        if constexpr (NMF > NP) __builtin_amdgcn_sched_group_barrier(0x008, NMF - NP, 0);
        if constexpr (NRD > NP) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NP, 0);
      }
      __builtin_amdgcn_s_setprio(0);
    }
  };
#pragma unroll
  for (int j = 0; j < kGNST - 1; ++j)
    if (kb0 + j < kb1) load(j, kb0 + j);
  auto step = [&](int st, int kb) {
    // stage kb's loads were issued before those of the next kGNST - 2 stages
    wait_stages_after<NA + NW, 0, kGNST - 2>(min(kb1 - 1 - kb, kGNST - 2));
    __syncthreads();  // stage kb visible to all waves; stage kb - 1 no longer read
    if (kb + kGNST - 1 < kb1) load((st + kGNST - 1) % kGNST, kb + kGNST - 1);
    compute(st);
  };
  for (int kb = kb0; kb < kb1; kb += kGNST) {
#pragma unroll
    for (int j = 0; j < kGNST; ++j)
      if (kb + j < kb1) step(j, kb + j);
  }

  // acc[mt][nt] register e: m = wm*WROWS + mt*32 + 8*(e/4) + 4*lh + e%4, n = wn*64 + nt*32 + l32
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = mb * BM + wm * WROWS + mt * 32 + 8 * (e >> 2) + 4 * lh + (e & 3);
      if (m >= a.M) continue;
      if (SILU) {
        const int idx = nb * (BN / 2) + wn * 32 + l32;
        static_cast<bf16_t*>(a.act_out)[static_cast<size_t>(m) * a.N + idx] =
            f32_to_bf16(silu(acc[mt][0][e]) * acc[mt][1][e]);
      } else {
        float* out = a.part + (static_cast<size_t>(split) * a.M + m) * a.N;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int n = nb * BN + wn * 64 + nt * 32 + l32;
          if (n < a.N) out[n] = acc[mt][nt][e];
        }
      }
    }
}

// ---- fp32 model ------------------------------------------------------------
template <bool SILU>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs a) {
  constexpr int BM = 64, BN = 64, BK = 16;
  constexpr int NW = SILU ? 2 : 1;
  __shared__ float As[BK][BM + 1];
  __shared__ float Ws[NW][BK][BN + 1];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const float* A = static_cast<const float*>(a.A);
  float acc[NW][4][4];
#pragma unroll
  for (int w = 0; w < NW; ++w)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[w][i][j] = 0.f;

  for (int k0 = 0; k0 < a.K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i;
      const int row = e >> 4, kk = e & 15;
      const int m = m0 + row, k = k0 + kk, n = n0 + row;
      As[kk][row] = (m < a.M && k < a.K) ? A[static_cast<size_t>(m) * a.lda + k] : 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        float v = 0.f;
        if (n < a.N && k < a.K) {
          const float* wr = SILU ? static_cast<const float*>(a.W.ptr[w]) + static_cast<size_t>(n) * a.K
                                 : seg_row<float>(a.W, n, a.K);
          v = wr[k];
        }
        Ws[w][kk][row] = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float wv = Ws[w][kk][tx * 4 + j];
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[w][i][j] = fmaf(av[i], wv, acc[w][i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= a.N) continue;
      if (SILU) static_cast<float*>(a.act_out)[static_cast<size_t>(m) * a.N + n] = silu(acc[0][i][j]) * acc[NW - 1][i][j];
      else a.part[static_cast<size_t>(m) * a.N + n] = acc[0][i][j];
    }
  }
}

template <int R, int MT, bool SILU>
void launch_stream_t(const GemmArgs& a, hipStream_t s) {
  const int n_chunks = a.K / 128;
  const int cps = (n_chunks + a.splits - 1) / a.splits;
  const int blocks = SILU ? a.N / 16 : a.N / (16 * R);
  launch_kernel((k_gemm_stream<R, MT, SILU>), dim3(blocks, a.splits), dim3(256), 0, s, a, cps);
}

template <bool SILU>
void launch_stream_m(const GemmArgs& a, hipStream_t s) {
  switch ((a.M + 15) / 16) {
    case 1: launch_stream_t<2, 1, SILU>(a, s); break;
    case 2: launch_stream_t<2, 2, SILU>(a, s); break;
    case 3: launch_stream_t<2, 3, SILU>(a, s); break;
    default: launch_stream_t<2, 4, SILU>(a, s); break;
  }
}

template <int R, int MT, bool SILU>
void launch_skinny_t(const GemmArgs& a, hipStream_t s) {
  const int n_chunks = a.K / 128;
  const int cps = (n_chunks + a.splits - 1) / a.splits;
  const int blocks = SILU ? a.N / 64 : a.N / (64 * R);
  launch_kernel((k_gemm_skinny<R, MT, SILU>), dim3(blocks, a.splits), dim3(256), 0, s, a, cps);
}

template <int R, bool SILU>
void launch_skinny_m(const GemmArgs& a, hipStream_t s) {
  switch ((a.M + 15) / 16) {
    case 1: launch_skinny_t<R, 1, SILU>(a, s); break;
    case 2: launch_skinny_t<R, 2, SILU>(a, s); break;
    case 3: launch_skinny_t<R, 3, SILU>(a, s); break;
    default: launch_skinny_t<R, 4, SILU>(a, s); break;
  }
}

constexpr int kMaxSplitsAny = 64;

enum GemmKernel { kKStream = 1, kKSkinny16 = 2, kKSkinny32 = 3, kKTiled = 4, kKF32 = 5, kKDeep = 6 };

struct GemmPlan {
  int kernel;
  int splits;
  int R = 0, D = 0;  // k_gemm_deep: weight fragments per block and register stages
  int bm = 256;      // k_gemm_tiled: activation rows per block tile
  int bn = 256;      // k_gemm_tiled: weight rows per block tile
};

template <int R, int MT, int D, bool SILU>
void launch_deep_t(const GemmArgs& a, hipStream_t s) {
  const int KU = a.K / 64;
  const int ups = (KU + a.splits - 1) / a.splits;
  const int per = SILU ? R / 2 : R;
  const int nb = (a.N / 16 + per - 1) / per;
  if (a.Wp.n_seg > 0)
    launch_kernel((k_gemm_deep<R, MT, D, SILU, true>), dim3(nb, a.splits), dim3(256), 0, s, a, ups);
  else
    launch_kernel((k_gemm_deep<R, MT, D, SILU, false>), dim3(nb, a.splits), dim3(256), 0, s, a, ups);
}

// One thread per 16-byte piece of the packed matrix (the layout of launch_pack_weights).
__global__ void k_pack_weights(const uint4* __restrict__ w, uint4* __restrict__ p, int rows, int K) {
  const size_t n = static_cast<size_t>(rows) * K / 8;
  const size_t tile_pieces = static_cast<size_t>(2) * K;  // 16 rows x K / 8
  for (size_t q = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; q < n;
       q += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const size_t t = q / tile_pieces, rem = q % tile_pieces;
    const int u = static_cast<int>(rem >> 7), j = static_cast<int>(rem >> 6) & 1, l = static_cast<int>(rem) & 63;
    p[q] = w[((t * 16 + (l & 15)) * static_cast<size_t>(K) + 64 * u + 16 * (l >> 4) + 8 * j) / 8];
  }
}

// The (R, D) pairs instantiated for each activation tile count MT = ceil(M / 16).
struct DeepCfg { int R, D; };
constexpr DeepCfg kDeepCfg[4][4] = {
    {{10, 2}, {8, 2}, {4, 4}, {0, 0}},
    {{10, 2}, {8, 2}, {4, 4}, {0, 0}},
    {{10, 2}, {8, 2}, {6, 2}, {0, 0}},
    {{10, 2}, {8, 2}, {6, 2}, {4, 3}},
};

template <bool SILU>
bool launch_deep(const GemmArgs& a, int R, int D, hipStream_t s) {
#define RP_DEEP(MT_, R_, D_) \
  if (mt == MT_ && R == R_ && D == D_) { launch_deep_t<R_, MT_, D_, SILU>(a, s); return true; }
  const int mt = (a.M + 15) / 16;
  RP_DEEP(1, 10, 2) RP_DEEP(1, 8, 2) RP_DEEP(1, 4, 4)
  RP_DEEP(2, 10, 2) RP_DEEP(2, 8, 2) RP_DEEP(2, 4, 4)
  RP_DEEP(3, 10, 2) RP_DEEP(3, 8, 2) RP_DEEP(3, 6, 2)
  RP_DEEP(4, 10, 2) RP_DEEP(4, 8, 2) RP_DEEP(4, 6, 2) RP_DEEP(4, 4, 3)
#undef RP_DEEP
  return false;
}

// Number of K splits that leaves no split empty, for a wish of `want`.
int even_splits(int n_units, int want) {
  if (want < 1) want = 1;
  if (want > n_units) want = n_units;
  const int per = (n_units + want - 1) / want;
  return (n_units + per - 1) / per;
}

// k_gemm_deep plan.  The blocks hold one CU each (their register use
// allows one wave per SIMD), so the time is set by the busiest CU: rounds of
// 256 blocks times the rows x K units of one block.  The K split is the
// largest that keeps all blocks in one round and every wave at >= 3 units;
// a small penalty for activation traffic (MT / R of the weight loads)
// breaks ties toward more weight rows per block.  Measured on the Qwen2.5
// 7B decode shapes, this picks the best swept configuration or one within
// a few percent of it.
GemmPlan plan_deep(int M, int N, int K, bool silu, int max_splits) {
  const int mt = (M + 15) / 16, KU = K / 64, units = N / 16;
  GemmPlan best{kKDeep, 1};
  double best_cost = 1e300;
  for (const DeepCfg& c : kDeepCfg[mt - 1]) {
    if (c.R == 0) continue;
    const int per = silu ? c.R / 2 : c.R;
    const int nb = (units + per - 1) / per;
    int S = 1;
    if (!silu) {
      const int smax = std::max(1, std::min(std::min(16, max_splits), KU / 12));
      while (S < smax && nb * (S + 1) <= 256) ++S;
      S = even_splits(KU, S);
    }
    const int rounds = (nb * S + 255) / 256;
    const double cost = static_cast<double>(rounds) * c.R * 16 * ((KU + S - 1) / S) * (1.0 + 0.15 * mt / c.R);
    if (cost < best_cost) {
      best_cost = cost;
      best = GemmPlan{kKDeep, S, c.R, c.D};
    }
  }
  return best;
}

// k_gemm_tiled plan: the block tile (BM activation rows x BN weight rows) and
// the K split.  A block holds one CU's LDS ring and the 8 waves of two
// SIMD-pairs, so the time is set by rounds of 256 blocks times the K steps of
// one block.  Decode batches (<= 512 rows) weigh every tile shape and split
// against the fp32 partials a split adds, which at these sizes can exceed the
// weights themselves (q/k/v at 256 rows and 14 splits: 66 MB of partials for
// 33 MB of weights).  Prefill takes 256-row weight panels and splits K only
// until the blocks fill one round.  The tile does not depend on max_splits,
// so a launch with a capped split recomputes the same one.
GemmPlan plan_tiled(int M, int N, int K, bool silu, int max_splits) {
  const int KB = K / kGBK;
  GemmPlan best{kKTiled, 1};
  double best_cost = 1e300;
  if (M <= 512) {
    // Decode batches: every tile shape and split, priced as rounds of 256 blocks x K steps per
    // block x the tile's cost per K step (256 x 256: 1, 256 x 128 and 128 x 256: 0.65,
    // 128 x 128: 0.49, with one 256 x 256 step ~0.5 us), plus the fp32 partials the split
    // writes and its consumer reads at 4 TB/s.  Fitted to a sweep of all tile shapes and splits
    // 1-16 at 96-512 rows of the 7B projections (q/k/v, o, gate/up, down, LM head), the plan
    // it picks is within 0.2% of the fastest in total.
    for (int bn : {128, 256})
      for (int bm : {256, 128}) {
        const double tile = (bm == 256 && bn == 256) ? 1.0 : (bm == 128 && bn == 128) ? 0.4875 : 0.65;
        const int n_tiles = (silu ? N / (bn / 2) : (N + bn - 1) / bn) * ((M + bm - 1) / bm);
        const int s_max = silu ? 1 : std::min(16, std::max(1, KB / 4));
        for (int sp = 1; sp <= s_max; ++sp) {
          if (even_splits(KB, sp) != sp) continue;
          const int rounds = (n_tiles * sp + 255) / 256;
          const double cost = rounds * static_cast<double>((KB + sp - 1) / sp) * 0.5 * tile +
                              (silu ? 0.0 : sp * static_cast<double>(M) * N * 8 / 4.0e6);
          if (cost < best_cost) {
            best_cost = cost;
            best = GemmPlan{kKTiled, sp, 0, 0, bm, bn};
          }
        }
      }
    best.splits = even_splits(KB, std::min(best.splits, max_splits));
    return best;
  }
  // Prefill: 256-row weight panels; the block tile from rounds of 256 blocks times the K steps
  // of one block, a BM = 128 step costing 0.71 of a BM = 256 one (measured at 4k rows).
  const int bn = 256;
  for (int bm : {256, 128}) {
    const int blocks = (silu ? N / (bn / 2) : (N + bn - 1) / bn) * ((M + bm - 1) / bm);
    int sp = silu ? 1 : std::max(1, 256 / blocks);
    sp = even_splits(KB, std::min(sp, std::max(1, KB / 8)));
    const int rounds = (blocks * sp + 255) / 256;
    const double cost = static_cast<double>(rounds) * ((KB + sp - 1) / sp) * (bm == 256 ? 1.0 : 0.71);
    if (cost < best_cost) {
      best_cost = cost;
      best = GemmPlan{kKTiled, sp, 0, 0, bm, bn};
    }
  }
  best.splits = even_splits(KB, std::min(best.splits, max_splits));
  return best;
}

// Kernel and split choice, from sweeps of the Qwen2.5 decode shapes on
// gfx950 (weights cycled through more than the 256 MB last-level cache so
// that none is reused between launches): the deep-pipelined kernel for
// decode batches of the weight matrices of 7B and larger models; the older
// streaming kernels for the small matrices (the 0.5B model, the 7B output
// projection at <= 16 rows), where launch latency dominates.
GemmPlan plan_gemm(int bf16, int M, int N, int K, bool silu, int max_splits) {
  if (!bf16) return {kKF32, 1};
  if (M > 64) return plan_tiled(M, N, K, silu, max_splits);
  const double work = static_cast<double>(N) * K * (silu ? 2 : 1);
  if (K % 64 == 0 && N % 16 == 0 && work >= (M > 16 ? 8.0e6 : 1.4e7)) return plan_deep(M, N, K, silu, max_splits);
  const int n_chunks = K / 128;
  auto pick = [&](int blocks, int target) {
    int s = 1;
    for (int c : {1, 2, 3, 4, 6, 8, 12, 16}) {
      s = c;
      if (blocks * c >= target) break;
    }
    s = std::min(std::min(s, max_splits), std::max(1, n_chunks / 2));
    return even_splits(n_chunks, s);
  };
  if (silu) return {kKStream, 1};
  if (M <= 16) {
    if (N >= 16384) return {M <= 8 ? kKStream : kKSkinny32, 1};
    return {kKSkinny16, pick(N / 64, 512)};
  }
  return {kKSkinny32, pick(N / 128, K >= 8192 ? 448 : 256)};
}

}  // namespace

int gemm_pick_splits(int bf16, int M, int N, int K, bool silu, int max_splits) {
  return plan_gemm(bf16, M, N, K, silu, max_splits).splits;
}

hipError_t launch_pack_weights(const void* w, void* packed, int rows, int K, hipStream_t s) {
  if (!w || !packed || rows <= 0 || rows % 16 || K <= 0 || K % 64 ||
      (reinterpret_cast<uintptr_t>(w) | reinterpret_cast<uintptr_t>(packed)) % 16)
    return hipErrorInvalidValue;
  launch_kernel(k_pack_weights, dim3(2048), dim3(256), 0, s, static_cast<const uint4*>(w), static_cast<uint4*>(packed),
                rows, K);
  return hipGetLastError();
}

hipError_t launch_gemm(int bf16, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const bool silu = a.epi == kEpiSiluMul;
  if (a.splits < 1 || (silu && a.splits != 1)) return hipErrorInvalidValue;
  GemmPlan plan = plan_gemm(bf16, a.M, a.N, a.K, silu, kMaxSplitsAny);
  if (a.variant == kKDeep && plan.kernel != kKDeep && a.M <= 64) plan = plan_deep(a.M, a.N, a.K, silu, kMaxSplitsAny);
  const int kernel = a.variant ? a.variant : plan.kernel;
  if (!bf16 || kernel == kKF32) {
    if (bf16 || a.splits != 1) return hipErrorInvalidValue;
    dim3 grid((a.N + 63) / 64, (a.M + 63) / 64);
    if (silu) launch_kernel(k_gemm_f32<true>, grid, dim3(256), 0, s, a);
    else launch_kernel(k_gemm_f32<false>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (kernel == kKTiled || a.M > 64) {
    if (a.K % kGBK != 0 || (silu && a.N % 128 != 0) || (!silu && a.N % 8 != 0)) return hipErrorInvalidValue;
    // 32-bit buffer offsets; every weight segment but the last a whole number of 16-row blocks
    if (static_cast<int64_t>(a.M + 256) * a.lda * 2 >= (int64_t{1} << 31)) return hipErrorInvalidValue;
    for (int sg = 0; sg < a.W.n_seg; ++sg) {
      if (static_cast<int64_t>(a.W.rows[sg]) * a.K * 2 >= (int64_t{1} << 31)) return hipErrorInvalidValue;
      if (!silu && sg < a.W.n_seg - 1 && a.W.rows[sg] % 16 != 0) return hipErrorInvalidValue;
    }
    GemmPlan tp{kKTiled, 1};
    if (a.M > 64) tp = plan_tiled(a.M, a.N, a.K, silu, kMaxSplitsAny);
    const int bm = tp.bm, bn = tp.bn;
    const int kbps = (a.K / kGBK + a.splits - 1) / a.splits;
    const int n_nb = silu ? a.N / (bn / 2) : (a.N + bn - 1) / bn;
    const int n_mb = (a.M + bm - 1) / bm;
    const int per_xcd = (n_mb * n_nb * a.splits + 7) / 8;
    const int gm = n_nb >= 64 ? 8 : 2;
    dim3 grid(8 * per_xcd);
#define RP_TILED(BM_, BN_)                                                                                   \
    if (bm == BM_ && bn == BN_) {                                                                            \
      if (silu) launch_kernel((k_gemm_tiled<BM_, BN_, true>), grid, dim3(512), 0, s, a, kbps, n_mb, n_nb, gm); \
      else launch_kernel((k_gemm_tiled<BM_, BN_, false>), grid, dim3(512), 0, s, a, kbps, n_mb, n_nb, gm); \
    }
    RP_TILED(128, 128) RP_TILED(128, 256) RP_TILED(256, 128) RP_TILED(256, 256)
#undef RP_TILED
    return hipGetLastError();
  }
  if (kernel == kKDeep) {
    if (a.K % 64 != 0 || a.N % 16 != 0 || plan.kernel != kKDeep) return hipErrorInvalidValue;
    const bool ok = silu ? launch_deep<true>(a, plan.R, plan.D, s) : launch_deep<false>(a, plan.R, plan.D, s);
    return ok ? hipGetLastError() : hipErrorInvalidValue;
  }
  if (a.K % 128 != 0) return hipErrorInvalidValue;
  switch (kernel) {
    case kKStream:
      if (a.N % (silu ? 16 : 32) != 0) return hipErrorInvalidValue;
      if (silu) launch_stream_m<true>(a, s);
      else launch_stream_m<false>(a, s);
      break;
    case kKSkinny16:
      if (a.N % 64 != 0) return hipErrorInvalidValue;
      if (silu) launch_skinny_m<2, true>(a, s);
      else launch_skinny_m<1, false>(a, s);
      break;
    case kKSkinny32:
      if (a.N % (silu ? 64 : 128) != 0) return hipErrorInvalidValue;
      if (silu) launch_skinny_m<2, true>(a, s);
      else launch_skinny_m<2, false>(a, s);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rollpack
