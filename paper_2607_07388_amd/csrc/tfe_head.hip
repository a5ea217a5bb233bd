// Early-exit prefetch head on gfx950 (wave64, MFMA): the approximate
// next-token distribution p = softmax(W h) of an intermediate hidden state
// (Eq. 13) and its K most likely tokens (Eq. 14), which are the candidates
// the cache prefetch consumes.
//
// Three launches:
//   k_head_logits  logits = W h for up to 64 rows h per block: a dense
//                  contraction, so it runs on the matrix cores
//                  (v_mfma_f32_16x16x32_bf16).  W ([V x D] bf16, 311 MB for
//                  the 151936 x 1024 head) is streamed from HBM exactly once
//                  per 64 rows; the 64 hidden rows are staged in LDS and read
//                  by every wave.  One wave computes a 16-token x 64-row
//                  tile: it loads its 16 W rows whole (D/32 16-byte loads per
//                  lane, all in flight before the first MFMA), then runs D/32
//                  k-steps of 4 MFMAs.  fp32 logits go to a scratch buffer.
//   k_head_select  per (row, chunk of the vocabulary): the chunk's K largest
//                  (logit, -id) keys by an exact 8-bit radix select over
//                  64-bit keys, plus the chunk's max logit and sum of
//                  exp(logit - max).
//   k_head_merge   per row: bitonic sort of the chunks' candidates, the top
//                  K with their probabilities exp(l - M) / S, M and S merged
//                  from the chunk partials (a log-sum-exp merge).
// Ties in logit go to the lower token id, so the answer is unique.  The
// exponentials use the full-accuracy expf (about 1 ulp): their cost is small
// next to the logits, and the probabilities feed a priority score.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tfe_head.h"

namespace tfe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kLogitWaves = 8;   // waves per logits block
constexpr int kCols = 64;        // hidden rows per logits block (4 MFMA column tiles)
constexpr int kSelThreads = 256;
constexpr int kSelPer = kHeadChunkMax / kSelThreads;  // logits per thread in a chunk
constexpr int kMergeThreads = 256;
constexpr int kMergeMax = kHeadMaxChunks * kHeadMaxK;  // candidates per row

// Order-preserving float -> uint32 map (larger float, larger key).
__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
// (logit, token) -> 64-bit key: higher logit first, then lower token id.
__device__ __forceinline__ uint64_t make_key(float l, uint32_t id) {
  return ((uint64_t)f2key(l) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}

template <int KS>  // KS = D / 32 k-steps
__global__ __launch_bounds__(kLogitWaves * 64) void k_head_logits(const HeadArgs a) {
  constexpr int D = KS * 32;
  constexpr int STRIDE = D + 8;  // staged row pitch (elements): conflict-free b128 reads
  __shared__ __attribute__((aligned(16))) __bf16 hs[kCols * STRIDE];
  const uint32_t col0 = blockIdx.y * kCols;
  const int ncols = (int)min((uint32_t)kCols, a.B - col0);
  for (int e = threadIdx.x; e < kCols * (D / 8); e += kLogitWaves * 64) {
    const int j = e / (D / 8), c = e - j * (D / 8);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (j < ncols) v = *((const u32x4*)a.hidden + ((size_t)(col0 + j) * D) / 8 + c);
    *(u32x4*)(hs + j * STRIDE + c * 8) = v;
  }
  __syncthreads();
  const int nbt = (ncols + 15) >> 4;  // live 16-row column tiles
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const uint32_t ntiles = (a.V + 15) >> 4;
  for (uint32_t t = blockIdx.x * kLogitWaves + wave; t < ntiles; t += gridDim.x * kLogitWaves) {
    // A operand: W rows t*16 + r (clamped in the last tile), k = 32 s + 8 g.
    const uint32_t row = min(t * 16 + r, a.V - 1);
    const u32x4* wp = (const u32x4*)a.w + ((size_t)row * D) / 8 + g;
    u32x4 av[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) av[s] = __builtin_nontemporal_load(wp + 4 * s);
    f32x4 acc[4];
#pragma unroll
    for (int bt = 0; bt < 4; ++bt) acc[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int bt = 0; bt < 4; ++bt) {
        if (bt < nbt) {
          const u32x4 bv = *(const u32x4*)(hs + (bt * 16 + r) * STRIDE + 32 * s + 8 * g);
          acc[bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, av[s]), __builtin_bit_cast(bf16x8, bv), acc[bt], 0, 0,
              0);
        }
      }
    }
    // D operand: lane (r, g) holds tokens t*16 + 4 g + q, q = 0..3, of column r.
    const uint32_t i0 = t * 16 + 4 * g;
#pragma unroll
    for (int bt = 0; bt < 4; ++bt) {
      const int j = bt * 16 + r;
      if (bt < nbt && j < ncols) {
        float* dst = a.logits + (size_t)(col0 + j) * a.V + i0;
        if ((a.V & 3u) == 0 && i0 + 3 < a.V) {
          *(f32x4*)dst = acc[bt];
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (i0 + q < a.V) dst[q] = acc[bt][q];
        }
      }
    }
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x = fmaxf(x, __shfl_xor(x, d, 64));
  return x;
}
__device__ __forceinline__ float wave_add(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, 64);
  return x;
}

// Inclusive block prefix sum over kSelThreads values.
__device__ uint32_t sel_scan(uint32_t v, uint32_t* s_wave) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  uint32_t off = 0;
  for (int w = 0; w < wave; ++w) off += s_wave[w];
  __syncthreads();
  return x + off;
}

__global__ __launch_bounds__(kSelThreads) void k_head_select(const HeadArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_wave[kSelThreads / 64];
  __shared__ uint32_t s_bin, s_above, s_cnt, s_out;
  __shared__ float s_red[kSelThreads / 64];
  const uint32_t b = blockIdx.y, c = blockIdx.x;
  const uint32_t lo = (uint32_t)((uint64_t)a.V * c / a.C);
  const uint32_t hi = (uint32_t)((uint64_t)a.V * (c + 1) / a.C);
  const uint32_t n = hi - lo;
  const float* lg = a.logits + (size_t)b * a.V;
  const int tid = threadIdx.x;

  uint32_t key[kSelPer];
  uint32_t kmax = 0;
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) {
    const uint32_t e = tid + i * kSelThreads;
    key[i] = e < n ? f2key(lg[lo + e]) : 0u;
    kmax = max(kmax, key[i]);
  }
  // Chunk max and sum of exp(l - max).
  {
    float m = key2f(kmax);
    if (kmax == 0u) m = -INFINITY;
    m = wave_max(m);
    if ((tid & 63) == 0) s_red[tid >> 6] = m;
    __syncthreads();
    m = s_red[0];
    for (int w = 1; w < kSelThreads / 64; ++w) m = fmaxf(m, s_red[w]);
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kSelPer; ++i) {
      const uint32_t e = tid + i * kSelThreads;
      if (e < n) s += expf(key2f(key[i]) - m);
    }
    s = wave_add(s);
    if ((tid & 63) == 0) s_red[tid >> 6] = s;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
      for (int w = 0; w < kSelThreads / 64; ++w) t += s_red[w];
      a.part[((size_t)b * a.C + c) * 2] = m;
      a.part[((size_t)b * a.C + c) * 2 + 1] = t;
    }
  }

  // Exact radix select of the K-th largest 64-bit key, 8 bits per pass from
  // the top.  Keys are distinct (they contain the token id), so at the
  // latest the last pass leaves one key in the chosen bin.
  const uint32_t take = min(a.K, n);
  uint64_t prefix = 0, mask = 0;
  if (take < n) {
    uint32_t need = take;
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      hist[tid] = 0u;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kSelPer; ++i) {
        const uint32_t e = tid + i * kSelThreads;
        if (e < n) {
          const uint64_t k = ((uint64_t)key[i] << 32) | (uint64_t)(0xFFFFFFFFu - (lo + e));
          if ((k & mask) == prefix) atomicAdd(&hist[(uint32_t)(k >> shift) & 255u], 1u);
        }
      }
      __syncthreads();
      // Thread t looks at bin 255 - t: prefix sums count keys from the top.
      const uint32_t v = hist[255 - tid];
      const uint32_t incl = sel_scan(v, s_wave);
      if (incl - v < need && need <= incl) {
        s_bin = 255 - tid;
        s_above = incl - v;
        s_cnt = v;
      }
      __syncthreads();
      need -= s_above;
      prefix |= (uint64_t)s_bin << shift;
      mask |= (uint64_t)0xFF << shift;
      const bool done = s_cnt == need;  // the whole bin is taken
      __syncthreads();
      if (done) break;
    }
  }
  // Every key whose masked bits are at least the prefix is selected: exactly
  // `take` keys.
  if (tid == 0) s_out = 0u;
  __syncthreads();
  uint64_t* out = a.cand + ((size_t)b * a.C + c) * a.K;
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) {
    const uint32_t e = tid + i * kSelThreads;
    if (e < n) {
      const uint64_t k = ((uint64_t)key[i] << 32) | (uint64_t)(0xFFFFFFFFu - (lo + e));
      if ((k & mask) >= prefix) {
        const uint32_t slot = atomicAdd(&s_out, 1u);
        if (slot < a.K) out[slot] = k;
      }
    }
  }
  if (tid == 0) a.cnt[(size_t)b * a.C + c] = take;
}

__global__ __launch_bounds__(kMergeThreads) void k_head_merge(const HeadArgs a) {
  __shared__ uint64_t keys[kMergeMax];
  const uint32_t b = blockIdx.x;
  const uint32_t N = a.C * a.K;
  uint32_t N2 = 1;
  while (N2 < N) N2 <<= 1;
  for (uint32_t e = threadIdx.x; e < N2; e += kMergeThreads) {
    uint64_t k = 0;  // below every real key
    if (e < N) {
      const uint32_t c = e / a.K, i = e - c * a.K;
      if (i < a.cnt[(size_t)b * a.C + c]) k = a.cand[((size_t)b * a.C + c) * a.K + i];
    }
    keys[e] = k;
  }
  __syncthreads();
  // Bitonic sort, descending.
  for (uint32_t size = 2; size <= N2; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (uint32_t e = threadIdx.x; e < N2 / 2; e += kMergeThreads) {
        const uint32_t i = 2 * e - (e & (stride - 1));
        const uint32_t j = i + stride;
        const bool desc = (i & size) == 0;
        const uint64_t x = keys[i], y = keys[j];
        if ((x < y) == desc) {
          keys[i] = y;
          keys[j] = x;
        }
      }
      __syncthreads();
    }
  }
  // Log-sum-exp merge of the chunk partials.
  float M = -INFINITY;
  for (uint32_t c = 0; c < a.C; ++c) M = fmaxf(M, a.part[((size_t)b * a.C + c) * 2]);
  float S = 0.f;
  for (uint32_t c = 0; c < a.C; ++c) {
    const float mc = a.part[((size_t)b * a.C + c) * 2];
    const float sc = a.part[((size_t)b * a.C + c) * 2 + 1];
    if (sc > 0.f) S += sc * expf(mc - M);
  }
  const float invS = 1.0f / S;
  for (uint32_t i = threadIdx.x; i < a.K; i += kMergeThreads) {
    const uint64_t k = keys[i];
    a.top_ids[(size_t)b * a.K + i] = (int32_t)(0xFFFFFFFFu - (uint32_t)k);
    a.top_prob[(size_t)b * a.K + i] = expf(key2f((uint32_t)(k >> 32)) - M) * invS;
  }
}

}  // namespace

uint32_t head_chunks(uint32_t V) {
  uint32_t c = (V + 4095) / 4096;
  return c < 1 ? 1 : (c > (uint32_t)kHeadMaxChunks ? (uint32_t)kHeadMaxChunks : c);
}

bool head_dim_supported(int D) { return D == 256 || D == 512 || D == 1024; }

uint32_t head_lds_bytes(int D) { return (uint32_t)(kCols * (D + 8) * 2); }

hipError_t launch_head_logits(const HeadArgs& a, uint32_t blocks, hipStream_t s) {
  const dim3 grid(blocks, (a.B + kCols - 1) / kCols);
  switch (a.D) {
    case 256: hipLaunchKernelGGL(k_head_logits<8>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    case 512: hipLaunchKernelGGL(k_head_logits<16>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    case 1024: hipLaunchKernelGGL(k_head_logits<32>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_head_select(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_head_select, dim3(a.C, a.B), dim3(kSelThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_head_merge(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_head_merge, dim3(a.B), dim3(kMergeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace tfe
