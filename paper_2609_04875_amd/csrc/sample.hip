// Deterministic next-token sampling for re-decode: Gumbel-max over
// logits / T with noise from the counter-based generator Philox4x64-10
// (Salmon et al., SC 2011), so a (seed, stream, position) triple always picks
// the same token (assumption A1 of Theorem 1).  T = 0 is the greedy argmax.
//
// A row's vocabulary is cut into chunks of kChunk entries, one workgroup each;
// a thread draws one Philox block (4 words -> 4 entries) at a time.  Each
// candidate becomes a 64-bit key: the fp32 score mapped to an order-preserving
// unsigned integer in the high half, the complement of the vocabulary index in
// the low half.  The largest key is then the highest score with, among equal
// scores, the lowest index, whatever order the keys are reduced in, so the
// chunk partials (in a caller workspace) and the in-workgroup reductions are
// exact and deterministic.  NaN scores count as -inf.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace pgsr {

namespace {

constexpr int kThreads = 256;

struct Philox4 {
  uint64_t w[4];
};

// Ten Philox4x64 rounds on counter c with key k.
__device__ inline Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                        uint64_t k1) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t lo0 = M0 * c0, hi0 = __umul64hi(M0, c0);
    const uint64_t lo1 = M1 * c2, hi1 = __umul64hi(M1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += W0;
    k1 += W1;
  }
  return Philox4{{c0, c1, c2, c3}};
}

__device__ inline float load_logit(const float* p, int64_t i) { return p[i]; }
__device__ inline float load_logit(const uint16_t* p, int64_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}

// Order-preserving key: larger score, then lower index, gives a larger key.
__device__ inline uint64_t make_key(float score, int32_t v) {
  if (!(score == score)) score = -INFINITY;   // NaN never wins
  score += 0.f;                                // -0 -> +0: equal scores tie
  const uint32_t b = __float_as_uint(score);
  const uint32_t mono = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)mono << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)v);
}

__device__ inline uint64_t max_key_wave(uint64_t k) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(k, off);
    k = o > k ? o : k;
  }
  return k;
}

template <typename T>
__global__ void __launch_bounds__(kThreads) sample_chunk_kernel(SampleArgs a, const T* __restrict__ logits,
                                                                int32_t* __restrict__ tokens) {
  __shared__ uint64_t red[kThreads / 64];
  const int row = blockIdx.x / a.n_chunks, chunk = blockIdx.x % a.n_chunks;
  const int64_t grow = (int64_t)a.row0 + row;
  const T* lr = logits + grow * a.vocab;
  const int32_t v_lo = chunk * a.chunk_len;
  const int32_t v_hi = min(a.vocab, v_lo + a.chunk_len);
  const bool hot = a.temperature > 0.f;
  const uint64_t pos = (uint64_t)a.position[row], str = (uint64_t)a.stream[row];
  uint64_t best = 0;
  // Philox blocks of 4 entries; chunk_len is a multiple of 4, so blocks never
  // straddle two chunks.
  for (int32_t v0 = v_lo + 4 * (int32_t)threadIdx.x; v0 < v_hi; v0 += 4 * kThreads) {
    Philox4 r{};
    if (hot) r = philox4x64_10((uint64_t)(v0 / 4), pos, str, 0, a.seed, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int32_t v = v0 + j;
      if (v >= v_hi) break;
      float score = load_logit(lr, v);
      if (hot) {
        const float u = ((float)(uint32_t)(r.w[j] >> 41) + 0.5f) * (1.f / 8388608.f);
        score = score / a.temperature - logf(-logf(u));
      }
      const uint64_t k = make_key(score, v);
      best = k > best ? k : best;
    }
  }
  best = max_key_wave(best);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t k = red[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) k = red[w] > k ? red[w] : k;
    if (a.n_chunks == 1)
      tokens[grow] = (int32_t)(0xFFFFFFFFu - (uint32_t)k);
    else
      a.partial[grow * a.n_chunks + chunk] = k;
  }
}

// One thread per row: the largest of its chunk keys.
__global__ void __launch_bounds__(kThreads) sample_reduce_kernel(int32_t n, int32_t n_chunks,
                                                                 const uint64_t* __restrict__ partial,
                                                                 int32_t* __restrict__ tokens) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  uint64_t k = 0;
  for (int c = 0; c < n_chunks; ++c) {
    const uint64_t p = partial[(int64_t)i * n_chunks + c];
    k = p > k ? p : k;
  }
  tokens[i] = (int32_t)(0xFFFFFFFFu - (uint32_t)k);
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, int dtype, const void* logits, int32_t* tokens,
                         hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  dim3 grid(a.n * a.n_chunks);
  if (dtype == 1)
    hipLaunchKernelGGL(sample_chunk_kernel<uint16_t>, grid, dim3(kThreads), 0, s, a,
                       (const uint16_t*)logits, tokens);
  else
    hipLaunchKernelGGL(sample_chunk_kernel<float>, grid, dim3(kThreads), 0, s, a, (const float*)logits,
                       tokens);
  return hipGetLastError();
}

hipError_t launch_sample_reduce(int32_t n, int32_t n_chunks, const uint64_t* partial, int32_t* tokens,
                                hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(sample_reduce_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, s, n,
                     n_chunks, partial, tokens);
  return hipGetLastError();
}

}  // namespace pgsr
