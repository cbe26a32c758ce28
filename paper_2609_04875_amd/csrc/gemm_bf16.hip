// Dense bf16 projection Y = X W (+ R) for the stacked-layer transition F,
// fp32 accumulation on v_mfma_f32_32x32x16_bf16, one round-to-nearest-even
// store.  A workgroup of 4 waves computes a 128 x 128 output tile; each wave a
// 64 x 64 quarter as 2 x 2 MFMA tiles.  K advances 32 at a time through LDS:
// X rows are stored as read, W is stored transposed (n-major) so that both
// MFMA operands are contiguous 16-byte LDS reads.  The K loop never splits, so
// each output element's accumulation order is fixed.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace pgsr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDK = BK + 8;  // LDS row stride (elements) of both staged tiles

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__global__ void __launch_bounds__(256)
gemm_bf16_kernel(int M, int N, int K, const uint16_t* __restrict__ X,
                 const uint16_t* __restrict__ W, const uint16_t* R, uint16_t* Y) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t wt[BN * LDK];
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, r = lane & 31, hh = lane >> 5;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = (wv >> 1) * 64, wn = (wv & 1) * 64;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  for (int k0 = 0; k0 < K; k0 += BK) {
    __syncthreads();
    // X tile: 128 rows x 32 k = 512 chunks of 8 elements, 2 per thread.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256;
      const int row = c >> 2, kc = (c & 3) * 8;
      u32x4 v = {0, 0, 0, 0};
      if (m0 + row < M && k0 + kc < K) v = *(const u32x4*)(X + (int64_t)(m0 + row) * K + k0 + kc);
      *(u32x4*)&xs[row * LDK + kc] = v;
    }
    // W tile: 32 k x 128 n = 512 chunks of 8 n-values; stored transposed.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256;
      const int kk = c >> 4, nc = (c & 15) * 8;
      u32x4 v = {0, 0, 0, 0};
      if (k0 + kk < K && n0 + nc < N) v = *(const u32x4*)(W + (int64_t)(k0 + kk) * N + n0 + nc);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        wt[(nc + e) * LDK + kk] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = __builtin_bit_cast(bf16x8,
                                  *(const u32x4*)&xs[(wm + 32 * i + r) * LDK + ks * 16 + 8 * hh]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = __builtin_bit_cast(bf16x8,
                                  *(const u32x4*)&wt[(wn + 32 * j + r) * LDK + ks * 16 + 8 * hh]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  // Accumulator: lane holds column r, rows 8*(q/4) + 4*hh + q%4.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + 32 * j + r;
      if (col >= N) continue;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int rowi = m0 + wm + 32 * i + 8 * (q >> 2) + 4 * hh + (q & 3);
        if (rowi >= M) continue;
        float v = acc[i][j][q];
        const int64_t idx = (int64_t)rowi * N + col;
        if (R) v += bf16_to_f32(R[idx]);
        Y[idx] = __builtin_bit_cast(uint16_t, (__bf16)v);
      }
    }
}

}  // namespace

hipError_t launch_gemm_bf16(int m, int n, int k, const void* x, const void* w, const void* r,
                            void* y, hipStream_t s) {
  dim3 grid((n + BN - 1) / BN, (m + BM - 1) / BM);
  hipLaunchKernelGGL(gemm_bf16_kernel, grid, dim3(256), 0, s, m, n, k, (const uint16_t*)x,
                     (const uint16_t*)w, (const uint16_t*)r, (uint16_t*)y);
  return hipGetLastError();
}

}  // namespace pgsr
