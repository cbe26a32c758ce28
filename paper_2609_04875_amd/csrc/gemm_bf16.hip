// Dense bf16 projection Y = X W^T (+ R) for the stacked-layer transition F,
// with W in the linear-layer layout [n][k]: fp32 accumulation on
// v_mfma_f32_32x32x16_bf16 and one round-to-nearest-even store.
//
// A workgroup of 4 waves computes a 128 x 128 output tile, each wave a 64 x 64
// quarter as 2 x 2 MFMA tiles.  K advances 64 at a time through padded,
// double-buffered LDS tiles of X rows and W rows (both k-contiguous, so both
// MFMA operands are 16-byte reads); the next K step is loaded into registers
// while the current one is multiplied.  The product is formed transposed
// (A = W rows, B = X rows): a lane then holds one output row and groups of 4
// consecutive columns, stored as 8-byte writes.  The K loop never splits, so
// each output element's accumulation order is fixed (rows of Y are bitwise
// independent of which other rows share the launch).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace pgsr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDK = BK + 8;                      // LDS row stride (elements), 144 bytes
constexpr int CPT = BM * BK / 8 / 256;           // 16-byte chunks per thread per operand

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__global__ void __launch_bounds__(256, 2)
gemm_bf16_kernel(int M, int N, int K, const uint16_t* __restrict__ X,
                 const uint16_t* __restrict__ W, const uint16_t* R, uint16_t* Y) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t ws[2][BN * LDK];
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, r = lane & 31, hh = lane >> 5;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = (wv >> 1) * 64, wn = (wv & 1) * 64;

  u32x4 xr[CPT], wr[CPT];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * 256;
      const int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      const bool kin = k0 + kc < K;
      xr[i] = (m0 + row < M && kin) ? *(const u32x4*)(X + (int64_t)(m0 + row) * K + k0 + kc)
                                    : u32x4{0, 0, 0, 0};
      wr[i] = (n0 + row < N && kin) ? *(const u32x4*)(W + (int64_t)(n0 + row) * K + k0 + kc)
                                    : u32x4{0, 0, 0, 0};
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * 256;
      const int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      *(u32x4*)&xs[buf][row * LDK + kc] = xr[i];
      *(u32x4*)&ws[buf][row * LDK + kc] = wr[i];
    }
  };

  f32x16 acc[2][2];   // [n sub-tile][m sub-tile], element (n, m)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  const int nk = (K + BK - 1) / BK;
  load(0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    store(buf);                 // buffer last read two steps ago, one barrier before
    __syncthreads();
    if (kt + 1 < nk) load((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 wa[2], xb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        wa[i] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)&ws[buf][(wn + 32 * i + r) * LDK + ks * 16 + 8 * hh]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        xb[j] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)&xs[buf][(wm + 32 * j + r) * LDK + ks * 16 + 8 * hh]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[i], xb[j], acc[i][j], 0, 0, 0);
    }
  }
  // acc[i][j] lane (r, hh), register q: n = wn + 32i + 8(q/4) + 4hh + q%4,
  // m = wm + 32j + r.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = m0 + wm + 32 * j + r;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn + 32 * i + 8 * q4 + 4 * hh;
        if (n >= N) continue;                      // N is a multiple of 8: whole group in or out
        const int64_t idx = (int64_t)m * N + n;
        f32x4 v = {acc[i][j][4 * q4 + 0], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2],
                   acc[i][j][4 * q4 + 3]};
        if (R) {
          const u32x2 rb = *(const u32x2*)(R + idx);
          v[0] += bf16_to_f32((uint16_t)(rb[0] & 0xFFFF));
          v[1] += bf16_to_f32((uint16_t)(rb[0] >> 16));
          v[2] += bf16_to_f32((uint16_t)(rb[1] & 0xFFFF));
          v[3] += bf16_to_f32((uint16_t)(rb[1] >> 16));
        }
        *(bf16x4*)(Y + idx) = __builtin_convertvector(v, bf16x4);
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
