// Dense bf16 projection Y = X W^T (+ R) for the stacked-layer transition F,
// with W in the linear-layer layout [n][k]: fp32 accumulation on
// v_mfma_f32_16x16x32_bf16 (k in slices of 32 from 0) and one
// round-to-nearest-even store.  Products with at least 256 tiles of
// 256 x 256 (and K a multiple of 64) run the one-wave-per-SIMD kernel of
// gemm_bf16_wide.hip; this register-staged kernel takes every other product.
//
// A workgroup computes a BM x BN output tile with WGM x WGN waves, each wave a
// (TM * 32) x (TN * 32) block as (2 TM) x (2 TN) 16 x 16 MFMA tiles: 128 x 128
// with 4 waves of 64 x 64, two workgroups per CU; products with fewer than
// 128 such tiles take 128 x 32 (two waves) or, up to 64 rows, 64 x 32 (one
// wave) tiles, so that more workgroups stream W at once.  K advances 64 at a time
// through padded, double-buffered LDS tiles of X rows and W rows (both
// k-contiguous, so both MFMA operands are 16-byte reads); the next K steps
// are loaded into registers while the current one is multiplied.  The
// product is formed transposed (A = W rows, B = X rows): a lane then holds
// one output row and 4 consecutive columns per sub-tile, stored as 8-byte
// writes.  Output tiles are numbered so that each XCD (workgroup id mod 8)
// takes a contiguous run of them, walked in groups of 8 tile rows, and the
// workgroups sharing an XCD's L2 share their X and W panels.  The K loop
// never splits and both kernels run the same products in the same order, so
// each output element's accumulation order is fixed (rows of Y are bitwise
// independent of which other rows share the launch).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace pgsr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BK = 64;
constexpr int LDK = BK + 8;                      // LDS row stride (elements), 144 bytes
constexpr int kGroupM = 8;                       // tile rows per group of the tile order

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <int WGM, int WGN, int TM, int TN, int MINB>
__global__ void __launch_bounds__(WGM * WGN * 64, MINB)
gemm_bf16_kernel(int M, int N, int K, const uint16_t* __restrict__ X,
                 const uint16_t* __restrict__ W, const uint16_t* R, uint16_t* Y) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int BM = WGM * TM * 32, BN = WGN * TN * 32;
  constexpr int CPX = BM * BK / 8 / NT, CPW = BN * BK / 8 / NT;   // 16-byte chunks per thread
  static_assert(CPX * NT * 8 == BM * BK && CPW * NT * 8 == BN * BK, "tile split");
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t ws[2][BN * LDK];

  // output tile of this workgroup: XCD x = blockIdx % 8 takes tiles
  // [x * per_xcd, (x + 1) * per_xcd), in groups of kGroupM tile rows
  const int n_tm = (M + BM - 1) / BM, n_tn = (N + BN - 1) / BN;
  const int per_xcd = (n_tm * n_tn + 7) / 8;
  const int t = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
  if (t >= n_tm * n_tn) return;
  const int grp = t / (kGroupM * n_tn), first_m = grp * kGroupM;
  const int gsize = min(n_tm - first_m, kGroupM);
  const int idx = t - grp * kGroupM * n_tn;
  const int m0 = (first_m + idx % gsize) * BM, n0 = (idx / gsize) * BN;

  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, r16 = lane & 15, g4 = lane >> 4;
  const int wm = (wv % WGM) * TM * 32, wn = (wv / WGM) * TN * 32;

  // Loads read clamped (always valid) addresses, so the load sequence has no
  // branches: rows past M or N only feed output rows and columns that are
  // never stored, and chunks past K are zeroed when they are written to LDS.
  // Two register sets of staged chunks: the loads for K step kt+2 are issued
  // while step kt is multiplied, so each has two steps of products to arrive.
  u32x4 xr[2][CPX], wr[2][CPW];
  auto load = [&](int set, int k0) {
#pragma unroll
    for (int i = 0; i < CPX; ++i) {
      const int c = tid + i * NT;
      const int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      xr[set][i] = *(const u32x4*)(X + (int64_t)min(m0 + row, M - 1) * K + min(k0 + kc, K - 8));
    }
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int c = tid + i * NT;
      const int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      wr[set][i] = *(const u32x4*)(W + (int64_t)min(n0 + row, N - 1) * K + min(k0 + kc, K - 8));
    }
  };
  auto store = [&](int set, int buf, int k0) {
    const bool tail = k0 + BK > K;
#pragma unroll
    for (int i = 0; i < CPX; ++i) {
      const int c = tid + i * NT;
      const int kc = (c % (BK / 8)) * 8;
      const u32x4 v = tail && k0 + kc >= K ? u32x4{0, 0, 0, 0} : xr[set][i];
      *(u32x4*)&xs[buf][(c / (BK / 8)) * LDK + kc] = v;
    }
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int c = tid + i * NT;
      const int kc = (c % (BK / 8)) * 8;
      const u32x4 v = tail && k0 + kc >= K ? u32x4{0, 0, 0, 0} : wr[set][i];
      *(u32x4*)&ws[buf][(c / (BK / 8)) * LDK + kc] = v;
    }
  };

  // 16 x 16 output sub-tiles: a wave's (TM * 32) x (TN * 32) block is
  // (2 TM) x (2 TN) of them
  f32x4 acc[2 * TN][2 * TM];   // [n sub-tile][m sub-tile], element (n, m)
#pragma unroll
  for (int i = 0; i < 2 * TN; ++i)
#pragma unroll
    for (int j = 0; j < 2 * TM; ++j) acc[i][j] = f32x4{};

  const int nk = (K + BK - 1) / BK;
  // operand = 16 rows x 32 k (k slice ks): lane -> row r16, k 32 ks + 8 g4 .. +7
  auto mma = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 wa[2 * TN], xb[2 * TM];
#pragma unroll
      for (int i = 0; i < 2 * TN; ++i)
        wa[i] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)&ws[buf][(wn + 16 * i + r16) * LDK + ks * 32 + 8 * g4]);
#pragma unroll
      for (int j = 0; j < 2 * TM; ++j)
        xb[j] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)&xs[buf][(wm + 16 * j + r16) * LDK + ks * 32 + 8 * g4]);
#pragma unroll
      for (int i = 0; i < 2 * TN; ++i)
#pragma unroll
        for (int j = 0; j < 2 * TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[i], xb[j], acc[i][j], 0, 0, 0);
    }
  };
  // step kt: its chunks (register set kt % 2) go to LDS buffer kt % 2, last
  // read two steps ago with a barrier since; then step kt+2 is requested
  // into the same register set and step kt is multiplied.
  auto kstep = [&](int set, int kt) {
    store(set, set, kt * BK);
    if (kt + 2 < nk) load(set, (kt + 2) * BK);
    __syncthreads();
    mma(set);
  };
  load(0, 0);
  if (nk > 1) load(1, BK);
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    kstep(0, kt);
    kstep(1, kt + 1);
  }
  if (kt < nk) kstep(0, kt);
  // acc[i][j] lane (r16, g4), register q: n = wn + 16i + 4g4 + q,
  // m = wm + 16j + r16.
#pragma unroll
  for (int j = 0; j < 2 * TM; ++j) {
    const int m = m0 + wm + 16 * j + r16;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 2 * TN; ++i) {
      const int n = n0 + wn + 16 * i + 4 * g4;
      if (n >= N) continue;                        // N is a multiple of 8: whole group in or out
      const int64_t o = (int64_t)m * N + n;
      f32x4 v = acc[i][j];
      if (R) {
        const u32x2 rb = *(const u32x2*)(R + o);
        v[0] += bf16_to_f32((uint16_t)(rb[0] & 0xFFFF));
        v[1] += bf16_to_f32((uint16_t)(rb[0] >> 16));
        v[2] += bf16_to_f32((uint16_t)(rb[1] & 0xFFFF));
        v[3] += bf16_to_f32((uint16_t)(rb[1] >> 16));
      }
      *(bf16x4*)(Y + o) = __builtin_convertvector(v, bf16x4);
    }
  }
}

template <int WGM, int WGN, int TM, int TN, int MINB>
void launch_tiles(int m, int n, int k, const void* x, const void* w, const void* r, void* y,
                  hipStream_t s) {
  constexpr int BM = WGM * TM * 32, BN = WGN * TN * 32;
  const int tiles = ((m + BM - 1) / BM) * ((n + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_kernel<WGM, WGN, TM, TN, MINB>), dim3(8 * ((tiles + 7) / 8)),
                     dim3(WGM * WGN * 64), 0, s, m, n, k, (const uint16_t*)x, (const uint16_t*)w,
                     (const uint16_t*)r, (uint16_t*)y);
}

}  // namespace

hipError_t launch_gemm_bf16(int m, int n, int k, const void* x, const void* w, const void* r,
                            void* y, hipStream_t s) {
  if (gemm_bf16_wide_eligible(m, n, k)) return launch_gemm_bf16_wide(m, n, k, x, w, r, y, s);
  const int64_t tiles128 = (int64_t)((m + 127) / 128) * ((n + 127) / 128);
  if (tiles128 < 128) {
    // 128 x 128 tiles would leave most CUs idle (few rows: a short replayed
    // suffix against a model's weights): 32-column tiles, four times as many
    // workgroups streaming W at once; 64 x 32 for at most 64 rows
    if (m <= 64) launch_tiles<1, 1, 2, 1, 4>(m, n, k, x, w, r, y, s);
    else launch_tiles<2, 1, 2, 1, 3>(m, n, k, x, w, r, y, s);
  } else {
    // every other product: 128 x 128 tiles, two workgroups per CU
    launch_tiles<2, 2, 2, 2, 2>(m, n, k, x, w, r, y, s);
  }
  return hipGetLastError();
}

}  // namespace pgsr
