// Dense bf16 projection Y = X W^T (+ R), large-product path: one wave per
// SIMD, each owning a 128 x 128 block of a 256 x 256 output tile, the 256
// accumulators in AGPRs, X and W tiles brought to LDS by global->LDS loads,
// and every K step laid out as 32 fenced issue slots.
//
// K advances 32 at a time.  A step needs a 256 x 32 tile of X and one of W
// (16 KB each, one 32 KB LDS buffer); four buffers rotate and step kt
// requests step kt + 3 into the buffer step kt - 1 used.  A wave requests 4
// runs of 1 KB of each image per step (16 rows x 64 bytes per run) with
// global_load_lds_dwordx4: lane l's 16 bytes land at byte 16 l of the run, so
// the image layout is chosen through the global chunk each lane fetches:
// chunk c of row j sits at slot c ^ ((j / 4) mod 4), which spreads the 16
// rows an operand read touches over all 64 banks.
//
// Step schedule (slot s = one v_mfma_f32_32x32x16_bf16: k slice s / 16, W
// sub-tile (s / 4) mod 4, X sub-tile s mod 4).  Slots 0-15 multiply slice 0
// while the operands of slice 1 are read, one read every other slot; then
// this wave's requests of step kt - 2 are waited for (s_waitcnt vmcnt(8):
// only step kt - 1's are left) and the workgroup meets at a barrier, after
// which step kt + 1's tiles are in LDS and step kt - 1's buffer is free;
// slots 16-31 multiply slice 1 while this step's 8 requests go out and the
// operands of slice 0 of step kt + 1 are read.  Every operand register is
// rewritten at least six slots after the last product that read it.  The
// loop issues no other vector memory operation, so the vmcnt count is exact.
//
// The products are inline assembly (AGPR accumulators), and the wait states
// the compiler would insert before VALU reads of the accumulators are
// written out at the end of every step (they overlap the last product).  The
// requests are inline assembly too: the compiler's builtin would make every
// later LDS read wait for them.  Each request moves its LDS address into M0
// and waits one state before the load reads M0.
//
// Every output element is accumulated by the same products in the same
// order as in the register-staged kernel (A = W rows, B = X rows, k slices of
// 16 from 0), so both give identical bits and rows of Y do not depend on the
// launch.
#include <hip/hip_runtime.h>

#include <utility>

#include "internal.h"

#pragma clang diagnostic ignored "-Winline-asm"

namespace pgsr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kGB = 256;               // output tile edge (M and N)
constexpr int kGK = 32;                // K step
constexpr int kGNB = 4;                // LDS buffers
constexpr int kGImg = kGB * kGK;       // elements of one X or W image
constexpr int kGBuf = 2 * kGImg;       // elements of one buffer (X image, then W image)
constexpr int kGRuns = 4;              // 1 KB runs per wave and image per step
constexpr int kGGroupM = 8;            // tile rows per group of the tile order

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <class F, int... I>
__device__ __forceinline__ void static_for(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

// swizzle of the 16-byte chunk slot within a 64-byte image row
__device__ __forceinline__ int gsw(int row) { return (row >> 2) & 3; }

__global__ void __launch_bounds__(256, 1)
gemm_bf16_wide_kernel(int M, int N, int K, const uint16_t* __restrict__ X,
                      const uint16_t* __restrict__ W, const uint16_t* R, uint16_t* Y) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[kGNB * kGBuf];

  // output tile of this workgroup: XCD x = blockIdx % 8 takes tiles
  // [x * per_xcd, (x + 1) * per_xcd), in groups of kGGroupM tile rows
  const int n_tm = (M + kGB - 1) / kGB, n_tn = (N + kGB - 1) / kGB;
  const int per_xcd = (n_tm * n_tn + 7) / 8;
  const int t = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
  if (t >= n_tm * n_tn) return;
  const int grp = t / (kGGroupM * n_tn), first_m = grp * kGGroupM;
  const int gsize = min(n_tm - first_m, kGGroupM);
  const int idx = t - grp * kGGroupM * n_tn;
  const int m0 = (first_m + idx % gsize) * kGB, n0 = (idx / gsize) * kGB;

  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, r = lane & 31, hh = lane >> 5;
  const int wm = (w & 1) * 128, wn = (w >> 1) * 128;

  // Requests: wave w takes runs w, w + 4, w + 8, w + 12 of each image; run q
  // = rows 16 q .. 16 q + 15, lane l -> row 16 q + l / 4, slot l % 4, chunk
  // (l % 4) ^ gsw(row).  Rows past M or N read row M-1 or N-1 (their outputs
  // are never stored).  Byte offsets from the matrix start (the launcher
  // takes only M*K and N*K below 2^31 elements).
  uint32_t xoff[kGRuns], woff[kGRuns];
#pragma unroll
  for (int j = 0; j < kGRuns; ++j) {
    const int row = 16 * (w + 4 * j) + lane / 4;
    const int c = (lane & 3) ^ gsw(row);
    xoff[j] = 2u * ((uint32_t)min(m0 + row, M - 1) * (uint32_t)K + 8u * c);
    woff[j] = 2u * ((uint32_t)min(n0 + row, N - 1) * (uint32_t)K + 8u * c);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)&lds[0] + 1024u * w;
  const int nk = K / kGK;
  // request q (0..7) of step kt: X run q (q < 4) or W run q - 4, into buffer
  // kt mod kGNB; steps past the last read the last step again (its buffer is
  // never read), so every step issues the same number of requests
  auto request = [&](int kt, int q) {
    const int ks = min(kt, nk - 1);
    const char* src = (const char*)((q < 4 ? X : W) + (int64_t)ks * kGK);
    const uint32_t img = lds0 + 2u * ((kt % kGNB) * kGBuf + (q < 4 ? 0 : kGImg)) + 4096u * (q & 3);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(q < 4 ? xoff[q & 3] : woff[q & 3]), "s"(src), "s"(img) : "memory", "m0");
  };

  // Operand reads: 32 x 16 slice ks of rows base + r at slot (2 ks + hh) ^
  // gsw(r) (every base is a multiple of 16).
  int soff[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) soff[ks] = r * kGK + (((2 * ks + hh) ^ gsw(r)) << 3);
  bf16x8 wa[2][4], xb[2][4];
  // operand u (0..7) of slice ks from buffer buf: W sub-tile u / 2 for even u,
  // X sub-tile u / 2 for odd u
  auto read_op = [&](int buf, int ks, int u) {
    const uint16_t* img = &lds[buf * kGBuf + ((u & 1) ? 0 : kGImg)];
    const int base = ((u & 1) ? wm : wn) + 32 * (u >> 1);
    const bf16x8 v = __builtin_bit_cast(bf16x8, *(const u32x4*)&img[base * kGK + soff[ks]]);
    if (u & 1) xb[ks][u >> 1] = v;
    else wa[ks][u >> 1] = v;
  };

  f32x16 acc[4][4];     // [n sub-tile][m sub-tile], element (n, m)
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  // prologue: steps 0..2 requested, step 0 landed, its slice-0 operands read
  for (int kt = 0; kt < kGNB - 1; ++kt)
#pragma unroll
    for (int q = 0; q < 8; ++q) request(kt, q);
  asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
#pragma unroll
  for (int u = 0; u < 8; ++u) read_op(0, 0, u);

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt % kGNB, nxt = (kt + 1) % kGNB;
    auto slot = [&](auto ic) {
      constexpr int s = decltype(ic)::value;
      constexpr int ks = s / 16, i = (s / 4) % 4, j = s % 4;
      if constexpr (s == 16) {
        // step kt + 1 landed (all but this wave's latest 8 requests), and
        // every wave is past step kt - 1
        asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
      }
      if constexpr (s % 2 == 0) {
        if constexpr (ks == 0) read_op(cur, 1, s / 2);
        else read_op(nxt, 0, (s - 16) / 2);
      }
      if constexpr (s >= 16 && s < 24) request(kt + kGNB - 1, s - 16);
      asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc[i][j]) : "v"(wa[ks][i]), "v"(xb[ks][j]));
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for(slot, std::make_integer_sequence<int, 32>{});
    // 19 wait states before any VALU read of the accumulators (they run in
    // the shadow of the last product; at the loop's end they precede the
    // epilogue's reads)
    asm volatile("s_nop 15\n\ts_nop 3" ::: "memory");
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // requests past the end, before LDS is handed on

  // acc[i][j] lane (r, hh), register q: n = wn + 32i + 8(q/4) + 4hh + q%4,
  // m = wm + 32j + r.
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    // one m sub-tile's accumulators at a time: they count as written here, so
    // their reads cannot move above the previous sub-tile's stores
    asm volatile("" : "+a"(acc[0][j]), "+a"(acc[1][j]), "+a"(acc[2][j]), "+a"(acc[3][j]) :: "memory");
    const int m = m0 + wm + 32 * j + r;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn + 32 * i + 8 * q4 + 4 * hh;
        if (n >= N) continue;                      // N is a multiple of 8: whole group in or out
        const int64_t o = (int64_t)m * N + n;
        f32x4 v = {acc[i][j][4 * q4 + 0], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2],
                   acc[i][j][4 * q4 + 3]};
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

}  // namespace

bool gemm_bf16_wide_eligible(int m, int n, int k) {
  const int64_t tiles = (int64_t)((m + kGB - 1) / kGB) * ((n + kGB - 1) / kGB);
  return k >= kGK && k % kGK == 0 && tiles >= 256 && (int64_t)m * k < ((int64_t)1 << 31) &&
         (int64_t)n * k < ((int64_t)1 << 31);
}

hipError_t launch_gemm_bf16_wide(int m, int n, int k, const void* x, const void* w, const void* r,
                                 void* y, hipStream_t s) {
  if (!gemm_bf16_wide_eligible(m, n, k)) return hipErrorInvalidValue;
  const int tiles = ((m + kGB - 1) / kGB) * ((n + kGB - 1) / kGB);
  hipLaunchKernelGGL(gemm_bf16_wide_kernel, dim3(8 * ((tiles + 7) / 8)), dim3(256), 0, s, m, n, k,
                     (const uint16_t*)x, (const uint16_t*)w, (const uint16_t*)r, (uint16_t*)y);
  return hipGetLastError();
}

}  // namespace pgsr
