// Dense bf16 projection Y = X W^T (+ R), large-product path: one wave per
// SIMD, each owning a 128 x 128 block of a 256 x 256 output tile (8 x 8
// sub-tiles of 16 x 16, 256 accumulators in AGPRs), X and W tiles brought to
// LDS by global->LDS loads, and every K step laid out as 128 fenced issue
// slots.
//
// K advances 64 at a time.  A step needs a 256 x 64 tile of X and one of W
// (32 KB each, one 64 KB LDS buffer); two buffers alternate.  A wave
// requests 8 runs of 1 KB of each image per step (8 rows x 128 bytes per
// run, whole cache lines) with global_load_lds_dwordx4: lane l's 16 bytes
// land at byte 16 l of the run, so the image layout is chosen through the
// global chunk each lane fetches: chunk c of row j sits at slot
// c ^ ((j / 2) mod 8), which spreads the 16 rows an operand read touches
// over all 64 banks.
//
// Step schedule (slot s = one v_mfma_f32_16x16x32_bf16: k slice s / 64, W
// sub-tile (s / 8) mod 8, X sub-tile s mod 8; each slice's 16 operands in a
// register set of their own).  Slots 0-31 read slice 1 of this step, one
// operand every other slot.  At slot 40 the wave waits for its requests of
// step kt + 1 (issued in slots 40-100 of the previous step) and its LDS
// reads, and the workgroup meets at the step's one barrier: step kt + 1's
// tiles are then in LDS and every wave has read all of step kt's buffer.
// Slots 40-100 issue this step's 16 requests (step kt + 2, into the buffer
// just read), one every fourth slot, so that the four waves' loads reach the
// CU's load path spread over the step; slots 64-94 read slice 0 of step
// kt + 1 (after the last product that reads slice 0 of this step).  Every
// operand register is rewritten at least ten slots after its last reader.
// The loop is unrolled by two, so each buffer's operand addresses are
// loop-invariant registers plus immediates.  The loop issues no other
// vector memory operation, so the vmcnt count is exact.
//
// The products are inline assembly (AGPR accumulators); the 19 wait states
// the compiler would insert before VALU reads of the accumulators are
// written out after the loop, and the epilogue reads each m sub-tile's
// accumulators only after an assembly statement ordered after them.  The
// requests are inline assembly too: the compiler's builtin would make every
// later LDS read wait for them.  Each request moves its LDS address into M0
// and waits one state before the load reads M0.
//
// Every output element is accumulated by the same products in the same
// order as in the register-staged kernel (A = W rows, B = X rows, k slices of
// 32 from 0), so both give identical bits and rows of Y do not depend on the
// launch.
#include <hip/hip_runtime.h>

#include <utility>

#include "internal.h"

// The requests write M0 (the LDS address of a global->LDS load) from inline
// assembly that lists it as clobbered; nothing else in this file uses M0.
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
constexpr int kGK = 64;                // K step
constexpr int kGNB = 2;                // LDS buffers
constexpr int kGImg = kGB * kGK;       // elements of one X or W image
constexpr int kGBuf = 2 * kGImg;       // elements of one buffer (X image, then W image)
constexpr int kGRuns = 8;              // 1 KB runs per wave and image per step
constexpr int kGGroupM = 4;            // tile rows per group of the tile order

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <class F, int... I>
__device__ __forceinline__ void static_for(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

// swizzle of the 16-byte chunk slot within a 128-byte image row
__device__ __forceinline__ int gsw(int row) { return (row >> 1) & 7; }

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

  // Requests: wave w takes runs w, w + 4, ..., w + 28 of each image; run q =
  // rows 8 q .. 8 q + 7, lane l -> row 8 q + l / 8, slot l % 8, chunk
  // (l % 8) ^ gsw(row).  Rows past M or N read row M-1 or N-1 (their outputs
  // are never stored).  Byte offsets from the matrix start (the launcher
  // takes only M*K and N*K below 2^31 elements).
  uint32_t xoff[kGRuns], woff[kGRuns];
#pragma unroll
  for (int j = 0; j < kGRuns; ++j) {
    const int row = 8 * (w + 4 * j) + lane / 8;
    const int c = (lane & 7) ^ gsw(row);
    xoff[j] = 2u * ((uint32_t)min(m0 + row, M - 1) * (uint32_t)K + 8u * c);
    woff[j] = 2u * ((uint32_t)min(n0 + row, N - 1) * (uint32_t)K + 8u * c);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)&lds[0] + 1024u * w;
  const int nk = K / kGK;
  // request q (0..15) of step kt: X run q (q < 8) or W run q - 8, into buffer
  // kt mod kGNB; steps past the last read the last step again (its buffer is
  // never read), so every step issues the same number of requests
  auto request = [&](int kt, int q) {
    const int ks = min(kt, nk - 1);
    const char* src = (const char*)((q < 8 ? X : W) + (int64_t)ks * kGK);
    const uint32_t img = lds0 + 2u * ((kt % kGNB) * kGBuf + (q < 8 ? 0 : kGImg)) + 4096u * (q & 7);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(q < 8 ? xoff[q & 7] : woff[q & 7]), "s"(src), "s"(img) : "memory", "m0");
  };

  // Operand reads: 16 rows x 32 k (slice ks) of rows base + r16, lane l ->
  // row l % 16, k group l / 16 (8 values): chunk 4 ks + l / 16 of the row,
  // at slot (4 ks + l / 16) ^ gsw(r16) (every base is a multiple of 16)
  const int r16 = lane & 15, g4 = lane >> 4;
  int soff[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) soff[ks] = r16 * kGK + (((4 * ks + g4) ^ gsw(r16)) << 3);
  bf16x8 wa[2][8], xb[2][8];
  // operand u (0..15) of slice ks: W sub-tile u / 2 (even u), X sub-tile u / 2 (odd u)
  auto read_op = [&](int buf, int ks, int u) {
    const uint16_t* img = &lds[buf * kGBuf + ((u & 1) ? 0 : kGImg)];
    const int base = ((u & 1) ? wm : wn) + 16 * (u >> 1);
    const bf16x8 v = __builtin_bit_cast(bf16x8, *(const u32x4*)&img[base * kGK + soff[ks]]);
    if (u & 1) xb[ks][u >> 1] = v;
    else wa[ks][u >> 1] = v;
  };

  f32x4 acc[8][8];      // [n sub-tile][m sub-tile], element (n, m)
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{};

  // prologue: steps 0 and 1 requested, step 0 landed, its slice-0 operands read
#pragma unroll
  for (int q = 0; q < 16; ++q) request(0, q);
#pragma unroll
  for (int q = 0; q < 16; ++q) request(1, q);
  asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
#pragma unroll
  for (int u = 0; u < 16; ++u) read_op(0, 0, u);

  // step kt with its buffer parity CUR known at compile time, so that every
  // operand address is a loop-invariant register plus an immediate
  auto step = [&](auto cur_c, int kt) {
    constexpr int cur = decltype(cur_c)::value, nxt = 1 - cur;
    auto slot = [&](auto ic) {
      constexpr int s = decltype(ic)::value;
      constexpr int ks = s / 64, i = (s / 8) % 8, j = s % 8;
      if constexpr (s == 40) {
        // step kt + 1 landed (this wave's requests, and the barrier for the
        // other waves'), and every wave has read all of step kt's buffer,
        // which the requests below refill with step kt + 2
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      }
      if constexpr (s < 32 && s % 2 == 0) read_op(cur, 1, s / 2);
      else if constexpr (s >= 64 && s < 96 && s % 2 == 0) read_op(nxt, 0, (s - 64) / 2);
      if constexpr (s >= 40 && s < 104 && s % 4 == 0) request(kt + 2, (s - 40) / 4);
      asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc[i][j]) : "v"(wa[ks][i]), "v"(xb[ks][j]));
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for(slot, std::make_integer_sequence<int, 128>{});
  };
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(std::integral_constant<int, 0>{}, kt);
    step(std::integral_constant<int, 1>{}, kt + 1);
  }
  if (kt < nk) step(std::integral_constant<int, 0>{}, kt);
  // 19 wait states before any VALU read of the accumulators (the epilogue
  // reads each m sub-tile's after an assembly statement ordered after this)
  asm volatile("s_nop 15\n\ts_nop 3" ::: "memory");
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // requests past the end, before LDS is handed on

  // acc[i][j] lane l, register q: n = wn + 16 i + 4 (l / 16) + q, m = wm + 16 j + l % 16
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    // one m sub-tile's accumulators at a time: they count as written here, so
    // their reads cannot move above the previous sub-tile's stores
    asm volatile("" : "+a"(acc[0][j]), "+a"(acc[1][j]), "+a"(acc[2][j]), "+a"(acc[3][j]),
                 "+a"(acc[4][j]), "+a"(acc[5][j]), "+a"(acc[6][j]), "+a"(acc[7][j]) :: "memory");
    const int m = m0 + wm + 16 * j + r16;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
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
