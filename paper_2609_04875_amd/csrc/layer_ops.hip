// Elementwise steps of a full decoder layer around the projections: RMSNorm
// with a gain, rotary embedding of Q and K at absolute positions, and the
// SiLU-gated product of the MLP.  bf16 in and out, fp32 arithmetic, one
// rounding per stored value.  All three are HBM-bound streams: 16-byte loads
// and stores, fixed reduction order (results do not depend on timing).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace pgsr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN).
__device__ inline uint32_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ inline uint32_t pack(float a, float b) { return to_bf16(a) | (to_bf16(b) << 16); }

constexpr int kThreads = 256;

// y = x / sqrt(mean(x^2) + eps) * g, one workgroup per row; d_model % 8 == 0.
__global__ void __launch_bounds__(kThreads) rmsnorm_kernel(int32_t dm, const uint16_t* __restrict__ x,
                                                           const uint16_t* __restrict__ g, float eps,
                                                           uint16_t* __restrict__ y) {
  __shared__ float red[kThreads / 64];
  const int64_t row = blockIdx.x;
  const u32x4* xr = (const u32x4*)(x + row * dm);
  const u32x4* gr = (const u32x4*)g;
  u32x4* yr = (u32x4*)(y + row * dm);
  const int chunks = dm / 8;
  float ss = 0.f;
  for (int c = threadIdx.x; c < chunks; c += kThreads) {
    const u32x4 v = xr[c];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a = lo_bf16(v[j]), b = hi_bf16(v[j]);
      ss = fmaf(a, a, ss);
      ss = fmaf(b, b, ss);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float total = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.f / sqrtf(total / (float)dm + eps);
  for (int c = threadIdx.x; c < chunks; c += kThreads) {
    const u32x4 v = xr[c], w = gr[c];
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack(lo_bf16(v[j]) * inv * lo_bf16(w[j]), hi_bf16(v[j]) * inv * hi_bf16(w[j]));
    yr[c] = o;
  }
}

// Rotary embedding in place on x [n][heads][d]: for i < d/2 the pair
// (x_i, x_{i+d/2}) turns by pos * theta^(-2i/d).  The angle is formed and
// reduced to [-pi, pi] in fp64 (positions reach 10^5 radians), then sin and
// cos run in fp32 on the reduced angle.
__global__ void __launch_bounds__(kThreads) rope_kernel(int64_t n_pairs, int32_t heads, int32_t d,
                                                        uint16_t* __restrict__ x,
                                                        const int32_t* __restrict__ pos, double log2_theta) {
  const int half = d / 2;
  for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < n_pairs;
       p += (int64_t)gridDim.x * kThreads) {
    const int i = (int)(p % half);
    const int64_t th = p / half;                  // token * heads + head
    const int64_t tok = th / heads;
    const double inv = exp2(-2.0 * i / d * log2_theta);
    const double ang = (double)pos[tok] * inv;
    const double two_pi = 6.283185307179586476925287;
    const float r = (float)(ang - two_pi * rint(ang / two_pi));
    float s, c;
    sincosf(r, &s, &c);
    uint16_t* row = x + th * d;
    const float a = __uint_as_float((uint32_t)row[i] << 16);
    const float b = __uint_as_float((uint32_t)row[i + half] << 16);
    row[i] = (uint16_t)to_bf16(a * c - b * s);
    row[i + half] = (uint16_t)to_bf16(b * c + a * s);
  }
}

// out[r][j] = SiLU(gu[r][j]) * gu[r][d_ff + j], SiLU(g) = g / (1 + e^-g).
__global__ void __launch_bounds__(kThreads) silu_mul_kernel(int64_t n_chunks, int32_t dff,
                                                            const uint16_t* __restrict__ gu,
                                                            uint16_t* __restrict__ out) {
  const int per_row = dff / 8;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < n_chunks;
       c += (int64_t)gridDim.x * kThreads) {
    const int64_t r = c / per_row;
    const int j = (int)(c % per_row) * 8;
    const u32x4 g = *(const u32x4*)(gu + r * 2 * dff + j);
    const u32x4 u = *(const u32x4*)(gu + r * 2 * dff + dff + j);
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float g0 = lo_bf16(g[k]), g1 = hi_bf16(g[k]);
      const float s0 = g0 / (1.f + expf(-g0)), s1 = g1 / (1.f + expf(-g1));
      o[k] = pack(s0 * lo_bf16(u[k]), s1 * hi_bf16(u[k]));
    }
    *(u32x4*)(out + r * dff + j) = o;
  }
}

int grid_for(int64_t work) {
  int64_t g = (work + kThreads - 1) / kThreads;
  return (int)(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

}  // namespace

hipError_t launch_rmsnorm(int32_t n, int32_t dm, const void* x, const void* g, float eps, void* y,
                          hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(n), dim3(kThreads), 0, s, dm, (const uint16_t*)x,
                     (const uint16_t*)g, eps, (uint16_t*)y);
  return hipGetLastError();
}

hipError_t launch_rope(int32_t n, int32_t heads, int32_t d, void* x, const int32_t* pos, double theta,
                       hipStream_t s) {
  const int64_t pairs = (int64_t)n * heads * (d / 2);
  if (pairs <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_kernel, dim3(grid_for(pairs)), dim3(kThreads), 0, s, pairs, heads, d,
                     (uint16_t*)x, pos, log2(theta));
  return hipGetLastError();
}

hipError_t launch_silu_mul(int32_t n, int32_t dff, const void* gu, void* out, hipStream_t s) {
  const int64_t chunks = (int64_t)n * (dff / 8);
  if (chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL(silu_mul_kernel, dim3(grid_for(chunks)), dim3(kThreads), 0, s, chunks, dff,
                     (const uint16_t*)gu, (uint16_t*)out);
  return hipGetLastError();
}

}  // namespace pgsr
