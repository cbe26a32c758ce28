// fp32 prefix + causal prefill attention over the paged cache.
//
// One wave64 workgroup handles 64 consecutive query tokens of one query head;
// each lane owns one query row.  Keys are visited in tiles of KT at absolute
// positions 0, KT, 2KT, ... (the same tiling for any prefix length, so a row's
// result depends only on its absolute position: a selective replay and a full
// reset produce identical bits for the same query).  Each tile is gathered
// through the block table into LDS; a lane computes its KT logits with FMAs,
// masks keys past its position by select, and folds the tile into an online
// softmax (running max m, running sum l, rescaled accumulator) in the base-2
// domain.  Keys at or beyond the sequence length are never loaded: their LDS
// rows are zero, so stale or NaN slots cannot leak into the result.
//
// This path exists for fp32 accuracy (the fp32 tolerance is 1e-4 against fp64);
// the bf16 MFMA kernel is the performance path.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace pgsr {

namespace {

constexpr int kTokens = 64;  // query tokens per workgroup (one per lane)

template <int D, int KT>
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a) {
  __shared__ float ks[KT][D + 1];
  __shared__ float vs[KT][D + 1];

  const int tile = blockIdx.x;
  const int hq = blockIdx.y;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].tile_start <= tile) ++ei;
  const AttnEntry e = a.e[ei];
  const int lt = tile - e.tile_start;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int g = hq / G;
  const int B = a.block_size;
  const int lane = threadIdx.x;
  const int t = lt * kTokens + lane;             // token index inside the suffix
  const bool valid = t < e.q_len;
  const int qpos = valid ? e.prefix + t : -1;    // absolute position (-1: padding row)
  const int t_last = min(e.q_len, (lt + 1) * kTokens) - 1;
  const int kv_len = e.prefix + e.q_len;
  const int key_end = e.prefix + t_last + 1;     // keys this workgroup needs: [0, key_end)

  const float* q = (const float*)a.q;
  float qr[D];
  if (valid) {
    const float* qp = q + ((int64_t)(e.q_off + t) * a.n_q_heads + hq) * D;
#pragma unroll
    for (int c = 0; c < D; ++c) qr[c] = qp[c];
  } else {
#pragma unroll
    for (int c = 0; c < D; ++c) qr[c] = 0.f;
  }
  float acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) acc[c] = 0.f;
  float m = -INFINITY, l = 0.f;

  const int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
  const int64_t layer_off = (int64_t)a.layer * a.n_blocks * a.n_kv_heads;
  const float* kc = (const float*)a.k_cache;
  const float* vc = (const float*)a.v_cache;
  const float c2 = a.scale_log2;

  for (int kb = 0; kb < key_end; kb += KT) {
    __syncthreads();
    for (int i = lane; i < KT * D; i += 64) {  // K rows: contiguous D per slot
      const int j = i / D, c = i % D;
      const int pos = kb + j;
      float val = 0.f;
      if (pos < kv_len) {
        const int32_t id = row[pos / B];
        val = kc[((layer_off + (int64_t)id * a.n_kv_heads + g) * B + pos % B) * D + c];
      }
      ks[j][c] = val;
    }
    for (int i = lane; i < KT * D; i += 64) {  // V^T rows: contiguous B per d
      const int c = i / KT, j = i % KT;
      const int pos = kb + j;
      float val = 0.f;
      if (pos < kv_len) {
        const int32_t id = row[pos / B];
        val = vc[((layer_off + (int64_t)id * a.n_kv_heads + g) * D + c) * B + pos % B];
      }
      vs[j][c] = val;
    }
    __syncthreads();
    float s[KT];
    float tmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float dot = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) dot = fmaf(qr[c], ks[j][c], dot);
      s[j] = (kb + j <= qpos) ? dot * c2 : -INFINITY;
      tmax = fmaxf(tmax, s[j]);
    }
    const float m_new = fmaxf(m, tmax);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m - m_use);
    l *= alpha;
#pragma unroll
    for (int c = 0; c < D; ++c) acc[c] *= alpha;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const float p = exp2f(s[j] - m_use);
      l += p;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(p, vs[j][c], acc[c]);
    }
    m = m_new;
  }
  if (valid) {
    float* op = (float*)a.o + ((int64_t)(e.q_off + t) * a.n_q_heads + hq) * D;
    const float inv = 1.f / l;
#pragma unroll
    for (int c = 0; c < D; ++c) op[c] = acc[c] * inv;
  }
}

}  // namespace

int attn_f32_tile_tokens(int, int) { return kTokens; }

hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  dim3 grid(a.n_tiles, a.n_q_heads);
  if (a.head_dim == 64)
    hipLaunchKernelGGL((attn_f32_kernel<64, 32>), grid, dim3(64), 0, s, a);
  else if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_f32_kernel<128, 16>), grid, dim3(64), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pgsr
