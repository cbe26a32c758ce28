// fp32 prefix + causal prefill attention over the paged cache.
//
// A workgroup of four waves handles 64 consecutive query tokens of one query
// head; in every wave, lane i owns query row i.  Keys are visited in tiles of
// KT at absolute positions 0, KT, 2KT, ...; wave w takes the tiles whose index
// is w mod 4, each into its own LDS region (no workgroup barrier in the loop),
// and keeps its own online softmax (running max m, running sum l, rescaled
// accumulator, base-2 domain).  The four partial states are merged at the end
// in the fixed order 0, 1, 2, 3.  Tile ownership depends only on absolute
// positions, so a row's result depends only on its position and its keys: a
// selective replay and a full reset produce identical bits.  Keys at or past
// the sequence length are never loaded: their LDS rows are zero, so stale or
// NaN slots cannot leak into the result.
//
// Tiles are gathered with 16-byte loads; K rows and V rows sit in LDS
// key-major without padding, read as 16-byte broadcasts (every lane reads the
// same key).  This path exists for fp32 accuracy (1e-4 against fp64); the
// bf16 MFMA kernel is the performance path.
//
// Split-key mode (a call too small to fill the chip, with a workspace): split
// s of a query tile covers the keys [s * split_len, (s+1) * split_len) at
// absolute positions and writes its merged unnormalised state (m, l, acc) in
// fp32 for the split combine, which adds the splits in increasing order.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace pgsr {

namespace {

constexpr int kTokens = 64;  // query tokens per workgroup (one per lane)
constexpr int kWaves = 4;

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int D, int KT>
__global__ void __launch_bounds__(kWaves * 64) attn_f32_kernel(AttnArgs a) {
  constexpr int KV = KT * D;                      // floats per tile operand
  __shared__ __attribute__((aligned(16))) float lds[kWaves][2][KV];

  const int tile = blockIdx.x / a.n_splits;
  const int split = blockIdx.x % a.n_splits;
  const int hq = blockIdx.y;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].tile_start <= tile) ++ei;
  const AttnEntry e = a.e[ei];
  const int lt = tile - e.tile_start;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int g = hq / G;
  const int B = a.block_size;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = lt * kTokens + lane;             // token index inside the suffix
  const bool valid = t < e.q_len;
  const int qpos = valid ? e.prefix + t : -1;    // absolute position (-1: padding row)
  const int t_last = min(e.q_len, (lt + 1) * kTokens) - 1;
  const int kv_len = e.prefix + e.q_len;
  // keys this workgroup visits: [key_lo, key_end), whole tiles at absolute
  // positions (split_len is a multiple of KT)
  const int key_lo = a.n_splits > 1 ? split * a.split_len : 0;
  const int key_end = a.n_splits > 1 ? min(e.prefix + t_last + 1, key_lo + a.split_len) : e.prefix + t_last + 1;
  if (key_lo >= key_end) return;                   // the whole workgroup: no barrier is skipped
  const int kt0 = key_lo / KT;
  const int n_kt = (key_end + KT - 1) / KT;

  float qr[D];
  {
    const float* qp = (const float*)a.q + ((int64_t)(e.q_off + (valid ? t : 0)) * a.n_q_heads + hq) * D;
#pragma unroll
    for (int c = 0; c < D; c += 4) {
      const f32x4 v = valid ? *(const f32x4*)(qp + c) : f32x4{0, 0, 0, 0};
      qr[c] = v[0]; qr[c + 1] = v[1]; qr[c + 2] = v[2]; qr[c + 3] = v[3];
    }
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
  float* ks = lds[w][0];
  float* vs = lds[w][1];

  for (int kt = kt0 + w; kt < n_kt; kt += kWaves) {
    const int kb = kt * KT;
    // K: slot rows of D floats, 4 at a time
    for (int i = lane; i < KV / 4; i += 64) {
      const int j = i / (D / 4), c = (i % (D / 4)) * 4;
      const int pos = kb + j;
      f32x4 val = {0, 0, 0, 0};
      if (pos < kv_len) {
        const int32_t id = blk_id(row[pos / B], a.n_blocks, a.chk);
        val = *(const f32x4*)(kc + ((layer_off + (int64_t)id * a.n_kv_heads + g) * B + pos % B) * D + c);
      }
      *(f32x4*)(ks + j * D + c) = val;
    }
    // V: stored [d][slot] per block; 4 consecutive slots of one d at a time
    for (int i = lane; i < KV / 4; i += 64) {
      const int c = i / (KT / 4), j = (i % (KT / 4)) * 4;
      const int pos = kb + j;                    // 4 slots of one block (B % 4 == 0)
      f32x4 val = {0, 0, 0, 0};
      if (pos < kv_len) {
        const int32_t id = blk_id(row[pos / B], a.n_blocks, a.chk);
        val = *(const f32x4*)(vc + ((layer_off + (int64_t)id * a.n_kv_heads + g) * D + c) * B + pos % B);
#pragma unroll
        for (int r = 1; r < 4; ++r)
          if (pos + r >= kv_len) val[r] = 0.f;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) vs[(j + r) * D + c] = val[r];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float s[KT];
    float tmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float d0 = 0.f, d1 = 0.f;
#pragma unroll
      for (int c = 0; c < D; c += 4) {
        const f32x4 kv = *(const f32x4*)(ks + j * D + c);
        d0 = fmaf(qr[c], kv[0], d0);
        d1 = fmaf(qr[c + 1], kv[1], d1);
        d0 = fmaf(qr[c + 2], kv[2], d0);
        d1 = fmaf(qr[c + 3], kv[3], d1);
      }
      s[j] = (kb + j <= qpos && kb + j < key_end) ? (d0 + d1) * c2 : -INFINITY;
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
      for (int c = 0; c < D; c += 4) {
        const f32x4 vv = *(const f32x4*)(vs + j * D + c);
        acc[c] = fmaf(p, vv[0], acc[c]);
        acc[c + 1] = fmaf(p, vv[1], acc[c + 1]);
        acc[c + 2] = fmaf(p, vv[2], acc[c + 2]);
        acc[c + 3] = fmaf(p, vv[3], acc[c + 3]);
      }
    }
    m = m_new;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // reads done before the next tile's writes
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Merge the four partial states in order 0, 1, 2, 3 through LDS (the tile
  // buffers are free now): wave w >= 1 publishes, wave 0 folds it in.
  float* pub = &lds[0][0][0];                    // [64][D + 2]
  static_assert(kWaves * 2 * KV >= 64 * (D + 2), "merge buffer");
  for (int src = 1; src < kWaves; ++src) {
    __syncthreads();
    if (w == src) {
      float* p = pub + lane * (D + 2);
#pragma unroll
      for (int c = 0; c < D; ++c) p[c] = acc[c];
      p[D] = m;
      p[D + 1] = l;
    }
    __syncthreads();
    if (w == 0) {
      const float* p = pub + lane * (D + 2);
      const float mo = p[D], lo = p[D + 1];
      const float mn = fmaxf(m, mo);
      const float mu = (mn == -INFINITY) ? 0.f : mn;
      const float a0 = exp2f(m - mu), a1 = exp2f(mo - mu);
      l = l * a0 + lo * a1;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = acc[c] * a0 + p[c] * a1;
      m = mn;
    }
  }
  if (w == 0 && valid && a.n_splits > 1) {        // unnormalised partials
    const int64_t prow = (int64_t)split * a.n_rows + (int64_t)(e.q_off + t) * a.n_q_heads + hq;
    float* acc_out = a.ws_acc + prow * D;
#pragma unroll
    for (int c = 0; c < D; c += 4) *(f32x4*)(acc_out + c) = f32x4{acc[c], acc[c + 1], acc[c + 2], acc[c + 3]};
    a.ws_ml[2 * prow] = m;
    a.ws_ml[2 * prow + 1] = l;
  } else if (w == 0 && valid) {
    float* op = (float*)a.o + ((int64_t)(e.q_off + t) * a.n_q_heads + hq) * D;
    const float inv = 1.f / l;
#pragma unroll
    for (int c = 0; c < D; c += 4)
      *(f32x4*)(op + c) = f32x4{acc[c] * inv, acc[c + 1] * inv, acc[c + 2] * inv, acc[c + 3] * inv};
  }
}

}  // namespace

int attn_f32_tile_tokens(int, int) { return kTokens; }

hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  dim3 grid(a.n_tiles * a.n_splits, a.n_q_heads);
  if (a.head_dim == 64)
    hipLaunchKernelGGL((attn_f32_kernel<64, 32>), grid, dim3(kWaves * 64), 0, s, a);
  else if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_f32_kernel<128, 16>), grid, dim3(kWaves * 64), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pgsr
