// Decode attention on CDNA4 matrix cores (gfx950): a few query tokens per
// sequence (a re-decode step) against the whole paged cache, without LDS.
//
// One wave per (sequence, KV head, key split).  Its 32 query rows are the
// sequence's TPW = floor(32 / G) tokens times the G query heads sharing the KV
// head (rows past TPW * G or past the sequence's tokens are padding).  The
// wave walks its split's keys in tiles of 32 and gathers each tile's MFMA
// operands straight from the paged cache into registers, one tile ahead: no
// LDS and no barrier, so waves never wait for each other and the loads of all
// resident waves keep HBM busy.  Four independent waves share a workgroup
// only for launch efficiency.
//
// S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16.  Two free
// choices make every gather a 16-byte load of contiguous cache bytes:
//  * the reduction order over d: lane half h of MFMA step ds holds
//    d in [h * D/2 + 8 ds, +8), so the K row piece a lane needs for successive
//    steps is contiguous (one load per step for bf16, per two steps for FP8);
//    Q^T is held in the same order;
//  * which key each K operand row is: row i holds key
//    16 ((i / 4) mod 2) + 4 (i / 8) + i mod 4 of the tile, which leaves keys
//    16h .. 16h+15, in order, in the S^T registers of lane half h.  The P
//    values of a 16-key PV step are then 8 consecutive keys per lane, and the
//    matching V^T operand is 8 consecutive slots of one d row of the
//    [d][slot] block layout (both steps in one 16-byte load for FP8).
// With bf16 codes at d = 128 the two tiles in flight, the accumulators and
// Q^T exceed 256 registers, so Q^T is parked in LDS (each wave its own rows,
// padded) and read per MFMA step; the other variants keep it in registers.
// FP8 E4M3 codes widen to bf16 exactly in registers (at most 4 significant
// bits each); the K scale rides in the softmax scale and the V scale in the
// output normalisation.
//
// Keys at or past the sequence length: addresses are clamped to valid slots,
// their scores are masked, and their V elements are zeroed, so stale or NaN
// slots never reach the result.  The online softmax (base 2, lazy rescale,
// row sum of the bf16-rounded P) is the prefill kernel's.  With several
// splits a wave writes unnormalised partials (m, l, acc) of its split and the
// split combine merges them in increasing split order; with one split it
// writes O.
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "attn_common.h"
#include "internal.h"

namespace pgsr {

namespace {

constexpr int kDecKT = 32;          // keys per tile
constexpr float kDecSlack = 8.f;    // lazy rescale threshold, log2 units

template <int D, int B, bool F8>
__global__ void __launch_bounds__(256, 2)
attn_decode_kernel(AttnArgs a, const int32_t* __restrict__ tables, const uint16_t* __restrict__ qg_,
                   const std::conditional_t<F8, uint8_t, uint16_t>* __restrict__ kc,
                   const std::conditional_t<F8, uint8_t, uint16_t>* __restrict__ vc,
                   uint16_t* __restrict__ og) {
  constexpr int KT = kDecKT;
  constexpr int NDS = D / 16;                    // S^T MFMA steps over d
  constexpr int NDB = D / 32;                    // 32-row blocks of O^T
  constexpr int NK = F8 ? NDS / 2 : NDS;         // 16-byte K loads per tile
  constexpr int NV = F8 ? NDB : 2 * NDB;         // 16-byte V loads per tile
  constexpr int EK = F8 ? 16 : 8;                // cache elements per 16-byte load
  static_assert(B % 16 == 0, "a 16-key group never straddles two blocks");
  constexpr bool kQLds = !F8 && D == 128;        // Q^T in LDS instead of registers
  constexpr int QLD = D + 8;                     // padded LDS row of Q (elements)
  __shared__ __attribute__((aligned(16))) uint16_t q_lds[kQLds ? 4 * 32 * QLD : 1];

  const int lane = threadIdx.x & 63, r = lane & 31, hh = lane >> 5;
  const int hkv = a.n_kv_heads;
  const int64_t wid = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wid >= (int64_t)a.n * hkv * a.n_splits) return;
  const int split = (int)(wid % a.n_splits);
  const int unit = (int)(wid / a.n_splits);
  const int g = unit % hkv;
  const AttnEntry e = a.e[unit / hkv];
  const int G = a.n_q_heads / hkv;
  const int TPW = 32 / G;
  const int tok = r / G, hq = g * G + r % G;
  const bool valid = r < TPW * G && tok < e.q_len;
  const int qpos = valid ? e.prefix + tok : -1;
  const int kv_len = e.prefix + e.q_len;
  // Keys of this split: [key_lo, key_hi); split_len is a multiple of the
  // tile, so tiles never cross a split boundary (only kv_len is unaligned).
  const int key_lo = a.n_splits > 1 ? split * a.split_len : 0;
  const int key_hi = a.n_splits > 1 ? min(kv_len, key_lo + a.split_len) : kv_len;
  if (key_lo >= key_hi) return;

  // Q^T operand: lane (row r, half hh) holds d in [hh D/2 + 8 ds, +8).
  bf16x8 qb[kQLds ? 1 : NDS];
  uint16_t* const q_mine = &q_lds[kQLds ? ((threadIdx.x >> 6) * 32 + r) * QLD + hh * (D / 2) : 0];
  {
    const uint16_t* qp = qg_ + ((int64_t)(e.q_off + (valid ? tok : 0)) * a.n_q_heads + hq) * D + hh * (D / 2);
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) {
      const u32x4 raw = valid ? *(const u32x4*)(qp + 8 * ds) : u32x4{0, 0, 0, 0};
      if constexpr (kQLds)
        *(u32x4*)(q_mine + 8 * ds) = raw;          // read back by this lane only
      else
        qb[ds] = __builtin_bit_cast(bf16x8, raw);
    }
  }
  auto q_operand = [&](int ds) {
    if constexpr (kQLds) return __builtin_bit_cast(bf16x8, *(const u32x4*)(q_mine + 8 * ds));
    else return qb[ds];
  };

  const int32_t* __restrict__ row = tables + (int64_t)e.seq * a.max_bps;
  const int64_t head_base = (int64_t)a.layer * a.n_blocks * hkv + g;   // + id * hkv
  const int kperm = 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3);     // key of K operand row r
  auto k_key = [&](int kb) { return min(kb + kperm, kv_len - 1); };
  auto v_key = [&](int kb) {                                           // first of this lane's 16 V keys
    const int k0 = kb + 16 * hh;
    return k0 < kv_len ? k0 : ((kv_len - 1) & ~15);
  };
  auto k_id = [&](int kb) { return blk_id(row[k_key(kb) / B], a.n_blocks, a.chk); };
  auto v_id = [&](int kb) { return blk_id(row[v_key(kb) / B], a.n_blocks, a.chk); };

  u32x4 kr[NK], vr[NV];
  auto load_k = [&](int kb, int idk) {
    const int kk = k_key(kb);
    const auto* kp = kc + ((head_base + (int64_t)idk * hkv) * B + kk % B) * D + hh * (D / 2);
#pragma unroll
    for (int c = 0; c < NK; ++c) kr[c] = *(const u32x4*)(kp + c * EK);
  };
  auto load_v = [&](int kb, int idv) {
    const auto* vp = vc + ((head_base + (int64_t)idv * hkv) * D + r) * B + v_key(kb) % B;
#pragma unroll
    for (int c = 0; c < NV; ++c) {
      const int db = F8 ? c : c / 2, ks = F8 ? 0 : c % 2;
      vr[c] = *(const u32x4*)(vp + (int64_t)db * 32 * B + 8 * ks);
    }
  };
  auto k_operand = [&](const u32x4 (&k)[NK], int ds) {
    if constexpr (F8) {
      const u32x4 w = k[ds / 2];
      return __builtin_bit_cast(bf16x8, widen_fp8(ds % 2 ? u32x2{w[2], w[3]} : u32x2{w[0], w[1]}));
    } else {
      return __builtin_bit_cast(bf16x8, k[ds]);
    }
  };
  auto v_operand = [&](const u32x4 (&v)[NV], int ks, int db) {
    if constexpr (F8) {
      const u32x4 w = v[db];
      return widen_fp8(ks ? u32x2{w[2], w[3]} : u32x2{w[0], w[1]});
    } else {
      return v[2 * db + ks];
    }
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m = -INFINITY, l = 0.f;
  const float c2 = a.scale_log2;

  // Tile j+1's K is requested before tile j's S products and its V right
  // after them (tile j's K is dead by then), with block ids a tile earlier
  // still.  The requests for the last tile are skipped, so the compiler waits
  // for all outstanding loads before the last S product: K's latency is
  // covered by the S products, V's by a whole tile.  Measured on 32 x 8192
  // keys this beats unconditional requests (both covered by a whole tile) by
  // 6% for bf16 and ties for FP8: fewer bytes in flight per CU keep the HBM
  // queues shorter.
  const int n_kt = (key_hi - key_lo + KT - 1) / KT;
  load_k(key_lo, k_id(key_lo));
  load_v(key_lo, v_id(key_lo));
  int idk_n = 0, idv_n = 0;
  if (n_kt > 1) {
    idk_n = k_id(key_lo + KT);
    idv_n = v_id(key_lo + KT);
  }
  for (int j = 0; j < n_kt; ++j) {
    const int kb = key_lo + j * KT;
    const bool more = j + 1 < n_kt;
    u32x4 kcur[NK], vcur[NV];
#pragma unroll
    for (int c = 0; c < NK; ++c) kcur[c] = kr[c];
    if (more) load_k(kb + KT, idk_n);
    f32x16 s = f32x16{};
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_operand(kcur, ds), q_operand(ds), s, 0, 0, 0);
#pragma unroll
    for (int c = 0; c < NV; ++c) vcur[c] = vr[c];
    if (more) {
      load_v(kb + KT, idv_n);
      if (j + 2 < n_kt) {
        idk_n = k_id(kb + 2 * KT);
        idv_n = v_id(kb + 2 * KT);
      }
    }
    // lane half hh holds keys kb + 16 hh + v; mask those past the row's position
    if (kb + KT - 1 > e.prefix) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[v] = kb + 16 * hh + v > qpos ? -INFINITY : s[v];
    }
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[v]);
    mx = fmaxf(mx, xor32(mx)) * c2;
    const bool bump = mx > m + kDecSlack;
    const float m_new = bump ? mx : m;
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = bump ? __builtin_amdgcn_exp2f(m - m_use) : 1.f;
    m = m_new;
    bf16x8 pb[2];
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      f32x8 p8;
#pragma unroll
      for (int t = 0; t < 8; ++t) p8[t] = __builtin_amdgcn_exp2f(fmaf(s[8 * ks + t], c2, -m_use));
      pb[ks] = __builtin_convertvector(p8, bf16x8);
      const bf16x2* p2 = (const bf16x2*)&pb[ks];
      ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[0], kOnes, ps0, false);
      ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[1], kOnes, ps1, false);
      ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[2], kOnes, ps0, false);
      ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[3], kOnes, ps1, false);
    }
    l = fmaf(l, alpha, ps0 + ps1);
    if (__ballot(bump)) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
    }
    const bool tail = kb + KT > kv_len;            // V of keys >= kv_len must read as 0
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        u32x4 vv = v_operand(vcur, ks, db);
        if (tail) vv = zero_tail(vv, kb + 16 * hh + 8 * ks, kv_len);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pb[ks], oacc[db],
                                                           0, 0, 0);
      }
  }

  const float l_tot = l + xor32(l);
  if (!valid) return;
  const int64_t qrow = (int64_t)(e.q_off + tok) * a.n_q_heads + hq;
  if (a.n_splits > 1) {                            // unnormalised partials, fp32
    const int64_t prow = (int64_t)split * a.n_rows + qrow;
    float* acc = a.ws_acc + prow * D + 4 * hh;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
        *(f32x4*)(acc + db * 32 + 8 * i4) =
            f32x4{oacc[db][4 * i4 + 0], oacc[db][4 * i4 + 1], oacc[db][4 * i4 + 2], oacc[db][4 * i4 + 3]};
    if (hh == 0) *(f32x2*)(a.ws_ml + 2 * prow) = f32x2{m, l_tot};
  } else {
    const float inv = a.o_scale / l_tot;
    uint16_t* op = og + qrow * D + 4 * hh;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        f32x4 v4 = {oacc[db][4 * i4 + 0] * inv, oacc[db][4 * i4 + 1] * inv, oacc[db][4 * i4 + 2] * inv,
                    oacc[db][4 * i4 + 3] * inv};
        *(bf16x4*)(op + db * 32 + 8 * i4) = __builtin_convertvector(v4, bf16x4);
      }
  }
}

template <int D, int B, bool F8>
void launch_dec(const AttnArgs& a, hipStream_t s) {
  using CT = std::conditional_t<F8, uint8_t, uint16_t>;
  const int64_t waves = (int64_t)a.n * a.n_kv_heads * a.n_splits;
  hipLaunchKernelGGL((attn_decode_kernel<D, B, F8>), dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, a,
                     a.tables, (const uint16_t*)a.q, (const CT*)a.k_cache, (const CT*)a.v_cache,
                     (uint16_t*)a.o);
}

template <int D, bool F8>
hipError_t launch_dec_d(const AttnArgs& a, hipStream_t s) {
  switch (a.block_size) {
    case 16: launch_dec<D, 16, F8>(a, s); break;
    case 32: launch_dec<D, 32, F8>(a, s); break;
    case 64: launch_dec<D, 64, F8>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int attn_decode_keys_per_tile() { return kDecKT; }

hipError_t launch_attn_decode(const AttnArgs& a, bool fp8, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.head_dim == 128) return fp8 ? launch_dec_d<128, true>(a, s) : launch_dec_d<128, false>(a, s);
  if (a.head_dim == 64) return fp8 ? launch_dec_d<64, true>(a, s) : launch_dec_d<64, false>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace pgsr
