// bf16 prefix + causal prefill attention for head_dim 128 on CDNA4 matrix
// cores (gfx950), software-pipelined so that each wave overlaps its own
// matrix products with its own softmax arithmetic.
//
// Work decomposition.  A workgroup of 8 wave64s, two per SIMD (each wave
// holds up to 256 VGPRs), owns one KV head g and a tile of 8 * 32 / G
// consecutive suffix tokens with the G query heads sharing g (G divides 32);
// each wave owns one 32-row block of (token, head) query rows, and the two
// waves of a SIMD interleave their matrix products with each other's softmax
// arithmetic.  Three 35 KB LDS tile buffers keep one workgroup per CU.
// blockIdx.x = tile * n_kv_heads + g, so all tiles of a KV head land on one
// XCD and share its L2 copy of the head's keys and values; tiles are issued
// costliest first.
//
// Per 64-key tile at absolute positions kb .. kb+63, in fp32:
//   S^T = K Q^T (v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q^T in
//   registers); a lane holds one query column and 16 keys of each 32-key half,
//   so row max and row sum are in-lane plus one exchange between lane halves.
//   Online softmax in base 2 with a lazy rescale (the running max moves only
//   when a tile exceeds it by more than 2^8).  Q is scaled by the softmax
//   scale * log2(e) once, when it is loaded, and every S accumulator starts
//   at -m (m: the row's current reference max), so S holds s * c - m and the
//   exponentials take it directly; when m moves, the tile that moved it is
//   shifted by the same amount.  P is rounded to bf16 and the row sum adds
//   exactly those values; O^T += V^T P^T.  Accumulator row i of S^T
//   is key pi(i) (bits 2 and 3 of i swapped), so a lane's P^T registers hold
//   8 consecutive keys of each 16-key group and V^T sits in LDS in natural
//   key order: every operand is one 16-byte read.
//
// Pipeline.  Tiles whose keys all precede the workgroup's first query need no
// causal mask.  For those, step t issues the products S(t+1) = K(t+1) Q^T
// interleaved with the exponentials of S(t)'s first 32 keys, then
// O += V(t) P(t) interleaved with the exponentials of the last 32 keys and the
// row max of S(t+1); the softmax of one tile thus runs in the shadow of
// another tile's products.  The (at most a few) tiles that straddle the
// diagonal run unpipelined with the mask applied by select.  Three LDS tile
// buffers rotate, so a step needs one barrier: tile t+2 is gathered through
// the block table into registers at the start of step t and written to LDS at
// its end, into the buffer tile t-1 occupied.
//
// Every row's arithmetic (accumulation order of the products, max, rounding
// of P, row-sum order, rescale, final division) is the same sequence of
// operations whichever kernel, tile or wave holds the row, so results depend
// only on a query's absolute position and its keys: selective replay and
// full reset agree bitwise, and so does the four-wave kernel of attn_bf16.hip.
#include <hip/hip_runtime.h>

#include <cmath>

#include "attn_common.h"
#include "internal.h"

namespace pgsr {

namespace {

constexpr int kPW = 8;          // waves per workgroup, two per SIMD
constexpr int kPQB = 1;         // 32-row query blocks per wave
constexpr int kPKT = 64;        // keys per tile
constexpr int kPBuf = 3;        // LDS tile buffers
constexpr float kPSlack = 8.f;  // lazy rescale threshold, log2 units

template <int B>
__global__ void __launch_bounds__(kPW * 64, 1)
attn_bf16_pipe_kernel(AttnArgs a, const int32_t* __restrict__ tables, const uint16_t* __restrict__ qg_,
                      const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
                      uint16_t* __restrict__ og) {
  constexpr int D = 128, NW = kPW, QB = kPQB, KT = kPKT;
  constexpr int KB = KT / B;               // blocks per key tile
  constexpr int KLD = D + 8;               // LDS row stride of the K tile (elements)
  constexpr int VLD = KT + 8;              // LDS row stride of the V^T tile (elements)
  constexpr int NT = NW * 64;
  constexpr int CHB = B * D / 8;           // 16-byte chunks per block-head (K or V)
  constexpr int CPT = KT * D / 8 / NT;     // chunks per thread per tile (K or V)
  constexpr int NDS = D / 16;              // reduction steps of S
  constexpr int NDB = D / 32;              // 32-row blocks of O^T
  constexpr int NKS = KT / 16;             // 16-key steps of PV
  // phase A takes the exponentials of keys 0..31 of every block: 2 * QB
  // (block, 16-key group) pairs, one every kEvery reduction steps of S(t+1)
  constexpr int kEvery = NDS / (2 * QB);
  static_assert(kEvery >= 1 && NDS % (2 * QB) == 0, "phase A placement");
  static_assert(CPT * NT * 8 == KT * D, "tile split");
  static_assert(KB >= 1 && KB <= 4, "block size 16, 32 or 64");
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kPBuf][KT * KLD];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kPBuf][D * VLD];

  uint64_t clk0 = 0, rt0 = 0;
  if (a.clk) {
    clk0 = __builtin_amdgcn_s_memtime();
    rt0 = __builtin_amdgcn_s_memrealtime();
  }
  const int hkv = a.n_kv_heads;
  const int g = blockIdx.x % hkv;
  const int split = (blockIdx.x / hkv) % a.n_splits;
  const int tile = blockIdx.x / hkv / a.n_splits;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].tile_start <= tile) ++ei;
  const AttnEntry e = a.e[ei];
  const int G = a.n_q_heads / hkv;
  const int TPB = 32 / G;                           // tokens per 32-row block
  const int TW = NW * QB * TPB;                     // tokens per tile
  const int n_tiles_e = (e.q_len + TW - 1) / TW;
  const int lt = n_tiles_e - 1 - (tile - e.tile_start);
  const int t0 = lt * TW;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, r = lane & 31, hh = lane >> 5;
  const int hq = g * G + r % G;
  int tok[QB], qpos[QB];
  bool valid[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    tok[b] = t0 + (w * QB + b) * TPB + r / G;
    valid[b] = tok[b] < e.q_len;
    qpos[b] = valid[b] ? e.prefix + tok[b] : -1;
  }
  const int t_last = min(e.q_len, t0 + TW) - 1;
  const int kv_len = e.prefix + e.q_len;
  const int first_q = e.prefix + t0;
  const int key_lo = split * a.split_len;
  const int key_end = min(e.prefix + t_last + 1, a.n_splits > 1 ? key_lo + a.split_len : INT32_MAX);
  if (key_lo >= key_end) return;                   // nothing of this tile in this split
  const int kt0 = key_lo / KT;
  const int n_kt = (key_end + KT - 1) / KT;
  // tiles [kt0, nu) hold only keys at or before every query of the workgroup
  const int nu = min(max((first_q + 1) / KT, kt0), n_kt);

  // Q^T operands: lane holds Q[row][16*ds + 8*hh .. +7].
  bf16x8 qf[QB][NDS];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const uint16_t* qg = qg_ + ((int64_t)(e.q_off + tok[b]) * a.n_q_heads + hq) * D + 8 * hh;
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) {
      u32x4 raw = valid[b] ? *(const u32x4*)(qg + 16 * ds) : u32x4{0, 0, 0, 0};
      f32x8 qx = __builtin_convertvector(__builtin_bit_cast(bf16x8, raw), f32x8) * a.scale_log2;
      qf[b][ds] = __builtin_convertvector(qx, bf16x8);   // Q scaled by scale * log2(e), rounded once
    }
  }

  const int32_t* __restrict__ row = tables + (int64_t)e.seq * a.max_bps;
  const int64_t head_base = (int64_t)a.layer * a.n_blocks * hkv + g;
  const int last_blk = (kv_len - 1) / B;

  // Chunk i of thread tid belongs to block chunk_blk(i) of the tile; when a
  // block-head has fewer chunks than the workgroup has threads, that block
  // depends on the wave only (CHB is a multiple of 64), so it is taken as a
  // scalar and selecting its id needs no per-lane branch.
  constexpr bool kBlkConst = CHB % NT == 0;
  static_assert(kBlkConst || CHB % 64 == 0, "block-head chunks per wave");
  const int wave_blk = __builtin_amdgcn_readfirstlane(tid / CHB);
  auto chunk_blk = [&](int i) {
    if constexpr (kBlkConst) return i / (CHB / NT);
    else return i * (NT / CHB) + wave_blk;
  };
  auto chunk_in = [&](int i) {
    if constexpr (kBlkConst) return tid + (i % (CHB / NT)) * NT;
    else return tid % CHB;
  };
  // Block ids of a tile: a per-lane load (lane bi holds block bi's id) one
  // step ahead; each chunk reads its block's id with readlane at a scalar
  // lane index.
  int idv = 0;
  auto fetch_ids = [&](int kt) {
    idv = blk_id(row[min(kt * KB + (lane < KB ? lane : 0), last_blk)], a.n_blocks, a.chk);
  };
  // Per-lane element offsets of a thread's chunks inside a block-head (K:
  // slot-major rows of D; V: d-major rows of B slots), fixed for the kernel;
  // a load is then a scalar block pointer plus this offset.
  int koff[CPT], voff[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int in = chunk_in(i);
    koff[i] = (in / (D / 8)) * D + (in % (D / 8)) * 8;
    voff[i] = (in / (B / 8)) * B + (in % (B / 8)) * 8;
  }
  u32x4 kreg[CPT], vreg[CPT];
  auto load_tile = [&](int ids) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int id = __builtin_amdgcn_readlane(ids, chunk_blk(i));
      const int64_t base = (head_base + (int64_t)id * hkv) * (B * D);
      kreg[i] = *(const u32x4*)((kc + base) + koff[i]);
      vreg[i] = *(const u32x4*)((vc + base) + voff[i]);
    }
  };
  auto store_tile = [&](int buf, int kb) {
    const bool tail = kb + KT > kv_len;   // V slots at or past kv_len must read as 0
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int blk = chunk_blk(i), in = chunk_in(i);
      *(u32x4*)&k_lds[buf][(blk * B + in / (D / 8)) * KLD + (in % (D / 8)) * 8] = kreg[i];
      const int dd = in / (B / 8), key0 = blk * B + (in % (B / 8)) * 8;
      u32x4 val = vreg[i];
      if (tail) val = zero_tail(val, kb + key0, kv_len);   // selects only: no per-lane branch
      *(u32x4*)&v_lds[buf][dd * VLD + key0] = val;
    }
  };
  // One pipeline step's memory work around its compute: gather tile x+2 at
  // the start, write it to LDS at the end.  Both run unconditionally, so every
  // load is consumed on every path and no load is outstanding across steps: a
  // tile past the last reads clamped (valid) block ids and lands in the buffer
  // of tile x-1, which no later step reads.
  auto gather_next = [&](int x) {
    const int ids = idv;                         // tile x+2, fetched a step ago
    fetch_ids(x + 3);
    load_tile(ids);
  };
  auto commit_next = [&](int x) { store_tile((x + 2) % kPBuf, (x + 2) * KT); };

  f32x16 oacc[QB][NDB];
#pragma unroll
  for (int b = 0; b < QB; ++b)
#pragma unroll
    for (int db = 0; db < NDB; ++db) oacc[b][db] = f32x16{};
  float m[QB], l[QB], alpha[QB], m_use[QB];
  f32x16 cinit[QB];     // -m_use in every element: the start value of each S accumulator
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    m[b] = -INFINITY;
    l[b] = 0.f;
    alpha[b] = 1.f;
    m_use[b] = 0.f;
    cinit[b] = f32x16{};
  }

  const int kr = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);   // pi(r): bits 2 and 3 swapped
  auto k_op = [&](int buf, int kh, int ds) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)&k_lds[buf][(kh * 32 + kr) * KLD + 16 * ds + 8 * hh]);
  };
  auto v_op = [&](int buf, int ks, int db) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)&v_lds[buf][(db * 32 + r) * VLD + ks * 16 + 8 * hh]);
  };
  auto mfma = [](bf16x8 x, bf16x8 y, f32x16 c) { return __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c, 0, 0, 0); };

  // Row max of a tile (log2 units), branch-free, and the lazy-rescale
  // decision; the wave rescales O when any of its rows moved its maximum.
  auto row_max = [&](const f32x16 (&s)[QB][2], float (&mx)[QB]) {
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      float x = -INFINITY;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int i = 0; i < 16; ++i) x = fmaxf(x, s[b][kh][i]);
      mx[b] = fmaxf(x, xor32(x)) + m_use[b];   // S holds s * c - m_use
    }
  };
  auto apply_max = [&](const float (&mx)[QB], f32x16 (&st)[QB][2]) {
    bool any = false;
    float delta[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const bool bump = mx[b] > m[b] + kPSlack;
      const float m_new = bump ? mx[b] : m[b];
      const float mu = m_new == -INFINITY ? 0.f : m_new;
      delta[b] = mu - m_use[b];
      m_use[b] = mu;
      alpha[b] = bump ? __builtin_amdgcn_exp2f(m[b] - m_use[b]) : 1.f;
      m[b] = m_new;
      any = any || bump;
    }
    if (__ballot(any)) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[b][db] *= alpha[b];
        st[b][0] -= delta[b];
        st[b][1] -= delta[b];
#pragma unroll
        for (int i = 0; i < 16; ++i) cinit[b][i] = -m_use[b];
      }
    }
  };
  auto update_max = [&](f32x16 (&s)[QB][2]) {
    float mx[QB];
    row_max(s, mx);
    apply_max(mx, s);
  };
  // P for 16 keys (registers o8 .. o8+7 of one 32-key half), rounded to bf16,
  // with the row-sum terms added in the fixed order.
  auto expo = [&](const f32x16& s, int o8, int b, float& ps0, float& ps1) {
    f32x8 pv8;
#pragma unroll
    for (int j = 0; j < 8; ++j) pv8[j] = __builtin_amdgcn_exp2f(s[o8 + j]);
    const bf16x8 p = __builtin_convertvector(pv8, bf16x8);
    const bf16x2* p2 = (const bf16x2*)&p;
    ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[0], kOnes, ps0, false);
    ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[1], kOnes, ps1, false);
    ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[2], kOnes, ps0, false);
    ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[3], kOnes, ps1, false);
    return p;
  };

  // ---- prologue: tiles kt0 and kt0+1 into LDS -------------------------- //
  fetch_ids(kt0);
  {
    const int ids = idv;
    fetch_ids(kt0 + 1);
    load_tile(ids);
    store_tile(kt0 % kPBuf, kt0 * KT);
  }
  {
    const int ids = idv;
    fetch_ids(kt0 + 2);
    load_tile(ids);
    store_tile((kt0 + 1) % kPBuf, (kt0 + 1) * KT);
  }
  __syncthreads();

  f32x16 sa[QB][2], sb[QB][2];
  auto qk = [&](int buf, f32x16 (&s)[QB][2]) {
#pragma unroll
    for (int b = 0; b < QB; ++b) s[b][0] = s[b][1] = cinit[b];
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        const bf16x8 kx = k_op(buf, kh, ds);
#pragma unroll
        for (int b = 0; b < QB; ++b) s[b][kh] = mfma(kx, qf[b][ds], s[b][kh]);
      }
  };
  if (nu > kt0) {
    qk(kt0 % kPBuf, sa);
    update_max(sa);
  }

  // ---- pipelined steps over unmasked tiles ----------------------------- //
  // Step t: S(t+1) = K(t+1) Q^T with P(t) keys 0..31; O += V(t) P(t) with
  // P(t) keys 32..63 and the row max of S(t+1).
  auto step = [&](int t, const f32x16 (&sc)[QB][2], f32x16 (&sn)[QB][2]) {
    __syncthreads();
    gather_next(t);
    const int cb = t % kPBuf, nb = (t + 1) % kPBuf;
    bf16x8 p[QB][NKS];
    float ps0[QB], ps1[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      ps0[b] = 0.f;
      ps1[b] = 0.f;
      sn[b][0] = sn[b][1] = cinit[b];
    }
    // phase A: 32 products of S(t+1), 16 K operand reads; exponentials of
    // keys 0..31 of S(t) (both blocks)
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) {
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        const bf16x8 kx = k_op(nb, kh, ds);
#pragma unroll
        for (int b = 0; b < QB; ++b) sn[b][kh] = mfma(kx, qf[b][ds], sn[b][kh]);
      }
      if (ds % kEvery == 0) {                  // pair j = (block j / 2, 16-key group j % 2)
        const int j = ds / kEvery, b = j / 2, ks = j % 2;
        p[b][ks] = expo(sc[b][0], 8 * ks, b, ps0[b], ps1[b]);
      }
    }
    // phase B: 32 products of O; exponentials of keys 32..63, row max of S(t+1)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 vx = v_op(cb, ks, db);
#pragma unroll
        for (int b = 0; b < QB; ++b) oacc[b][db] = mfma(vx, p[b][ks], oacc[b][db]);
      }
      if (ks < 2) {                            // keys 32..63, needed by ks = 2, 3
#pragma unroll
        for (int b = 0; b < QB; ++b) p[b][2 + ks] = expo(sc[b][1], 8 * ks, b, ps0[b], ps1[b]);
      }
    }
    float mx[QB];
    row_max(sn, mx);
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      l[b] = fmaf(l[b], alpha[b], ps0[b] + ps1[b]);
      // Keep this step's row sum in this step: otherwise the compiler sinks
      // the dot products of both unrolled steps to the loop's end, where they
      // run with no products to overlap and hold P live across a step.
      asm volatile("" ::"v"(l[b]));
    }
    commit_next(t);
    apply_max(mx, sn);
  };
  // Finish a tile whose S is computed and whose max is taken.
  auto finish = [&](int t, const f32x16 (&sc)[QB][2]) {
    __syncthreads();
    gather_next(t);
    const int cb = t % kPBuf;
    bf16x8 p[QB][NKS];
    float ps0[QB], ps1[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      ps0[b] = 0.f;
      ps1[b] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) p[b][ks] = expo(sc[b][ks / 2], 8 * (ks % 2), b, ps0[b], ps1[b]);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 vx = v_op(cb, ks, db);
#pragma unroll
        for (int b = 0; b < QB; ++b) oacc[b][db] = mfma(vx, p[b][ks], oacc[b][db]);
      }
#pragma unroll
    for (int b = 0; b < QB; ++b) l[b] = fmaf(l[b], alpha[b], ps0[b] + ps1[b]);
    commit_next(t);
  };

  int t = kt0;
  for (; t + 2 < nu; t += 2) {
    step(t, sa, sb);
    step(t + 1, sb, sa);
  }
  if (t + 1 < nu) {
    step(t, sa, sb);
    ++t;
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      sa[b][0] = sb[b][0];
      sa[b][1] = sb[b][1];
    }
  }
  if (nu > kt0) finish(t, sa);

  // ---- tiles on the diagonal: mask by select, unpipelined -------------- //
  for (int u = nu; u < n_kt; ++u) {
    __syncthreads();
    gather_next(u);
    const int cb = u % kPBuf, kb = u * KT;
    qk(cb, sa);
#pragma unroll
    for (int b = 0; b < QB; ++b)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb + kh * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
          sa[b][kh][i] = key > qpos[b] ? -INFINITY : sa[b][kh][i];
        }
    update_max(sa);
    bf16x8 p[QB][NKS];
    float ps0[QB], ps1[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      ps0[b] = 0.f;
      ps1[b] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) p[b][ks] = expo(sa[b][ks / 2], 8 * (ks % 2), b, ps0[b], ps1[b]);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 vx = v_op(cb, ks, db);
#pragma unroll
        for (int b = 0; b < QB; ++b) oacc[b][db] = mfma(vx, p[b][ks], oacc[b][db]);
      }
#pragma unroll
    for (int b = 0; b < QB; ++b) l[b] = fmaf(l[b], alpha[b], ps0[b] + ps1[b]);
    commit_next(u);
  }

  // ---- epilogue: normalise and store (or write split partials) --------- //
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const float l_tot = l[b] + xor32(l[b]);
    if (valid[b] && a.n_splits > 1) {
      const int64_t prow = (int64_t)split * a.n_rows + (int64_t)(e.q_off + tok[b]) * a.n_q_heads + hq;
      float* acc = a.ws_acc + prow * D + 4 * hh;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4)
          *(f32x4*)(acc + db * 32 + 8 * i4) =
              f32x4{oacc[b][db][4 * i4 + 0], oacc[b][db][4 * i4 + 1], oacc[b][db][4 * i4 + 2],
                    oacc[b][db][4 * i4 + 3]};
      if (hh == 0) *(f32x2*)(a.ws_ml + 2 * prow) = f32x2{m[b], l_tot};
    } else if (valid[b]) {
      const float inv = a.o_scale / l_tot;
      uint16_t* op = og + ((int64_t)(e.q_off + tok[b]) * a.n_q_heads + hq) * D + 4 * hh;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          f32x4 v4 = {oacc[b][db][4 * i4 + 0] * inv, oacc[b][db][4 * i4 + 1] * inv,
                      oacc[b][db][4 * i4 + 2] * inv, oacc[b][db][4 * i4 + 3] * inv};
          *(bf16x4*)(op + db * 32 + 8 * i4) = __builtin_convertvector(v4, bf16x4);
        }
    }
  }
  if (a.clk && tid == 0 && (int)blockIdx.x < a.clk_n) {
    const uint64_t clk1 = __builtin_amdgcn_s_memtime(), rt1 = __builtin_amdgcn_s_memrealtime();
    uint64_t* c = a.clk + 4 * (int64_t)blockIdx.x;
    c[0] = clk0;
    c[1] = clk1;
    c[2] = rt0;
    c[3] = rt1;
  }
}

}  // namespace

bool attn_bf16_pipe_eligible(int head_dim, int group) {
  return head_dim == 128 && group >= 1 && group <= 32 && 32 % group == 0;
}

int attn_bf16_pipe_tile_tokens(int group) { return kPW * kPQB * (32 / group); }

hipError_t launch_attn_bf16_pipe(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  const int group = a.n_q_heads / a.n_kv_heads;
  if (!attn_bf16_pipe_eligible(a.head_dim, group)) return hipErrorInvalidValue;
  const dim3 grid(a.n_tiles * a.n_kv_heads * a.n_splits), blk(kPW * 64);
  const auto* q = (const uint16_t*)a.q;
  const auto* kc = (const uint16_t*)a.k_cache;
  const auto* vc = (const uint16_t*)a.v_cache;
  auto* o = (uint16_t*)a.o;
  switch (a.block_size) {
    case 16: hipLaunchKernelGGL(attn_bf16_pipe_kernel<16>, grid, blk, 0, s, a, a.tables, q, kc, vc, o); break;
    case 32: hipLaunchKernelGGL(attn_bf16_pipe_kernel<32>, grid, blk, 0, s, a, a.tables, q, kc, vc, o); break;
    case 64: hipLaunchKernelGGL(attn_bf16_pipe_kernel<64>, grid, blk, 0, s, a, a.tables, q, kc, vc, o); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pgsr
