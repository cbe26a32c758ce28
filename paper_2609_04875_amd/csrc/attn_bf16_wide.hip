// bf16 prefix + causal prefill attention for head_dim 128 and 16-token cache
// blocks on CDNA4 matrix cores (gfx950): one wave per SIMD holding 64 query
// rows, so every K and V^T operand read from LDS feeds two products.
//
// Work decomposition.  A workgroup of 4 wave64s (one per SIMD, up to 512
// registers each) owns one KV head g and a tile of 4 * 64 / G consecutive
// suffix tokens with the G query heads sharing g (G divides 32); wave w owns
// two 32-row blocks of (token, head) query rows.  blockIdx.x = tile *
// n_kv_heads + g keeps every tile of a KV head on one XCD; tiles are issued
// costliest first.  The query tiling, the key tiling, the per-row arithmetic
// and therefore every output bit are those of the two-wave pipelined kernel
// (attn_bf16_pipe.hip) and of the four-wave kernel (attn_bf16.hip): scores
// S^T = K Q^T and O^T += V^T P^T on v_mfma_f32_32x32x16_bf16 with Q scaled by
// softmax scale * log2(e) at load, accumulators started at -m, the 64-key
// row max with a lazy rescale (the reference max moves only when a tile
// exceeds it by more than 2^8), P rounded to bf16 and summed as rounded.
//
// Registers.  64 rows per wave need O (128 registers), Q (64), two S tiles
// (128: the next tile's products run during this tile's softmax), P (32) and
// the -m splat (32).  O and Q live in AGPRs: the products are written as
// inline assembly with AGPR operands (O as accumulator, Q as the B operand of
// S^T = K Q^T), which the compiler cannot express for a mix of VGPR and AGPR
// accumulators.  The compiler does not see those products as matrix
// instructions, so the wait states it would otherwise insert are written out:
// 19 before any VALU read of S or O after its last product (s_sync,
// oacc_sync), 4 after VALU writes that a product reads as accumulator or
// operand (rescale, -m splat, Q), and a fresh P is written at least three
// products before its first use.
//
// K/V tiles.  Each 64-key tile (four 16-key blocks) reaches LDS through
// global_load_lds_dwordx4: no staging registers and no LDS stores.  A wave's
// request writes a contiguous 1 KB run (lane l's 16 bytes at byte 16 l), so
// the LDS images are laid out for the readers by choosing which global chunk
// each lane fetches: K keeps the cache's [key][d] rows but chunk c of key row
// j sits at slot c ^ j (the 16 rows an operand read touches hit 16 different
// bank groups); V^T keeps the cache's per-block [d][16 slots] but puts slots
// 0-7 of 32 consecutive d rows in one 512-byte half and slots 8-15 in the
// other, so a V^T operand read is 1 KB of contiguous LDS.  Four 32 KB buffers
// rotate: the step that works on tile x requests tile x + 3 into the buffer
// of tile x - 1, so a request has two steps to land.  The requests are inline
// assembly too; the loop issues no other vector memory operation, so "all but
// the latest 8 requests complete" (s_waitcnt vmcnt(8)) before the one barrier
// of a step proves the tiles the next step reads are in LDS.  Block ids come
// from a copy of the workgroup's part of the block table in LDS (one 16-byte
// read per tile, in order with the operand reads); the loop issues no scalar
// load (one in flight would turn every LDS wait into a full wait).
//
// Step schedule.  Tiles whose keys all precede the workgroup's first query
// need no mask.  Step t is 64 issue slots fenced by sched_barrier, one product
// each: slots 0-3 the last four products of O += V(t-1) P(t-1), deferred
// from the step before so that the matrix pipe has work while the first K
// operands of this step come from LDS (they can only be read after the
// step's barrier); slots 4-35 the products of S(t+1); slots 36-63 the first
// 28 products of O += V(t) P(t).  Around them: the eight requests of tile
// t+3 (slots 0-7), LDS operand reads two operands ahead, the exponentials of
// P(t) (two per item, their bf16 rounding two slots later) and the row max
// of S(t+1) (slots 38-63, after its last product).  Every O accumulator
// still receives its products in the same order; when a row moves its
// reference max, the deferred products are issued before O is rescaled.  A
// single wave has no partner wave to fill the matrix pipe while it waits,
// so the order is fixed here rather than left to the scheduler.  Tiles that
// straddle the diagonal run unpipelined with the mask applied by select; a
// tile past kv_len gets its V^T slots zeroed in LDS.
#include <hip/hip_runtime.h>

#include <cmath>
#include <utility>

#include "attn_common.h"
#include "internal.h"

// The requests write M0 (the LDS address of a global->LDS load) from inline
// assembly that lists it as clobbered; nothing else in this file uses M0.
#pragma clang diagnostic ignored "-Winline-asm"

namespace pgsr {

namespace {

constexpr int kWW = 4;              // waves per workgroup, one per SIMD
constexpr int kWQB = 2;             // 32-row query blocks per wave
constexpr int kWKT = 64;            // keys per tile
constexpr int kWBufElems = 16384;   // elements per LDS tile buffer (K 8192, V^T 8192)
constexpr float kWSlack = 8.f;      // lazy rescale threshold, log2 units
constexpr int kWMaxIdt = 8192;      // block-table entries a workgroup keeps in LDS
// products of O += V P deferred past the next step's barrier (0, 2, 4, 6 or
// 8; 4 and 8 measured alike, both 1% faster than none)
#ifndef PGSR_WIDE_DEFER
#define PGSR_WIDE_DEFER 4
#endif
constexpr int kWDefer = PGSR_WIDE_DEFER;

// f(integral_constant<int, I>) for I = 0, 1, ... in order, at compile time.
template <class F, int... I>
__device__ __forceinline__ void static_for(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

__global__ void __launch_bounds__(kWW * 64, 1)
attn_bf16_wide_kernel(AttnArgs a, const int32_t* __restrict__ tables, const uint16_t* __restrict__ qg_,
                      const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
                      uint16_t* __restrict__ og) {
  constexpr int B = 16, D = 128, NW = kWW, QB = kWQB, KT = kWKT;
  constexpr int KB = KT / B;               // blocks per key tile
  constexpr int NDS = D / 16;              // reduction steps of S
  constexpr int NDB = D / 32;              // 32-row blocks of O^T
  constexpr int NKS = KT / 16;             // 16-key steps of PV
  static_assert(KB == 4 && NW == 4 && QB == 2 && NDS == 8 && NDB == 4 && NKS == 4, "slot layout");
  __shared__ __attribute__((aligned(16))) uint16_t lds[4 * kWBufElems];
  __shared__ __attribute__((aligned(16))) uint32_t idt[kWMaxIdt];

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
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, r = lane & 31, hh = lane >> 5;
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

  // Q rows (lane: Q[row][16*ds + 8*hh .. +7]), requested first; they are
  // scaled and moved to AGPRs after the first tile requests are issued, so
  // the latencies of both overlap.
  u32x4 qraw[QB][NDS];
  bf16x8 qf[QB][NDS];                             // Q^T operands, in AGPRs once filled below
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const uint16_t* qg = qg_ + ((int64_t)(e.q_off + tok[b]) * a.n_q_heads + hq) * D + 8 * hh;
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) qraw[b][ds] = valid[b] ? *(const u32x4*)(qg + 16 * ds) : u32x4{0, 0, 0, 0};
  }

  const int32_t* __restrict__ row = tables + (int64_t)e.seq * a.max_bps;
  const int64_t head_base = (int64_t)a.layer * a.n_blocks * hkv + g;
  const int last_blk = (kv_len - 1) / B;

  // A tile's blocks as byte offsets from block 0 of this layer and head (a
  // 32-bit range: the launcher takes only pools with n_blocks * n_kv_heads *
  // 4 KB < 4 GB); ids past the sequence's last block are clamped to it.
  const uint32_t blk_bytes = (uint32_t)hkv * (B * D * 2);
  auto tile_ids_s = [&](int kt, int (&id)[KB]) {
#pragma unroll
    for (int j = 0; j < KB; ++j)
      id[j] = __builtin_amdgcn_readfirstlane(
          (int)((uint32_t)blk_id(row[min(kt * KB + j, last_blk)], a.n_blocks, a.chk) * blk_bytes));
  };
  // The workgroup's block offsets (blocks kt0 * KB .. last_blk) in LDS, so
  // that the loop takes its block ids with LDS reads (in order with the
  // operand reads) instead of scalar loads (a scalar load in flight turns
  // every LDS wait into a full wait).  Filled before the first barrier.
  // Entries past last_blk repeat it (tiles up to n_kt + 3 are requested).
  const int blk0 = kt0 * KB;
  for (int i = tid; i < (n_kt + 4 - kt0) * KB; i += NW * 64)
    idt[i] = (uint32_t)blk_id(row[min(blk0 + i, last_blk)], a.n_blocks, a.chk) * blk_bytes;
  auto ids_fetch = [&](int kt) { return *(const u32x4*)&idt[(kt - kt0) * KB]; };
  auto ids_use = [&](const u32x4& v, int (&id)[KB]) {
#pragma unroll
    for (int j = 0; j < KB; ++j) id[j] = __builtin_amdgcn_readfirstlane((int)v[j]);
  };
  auto tile_ids = [&](int kt, int (&id)[KB]) { ids_use(ids_fetch(kt), id); };
  const char* kc_h = (const char*)(kc + head_base * (B * D));
  const char* vc_h = (const char*)(vc + head_base * (B * D));
  const uint32_t wofs = (uint32_t)w * 1024;         // byte offset of wave w's run in an image
  const uint32_t lds0 = (uint32_t)(uintptr_t)&lds[0];
  // Wave w writes run w (1 KB) of each block's K and V^T image.  K run w =
  // key rows 4w .. 4w+3; lane l -> row 4w + l / 16, LDS slot l % 16, so it
  // fetches chunk (l % 16) ^ row of that row.  V^T run w = d rows 32w ..
  // 32w+31; lane l -> d row 32w + l % 32, slots 8 (l / 32) .. +7.
  const int krow = w * 4 + (lane >> 4);
  const uint32_t kdma = 2u * (krow * D + ((lane & 15) ^ krow) * 8);
  const uint32_t vdma = 2u * ((w * 32 + (lane & 31)) * B + (lane >> 5) * 8);
  // j: 0..3 K of block j, 4..7 V^T of block j - 4, into the buffer at element buf
  auto request = [&](int buf, const int (&id)[KB], int j) {
    const int blk = j & 3;
    const char* src = (j < 4 ? kc_h : vc_h) + (uint32_t)id[blk];
    const uint32_t img = lds0 + 2u * (buf + (j < 4 ? 0 : 8192) + blk * 2048);
    // the add sets SCC (declared, so that no carry of the compiler's 64-bit
    // address arithmetic is held across it), and a load that reads M0 needs
    // one wait state after an SALU write of M0
    asm volatile("s_add_u32 m0, %2, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(j < 4 ? kdma : vdma), "s"(src), "s"(img), "s"(wofs) : "memory", "m0", "scc");
  };
  auto request_all = [&](int buf, const int (&id)[KB]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) request(buf, id, j);
  };
  // Workgroup barrier once this wave's LDS traffic and all but its latest 8
  // requests (the current step's) have completed.
  auto bar = [&]() { asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  auto buf_of = [&](int x) { return ((x - kt0) & 3) * kWBufElems; };

  f32x16 oacc[QB][NDB];
#pragma unroll
  for (int b = 0; b < QB; ++b)
#pragma unroll
    for (int db = 0; db < NDB; ++db) oacc[b][db] = f32x16{};
  auto oacc_sync = [&](bool long_wait) {
    if (long_wait)
      asm volatile("s_nop 15\n\ts_nop 3"
                   : "+a"(oacc[0][0]), "+a"(oacc[0][1]), "+a"(oacc[0][2]), "+a"(oacc[0][3]),
                     "+a"(oacc[1][0]), "+a"(oacc[1][1]), "+a"(oacc[1][2]), "+a"(oacc[1][3]));
    else
      asm volatile("s_nop 3"
                   : "+a"(oacc[0][0]), "+a"(oacc[0][1]), "+a"(oacc[0][2]), "+a"(oacc[0][3]),
                     "+a"(oacc[1][0]), "+a"(oacc[1][1]), "+a"(oacc[1][2]), "+a"(oacc[1][3]));
  };
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

  // Operand addresses (elements within a buffer).  K operand row i of a
  // 32-key half is key pi(i) (bits 2 and 3 of i swapped): block 2 kh + i / 16,
  // row pi(i) % 16, chunk 2 ds + hh at slot (2 ds + hh) ^ row.  V^T operand
  // (ks, db): block ks, d row 32 db + r, slots 8 hh .. +7 at 8 (r + 32 hh) of
  // group db.
  const int kr = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
  const int krow_r = kr & 15;
  int kaddr[NDS];
#pragma unroll
  for (int ds = 0; ds < NDS; ++ds) kaddr[ds] = (r >> 4) * 2048 + krow_r * 128 + ((2 * ds + hh) ^ krow_r) * 8;
  const int vaddr = (r + 32 * hh) * 8;
  auto k_op = [&](int buf, int kh, int ds) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)&lds[buf + kh * 4096 + kaddr[ds]]);
  };
  auto v_op = [&](int buf, int ks, int db) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)&lds[buf + 8192 + ks * 2048 + db * 512 + vaddr]);
  };
  // S^T products: the first of a chain reads the -m splat and writes a fresh
  // accumulator (early clobber: a product's accumulator and result may not
  // partly overlap); the Q^T operand comes from AGPRs.
  auto mfma_s0 = [](bf16x8 x, bf16x8 y, const f32x16& c) {
    f32x16 d;
    asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=&v"(d) : "v"(x), "a"(y), "v"(c));
    return d;
  };
  auto mfma_s = [](bf16x8 x, bf16x8 y, f32x16& c) {
    asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(x), "a"(y));
  };
  auto s_sync = [](f32x16 (&s)[QB][2]) {
    asm volatile("s_nop 15\n\ts_nop 3" : "+v"(s[0][0]), "+v"(s[0][1]), "+v"(s[1][0]), "+v"(s[1][1]));
  };
  // O^T products, accumulator in AGPRs; mfma_o1 for a P that may have just
  // been written.
  auto mfma_o = [](bf16x8 x, bf16x8 y, f32x16& c) {
    asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(x), "v"(y));
  };
  auto mfma_o1 = [](bf16x8 x, bf16x8& y, f32x16& c) {
    asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %2, %1, %0" : "+a"(c), "+v"(y) : "v"(x));
  };

  // Row max of a tile (log2 units) and the lazy-rescale decision; the wave
  // rescales O when any of its rows moved its reference max.
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
  // The last kWDefer products of O += V(t) P(t) (16-key step 3) are issued
  // after the next step's barrier, so that they keep the matrix pipe busy
  // while the first operands of that step are read from LDS; their V^T
  // operands and P stay in registers until then.  Each accumulator still
  // receives its products in the same order.  Before zero: no pending work.
  constexpr int ND = kWDefer;
  static_assert(ND % 2 == 0 && ND >= 0 && ND <= 8, "deferred products");
  bf16x8 dv[ND > 0 ? ND / 2 : 1];
  u32x4 dp[QB];
#pragma unroll
  for (int k = 0; k < (ND > 0 ? ND / 2 : 1); ++k) dv[k] = bf16x8{};
#pragma unroll
  for (int b = 0; b < QB; ++b) dp[b] = u32x4{0, 0, 0, 0};
  auto deferred = [&](auto kc) {
    constexpr int k = decltype(kc)::value;       // product k of the deferred ones
    constexpr int j = 32 - ND + k, db = (j / 2) % 4, b = j % 2;
    // the first may follow right after VALU writes of dv / dp
    if constexpr (k == 0) asm volatile("s_nop 1");
    mfma_o(dv[k / 2], __builtin_bit_cast(bf16x8, dp[b]), oacc[b][db]);
  };
  auto deferred_all = [&]() {
    if constexpr (ND > 0) static_for(deferred, std::make_integer_sequence<int, ND>{});
  };

  // New reference max per row; when any row of the wave moves it, rescale O
  // (after the deferred products when flush is set; they are then issued
  // here and zeroed, so that the next step adds nothing with them).
  auto apply_max = [&](const float (&mx)[QB], f32x16 (&st)[QB][2], auto flush) {
    bool any = false;
    bool bump[QB];
    float delta[QB], m_old[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      bump[b] = mx[b] > m[b] + kWSlack;
      const float m_new = bump[b] ? mx[b] : m[b];
      const float mu = m_new == -INFINITY ? 0.f : m_new;
      delta[b] = mu - m_use[b];
      m_old[b] = m[b];
      m_use[b] = mu;
      alpha[b] = 1.f;
      m[b] = m_new;
      any = any || bump[b];
    }
    if (__ballot(any)) {
      if constexpr (decltype(flush)::value) deferred_all();
      oacc_sync(true);
      if constexpr (decltype(flush)::value && ND > 0) {
#pragma unroll
        for (int k = 0; k < ND / 2; ++k) dv[k] = bf16x8{};
#pragma unroll
        for (int b = 0; b < QB; ++b) dp[b] = u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        alpha[b] = bump[b] ? __builtin_amdgcn_exp2f(m_old[b] - m_use[b]) : 1.f;
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[b][db] *= alpha[b];
        st[b][0] -= delta[b];
        st[b][1] -= delta[b];
#pragma unroll
        for (int i = 0; i < 16; ++i) cinit[b][i] = -m_use[b];
      }
      oacc_sync(false);
      asm volatile("s_nop 3" : "+v"(cinit[0]), "+v"(cinit[1]));
    }
  };
  auto update_max = [&](f32x16 (&s)[QB][2]) {
    float mx[QB];
    row_max(s, mx);
    apply_max(mx, s, std::false_type{});
  };
  // P for 16 keys (registers o8 .. o8+7 of one 32-key half), rounded to bf16,
  // with the row-sum terms added in the fixed order.
  auto expo = [&](const f32x16& s, int o8, float& ps0, float& ps1) {
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
  auto qk = [&](int tb, f32x16 (&s)[QB][2]) {
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        const bf16x8 kx = k_op(tb, kh, ds);
#pragma unroll
        for (int b = 0; b < QB; ++b) {
          if (ds == 0) s[b][kh] = mfma_s0(kx, qf[b][ds], cinit[b]);
          else mfma_s(kx, qf[b][ds], s[b][kh]);
        }
      }
    s_sync(s);
  };
  // exponentials of a whole tile, then O += V P
  auto pv_tile = [&](int tb, const f32x16 (&sc)[QB][2]) {
    bf16x8 p[QB][NKS];
    float ps0[QB], ps1[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      ps0[b] = 0.f;
      ps1[b] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) p[b][ks] = expo(sc[b][ks / 2], 8 * (ks % 2), ps0[b], ps1[b]);
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 vx = v_op(tb, ks, db);
#pragma unroll
        for (int b = 0; b < QB; ++b) {
          if (db == 0) mfma_o1(vx, p[b][ks], oacc[b][db]);
          else mfma_o(vx, p[b][ks], oacc[b][db]);
        }
      }
#pragma unroll
    for (int b = 0; b < QB; ++b) l[b] = fmaf(l[b], alpha[b], ps0[b] + ps1[b]);
  };

  // ---- prologue: tiles kt0 .. kt0+2 requested, kt0 and kt0+1 landed ---- //
  // Tile x lives in buffer (x - kt0) % 4; the step that works on tile x
  // requests tile x + 3 into the buffer tile x - 1 used.
  int idn[KB];
  {
    int id0[KB], id1[KB], id2[KB];
    tile_ids_s(kt0, id0);
    tile_ids_s(kt0 + 1, id1);
    tile_ids_s(kt0 + 2, id2);
    tile_ids_s(kt0 + 3, idn);
    request_all(buf_of(kt0), id0);
    request_all(buf_of(kt0 + 1), id1);
    request_all(buf_of(kt0 + 2), id2);
  }
  // Q^T operands in AGPRs, Q scaled by scale * log2(e) and rounded once
#pragma unroll
  for (int b = 0; b < QB; ++b)
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) {
      asm volatile("" : "+v"(qraw[b][ds]));     // after the requests above
      f32x8 qx = __builtin_convertvector(__builtin_bit_cast(bf16x8, qraw[b][ds]), f32x8) * a.scale_log2;
      const bf16x8 qv = __builtin_convertvector(qx, bf16x8);
      asm("; Q operand to AGPRs" : "=a"(qf[b][ds]) : "0"(qv));
    }
  asm volatile("s_nop 3"
               : "+a"(qf[0][0]), "+a"(qf[0][1]), "+a"(qf[0][2]), "+a"(qf[0][3]), "+a"(qf[0][4]),
                 "+a"(qf[0][5]), "+a"(qf[0][6]), "+a"(qf[0][7]), "+a"(qf[1][0]), "+a"(qf[1][1]),
                 "+a"(qf[1][2]), "+a"(qf[1][3]), "+a"(qf[1][4]), "+a"(qf[1][5]), "+a"(qf[1][6]),
                 "+a"(qf[1][7]));
  bar();

  f32x16 sa[QB][2], sb[QB][2];
  if (nu > kt0) {
    qk(buf_of(kt0), sa);
    update_max(sa);
  }

  // ---- pipelined steps over unmasked tiles ----------------------------- //
  auto step = [&](int t, const f32x16 (&sc)[QB][2], f32x16 (&sn)[QB][2]) {
    constexpr int kPF = 2;                      // operands read ahead
    constexpr int NU = 32 - ND / 2;             // operands of this step's own products
    bar();
    int ids[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) ids[j] = idn[j];
    const int tk = buf_of(t + 1), tv = buf_of(t), tr = buf_of(t + 3);
    u32x4 pw[QB][NKS];                          // P(t), bf16 pairs
    float ps[QB][2], mxa[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      ps[b][0] = ps[b][1] = 0.f;
      mxa[b] = -INFINITY;
    }
    // operand u (16 K, then the V^T operands of the products issued in this
    // step) feeds the products of slots ND + 2u and ND + 2u + 1
    bf16x8 opnd[NU];
    bf16x8 dvn[ND > 0 ? ND / 2 : 1];            // V^T operands of the products deferred to the next step
    u32x4 idv;                                  // block offsets of tile t + 4
    f32x2 ex[4];                                // exponentials awaiting their rounding
    auto read_op = [&](int u) {
      opnd[u] = u < 16 ? k_op(tk, u % 2, u / 2) : v_op(tv, (u - 16) / 4, (u - 16) % 4);
    };
#pragma unroll
    for (int u = 0; u < kPF - ND / 2; ++u) read_op(u);
    auto slot = [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i < 8) request(tr, ids, i);
      if constexpr (i % 2 == 0) {
        constexpr int u = (i - ND) / 2 + kPF;
        if constexpr (u >= 0 && u < NU) read_op(u);
      }
      if constexpr (ND > 0 && i >= 64 - ND && (i - (64 - ND)) % 2 == 0) {
        constexpr int k = (i - (64 - ND)) / 2, j = 32 - ND + 2 * k;
        dvn[k] = v_op(tv, j / 8, (j / 2) % 4);
      }
      if constexpr (i < ND) {
        deferred(ic);
      } else if constexpr (i < ND + 32) {
        constexpr int q = i - ND, ds = q / 4, kh = (q / 2) % 2, b = q % 2;
        if constexpr (ds == 0) sn[b][kh] = mfma_s0(opnd[q / 2], qf[b][ds], cinit[b]);
        else mfma_s(opnd[q / 2], qf[b][ds], sn[b][kh]);
      } else {
        constexpr int j = i - ND - 32, ks = j / 8, db = (j / 2) % 4, b = j % 2;
        // the last pair of P(t) for (b, ks) was rounded at least 3 slots
        // earlier (item placement below): past the VALU -> matrix wait states
        mfma_o(opnd[16 + j / 2], __builtin_bit_cast(bf16x8, pw[b][ks]), oacc[b][db]);
      }
      if constexpr (i == ND + 33) s_sync(sn);
      if constexpr (i == 40) idv = ids_fetch(t + 4);
      // keep the operand of slots i-3 and i-2 allocated until here, so that
      // no VALU result lands in registers a product may still be reading
      if constexpr (i >= 3) {
        constexpr int pp = i - 3;
        if constexpr (pp < ND) {
          if constexpr (pp % 2 == 0) asm volatile("" ::"v"(dv[pp / 2]));
        } else if constexpr ((pp - ND) % 2 == 0) {
          asm volatile("" ::"v"(opnd[(pp - ND) / 2]));
        }
      }
      // key pairs of P(t): item w = (ks, m, b) in ks-major order; its two
      // exponentials at slot floor(52 w / 32), their bf16 rounding two slots
      // later, so p[b][ks] is complete three slots before its first product
      constexpr int we = (32 * i + 51) / 52;
      if constexpr (we < 32 && (we * 52) / 32 == i) {
        constexpr int ks = we / 8, mm = (we / 2) % 4, b = we % 2;
        constexpr int o = 8 * (ks % 2) + 2 * mm;
        ex[we % 4] = f32x2{__builtin_amdgcn_exp2f(sc[b][ks / 2][o]), __builtin_amdgcn_exp2f(sc[b][ks / 2][o + 1])};
      }
      constexpr int wc = (32 * (i - 2) + 51) / 52;
      if constexpr (i >= 2 && wc < 32 && (wc * 52) / 32 == i - 2) {
        constexpr int ks = wc / 8, mm = (wc / 2) % 4, b = wc % 2;
        pw[b][ks][mm] = __builtin_bit_cast(uint32_t, __builtin_convertvector(ex[wc % 4], bf16x2));
      }
      // row max of S(t+1): 32 v_max3 items spread over the slots after its
      // last product and the wait for its results, as inline assembly (S
      // comes from inline assembly, so fmaxf would first quiet every input)
      constexpr int MB = ND + 34, MS = 64 - MB;
      if constexpr (i >= MB) {
        constexpr int w0 = (32 * (i - MB) + MS - 1) / MS;
        if constexpr (w0 < 32 && MB + (w0 * MS) / 32 == i) {
          constexpr int b = w0 % 2, q = w0 / 2, kh = q / 8, o = 2 * (q % 8);
          asm("v_max3_f32 %0, %0, %1, %2" : "+v"(mxa[b]) : "v"(sn[b][kh][o]), "v"(sn[b][kh][o + 1]));
        }
        constexpr int w1 = w0 + 1;
        if constexpr (w1 < 32 && MB + (w1 * MS) / 32 == i) {
          constexpr int b = w1 % 2, q = w1 / 2, kh = q / 8, o = 2 * (q % 8);
          asm("v_max3_f32 %0, %0, %1, %2" : "+v"(mxa[b]) : "v"(sn[b][kh][o]), "v"(sn[b][kh][o + 1]));
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for(slot, std::make_integer_sequence<int, 64>{});
    ids_use(idv, idn);
    // row-sum terms of P(t) in the fixed order (per row block: ks, then the
    // 4 pairs alternating between two partial sums)
#pragma unroll
    for (int w2 = 0; w2 < 32; ++w2) {
      const int ks = w2 / 8, mm = (w2 / 2) % 4, b = w2 % 2;
      // through a scalar: this compiler's bit cast of a vector element
      // lvalue reads element 0
      const uint32_t pair = pw[b][ks][mm];
      ps[b][mm % 2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), kOnes, ps[b][mm % 2], false);
    }
    float mx[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      mx[b] = fmaxf(mxa[b], xor32(mxa[b])) + m_use[b];
      l[b] = fmaf(l[b], alpha[b], ps[b][0] + ps[b][1]);
      // keep this step's row sum in this step (the compiler would otherwise
      // sink both unrolled steps' sums to the loop's end)
      asm volatile("" ::"v"(l[b]));
    }
    if constexpr (ND > 0) {
#pragma unroll
      for (int k = 0; k < ND / 2; ++k) dv[k] = dvn[k];
#pragma unroll
      for (int b = 0; b < QB; ++b) dp[b] = pw[b][NKS - 1];
    }
    apply_max(mx, sn, std::true_type{});
  };
  // Request tile x + 3 with the ids taken a step ago, take the next ids.
  auto advance = [&](int x) {
    int ids[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) ids[j] = idn[j];
    request_all(buf_of(x + 3), ids);
    tile_ids(x + 4, idn);
  };
  // Tile t's S is computed and its max taken: finish it unpipelined.
  auto finish = [&](int t, const f32x16 (&sc)[QB][2]) {
    bar();
    advance(t);
    deferred_all();
    pv_tile(buf_of(t), sc);
  };
  // A tile on the diagonal: S, causal mask by select, max, then P V.
  auto diag = [&](int u) {
    bar();
    advance(u);
    const int tb = buf_of(u);
    const int kb = u * KT;
    if (kb + KT > kv_len) {
      // V^T slots at or past kv_len must read as 0 (P is 0 there; a stale or
      // poisoned slot need not be finite): 1024 runs of 8 slots, 4 per thread
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = tid + 256 * j, blk = c >> 8, d = (c & 255) >> 1, half = c & 1;
        const int key0 = blk * B + half * 8;
        if (kb + key0 + 8 > kv_len) {
          u32x4* p = (u32x4*)&lds[tb + 8192 + blk * 2048 + (d >> 5) * 512 + ((d & 31) + 32 * half) * 8];
          *p = zero_tail(*p, kb + key0, kv_len);
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    qk(tb, sa);
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
    pv_tile(tb, sa);
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
  for (int u = nu; u < n_kt; ++u) diag(u);
  // requests past the last tile land in buffers nobody reads; they must
  // complete before the workgroup ends and its LDS is handed on
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // ---- epilogue: normalise and store (or write split partials) --------- //
  oacc_sync(true);
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

bool attn_bf16_wide_eligible(int head_dim, int group, int block_size, int64_t n_blocks, int n_kv_heads,
                             int64_t max_kv_len) {
  // a workgroup's LDS block table holds (key tiles + 4) * 4 entries
  if ((max_kv_len + kWKT - 1) / kWKT + 4 > kWMaxIdt / 4) return false;
  return head_dim == 128 && block_size == 16 && group >= 1 && group <= 32 && 32 % group == 0 &&
         n_blocks * n_kv_heads * 4096 <= ((int64_t)1 << 32);
}

hipError_t launch_attn_bf16_wide(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  const int group = a.n_q_heads / a.n_kv_heads;
  int64_t max_kv = 0;
  for (int i = 0; i < a.n; ++i) max_kv = max(max_kv, (int64_t)a.e[i].prefix + a.e[i].q_len);
  if (!attn_bf16_wide_eligible(a.head_dim, group, a.block_size, a.n_blocks, a.n_kv_heads, max_kv))
    return hipErrorInvalidValue;
  const dim3 grid(a.n_tiles * a.n_kv_heads * a.n_splits), blk(kWW * 64);
  hipLaunchKernelGGL(attn_bf16_wide_kernel, grid, blk, 0, s, a, a.tables, (const uint16_t*)a.q,
                     (const uint16_t*)a.k_cache, (const uint16_t*)a.v_cache, (uint16_t*)a.o);
  return hipGetLastError();
}

}  // namespace pgsr
