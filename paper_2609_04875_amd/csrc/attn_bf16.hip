// bf16 prefix + causal prefill attention on CDNA4 matrix cores (gfx950).
//
// Work decomposition.  A workgroup of NW wave64s owns one KV head g and a tile
// of TW = NW*32/G consecutive suffix tokens together with the G query heads
// that share g (GQA packing: every query row of the workgroup reads the same
// K/V tiles).  Each wave owns 32 query rows (token, head).  blockIdx.x =
// tile * n_kv_heads + g, so with 8 KV heads all tiles of one head land on the
// same XCD (workgroups are dealt to the 8 XCDs round-robin) and share that
// XCD's L2 copy of the head's keys and values.  Tiles are issued costliest
// first (sequences sorted by work on the host, tiles within a sequence from
// the last, longest-context one down).  Two workgroups share a CU.
//
// Per key tile (KT = 64 keys at absolute positions kb .. kb+63):
//   * K and V^T are gathered through the block table from HBM into registers
//     one tile ahead (block ids two tiles ahead), then stored to a
//     double-buffered LDS tile: one barrier per tile.  Every load is
//     unconditional (block index clamped to the sequence's last block); V
//     entries of keys at or past the sequence length are zeroed before the
//     LDS store, and such keys are masked out of S, so stale or NaN slots never
//     reach the result.
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = Q^T
//     held in registers for the whole kernel).  In the 32x32 accumulator a lane
//     holds one query column and 16 keys, so the row max and row sum are
//     in-lane reductions plus one exchange between the two 32-lane halves.
//     Operand reads are issued several MFMAs ahead of use.
//   * Online softmax in the base-2 domain (log2(e) folded into the scale);
//     the causal mask is a select to -inf on diagonal tiles only.  A row keeps
//     its running maximum until a tile exceeds it by more than 2^8 (weights
//     then stay below 256, harmless in fp32 / bf16), so the O rescale is rare;
//     when any row of the wave needs it the wave rescales (alpha = 1 exactly
//     for the others).  The row sum adds the bf16-rounded P values that enter
//     the PV product (v_dot2_f32_bf16 against ones).
//   * O^T += V^T P^T with the same MFMA (A = V^T rows from LDS, B = P^T taken
//     straight from the S^T registers after rounding to bf16).  The reduction
//     index of a B operand must match the A operand's.  In the 32x32
//     accumulator, lane half h holds rows {8a + 4h + c} (a = 0..3, c = 0..3);
//     the K operand therefore reads, for accumulator row i, key pi(i), where pi
//     swaps bits 2 and 3 of i.  Then lane half h holds keys 8h..8h+7 of each
//     16-key group in order, and the matching V^T operand is 8 consecutive keys
//     of one d row: V^T sits in LDS in natural key order and every operand is
//     one 16-byte read.
// LDS rows are padded by 16 bytes (K: D+8 elements, V^T: 72), which spreads
// the 32 rows one MFMA operand read touches over distinct bank groups and keeps
// every operand address a base plus an immediate offset.
//
// FP8 cache (E4M3 codes): the tile loads fetch 8 bytes where the bf16 path
// fetches 16, and the codes widen to bf16 exactly (every E4M3 value has at
// most 4 significant bits) before the LDS store, so everything after the store
// is the bf16 kernel.  The K scale rides in the softmax scale, the V scale in
// the output normalisation.
//
// Key tiles sit at absolute positions and rows never interact, so a query's
// output bits depend only on its absolute position and its own keys: selective
// replay and full reset agree bitwise, and repeated runs are bitwise identical.
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "attn_common.h"
#include "internal.h"

namespace pgsr {

namespace {

constexpr int kNW = 4;      // waves per workgroup
constexpr int kKT = 64;     // keys per tile
constexpr int kAhead = 3;   // LDS operand reads issued this many MFMAs ahead
constexpr float kSlack = 8.f;   // lazy rescale threshold, log2 units

// Block ids of one key tile (up to four blocks), indexed with a wave-uniform
// value through selects rather than as an array, which would live in memory.
struct Ids {
  int32_t v0, v1, v2, v3;
  __device__ int32_t get(int i) const { return i == 0 ? v0 : i == 1 ? v1 : i == 2 ? v2 : v3; }
};

template <int D, int NW, int B, bool F8>
__global__ void __launch_bounds__(NW * 64, 2)
attn_bf16_kernel(AttnArgs a, const int32_t* __restrict__ tables, const uint16_t* __restrict__ qg_,
                 const std::conditional_t<F8, uint8_t, uint16_t>* __restrict__ kc,
                 const std::conditional_t<F8, uint8_t, uint16_t>* __restrict__ vc,
                 uint16_t* __restrict__ og) {
  using Raw = std::conditional_t<F8, u32x2, u32x4>;   // 8 cache elements
  constexpr int KT = kKT;
  constexpr int KB = KT / B;               // blocks per key tile
  constexpr int KLD = D + 8;               // LDS row stride of the K tile (elements)
  constexpr int VLD = KT + 8;              // LDS row stride of the V^T tile (elements)
  constexpr int NT = NW * 64;
  constexpr int CHB = B * D / 8;           // 16-byte chunks per block-head (K or V)
  constexpr int CPT = KT * D / 8 / NT;     // chunks per thread per tile (K or V)
  static_assert(CPT * NT * 8 == KT * D, "tile split");
  static_assert(KB >= 1 && KB <= 4, "block size 16, 32 or 64");
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][KT * KLD];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][D * VLD];

  const int hkv = a.n_kv_heads;
  const int g = blockIdx.x % hkv;
  const int split = (blockIdx.x / hkv) % a.n_splits;
  const int tile = blockIdx.x / hkv / a.n_splits;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].tile_start <= tile) ++ei;
  const AttnEntry e = a.e[ei];
  const int G = a.n_q_heads / hkv;
  // A wave holds TPW = floor(32 / G) tokens x G heads; when G does not divide
  // 32 (e.g. 7) its last 32 - TPW * G rows are padding and never written.
  const int TPW = 32 / G;
  const int TW = NW * TPW;                          // tokens per tile
  const int n_tiles_e = (e.q_len + TW - 1) / TW;
  const int lt = n_tiles_e - 1 - (tile - e.tile_start);
  const int t0 = lt * TW;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, r = lane & 31, hh = lane >> 5;
  const int tok = t0 + w * TPW + r / G;
  const int hq = g * G + r % G;
  const bool valid = r < TPW * G && tok < e.q_len;
  // A wave whose 32 rows all lie past the tile's last query (a decode step or
  // a ragged last tile) still loads and stores its share of every tile but
  // skips the products.
  const bool wave_active = __ballot(valid) != 0;
  const int qpos = valid ? e.prefix + tok : -1;
  const int t_last = min(e.q_len, t0 + TW) - 1;
  const int kv_len = e.prefix + e.q_len;
  const int first_q = e.prefix + t0;               // smallest query position here
  // Keys this workgroup visits: [key_lo, key_end), whole tiles at absolute
  // positions (a split boundary is a multiple of the tile size).
  const int key_lo = split * a.split_len;
  const int key_end = min(e.prefix + t_last + 1, a.n_splits > 1 ? key_lo + a.split_len : INT32_MAX);
  if (key_lo >= key_end) return;                   // nothing of this tile in this split
  const int kt0 = key_lo / KT;
  const int n_kt = (key_end + KT - 1) / KT;

  // Q^T operand: lane holds Q[row][16*ds + 8*hh .. +7] for each ds.
  bf16x8 qb[D / 16];
  {
    const uint16_t* qg = qg_ + ((int64_t)(e.q_off + tok) * a.n_q_heads + hq) * D + 8 * hh;
#pragma unroll
    for (int ds = 0; ds < D / 16; ++ds) {
      u32x4 raw = valid ? *(const u32x4*)(qg + 16 * ds) : u32x4{0, 0, 0, 0};
      const f32x8 qx = __builtin_convertvector(__builtin_bit_cast(bf16x8, raw), f32x8) * a.scale_log2;
      qb[ds] = __builtin_convertvector(qx, bf16x8);   // Q scaled by the softmax scale * log2(e), rounded once
    }
  }

  const int32_t* __restrict__ row = tables + (int64_t)e.seq * a.max_bps;
  const int64_t head_base = (int64_t)a.layer * a.n_blocks * hkv + g;  // + id * hkv
  const int last_blk = (kv_len - 1) / B;   // blocks past it are clamped to it

  // Tile chunking.  A tile is KB block-heads of CHB 16-byte chunks each (K:
  // (slot, 8 columns); V^T: (d, 8 slots)); thread tid takes chunks
  // tid + i * NT.  When a block-head has at least NT chunks the block of chunk
  // i is a compile-time constant, otherwise it depends on tid.
  constexpr bool kBlkConst = CHB % NT == 0;
  auto chunk_blk = [&](int i) {
    if constexpr (kBlkConst) return i / (CHB / NT);
    else return i * (NT / CHB) + tid / CHB;
  };
  auto chunk_in = [&](int i) {
    if constexpr (kBlkConst) return tid + (i % (CHB / NT)) * NT;
    else return tid % CHB;
  };

  // Block ids of a key tile, clamped in range.  They are fetched as a
  // per-lane vector load (lane bi holds block bi's id) one tile before use,
  // issued ahead of that tile's data loads so waiting for the data implies
  // they have arrived, then broadcast to scalar registers with readlane.
  int idv = 0;
  auto fetch_ids = [&](int kt) {
    idv = blk_id(row[min(kt * KB + (lane < KB ? lane : 0), last_blk)], a.n_blocks, a.chk);
  };
  auto take_ids = [&]() {
    Ids ids;
    ids.v0 = __builtin_amdgcn_readlane(idv, 0);
    ids.v1 = KB > 1 ? __builtin_amdgcn_readlane(idv, 1) : 0;
    ids.v2 = KB > 2 ? __builtin_amdgcn_readlane(idv, 2) : 0;
    ids.v3 = KB > 3 ? __builtin_amdgcn_readlane(idv, 3) : 0;
    return ids;
  };

  Raw kreg[CPT], vreg[CPT];
  auto load_tile = [&](const Ids& ids) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int in = chunk_in(i);
      const int64_t base = (head_base + (int64_t)ids.get(chunk_blk(i)) * hkv) * (B * D);
      kreg[i] = *(const Raw*)(kc + base + (in / (D / 8)) * D + (in % (D / 8)) * 8);
      vreg[i] = *(const Raw*)(vc + base + (in / (B / 8)) * B + (in % (B / 8)) * 8);
    }
  };
  auto as_bf16 = [](const Raw& x) {
    if constexpr (F8) return widen_fp8(x);
    else return x;
  };
  auto store_tile = [&](int buf, int kb) {
    const bool tail = kb + KT > kv_len;   // V slots at or past kv_len must read as 0
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int blk = chunk_blk(i), in = chunk_in(i);
      *(u32x4*)&k_lds[buf][(blk * B + in / (D / 8)) * KLD + (in % (D / 8)) * 8] = as_bf16(kreg[i]);
      const int dd = in / (B / 8), key0 = blk * B + (in % (B / 8)) * 8;
      u32x4 val = as_bf16(vreg[i]);
      if (tail) {
        const int pos0 = kb + key0;
        if (pos0 >= kv_len) val = u32x4{0, 0, 0, 0};
        else if (pos0 + 8 > kv_len) val = zero_tail(val, pos0, kv_len);
      }
      *(u32x4*)&v_lds[buf][dd * VLD + key0] = val;
    }
  };

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db) oacc[db] = f32x16{};
  // S^T accumulators start at -m_use, so they hold s * c - m_use and the
  // exponentials need no subtraction; m_use moves only with the lazy
  // rescale, when the tile just computed is shifted by the same amount.
  float m = -INFINITY, l = 0.f, m_use = 0.f;

  // S^T = K Q^T for one 64-key tile: two independent 32-key accumulators.
  auto qk = [&](int buf, f32x16 (&s)[2]) {
#pragma unroll
    for (int i = 0; i < 16; ++i) s[0][i] = s[1][i] = -m_use;
    const int kr = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);   // pi(r): bits 2 and 3 swapped
    const uint16_t* kp = &k_lds[buf][kr * KLD + 8 * hh];
    constexpr int N = D / 16;
    bf16x8 k0[N], k1[N];
#pragma unroll
    for (int ds = 0; ds < N; ++ds) {
      k0[ds] = __builtin_bit_cast(bf16x8, *(const u32x4*)(kp + 16 * ds));
      k1[ds] = __builtin_bit_cast(bf16x8, *(const u32x4*)(kp + 32 * KLD + 16 * ds));
    }
#pragma unroll
    for (int ds = 0; ds < N; ++ds) {
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0[ds], qb[ds], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1[ds], qb[ds], s[1], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * kAhead, 1);   // DS reads
#pragma unroll
    for (int ds = 0; ds < N; ++ds) {
      if (ds + kAhead < N) __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);          // MFMAs
    }
  };
  // V^T operands of one tile.  The first NVE are read right after the S
  // products are issued, so their LDS latency overlaps the softmax and the PV
  // products can start as soon as each 16-key slice of P is ready; the rest
  // (where registers are short) are read with the PV products.
  constexpr int NV = KT / 16 * (D / 32);
  constexpr int NVE = (D == 128 && B > 16) ? 8 : NV;   // wider blocks need more address registers
  auto read_v = [&](int buf, bf16x8 (&va)[NV], int lo, int hi) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (i >= lo && i < hi)
        va[i] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)&v_lds[buf][((i % (D / 32)) * 32 + r) * VLD +
                                                (i / (D / 32)) * 16 + 8 * hh]);
  };
  // O^T += V^T P^T for one tile: 16 keys per step.
  auto pv = [&](int buf, bf16x8 (&va)[NV], const bf16x8 (&pb)[KT / 16]) {
    read_v(buf, va, NVE, NV);
#pragma unroll
    for (int ks = 0; ks < KT / 16; ++ks)
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[ks * (D / 32) + db], pb[ks],
                                                           oacc[db], 0, 0, 0);
  };

  // Prologue: tile kt0 in registers, ids of the next taken, the one after in
  // flight.
  Ids ids_n{};
  {
    fetch_ids(kt0);
    const Ids ids0 = take_ids();
    if (kt0 + 1 < n_kt) fetch_ids(kt0 + 1);
    load_tile(ids0);
    if (kt0 + 1 < n_kt) ids_n = take_ids();
    if (kt0 + 2 < n_kt) fetch_ids(kt0 + 2);
  }
  // One step per key tile.  LDS buffer kt&1 receives tile kt before the
  // barrier; it was last read two steps earlier, one barrier before.
  for (int kt = kt0; kt < n_kt; ++kt) {
    const int kb = kt * KT, buf = kt & 1;
    store_tile(buf, kb);
    __syncthreads();
    if (kt + 1 < n_kt) {
      const Ids ids = ids_n;                       // tile kt+1
      if (kt + 2 < n_kt) ids_n = take_ids();       // tile kt+2, fetched a step ago
      if (kt + 3 < n_kt) fetch_ids(kt + 3);
      load_tile(ids);
    }
    if (!wave_active) continue;
    f32x16 s[2];
    qk(buf, s);
    bf16x8 va[NV];
    read_v(buf, va, 0, NVE);
    // Causal mask (select) where some key may lie past some row's position.
    if (kb + KT - 1 > first_q) {
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb + kh * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
          s[kh][i] = key > qpos ? -INFINITY : s[kh][i];
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kh][i]);
    mx = fmaxf(mx, xor32(mx)) + m_use;             // tile max of the row, log2 units
    const bool bump = mx > m + kSlack;             // first tile: m = -inf
    const float m_new = bump ? mx : m;
    const float mu = m_new == -INFINITY ? 0.f : m_new;
    const float delta = mu - m_use;                // 0 unless this row moved its max
    m_use = mu;
    const float alpha = bump ? __builtin_amdgcn_exp2f(m - m_use) : 1.f;
    m = m_new;
    if (__ballot(bump)) {
      s[0] -= delta;
      s[1] -= delta;
    }
    // P = exp2(s*c - m) rounded to bf16; the row sum adds exactly those values.
    bf16x8 pb[KT / 16];
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int ks = 0; ks < KT / 16; ++ks) {
      const int kh = ks >> 1, o8 = (ks & 1) * 8;
      f32x8 pv8;
#pragma unroll
      for (int j = 0; j < 8; ++j) pv8[j] = __builtin_amdgcn_exp2f(s[kh][o8 + j]);
      pb[ks] = __builtin_convertvector(pv8, bf16x8);
      const bf16x2* p2 = (const bf16x2*)&pb[ks];
      ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[0], kOnes, ps0, false);
      ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[1], kOnes, ps1, false);
      ps0 = __builtin_amdgcn_fdot2_f32_bf16(p2[2], kOnes, ps0, false);
      ps1 = __builtin_amdgcn_fdot2_f32_bf16(p2[3], kOnes, ps1, false);
    }
    l = fmaf(l, alpha, ps0 + ps1);
    if (__ballot(bump)) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db) oacc[db] *= alpha;
    }
    pv(buf, va, pb);
  }

  const float l_tot = l + xor32(l);
  if (valid && a.n_splits > 1) {                   // unnormalised partials, fp32
    const int64_t prow = (int64_t)split * a.n_rows + (int64_t)(e.q_off + tok) * a.n_q_heads + hq;
    float* acc = a.ws_acc + prow * D + 4 * hh;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4)
        *(f32x4*)(acc + db * 32 + 8 * i4) =
            f32x4{oacc[db][4 * i4 + 0], oacc[db][4 * i4 + 1], oacc[db][4 * i4 + 2],
                  oacc[db][4 * i4 + 3]};
    if (hh == 0) *(f32x2*)(a.ws_ml + 2 * prow) = f32x2{m, l_tot};
  } else if (valid) {
    const float inv = a.o_scale / l_tot;
    uint16_t* op = og + ((int64_t)(e.q_off + tok) * a.n_q_heads + hq) * D + 4 * hh;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        f32x4 v4 = {oacc[db][4 * i4 + 0] * inv, oacc[db][4 * i4 + 1] * inv,
                    oacc[db][4 * i4 + 2] * inv, oacc[db][4 * i4 + 3] * inv};
        *(bf16x4*)(op + db * 32 + 8 * i4) = __builtin_convertvector(v4, bf16x4);
      }
  }
}

// Split-key combine: for query row r with position p, the splits s with
// s * split_len <= p hold partials (m_s, l_s, acc_s); splits starting past p
// saw no visible key and may hold stale data, so they are skipped.
//   M = max m_s,  w_s = 2^(m_s - M),  o = sum_s w_s acc_s / sum_s w_s l_s,
// summed in increasing s.  16 threads per row, 8 columns each.  The partials
// are read kGroup splits at a time, all loads of a group issued before any is
// used, so a row with many splits (a decode step) waits on few round trips;
// the sums still run in increasing s.
constexpr int kGroup = 8;

template <int D, typename TO>
__global__ void __launch_bounds__(256) split_combine_kernel(AttnArgs a, TO* __restrict__ og) {
  constexpr int TPR = D / 8;                       // threads per row
  const int64_t row = a.row_begin + (int64_t)blockIdx.x * (blockDim.x / TPR) + threadIdx.x / TPR;
  const int c0 = (threadIdx.x % TPR) * 8;
  if (row >= a.row_end) return;
  const int tok = (int)(row / a.n_q_heads);        // packed query token
  int ei = -1;                                     // entries are not sorted by q_off
  for (int i = 0; i < a.n; ++i)
    if (tok >= a.e[i].q_off && tok < a.e[i].q_off + a.e[i].q_len) ei = i;
  if (ei < 0) return;                              // a row of no entry of this launch
  const AttnEntry e = a.e[ei];
  const int qpos = e.prefix + (tok - e.q_off);
  const int ns = min(a.n_splits, qpos / a.split_len + 1);
  const float* __restrict__ ml = a.ws_ml;
  const float* __restrict__ acc = a.ws_acc;
  // Indices past the last split are clamped to it (always a valid address)
  // and weighted 0, so each group's loads are unconditional and issue together.
  float M = -INFINITY;
  float L = 0.f;
  f32x4 o0 = {0, 0, 0, 0}, o1 = {0, 0, 0, 0};
  if (ns <= kGroup) {
    // one group (every decode call): all loads in one round trip, then the
    // same max, weights and sums in the same order as the general loop below
    float mg[kGroup], lg[kGroup];
    f32x4 a0[kGroup], a1[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int64_t prow = (int64_t)min(j, ns - 1) * a.n_rows + row;
      mg[j] = ml[2 * prow];
      lg[j] = ml[2 * prow + 1];
      a0[j] = *(const f32x4*)(acc + prow * D + c0);
      a1[j] = *(const f32x4*)(acc + prow * D + c0 + 4);
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) M = fmaxf(M, mg[j]);
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const float wgt = j < ns ? __builtin_amdgcn_exp2f(mg[j] - M) : 0.f;
      L = fmaf(wgt, lg[j], L);
      o0 += wgt * a0[j];
      o1 += wgt * a1[j];
    }
  }
  for (int s0 = 0; s0 < ns && ns > kGroup; s0 += kGroup) {
    float mg[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
      mg[j] = ml[2 * ((int64_t)min(s0 + j, ns - 1) * a.n_rows + row)];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) M = fmaxf(M, mg[j]);
  }
  for (int s0 = 0; s0 < ns && ns > kGroup; s0 += kGroup) {
    float mg[kGroup], lg[kGroup];
    f32x4 a0[kGroup], a1[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int64_t prow = (int64_t)min(s0 + j, ns - 1) * a.n_rows + row;
      mg[j] = ml[2 * prow];
      lg[j] = ml[2 * prow + 1];
      a0[j] = *(const f32x4*)(acc + prow * D + c0);
      a1[j] = *(const f32x4*)(acc + prow * D + c0 + 4);
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const float wgt = s0 + j < ns ? __builtin_amdgcn_exp2f(mg[j] - M) : 0.f;
      L = fmaf(wgt, lg[j], L);
      o0 += wgt * a0[j];
      o1 += wgt * a1[j];
    }
  }
  const float inv = a.o_scale / L;
  if constexpr (std::is_same_v<TO, float>) {       // fp32 pools
    *(f32x4*)(og + row * D + c0) = o0 * inv;
    *(f32x4*)(og + row * D + c0 + 4) = o1 * inv;
  } else {
    bf16x8 out;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[j] = (__bf16)(o0[j] * inv);
      out[4 + j] = (__bf16)(o1[j] * inv);
    }
    *(bf16x8*)(og + row * D + c0) = out;
  }
}

}  // namespace

int attn_bf16_tile_tokens(int, int group) { return kNW * (32 / group); }

template <int D, int B, bool F8>
static void launch_d_b(const AttnArgs& a, hipStream_t s) {
  using CT = std::conditional_t<F8, uint8_t, uint16_t>;
  dim3 grid(a.n_tiles * a.n_kv_heads * a.n_splits);
  hipLaunchKernelGGL((attn_bf16_kernel<D, kNW, B, F8>), grid, dim3(kNW * 64), 0, s, a, a.tables,
                     (const uint16_t*)a.q, (const CT*)a.k_cache, (const CT*)a.v_cache,
                     (uint16_t*)a.o);
}

template <int D, bool F8>
static hipError_t launch_d(const AttnArgs& a, hipStream_t s) {
  switch (a.block_size) {
    case 16: launch_d_b<D, 16, F8>(a, s); break;
    case 32: launch_d_b<D, 32, F8>(a, s); break;
    case 64: launch_d_b<D, 64, F8>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_split_combine(const AttnArgs& a, bool f32_out, hipStream_t s) {
  if (a.row_begin < 0 || a.row_end > a.n_rows) return hipErrorInvalidValue;
  if (a.row_end <= a.row_begin) return hipSuccess;
  // 256 threads per block, or 64 when that would leave CUs idle (decode
  // calls have a few thousand rows)
  const int64_t rows = a.row_end - a.row_begin;
  const int tpr = a.head_dim / 8;
  const int threads = (rows + 256 / tpr - 1) / (256 / tpr) >= 1024 ? 256 : 64;
  const int rows_per_block = threads / tpr;
  dim3 grid((rows + rows_per_block - 1) / rows_per_block);
  if (a.head_dim == 128 && f32_out)
    hipLaunchKernelGGL((split_combine_kernel<128, float>), grid, dim3(threads), 0, s, a, (float*)a.o);
  else if (a.head_dim == 64 && f32_out)
    hipLaunchKernelGGL((split_combine_kernel<64, float>), grid, dim3(threads), 0, s, a, (float*)a.o);
  else if (a.head_dim == 128)
    hipLaunchKernelGGL((split_combine_kernel<128, uint16_t>), grid, dim3(threads), 0, s, a, (uint16_t*)a.o);
  else if (a.head_dim == 64)
    hipLaunchKernelGGL((split_combine_kernel<64, uint16_t>), grid, dim3(threads), 0, s, a, (uint16_t*)a.o);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  if (a.head_dim == 128) return launch_d<128, false>(a, s);
  if (a.head_dim == 64) return launch_d<64, false>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_attn_fp8(const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.n_tiles <= 0) return hipSuccess;
  if (a.head_dim == 128) return launch_d<128, true>(a, s);
  if (a.head_dim == 64) return launch_d<64, true>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace pgsr
