// Paged KV pool kernels: initial state, restore-by-crop (block-table truncation
// and compaction of the released ids onto the free-list stack), NaN poisoning
// of released slots, copy-on-write fork, and the reserve + append step of a
// replay.  Every block carries a count of the table entries that name it: a
// crop pushes a block only when its count reaches 0, and an append that would
// write into a shared partial tail block first copies it into a private one.
//
// All of this is integer bookkeeping and bit copies (an FP8 cache adds a
// rounding to E4M3 defined bit for bit): results are exact and do not depend
// on the launch shape.  Work per call is tiny (a crop touches at
// most a few KB of int32), so these kernels are launch-latency bound; they are
// written for clarity and coalescing, not occupancy.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace pgsr {

namespace {

__global__ void __launch_bounds__(256)
pool_init_kernel(int32_t* tables, int64_t n_table, int32_t* lens, int32_t max_seqs,
                 int32_t* free_list, int32_t n_blocks, int32_t* free_top, int32_t* refs) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_table; i += stride)
    tables[i] = -1;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < max_seqs; i += stride)
    lens[i] = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_blocks; i += stride) {
    refs[i] = 0;
    if (free_list)  // default stack: bottom n_blocks-1 ... top 0, so pops yield 0, 1, 2, ...
      free_list[i] = n_blocks - 1 - (int32_t)i;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *free_top = n_blocks;
}

// One workgroup takes the entries in call order (a block named by two of the
// cropped rows must reach 0 in the later one).  Within a row the released
// entries j = keep .. nalloc-1 name distinct blocks, so 256 of them are
// decremented at once; those reaching 0 are pushed in ascending j through a
// prefix count over the workgroup.
__global__ void __launch_bounds__(256) crop_kernel(CropArgs a) {
  __shared__ int32_t wave_cnt[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int32_t top = a.top_before;
  for (int i = 0; i < a.n; ++i) {
    const CropEntry e = a.e[i];
    int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
    for (int32_t j0 = e.keep; j0 < e.nalloc; j0 += 256) {
      const int32_t j = j0 + (int32_t)threadIdx.x;
      bool freed = false;
      int32_t b = -1;
      if (j < e.nalloc) {
        b = blk_id(row[j], a.n_blocks, a.chk);
        row[j] = -1;
        const int32_t r = a.refs[b] - 1;
        a.refs[b] = r;
        freed = r == 0;
      }
      const uint64_t m = __ballot(freed);
      if (lane == 0) wave_cnt[w] = __popcll(m);
      __syncthreads();
      int32_t before = __popcll(m & ((1ull << lane) - 1ull));
      for (int ww = 0; ww < w; ++ww) before += wave_cnt[ww];
      const int32_t total = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
      if (freed) a.free_list[top + before] = b;
      top += total;
      __syncthreads();   // wave_cnt is reused; count writes precede the next row's reads
    }
    if (threadIdx.x == 0) a.lens[e.seq] = e.new_len;
  }
  if (threadIdx.x == 0) *a.free_top = top;
}

// One workgroup per pair: dst (empty) takes src's row and length; every shared
// block's count grows by 1 (atomics: several pairs may share a source).
__global__ void __launch_bounds__(256) fork_kernel(ForkArgs a) {
  const ForkEntry e = a.e[blockIdx.x];
  const int32_t* src = a.tables + (int64_t)e.src * a.max_bps;
  int32_t* dst = a.tables + (int64_t)e.dst * a.max_bps;
  for (int32_t j = threadIdx.x; j < e.nalloc; j += blockDim.x) {
    const int32_t b = blk_id(src[j], a.n_blocks, a.chk);
    dst[j] = b;
    atomicAdd(&a.refs[b], 1);
  }
  if (threadIdx.x == 0) a.lens[e.dst] = e.len;
}

template <typename T>
__device__ void fill_nan(T* p, int64_t n, T nan, int tid, int nthreads) {
  for (int64_t i = tid; i < n; i += nthreads) p[i] = nan;
}

// blockIdx.x < n_freed: a pushed block; above: a cropped entry's tail slots
// (private kept partial blocks only).  blockIdx.y: layer.  Runs after
// crop_kernel on the same stream.
template <typename T>
__global__ void __launch_bounds__(256) poison_kernel(PoisonArgs a, T nan) {
  const int layer = blockIdx.y;
  const int64_t blk_elems = (int64_t)a.n_kv_heads * a.block_size * a.head_dim;
  T* kc = (T*)a.k_cache + (int64_t)layer * a.n_blocks * blk_elems;
  T* vc = (T*)a.v_cache + (int64_t)layer * a.n_blocks * blk_elems;
  if ((int)blockIdx.x < a.n_freed) {
    const int32_t id = blk_id(a.free_list[a.top_before + blockIdx.x], a.n_blocks, a.chk);
    fill_nan(kc + (int64_t)id * blk_elems, blk_elems, nan, threadIdx.x, blockDim.x);
    fill_nan(vc + (int64_t)id * blk_elems, blk_elems, nan, threadIdx.x, blockDim.x);
    return;
  }
  const CropEntry e = a.e[blockIdx.x - a.n_freed];
  const int32_t tail = e.new_len % a.block_size;
  if (tail != 0 && e.tail_private) {  // slots tail .. B-1 of the kept partial block
    const int32_t id = blk_id(a.tables[(int64_t)e.seq * a.max_bps + e.keep - 1], a.n_blocks, a.chk);
    const int B = a.block_size, D = a.head_dim;
    const int per_head = (B - tail) * D;
    for (int i = threadIdx.x; i < a.n_kv_heads * per_head; i += blockDim.x) {
      const int h = i / per_head, r = i % per_head;
      const int slot = tail + r / D, c = r % D;
      kc[(int64_t)id * blk_elems + ((int64_t)h * B + slot) * D + c] = nan;
      vc[(int64_t)id * blk_elems + ((int64_t)h * D + c) * B + slot] = nan;
    }
  }
}

// Copy-on-write before an append: for an entry whose next write lands in a
// shared partial tail block (cow_old), the first block popped for it becomes
// the row's private copy of slots 0 .. P mod B - 1 of every layer (this
// workgroup: one KV head).  Launched before append_kernel on the same stream,
// so every copy has read the shared block before any entry of the call writes
// into it (a later entry may own that block outright once this one has left).
template <typename T>
__global__ void __launch_bounds__(256) cow_kernel(AppendArgs a) {
  const AppendEntry e = a.e[blockIdx.x];
  if (e.cow_old < 0) return;
  const int B = a.block_size, D = a.head_dim, h = blockIdx.y;
  const int32_t id = blk_id(a.free_list[e.stack_before - 1], a.n_blocks, a.chk);
  const int s0 = e.prefix - e.lb_first * B;
  if (h == 0 && threadIdx.x == 0) {
    a.tables[(int64_t)e.seq * a.max_bps + e.lb_first] = id;
    a.refs[id] = 1;
    atomicSub(&a.refs[e.cow_old], 1);   // rows of several entries may share it
  }
  for (int L = 0; L < a.n_layers; ++L) {
    const int64_t ob = ((int64_t)L * a.n_blocks + e.cow_old) * a.n_kv_heads + h;
    const int64_t nb = ((int64_t)L * a.n_blocks + id) * a.n_kv_heads + h;
    const T* ko = (const T*)a.k_cache + ob * B * D;
    const T* vo = (const T*)a.v_cache + ob * D * B;
    T* kn = (T*)a.k_cache + nb * B * D;
    T* vn = (T*)a.v_cache + nb * D * B;
    for (int i = threadIdx.x; i < s0 * D; i += blockDim.x) kn[i] = ko[i];   // K: [slot][d]
    for (int i = threadIdx.x; i < D * s0; i += blockDim.x) {                // V: [d][slot]
      const int c = i / s0, t = i % s0;
      vn[(int64_t)c * B + t] = vo[(int64_t)c * B + t];
    }
  }
}

// FP8 E4M3 code of x (OCP "e4m3fn": bias 7, 3 mantissa bits, largest finite
// 448, NaN = 0x7F), round to nearest even, magnitudes from 464 on saturating
// to 448 (464 itself is the tie between 448 and the next step, 480, which the
// format lacks; ties go to the even mantissa 448 anyway).  Written from the
// format's definition on the fp32 bits.
__device__ inline uint8_t e4m3_code(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const float a = fabsf(x);
  if (!(a == a)) return (uint8_t)(sign | 0x7Fu);
  if (a >= 464.f) return (uint8_t)(sign | 0x7Eu);
  if (a < 0.015625f)                               // below 2^-6: subnormal steps of 2^-9
    return (uint8_t)(sign | (uint32_t)__builtin_rintf(a * 512.f));   // exact product; 8 is 2^-6
  const uint32_t au = u & 0x7FFFFFFFu;
  uint32_t code = (((au >> 23) - 120u) << 3) | ((au >> 20) & 7u);   // exponent rebiased 127 -> 7
  const uint32_t rest = au & 0xFFFFFu;                               // the 20 dropped mantissa bits
  if (rest > 0x80000u || (rest == 0x80000u && (code & 1u))) ++code;  // a carry moves up a binade
  return (uint8_t)(sign | code);
}

// Cache element for input element x: a bit copy, or (bf16 -> FP8) the code of
// the correctly rounded fp32 quotient x / scale.
template <typename TI, typename TC>
__device__ inline TC to_cache(TI x, float) {
  return x;
}
template <>
__device__ inline uint8_t to_cache<uint16_t, uint8_t>(uint16_t x, float scale) {
  return e4m3_code(__uint_as_float((uint32_t)x << 16) / scale);
}

// Reserve + append.  blockIdx.x enumerates (sequence, logical block) items,
// blockIdx.y the KV head.  The physical id of a newly reserved logical block
// lb is read straight from the stack (free_list[stack_before - 1 - k] for the
// k-th new block of the sequence), so no workgroup depends on another's table
// write; the kv-head-0 workgroup records it in the table.
//   K: token p -> k_cache[layer][id][h][p % B][:]      (row copy)
//   V: token p -> v_cache[layer][id][h][:][p % B]      (transposed via LDS)
template <typename TI, typename T>
__global__ void __launch_bounds__(256) append_kernel(AppendArgs a) {
  // [slot][d] staging of V, rows padded by 8 elements on the 16-byte path
  // (block_size <= 64, head_dim <= 128)
  __shared__ __attribute__((aligned(16))) T vstage[64 * (128 + 8)];
  const int item = blockIdx.x;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].item_start <= item) ++ei;
  const AppendEntry e = a.e[ei];
  const int B = a.block_size, D = a.head_dim, h = blockIdx.y;
  const int32_t lb = e.lb_first + (item - e.item_start);
  int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
  const int32_t cow_pops = e.cow_old >= 0 ? 1 : 0;   // cow_kernel took the first pop
  int32_t id;
  if (lb < e.nalloc_before) {
    id = blk_id(row[lb], a.n_blocks, a.chk);
  } else {
    id = blk_id(a.free_list[e.stack_before - 1 - cow_pops - (lb - e.nalloc_before)], a.n_blocks, a.chk);
    if (h == 0 && threadIdx.x == 0) {
      row[lb] = id;
      a.refs[id] = 1;
    }
  }
  if (threadIdx.x == 0 && h == 0) {
    if (a.commit && item == e.item_start) a.lens[e.seq] = e.prefix + e.q_len;
    if (a.write_top && item == 0) *a.free_top = a.top_after;
  }
  const int32_t p0 = max(e.prefix, lb * B);
  const int32_t p1 = min(e.prefix + e.q_len, (lb + 1) * B);
  const int nt = p1 - p0;  // tokens landing in this block (>= 1)
  const int s0 = p0 - lb * B;
  const int64_t blk = ((int64_t)a.layer * a.n_blocks + id) * a.n_kv_heads + h;
  const TI* kin = (const TI*)a.k_in;
  const TI* vin = (const TI*)a.v_in;
  T* kc = (T*)a.k_cache + blk * B * D;
  T* vc = (T*)a.v_cache + blk * D * B;
  if constexpr (sizeof(TI) == 2 && sizeof(T) == 2) {
    // bf16 pool, span starting and ending on 8-slot boundaries: K rows move in
    // 16-byte chunks; V is staged [slot][d] (rows padded to D + 8, so the
    // transposing reads of 8 slots at one d fall in distinct banks) and each
    // d row's 8-slot runs are written as 16-byte chunks.
    if ((s0 & 7) == 0 && (nt & 7) == 0 && (D & 7) == 0) {
      typedef uint32_t u4 __attribute__((ext_vector_type(4)));
      const int C8 = D / 8, DP = D + 8, S8 = nt / 8;
      const int64_t row_stride = (int64_t)a.n_kv_heads * D;
      const int64_t src0 = ((int64_t)(e.q_off + (p0 - e.prefix)) * a.n_kv_heads + h) * D;
      for (int i = threadIdx.x; i < nt * C8; i += blockDim.x) {
        const int t = i / C8, c = (i % C8) * 8;
        const int64_t src = src0 + t * row_stride + c;
        *(u4*)(kc + (int64_t)(s0 + t) * D + c) = *(const u4*)((const TI*)a.k_in + src);
        *(u4*)(&vstage[t * DP + c]) = *(const u4*)((const TI*)a.v_in + src);
      }
      __syncthreads();
      for (int i = threadIdx.x; i < D * S8; i += blockDim.x) {
        const int d = i / S8, t0 = (i % S8) * 8;
        u4 out;
#pragma unroll
        for (int w = 0; w < 4; ++w)
          out[w] = (uint32_t)vstage[(t0 + 2 * w) * DP + d] | ((uint32_t)vstage[(t0 + 2 * w + 1) * DP + d] << 16);
        *(u4*)(vc + (int64_t)d * B + s0 + t0) = out;
      }
      return;
    }
  }
  for (int i = threadIdx.x; i < nt * D; i += blockDim.x) {
    const int t = i / D, c = i % D;
    const int64_t src = ((int64_t)(e.q_off + (p0 - e.prefix) + t) * a.n_kv_heads + h) * D + c;
    kc[(int64_t)(s0 + t) * D + c] = to_cache<TI, T>(kin[src], a.k_scale);
    vstage[t * D + c] = to_cache<TI, T>(vin[src], a.v_scale);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nt * D; i += blockDim.x) {
    const int c = i / nt, t = i % nt;
    vc[(int64_t)c * B + s0 + t] = vstage[t * D + c];
  }
}

// K/V of the tokens of one (sequence, logical block) item for one KV head,
// bf16 pools, one wave: tokens p0 .. p0+nt-1 (block slots s0 .. s0+nt-1) from
// the packed inputs (rows of n_kv_heads * D elements) into the block-head at
// kc (K, [slot][d]) and vc (V, [d][slot]).  Every lane issues all of its loads
// (up to four 16-byte chunks of K and four of V per round) before any store;
// V is staged [slot][d] in LDS (rows padded to D + 8) and written back along d
// rows: 16-byte runs of 8 slots when the span starts and ends on 8-slot
// boundaries, else slot by slot (the partial first and last blocks).
template <int B, int D>
__device__ inline void copy_block_head(const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
                                       int64_t row_stride, uint16_t* __restrict__ kc,
                                       uint16_t* __restrict__ vc, int s0, int nt, uint16_t* vstage) {
  typedef uint32_t u4 __attribute__((ext_vector_type(4)));
  constexpr int C8 = D / 8, DP = D + 8;
  const int lane = threadIdx.x;
  const int nck = nt * C8;                   // 16-byte chunks of K (and of V) here
  if (nt == B && B * C8 <= 4 * 64) {         // a whole block in one round, constant indices
    u4 kk[B * C8 / 64], vv[B * C8 / 64];
#pragma unroll
    for (int j = 0; j < B * C8 / 64; ++j) {
      const int i = j * 64 + lane;
      const int64_t off = (i / C8) * row_stride + (i % C8) * 8;
      kk[j] = *(const u4*)(kin + off);
      vv[j] = *(const u4*)(vin + off);
    }
#pragma unroll
    for (int j = 0; j < B * C8 / 64; ++j) {
      const int i = j * 64 + lane, t = i / C8, c = (i % C8) * 8;
      *(u4*)(kc + (int64_t)t * D + c) = kk[j];
      *(u4*)(&vstage[t * DP + c]) = vv[j];
    }
  }
  for (int i0 = 0; i0 < nck && !(nt == B && B * C8 <= 4 * 64); i0 += 4 * 64) {
    u4 kk[4], vv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = i0 + j * 64 + lane;
      if (i < nck) {
        const int64_t off = (i / C8) * row_stride + (i % C8) * 8;
        kk[j] = *(const u4*)(kin + off);
        vv[j] = *(const u4*)(vin + off);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = i0 + j * 64 + lane;
      if (i < nck) {
        const int t = i / C8, c = (i % C8) * 8;
        *(u4*)(kc + (int64_t)(s0 + t) * D + c) = kk[j];
        *(u4*)(&vstage[t * DP + c]) = vv[j];
      }
    }
  }
  __syncthreads();
  if (nt == B) {                             // a whole block: constant trip counts
    constexpr int S8 = B / 8;
#pragma unroll
    for (int i = lane; i < D * S8; i += 64) {
      const int d = i / S8, t0 = (i % S8) * 8;
      u4 out;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        out[w] = (uint32_t)vstage[(t0 + 2 * w) * DP + d] | ((uint32_t)vstage[(t0 + 2 * w + 1) * DP + d] << 16);
      *(u4*)(vc + (int64_t)d * B + t0) = out;
    }
  } else if ((s0 & 7) == 0 && (nt & 7) == 0) {
    const int S8 = nt / 8;
    for (int i = lane; i < D * S8; i += 64) {
      const int d = i / S8, t0 = (i % S8) * 8;
      u4 out;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        out[w] = (uint32_t)vstage[(t0 + 2 * w) * DP + d] | ((uint32_t)vstage[(t0 + 2 * w + 1) * DP + d] << 16);
      *(u4*)(vc + (int64_t)d * B + s0 + t0) = out;
    }
  } else {
    // a partial first or last block: slot by slot, lanes along d (no division
    // by the run length; these two items per sequence set the launch's length)
    for (int t = 0; t < nt; ++t)
#pragma unroll
      for (int d = lane; d < D; d += 64) vc[(int64_t)d * B + s0 + t] = vstage[t * DP + d];
  }
}

// Reserve + append for bf16 pools: one wave per (sequence, logical block) item
// and KV head; block ids read from the table or straight from the stack
// (free_list[stack_before - 1 - k] for the k-th new block of the sequence), so
// no workgroup depends on another's table write.
template <int B, int D>
__global__ void __launch_bounds__(64) append_bf16_kernel(AppendArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vstage[B * (D + 8)];
  const int item = blockIdx.x, lane = threadIdx.x;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].item_start <= item) ++ei;
  const AppendEntry e = a.e[ei];
  const int h = blockIdx.y;
  const int32_t lb = e.lb_first + (item - e.item_start);
  const int32_t p0 = max(e.prefix, lb * B);
  const int32_t p1 = min(e.prefix + e.q_len, (lb + 1) * B);
  int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
  const int32_t cow_pops = e.cow_old >= 0 ? 1 : 0;   // cow_kernel took the first pop
  const int32_t id = blk_id(lb < e.nalloc_before
                                 ? row[lb]
                                 : a.free_list[e.stack_before - 1 - cow_pops - (lb - e.nalloc_before)],
                             a.n_blocks, a.chk);
  if (h == 0 && lane == 0) {
    if (lb >= e.nalloc_before) {
      row[lb] = id;
      a.refs[id] = 1;
    }
    if (a.commit && item == e.item_start) a.lens[e.seq] = e.prefix + e.q_len;
    if (a.write_top && item == 0) *a.free_top = a.top_after;
  }
  const int64_t row_stride = (int64_t)a.n_kv_heads * D;
  const int64_t src0 = ((int64_t)(e.q_off + (p0 - e.prefix)) * a.n_kv_heads + h) * D;
  const int64_t blk = ((int64_t)a.layer * a.n_blocks + id) * a.n_kv_heads + h;
  copy_block_head<B, D>((const uint16_t*)a.k_in + src0, (const uint16_t*)a.v_in + src0, row_stride,
                        (uint16_t*)a.k_cache + blk * B * D, (uint16_t*)a.v_cache + blk * D * B,
                        p0 - lb * B, p1 - p0, vstage);
}

// Restore + reserve + append in one launch.  Workgroup (0, 0) runs the crop of
// a.ce in call order (released entries of a row, 256 at a time: -1 into the
// table, count decremented, blocks reaching 0 pushed in ascending order by
// ballot prefix counts), then the reservation of a.e in call order (the k-th
// new block of an entry is free_list[stack_before - 1 - k] of the stack the
// crop just left, named in the table with count 1), then the lengths and the
// stack top; its accesses are ordered by the barriers between rounds.  Every
// other workgroup copies one item's K/V for one KV head into ids[item] and
// touches no metadata.
template <int B, int D>
__global__ void __launch_bounds__(64) fused_append_kernel(FusedAppendArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vstage[B * (D + 8)];
  const int lane = threadIdx.x, h = blockIdx.y;
  if (blockIdx.x == 0) {
    if (h != 0) return;
    // 256 entries per round, entry j0 + 64 r + lane in lane's slot r, so the
    // ascending push order is r-major: position = pushes of slots before r
    // plus pushes of lower lanes in slot r.
    constexpr int R = 4;
    const uint64_t below = (1ull << lane) - 1ull;
    int32_t top = a.top_before;
    for (int i = 0; i < a.n_crop; ++i) {
      const CropEntry c = a.ce[i];
      int32_t* row = a.tables + (int64_t)c.seq * a.max_bps;
      for (int32_t j0 = c.keep; j0 < c.nalloc; j0 += R * 64) {
        int32_t b[R], r[R];
#pragma unroll
        for (int k = 0; k < R; ++k) {
          const int32_t j = j0 + 64 * k + lane;
          b[k] = j < c.nalloc ? blk_id(row[j], a.n_blocks, a.chk) : -1;
        }
#pragma unroll
        for (int k = 0; k < R; ++k) r[k] = b[k] >= 0 ? a.refs[b[k]] - 1 : 1;
#pragma unroll
        for (int k = 0; k < R; ++k) {
          const int32_t j = j0 + 64 * k + lane;
          if (b[k] >= 0) {
            row[j] = -1;
            a.refs[b[k]] = r[k];
          }
          const uint64_t m = __ballot(r[k] == 0);
          if (r[k] == 0) a.free_list[top + __popcll(m & below)] = b[k];
          top += __popcll(m);
        }
        __syncthreads();   // this round's table, count and stack writes precede the next round's reads
      }
      if (lane == 0) a.lens[c.seq] = c.new_len;
    }
    for (int i = 0; i < a.n; ++i) {
      const AppendEntry e = a.e[i];
      int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
      const int32_t end = (e.prefix + e.q_len + B - 1) / B;
      for (int32_t lb0 = e.nalloc_before; lb0 < end; lb0 += R * 64) {
        int32_t id[R];
#pragma unroll
        for (int k = 0; k < R; ++k) {
          const int32_t lb = lb0 + 64 * k + lane;
          id[k] = lb < end ? blk_id(a.free_list[e.stack_before - 1 - (lb - e.nalloc_before)], a.n_blocks, a.chk)
                           : -1;
        }
#pragma unroll
        for (int k = 0; k < R; ++k) {
          if (id[k] >= 0) {
            row[lb0 + 64 * k + lane] = id[k];
            a.refs[id[k]] = 1;
          }
        }
      }
      if (lane == 0 && a.commit) a.lens[e.seq] = e.prefix + e.q_len;
    }
    if (lane == 0) *a.free_top = a.top_after;
    return;
  }
  const int item = blockIdx.x - 1;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].item_start <= item) ++ei;
  const AppendEntry e = a.e[ei];
  const int32_t lb = e.lb_first + (item - e.item_start);
  const int32_t p0 = max(e.prefix, lb * B);
  const int32_t p1 = min(e.prefix + e.q_len, (lb + 1) * B);
  const int64_t row_stride = (int64_t)a.n_kv_heads * D;
  const int64_t src0 = ((int64_t)(e.q_off + (p0 - e.prefix)) * a.n_kv_heads + h) * D;
  const int64_t blk = ((int64_t)a.layer * a.n_blocks + a.ids[item]) * a.n_kv_heads + h;
  copy_block_head<B, D>((const uint16_t*)a.k_in + src0, (const uint16_t*)a.v_in + src0, row_stride,
                        (uint16_t*)a.k_cache + blk * B * D, (uint16_t*)a.v_cache + blk * D * B,
                        p0 - lb * B, p1 - p0, vstage);
}

}  // namespace

hipError_t launch_pool_init(int32_t* tables, int64_t n_table, int32_t* lens, int32_t max_seqs,
                            int32_t* free_list, int32_t n_blocks, int32_t* free_top, int32_t* refs,
                            hipStream_t s) {
  int64_t biggest = n_table > n_blocks ? n_table : n_blocks;
  if (max_seqs > biggest) biggest = max_seqs;
  int grid = (int)((biggest + 255) / 256);
  if (grid > 4096) grid = 4096;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL(pool_init_kernel, dim3(grid), dim3(256), 0, s, tables, n_table, lens,
                     max_seqs, free_list, n_blocks, free_top, refs);
  return hipGetLastError();
}

hipError_t launch_crop(const CropArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(crop_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fork(const ForkArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fork_kernel, dim3(a.n), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_poison(const PoisonArgs& a, hipStream_t s) {
  if (a.n + a.n_freed <= 0) return hipSuccess;
  const dim3 grid(a.n_freed + a.n, a.n_layers);
  if (a.elem_bytes == 4)
    hipLaunchKernelGGL(poison_kernel<uint32_t>, grid, dim3(256), 0, s, a, (uint32_t)0x7FC00000u);
  else if (a.elem_bytes == 2)
    hipLaunchKernelGGL(poison_kernel<uint16_t>, grid, dim3(256), 0, s, a, (uint16_t)0x7FC0u);
  else
    hipLaunchKernelGGL(poison_kernel<uint8_t>, grid, dim3(256), 0, s, a, (uint8_t)0x7Fu);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, int elem_bytes, hipStream_t s) {
  if (a.n <= 0 || a.n_items <= 0) return hipSuccess;
  bool any_cow = false;
  for (int i = 0; i < a.n; ++i) any_cow |= a.e[i].cow_old >= 0;
  const dim3 cow_grid(a.n, a.n_kv_heads), grid(a.n_items, a.n_kv_heads);
  if (elem_bytes == 4) {
    if (any_cow) hipLaunchKernelGGL(cow_kernel<uint32_t>, cow_grid, dim3(256), 0, s, a);
    hipLaunchKernelGGL((append_kernel<uint32_t, uint32_t>), grid, dim3(256), 0, s, a);
  } else if (elem_bytes == 2) {
    if (any_cow) hipLaunchKernelGGL(cow_kernel<uint16_t>, cow_grid, dim3(256), 0, s, a);
    if (a.head_dim == 128 && a.block_size == 16)
      hipLaunchKernelGGL((append_bf16_kernel<16, 128>), grid, dim3(64), 0, s, a);
    else if (a.head_dim == 128 && a.block_size == 32)
      hipLaunchKernelGGL((append_bf16_kernel<32, 128>), grid, dim3(64), 0, s, a);
    else if (a.head_dim == 128 && a.block_size == 64)
      hipLaunchKernelGGL((append_bf16_kernel<64, 128>), grid, dim3(64), 0, s, a);
    else if (a.head_dim == 64 && a.block_size == 16)
      hipLaunchKernelGGL((append_bf16_kernel<16, 64>), grid, dim3(64), 0, s, a);
    else if (a.head_dim == 64 && a.block_size == 32)
      hipLaunchKernelGGL((append_bf16_kernel<32, 64>), grid, dim3(64), 0, s, a);
    else if (a.head_dim == 64 && a.block_size == 64)
      hipLaunchKernelGGL((append_bf16_kernel<64, 64>), grid, dim3(64), 0, s, a);
    else
      hipLaunchKernelGGL((append_kernel<uint16_t, uint16_t>), grid, dim3(256), 0, s, a);
  } else {                                          // FP8 cache, bf16 inputs
    if (any_cow) hipLaunchKernelGGL(cow_kernel<uint8_t>, cow_grid, dim3(256), 0, s, a);
    hipLaunchKernelGGL((append_kernel<uint16_t, uint8_t>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

bool fused_append_supported(int block_size, int head_dim) {
  return (head_dim == 128 || head_dim == 64) && (block_size == 16 || block_size == 32 || block_size == 64);
}

hipError_t launch_fused_append(const FusedAppendArgs& a, hipStream_t s) {
  const dim3 grid(1 + a.n_items, a.n_kv_heads);
#define PGSR_FUSED(BS, HD)                                                                      \
  if (a.block_size == BS && a.head_dim == HD) {                                                  \
    hipLaunchKernelGGL((fused_append_kernel<BS, HD>), grid, dim3(64), 0, s, a);                  \
    return hipGetLastError();                                                                    \
  }
  PGSR_FUSED(16, 128) PGSR_FUSED(32, 128) PGSR_FUSED(64, 128)
  PGSR_FUSED(16, 64) PGSR_FUSED(32, 64) PGSR_FUSED(64, 64)
#undef PGSR_FUSED
  return hipErrorInvalidValue;
}

}  // namespace pgsr
