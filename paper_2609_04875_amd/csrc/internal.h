// Internal interface between the host runtime (pgsr_host.cpp) and the kernels.
// Per-call sequence descriptors travel in the kernel-argument segment, so a
// call carries no host->device copy; calls with more sequences are split into
// several launches of at most kMaxSeqsPerLaunch sequences each.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

struct pgsr_pool;

namespace pgsr {

constexpr int kMaxSeqsPerLaunch = 64;

// ------------------------------------------------------- checked build --- //
// A library built with -DPGSR_CHECKED validates every block id it reads from
// the block table or the free stack before the id addresses the cache, the
// counts or the stack: an id outside [0, n_blocks) is replaced by block 0 and
// recorded in *chk (a device word the pool owns), and the call returns
// PGSR_ERANGE once its launches have finished.  Only memory written behind
// the library's back can hold such an id (the host mirror validates every
// call), so the default build reads ids unchecked; the checked one turns that
// corruption into an error instead of an access outside the pool.
__device__ __forceinline__ int32_t blk_id(int32_t id, int32_t n_blocks, int32_t* chk) {
#ifdef PGSR_CHECKED
  if ((uint32_t)id >= (uint32_t)n_blocks) {
    atomicOr(chk, 1);
    return 0;
  }
#else
  (void)n_blocks;
  (void)chk;
#endif
  return id;
}

// ---------------------------------------------------------------- crop ---- //
struct CropEntry {
  int32_t seq;       // row of the block table
  int32_t new_len;   // tokens kept
  int32_t keep;      // ceil(new_len / B): table entries kept
  int32_t nalloc;    // entries held before the crop
  int32_t tail_private;  // poison only: the kept partial block is named by this row alone
};

// One workgroup takes the entries in call order; each released table entry
// decrements its block's count, and blocks reaching 0 are pushed in ascending
// entry order starting at top_before.
struct CropArgs {
  int32_t* tables;
  int32_t* lens;
  int32_t* free_list;
  int32_t* free_top;
  int32_t* refs;
  int32_t* chk;        // checked build: out-of-range block id seen
  int32_t max_bps, n_blocks;
  int32_t top_before;  // stack height when this launch starts
  int32_t n;
  CropEntry e[kMaxSeqsPerLaunch];
};

// Debug aid: NaN-fill every slot a crop released: whole blocks it pushed
// (free_list[top_before .. top_before + n_freed)) in all layers, and the tail
// slots of a kept partial block that no other row names.
struct PoisonArgs {
  void* k_cache;
  void* v_cache;
  const int32_t* tables;
  const int32_t* free_list;
  int32_t* chk;
  int32_t max_bps, n_layers, n_blocks, n_kv_heads, block_size, head_dim, elem_bytes;
  int32_t top_before;
  int32_t n_freed;
  int32_t n;
  CropEntry e[kMaxSeqsPerLaunch];
};

// --------------------------------------------------------------- fork ----- //
struct ForkEntry {
  int32_t src, dst;
  int32_t nalloc;   // table entries of src, shared with dst
  int32_t len;      // tokens of src
};

struct ForkArgs {
  int32_t* tables;
  int32_t* lens;
  int32_t* refs;
  int32_t* chk;
  int32_t max_bps, n_blocks;
  int32_t n;
  ForkEntry e[kMaxSeqsPerLaunch];
};

// --------------------------------------------------------- reserve+append - //
struct AppendEntry {
  int32_t seq;
  int32_t prefix;         // committed length P (first new position)
  int32_t q_len;          // S new tokens
  int32_t q_off;          // first row of this sequence in the packed k/v inputs
  int32_t nalloc_before;  // table entries held before this call's reservation
  int32_t stack_before;   // stack height before this sequence's pops
  int32_t lb_first;       // first logical block touched: P / B
  int32_t item_start;     // prefix sum of logical blocks touched over entries
  int32_t cow_old;        // shared partial tail block to copy before writing, or -1;
                          // its private copy is the first block popped for this entry
};

struct AppendArgs {
  void* k_cache;
  void* v_cache;
  const void* k_in;
  const void* v_in;
  int32_t* tables;
  int32_t* lens;
  const int32_t* free_list;
  int32_t* free_top;
  int32_t* refs;
  int32_t* chk;
  int32_t max_bps, n_blocks, n_kv_heads, block_size, head_dim, layer, n_layers;
  int32_t commit;
  // FP8 E4M3 cache (1-byte elements) fed from bf16 inputs: each value is stored
  // as the code of fp32(x / scale), rounded to nearest even, saturating at 448.
  float k_scale, v_scale;
  int32_t write_top;   // 1: this launch writes free_top = top_after
  int32_t top_after;
  int32_t n;
  int32_t n_items;
  AppendEntry e[kMaxSeqsPerLaunch];
};

// Restore + reserve + append in one launch (bf16 pools, no copy-on-write, no
// poisoning): workgroup (0, 0) takes the crop of `ce` exactly as crop_kernel
// does, then the reservation pops of `e` from the stack it just pushed to
// (tables, counts, lengths, top); the other workgroups copy the K/V of item
// blockIdx.x - 1 and KV head blockIdx.y into block ids[item], which the host
// mirror computed by the same steps.
constexpr int kMaxFusedSeqs = 16;
constexpr int kMaxFusedItems = 512;

struct FusedAppendArgs {
  void* k_cache;
  void* v_cache;
  const void* k_in;
  const void* v_in;
  int32_t* tables;
  int32_t* lens;
  int32_t* free_list;
  int32_t* free_top;
  int32_t* refs;
  int32_t* chk;
  int32_t max_bps, n_blocks, n_kv_heads, block_size, head_dim, layer;
  int32_t commit;
  int32_t top_before;  // stack height before the crop
  int32_t top_after;   // after the reservation
  int32_t n_crop;
  int32_t n;
  int32_t n_items;
  CropEntry ce[kMaxFusedSeqs];
  AppendEntry e[kMaxFusedSeqs];
  int32_t ids[kMaxFusedItems];
};

// -------------------------------------------------------------- attention - //
struct AttnEntry {
  int32_t seq;
  int32_t prefix;      // P: queries sit at absolute positions P .. P+S-1
  int32_t q_len;       // S
  int32_t q_off;       // first row of this sequence in q / o
  int32_t tile_start;  // prefix sum of query tiles over entries
};

struct AttnArgs {
  const void* q;
  void* o;
  const void* k_cache;
  const void* v_cache;
  const int32_t* tables;
  int32_t* chk;
  int32_t max_bps, n_blocks, n_q_heads, n_kv_heads, block_size, head_dim, layer;
  float scale_log2;    // softmax_scale * log2(e) (times the K scale of an FP8 cache)
  float o_scale;       // output factor: the V scale of an FP8 cache, else 1
  int32_t n;
  int32_t n_tiles;
  // Split-key mode (n_splits > 1): split s of a query tile covers keys
  // [s * split_len, (s+1) * split_len) at absolute positions and writes
  // unnormalised partials for every query row r (r = token * n_q_heads + head
  // over the launch's packed queries): acc to ws_acc[(s * n_rows + r) * D],
  // the running max (log2 units) and row sum to ws_ml[2 * (s * n_rows + r)].
  int32_t n_splits;
  int32_t split_len;
  int32_t n_rows;
  // Packed query rows [row_begin, row_end) belong to this launch's entries
  // (a call with more than kMaxSeqsPerLaunch sequences is several launches,
  // each owning one contiguous run of rows); the combine touches only those.
  int32_t row_begin, row_end;
  float* ws_acc;
  float* ws_ml;
  // Clock probe (timing only, else null): workgroup b < clk_n writes
  // {s_memtime at start, at end, s_memrealtime at start, at end} to clk[4b..].
  uint64_t* clk;
  int32_t clk_n;
  AttnEntry e[kMaxSeqsPerLaunch];
};

// ------------------------------------------------------------- sampling -- //
struct SampleArgs {
  int32_t n;           // rows in this launch
  int32_t row0;        // first row of this launch in logits / tokens
  int32_t vocab;
  int32_t n_chunks;    // workgroups per row; > 1 writes partial keys
  int32_t chunk_len;   // vocabulary entries per chunk, a multiple of 4
  float temperature;   // 0: greedy
  uint64_t seed;
  uint64_t* partial;   // [rows][n_chunks] keys when n_chunks > 1
  int64_t stream[kMaxSeqsPerLaunch];
  int64_t position[kMaxSeqsPerLaunch];
};

hipError_t launch_sample(const SampleArgs& a, int dtype, const void* logits, int32_t* tokens,
                         hipStream_t s);
hipError_t launch_sample_reduce(int32_t n, int32_t n_chunks, const uint64_t* partial, int32_t* tokens,
                                hipStream_t s);

// Query tokens per workgroup tile for each kernel (the host sizes grids with these).
int attn_f32_tile_tokens(int head_dim, int group);
int attn_bf16_tile_tokens(int head_dim, int group);

hipError_t launch_crop(const CropArgs& a, hipStream_t s);
hipError_t launch_poison(const PoisonArgs& a, hipStream_t s);
hipError_t launch_fork(const ForkArgs& a, hipStream_t s);
hipError_t launch_append(const AppendArgs& a, int elem_bytes, hipStream_t s);
// False when the fused launch does not cover this geometry (the caller then
// launches crop and append separately).
bool fused_append_supported(int block_size, int head_dim);
hipError_t launch_fused_append(const FusedAppendArgs& a, hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s);
// Software-pipelined bf16 prefill for head_dim 128 and GQA groups dividing
// 32: two waves per SIMD, 32 query rows per wave, one workgroup per CU.
bool attn_bf16_pipe_eligible(int head_dim, int group);
int attn_bf16_pipe_tile_tokens(int group);
hipError_t launch_attn_bf16_pipe(const AttnArgs& a, hipStream_t s);
// The same tiles and bits with one wave per SIMD holding 64 query rows and
// global->LDS tile loads: 16-token blocks, pools whose layer-head block range
// fits 32-bit byte offsets, sequences of up to 130816 keys (a workgroup's
// part of the block table sits in LDS).  Tile tokens as
// attn_bf16_pipe_tile_tokens.
bool attn_bf16_wide_eligible(int head_dim, int group, int block_size, int64_t n_blocks, int n_kv_heads,
                             int64_t max_kv_len);
hipError_t launch_attn_bf16_wide(const AttnArgs& a, hipStream_t s);
// Same kernel over an FP8 E4M3 cache: codes widen to bf16 exactly on the way
// into LDS; the K scale is in scale_log2, the V scale in o_scale.
hipError_t launch_attn_fp8(const AttnArgs& a, hipStream_t s);
// Decode attention (every sequence of the launch has at most 32 / G query
// tokens): one wave per (sequence, KV head, split) gathering MFMA operands from
// the cache without LDS; with n_splits > 1 it writes split partials.
hipError_t launch_attn_decode(const AttnArgs& a, bool fp8, hipStream_t s);
int attn_decode_keys_per_tile();
// Merge split-key partials into O (bf16, or fp32 for fp32 pools), splits in
// increasing order.
hipError_t launch_split_combine(const AttnArgs& a, bool f32_out, hipStream_t s);
hipError_t launch_pool_init(int32_t* tables, int64_t n_table, int32_t* lens, int32_t max_seqs,
                            int32_t* free_list, int32_t n_blocks, int32_t* free_top, int32_t* refs,
                            hipStream_t s);
hipError_t launch_rmsnorm(int32_t n, int32_t dm, const void* x, const void* g, float eps, void* y,
                          hipStream_t s);
hipError_t launch_rope(int32_t n, int32_t heads, int32_t d, void* x, const int32_t* pos, double theta,
                       hipStream_t s);
hipError_t launch_silu_mul(int32_t n, int32_t dff, const void* gu, void* out, hipStream_t s);

// Text returned by pgsr_last_error() on this thread (host runtime).
void set_error(const char* msg);
void clear_error();
// Sets the error text and returns code.
int fail_with(int code, const char* msg);

// pgsr_replay_prefill with an explicit split-key / decode workspace (the
// pool's own, or the library's static scratch).
int replay_prefill_ws(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                      const int32_t* q_lens, const void* q, const void* k, const void* v, void* o,
                      float softmax_scale, unsigned flags, int64_t* recomputed_tokens, void* ws,
                      size_t ws_bytes, void* stream);

hipError_t launch_gemm_bf16(int m, int n, int k, const void* x, const void* w, const void* r,
                            void* y, hipStream_t s);
// One wave per SIMD, global->LDS tiles (products with at least 256 tiles of
// 256 x 256, K a multiple of 64, m*k and n*k below 2^31); same bits as above.
bool gemm_bf16_wide_eligible(int m, int n, int k);
hipError_t launch_gemm_bf16_wide(int m, int n, int k, const void* x, const void* w, const void* r,
                                 void* y, hipStream_t s);

}  // namespace pgsr
