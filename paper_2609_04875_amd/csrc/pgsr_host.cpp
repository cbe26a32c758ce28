// Host runtime of the C ABI declared in include/pgsr.h: argument validation
// against a host mirror of the pool, block reservation bookkeeping, and kernel
// launches on the caller's stream.  Every check runs before the first launch,
// so a rejected call changes neither the mirror nor device memory.
#include "pgsr.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <cfloat>
#include <string>
#include <unordered_map>
#include <vector>

#include "internal.h"

using namespace pgsr;

struct pgsr_pool {
  int32_t n_layers, hq, hkv, d, B, dtype, n_blocks, max_seqs, max_bps;
  void* k_cache;
  void* v_cache;
  int32_t* tables;
  int32_t* lens;
  int32_t* free_list;
  int32_t* free_top;
  int32_t* refs;
  void* workspace;
  size_t workspace_bytes;
  // host mirror of the metadata, updated at call time in enqueue order by the
  // same steps the kernels take
  std::vector<int32_t> h_len, h_nalloc;
  std::vector<int32_t> h_tab;    // [max_seqs][max_bps]
  std::vector<int32_t> h_free;   // stack storage
  std::vector<int32_t> h_ref;    // table entries naming each block
  int32_t h_top;
  // optional kernel timing: events around the append and attention launches
  bool timing = false, timed_call = false;
  // FP8 pools: per-layer K and V scales (stored code = x / scale, read = code * scale)
  std::vector<float> k_scale, v_scale;
  // bf16 prefill kernel choice (PGSR_PREFILL_AUTO / _FOUR_WAVE / _PIPELINED)
  int prefill_kind = PGSR_PREFILL_AUTO;
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
  // shader-clock probe (caller-owned device buffer, 4 uint64 per workgroup)
  uint64_t* clk = nullptr;
  int32_t clk_n = 0;
  bool clk_written = false;
  // checked build: device word the kernels set when a block id they read is
  // out of range (null in the default build)
  int32_t* chk = nullptr;
};

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return PGSR_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(PGSR_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// After a call's launches: in the checked build, wait for them and report a
// block id that a kernel found out of range (the flag is cleared for the next
// call); in the default build there is nothing to check.
int device_check(pgsr_pool* p, hipStream_t st) {
#ifdef PGSR_CHECKED
  int32_t h = 0;
  hipError_t err = hipMemcpyAsync(&h, p->chk, sizeof h, hipMemcpyDeviceToHost, st);
  if (err == hipSuccess) err = hipStreamSynchronize(st);
  if (err != hipSuccess) return hip_fail(err, "checked build: flag read");
  if (h != 0) {
    err = hipMemsetAsync(p->chk, 0, sizeof h, st);
    if (err == hipSuccess) err = hipStreamSynchronize(st);
    if (err != hipSuccess) return hip_fail(err, "checked build: flag reset");
    return fail(PGSR_ERANGE,
                "checked build: a kernel read a block id outside [0, %d) from the block table or the "
                "free stack (device metadata written outside the library); block 0 was used instead",
                p->n_blocks);
  }
#else
  (void)p;
  (void)st;
#endif
  return PGSR_OK;
}

inline int32_t cdiv(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }

int elem_bytes(const pgsr_pool* p) { return p->dtype == PGSR_F32 ? 4 : p->dtype == PGSR_BF16 ? 2 : 1; }

// Distinct, in-range sequence ids (a pairwise check for the few sequences of
// a typical call, a table past that).
int check_seqs(const pgsr_pool* p, int32_t n, const int32_t* seqs) {
  for (int32_t i = 0; i < n; ++i)
    if (seqs[i] < 0 || seqs[i] >= p->max_seqs)
      return fail(PGSR_EINVAL, "sequence id %d outside [0, %d)", seqs[i], p->max_seqs);
  if (n <= 32) {
    for (int32_t i = 0; i < n; ++i)
      for (int32_t j = 0; j < i; ++j)
        if (seqs[i] == seqs[j]) return fail(PGSR_EINVAL, "sequence id %d appears twice in one call", seqs[i]);
    return PGSR_OK;
  }
  std::vector<char> seen(p->max_seqs, 0);
  for (int32_t i = 0; i < n; ++i) {
    if (seen[seqs[i]]) return fail(PGSR_EINVAL, "sequence id %d appears twice in one call", seqs[i]);
    seen[seqs[i]] = 1;
  }
  return PGSR_OK;
}

// ------------------------------------------------------------------ crop -- //
// Mirror of a crop of sequence s to L tokens: released entries, ascending,
// decrement their block's count; blocks reaching 0 are pushed.
void mirror_crop(pgsr_pool* p, int32_t s, int32_t L) {
  const int32_t keep = cdiv(L, p->B);
  int32_t* row = &p->h_tab[(size_t)s * p->max_bps];
  for (int32_t j = keep; j < p->h_nalloc[s]; ++j) {
    const int32_t b = row[j];
    row[j] = -1;
    if (--p->h_ref[b] == 0) p->h_free[p->h_top++] = b;
  }
  p->h_nalloc[s] = keep;
  p->h_len[s] = L;
}

// Blocks a crop of these sequences would push (the mirror is left unchanged).
int64_t count_freed(const pgsr_pool* p, int32_t n, const int32_t* seqs, const int32_t* new_lens) {
  // without sharing (every released block named once) each release frees its block
  int64_t released = 0;
  bool shared = false;
  for (int32_t i = 0; i < n && !shared; ++i) {
    const int32_t s = seqs[i], keep = cdiv(new_lens[i], p->B);
    for (int32_t j = keep; j < p->h_nalloc[s]; ++j) {
      if (p->h_ref[p->h_tab[(size_t)s * p->max_bps + j]] != 1) {
        shared = true;
        break;
      }
      ++released;
    }
  }
  if (!shared) return released;
  std::unordered_map<int32_t, int32_t> dec;   // block -> decrements so far
  int64_t freed = 0;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = seqs[i], keep = cdiv(new_lens[i], p->B);
    for (int32_t j = keep; j < p->h_nalloc[s]; ++j) {
      const int32_t b = p->h_tab[(size_t)s * p->max_bps + j];
      if (p->h_ref[b] - ++dec[b] == 0) ++freed;
    }
  }
  return freed;
}

// Does the next write of sequence s (prefix P, S > 0 tokens) land in a partial
// tail block that other table entries also name?
bool shared_tail(const pgsr_pool* p, int32_t s, int32_t P, int32_t S) {
  if (S <= 0 || P % p->B == 0) return false;
  const int32_t b = p->h_tab[(size_t)s * p->max_bps + P / p->B];
  return b >= 0 && p->h_ref[b] > 1;
}

int do_crop(pgsr_pool* p, int32_t n, const int32_t* seqs, const int32_t* new_lens,
            unsigned flags, hipStream_t st) {
  for (int32_t base = 0; base < n; base += kMaxSeqsPerLaunch) {
    const int32_t cnt = std::min<int32_t>(kMaxSeqsPerLaunch, n - base);
    CropArgs a{};
    a.tables = p->tables;
    a.lens = p->lens;
    a.free_list = p->free_list;
    a.free_top = p->free_top;
    a.refs = p->refs;
    a.chk = p->chk;
    a.max_bps = p->max_bps;
    a.n_blocks = p->n_blocks;
    a.top_before = p->h_top;
    a.n = cnt;
    for (int32_t i = 0; i < cnt; ++i) {
      const int32_t s = seqs[base + i], L = new_lens[base + i];
      CropEntry& e = a.e[i];
      e.seq = s;
      e.new_len = L;
      e.keep = cdiv(L, p->B);
      e.nalloc = p->h_nalloc[s];
      mirror_crop(p, s, L);
      const int32_t tb = e.keep > 0 ? p->h_tab[(size_t)s * p->max_bps + e.keep - 1] : -1;
      e.tail_private = tb >= 0 && p->h_ref[tb] == 1;
    }
    hipError_t err = launch_crop(a, st);
    if (err != hipSuccess) return hip_fail(err, "crop launch");
    if (flags & PGSR_POISON) {
      PoisonArgs pa{};
      pa.k_cache = p->k_cache;
      pa.v_cache = p->v_cache;
      pa.tables = p->tables;
      pa.free_list = p->free_list;
      pa.chk = p->chk;
      pa.max_bps = p->max_bps;
      pa.n_layers = p->n_layers;
      pa.n_blocks = p->n_blocks;
      pa.n_kv_heads = p->hkv;
      pa.block_size = p->B;
      pa.head_dim = p->d;
      pa.elem_bytes = elem_bytes(p);
      pa.top_before = a.top_before;
      pa.n_freed = p->h_top - a.top_before;
      pa.n = cnt;
      std::memcpy(pa.e, a.e, sizeof(CropEntry) * cnt);
      err = launch_poison(pa, st);
      if (err != hipSuccess) return hip_fail(err, "poison launch");
    }
  }
  return PGSR_OK;
}

// ---------------------------------------------------------------- replay -- //
struct Seg {
  int32_t seq, prefix, q_len, q_off;
};

// Split-key attention: used when a launch has fewer workgroups than this (two
// per CU of the 256) and a workspace is available; at most kMaxSplits splits
// (a decode step of one sequence, 8 workgroups unsplit, then fills the chip),
// split boundaries at multiples of the 64-key tile.
constexpr int64_t kSplitTargetWorkgroups = 512;
// The pipelined bf16 kernel holds a CU alone (one wave per SIMD).
constexpr int64_t kSplitTargetWorkgroupsPipe = 256;
constexpr int64_t kMaxSplits = 32;
constexpr int32_t kSplitAlign = 64;
// Decode kernel (calls whose sequences all fit one wave's 32 query rows, with
// a workspace): aim for eight waves per CU, at most 64 splits of at least 256
// keys each.
#ifndef PGSR_DECODE_TARGET_WAVES
#define PGSR_DECODE_TARGET_WAVES 2048
#endif
#ifndef PGSR_DECODE_MIN_SPLIT_KEYS
#define PGSR_DECODE_MIN_SPLIT_KEYS 256
#endif
constexpr int64_t kDecodeTargetWaves = PGSR_DECODE_TARGET_WAVES;
constexpr int64_t kDecodeMaxSplits = 64;
constexpr int32_t kDecodeMinSplitKeys = PGSR_DECODE_MIN_SPLIT_KEYS;

// Validation of a replay step: lengths, table width, free blocks.
int check_replay(const pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                 const int32_t* q_lens, const void* q, const void* k, const void* v,
                 const void* o, const std::vector<int32_t>& prefix,
                 const std::vector<int32_t>& nalloc, int32_t free_blocks, float scale) {
  if (layer < 0 || layer >= p->n_layers)
    return fail(PGSR_EINVAL, "layer %d outside [0, %d)", layer, p->n_layers);
  if (!std::isfinite(scale)) return fail(PGSR_EINVAL, "softmax_scale is not finite");
  int64_t total = 0, need = 0;
  // Private tail copies are decided in call order: each copy releases one
  // entry of the shared block, so the last row naming it writes in place.
  std::unordered_map<int32_t, int32_t> released;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t S = q_lens[i];
    if (S < 0) return fail(PGSR_EINVAL, "q_lens[%d] = %d is negative", i, S);
    const int64_t end = (int64_t)prefix[i] + S;
    if (end > (int64_t)p->max_bps * p->B)
      return fail(PGSR_ERANGE, "sequence %d would reach %lld tokens; its row holds %lld",
                  seqs[i], (long long)end, (long long)p->max_bps * p->B);
    need += std::max<int64_t>(0, cdiv(end, p->B) - nalloc[i]);
    if (nalloc[i] > 0 && S > 0 && prefix[i] % p->B != 0) {
      const int32_t b = p->h_tab[(size_t)seqs[i] * p->max_bps + prefix[i] / p->B];
      if (b >= 0 && p->h_ref[b] - released[b] > 1) {   // private tail copy
        ++need;
        ++released[b];
      }
    }
    total += S;
  }
  if (total > INT32_MAX) return fail(PGSR_ERANGE, "more than 2^31-1 query tokens in one call");
  if (total > 0 && (!q || !k || !v || !o))
    return fail(PGSR_EINVAL, "null q/k/v/o pointer with %lld query tokens", (long long)total);
  if (need > free_blocks)
    return fail(PGSR_ENOMEM, "step needs %lld free blocks, %d available", (long long)need,
                free_blocks);
  return PGSR_OK;
}

// A crop whose device work rides in the replay's append launch: its entries
// (mirror already updated) and the stack height before it.
struct FoldedCrop {
  int32_t n = 0;
  int32_t top_before = 0;
  CropEntry e[kMaxFusedSeqs];
};

int do_replay(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
              const int32_t* q_lens, const void* q, const void* k, const void* v, void* o,
              float scale, unsigned flags, int64_t* recomputed, void* ws, size_t ws_bytes,
              hipStream_t st, const FoldedCrop* fold = nullptr) {
  if (ws == nullptr) ws_bytes = 0;
  // Segments with work, in call order (the packed inputs follow call order).
  std::vector<Seg> segs;
  segs.reserve(n);
  int32_t off = 0;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = seqs[i];
    if (q_lens[i] > 0) segs.push_back({s, p->h_len[s], q_lens[i], off});
    off += q_lens[i];
  }
  const bool commit = (flags & PGSR_COMMIT) != 0;
  const int eb = elem_bytes(p);

  if (p->timing) {
    hipError_t err = hipEventRecord(p->ev[0], st);
    if (err != hipSuccess) return hip_fail(err, "timing event");
  }
  // Restore + reserve + append in one launch (the caller checked that it
  // applies); the mirror takes the same pops in call order and records each
  // item's block for the copying workgroups.
  if (fold) {
    FusedAppendArgs a{};
    a.k_cache = p->k_cache;
    a.v_cache = p->v_cache;
    a.k_in = k;
    a.v_in = v;
    a.tables = p->tables;
    a.lens = p->lens;
    a.free_list = p->free_list;
    a.free_top = p->free_top;
    a.refs = p->refs;
    a.chk = p->chk;
    a.max_bps = p->max_bps;
    a.n_blocks = p->n_blocks;
    a.n_kv_heads = p->hkv;
    a.block_size = p->B;
    a.head_dim = p->d;
    a.layer = layer;
    a.commit = commit ? 1 : 0;
    a.top_before = fold->top_before;
    a.n_crop = fold->n;
    std::memcpy(a.ce, fold->e, sizeof(CropEntry) * fold->n);
    a.n = (int32_t)segs.size();
    int32_t items = 0;
    for (int32_t i = 0; i < a.n; ++i) {
      const Seg& g = segs[i];
      AppendEntry& e = a.e[i];
      int32_t* row = &p->h_tab[(size_t)g.seq * p->max_bps];
      e.seq = g.seq;
      e.prefix = g.prefix;
      e.q_len = g.q_len;
      e.q_off = g.q_off;
      e.nalloc_before = p->h_nalloc[g.seq];
      e.stack_before = p->h_top;
      e.lb_first = g.prefix / p->B;
      e.item_start = items;
      e.cow_old = -1;
      const int32_t end_blocks = cdiv((int64_t)g.prefix + g.q_len, p->B);
      for (int32_t lb = p->h_nalloc[g.seq]; lb < end_blocks; ++lb) {
        const int32_t nb = p->h_free[--p->h_top];
        p->h_ref[nb] = 1;
        row[lb] = nb;
      }
      p->h_nalloc[g.seq] = std::max(p->h_nalloc[g.seq], end_blocks);
      for (int32_t lb = e.lb_first; lb < end_blocks; ++lb) a.ids[items++] = row[lb];
    }
    a.n_items = items;
    a.top_after = p->h_top;
    hipError_t err = launch_fused_append(a, st);
    if (err != hipSuccess) return hip_fail(err, "restore + append launch");
  }
  // Reserve + append, chunked; the mirror takes the same pops in call order.
  for (size_t base = 0; !fold && base < segs.size(); base += kMaxSeqsPerLaunch) {
    const int32_t cnt = (int32_t)std::min<size_t>(kMaxSeqsPerLaunch, segs.size() - base);
    AppendArgs a{};
    a.k_cache = p->k_cache;
    a.v_cache = p->v_cache;
    a.k_in = k;
    a.v_in = v;
    a.tables = p->tables;
    a.lens = p->lens;
    a.free_list = p->free_list;
    a.free_top = p->free_top;
    a.refs = p->refs;
    a.chk = p->chk;
    a.max_bps = p->max_bps;
    a.n_blocks = p->n_blocks;
    a.n_kv_heads = p->hkv;
    a.block_size = p->B;
    a.head_dim = p->d;
    a.layer = layer;
    a.n_layers = p->n_layers;
    a.commit = commit ? 1 : 0;
    a.k_scale = p->k_scale[layer];
    a.v_scale = p->v_scale[layer];
    a.n = cnt;
    int32_t items = 0;
    for (int32_t i = 0; i < cnt; ++i) {
      const Seg& g = segs[base + i];
      AppendEntry& e = a.e[i];
      int32_t* row = &p->h_tab[(size_t)g.seq * p->max_bps];
      e.seq = g.seq;
      e.prefix = g.prefix;
      e.q_len = g.q_len;
      e.q_off = g.q_off;
      e.nalloc_before = p->h_nalloc[g.seq];
      e.stack_before = p->h_top;
      e.lb_first = g.prefix / p->B;
      e.item_start = items;
      e.cow_old = -1;
      const int32_t end_blocks = cdiv((int64_t)g.prefix + g.q_len, p->B);
      items += end_blocks - e.lb_first;
      if (shared_tail(p, g.seq, g.prefix, g.q_len)) {   // private copy first
        e.cow_old = row[e.lb_first];
        const int32_t nb = p->h_free[--p->h_top];
        --p->h_ref[e.cow_old];
        p->h_ref[nb] = 1;
        row[e.lb_first] = nb;
      }
      for (int32_t lb = p->h_nalloc[g.seq]; lb < end_blocks; ++lb) {
        const int32_t nb = p->h_free[--p->h_top];
        p->h_ref[nb] = 1;
        row[lb] = nb;
      }
      p->h_nalloc[g.seq] = std::max(p->h_nalloc[g.seq], end_blocks);
    }
    a.n_items = items;
    a.write_top = 1;
    a.top_after = p->h_top;
    hipError_t err = launch_append(a, eb, st);
    if (err != hipSuccess) return hip_fail(err, "append launch");
  }

  if (p->timing) {
    hipError_t err = hipEventRecord(p->ev[1], st);
    if (err == hipSuccess) err = hipEventRecord(p->ev[2], st);
    if (err != hipSuccess) return hip_fail(err, "timing event");
  }
  // Attention, chunked; within a launch, costlier sequences first.
  const int group = p->hq / p->hkv;
  // Decode path: every sequence's queries fit one wave (32 / G tokens) and the
  // pool has a workspace (so batching already decides the rounding order).
  bool decode = p->dtype != PGSR_F32 && ws_bytes > 0;
  for (const Seg& g : segs) decode = decode && g.q_len <= 32 / group;
  int64_t max_kv = 0;
  for (const Seg& g : segs) max_kv = std::max<int64_t>(max_kv, (int64_t)g.prefix + g.q_len);
  const bool wide = p->dtype == PGSR_BF16 && p->prefill_kind == PGSR_PREFILL_AUTO &&
                    attn_bf16_wide_eligible(p->d, group, p->B, p->n_blocks, p->hkv, max_kv);
  const bool pipe = !wide && p->dtype == PGSR_BF16 &&
                    (p->prefill_kind == PGSR_PREFILL_AUTO || p->prefill_kind == PGSR_PREFILL_PIPELINED) &&
                    attn_bf16_pipe_eligible(p->d, group);
  const int tile_tokens = p->dtype == PGSR_F32 ? attn_f32_tile_tokens(p->d, group)
                          : wide || pipe       ? attn_bf16_pipe_tile_tokens(group)
                                               : attn_bf16_tile_tokens(p->d, group);
  for (size_t base = 0; base < segs.size(); base += kMaxSeqsPerLaunch) {
    const int32_t cnt = (int32_t)std::min<size_t>(kMaxSeqsPerLaunch, segs.size() - base);
    std::vector<Seg> chunk(segs.begin() + base, segs.begin() + base + cnt);
    std::stable_sort(chunk.begin(), chunk.end(), [](const Seg& x, const Seg& y) {
      const double cx = (double)x.q_len * (x.prefix + 0.5 * x.q_len);
      const double cy = (double)y.q_len * (y.prefix + 0.5 * y.q_len);
      return cx > cy;
    });
    AttnArgs a{};
    a.q = q;
    a.o = o;
    a.k_cache = p->k_cache;
    a.v_cache = p->v_cache;
    a.tables = p->tables;
    a.chk = p->chk;
    a.max_bps = p->max_bps;
    a.n_blocks = p->n_blocks;
    a.n_q_heads = p->hq;
    a.n_kv_heads = p->hkv;
    a.block_size = p->B;
    a.head_dim = p->d;
    a.layer = layer;
    a.scale_log2 = (float)((double)scale * 1.4426950408889634 * (double)p->k_scale[layer]);
    a.o_scale = p->v_scale[layer];
    a.n = cnt;
    int32_t tiles = 0;
    for (int32_t i = 0; i < cnt; ++i) {
      a.e[i].seq = chunk[i].seq;
      a.e[i].prefix = chunk[i].prefix;
      a.e[i].q_len = chunk[i].q_len;
      a.e[i].q_off = chunk[i].q_off;
      a.e[i].tile_start = tiles;
      tiles += cdiv(chunk[i].q_len, tile_tokens);
    }
    a.n_tiles = tiles;
    a.n_splits = 1;
    a.split_len = 0;
    a.n_rows = off * p->hq;                        // packed query rows of the whole call
    // this launch's sequences are consecutive in call order, so their rows
    // form one contiguous run of the packed queries
    a.row_begin = segs[base].q_off * p->hq;
    a.row_end = (segs[base + cnt - 1].q_off + segs[base + cnt - 1].q_len) * p->hq;
    if (decode) {
      int32_t max_key = 0;
      for (int32_t i = 0; i < cnt; ++i) max_key = std::max(max_key, chunk[i].prefix + chunk[i].q_len);
      const int64_t units = (int64_t)cnt * p->hkv;
      const int64_t per_split = (int64_t)a.n_rows * ((int64_t)p->d + 2) * (int64_t)sizeof(float);
      int64_t ns = (kDecodeTargetWaves + units - 1) / units;
      ns = std::min<int64_t>(ns, kDecodeMaxSplits);
      ns = std::min<int64_t>(ns, std::max<int64_t>(1, max_key / kDecodeMinSplitKeys));
      ns = std::min<int64_t>(ns, (int64_t)(ws_bytes / std::max<int64_t>(per_split, 1)));
      if (ns > 1) {
        const int32_t kt = attn_decode_keys_per_tile();
        const int32_t len = cdiv(cdiv(max_key, ns), kt) * kt;
        a.n_splits = cdiv(max_key, len);
        a.split_len = len;
        a.ws_acc = (float*)ws;
        a.ws_ml = a.ws_acc + (int64_t)a.n_splits * a.n_rows * p->d;
      }
      hipError_t err = launch_attn_decode(a, p->dtype == PGSR_FP8_E4M3, st);
      if (err == hipSuccess && a.n_splits > 1) err = launch_split_combine(a, false, st);
      if (err != hipSuccess) return hip_fail(err, "decode attention launch");
      continue;
    }
    // Split-key mode when the launch would leave CUs idle and the caller gave
    // a workspace for the partials: splits at absolute multiples of split_len.
    // (the bf16 kernel packs a KV head's query heads into one workgroup, the
    // fp32 kernel takes one query head per workgroup)
    const int64_t wgs = (int64_t)tiles * (p->dtype == PGSR_F32 ? p->hq : p->hkv);
    const int64_t target = wide || pipe ? kSplitTargetWorkgroupsPipe : kSplitTargetWorkgroups;
    if (ws_bytes > 0 && wgs < target) {
      int32_t max_key = 0;
      for (int32_t i = 0; i < cnt; ++i) max_key = std::max(max_key, chunk[i].prefix + chunk[i].q_len);
      const int64_t per_split = (int64_t)a.n_rows * ((int64_t)p->d + 2) * (int64_t)sizeof(float);
      int64_t ns = std::min<int64_t>(kMaxSplits, (target + wgs - 1) / wgs);
      ns = std::min<int64_t>(ns, (int64_t)(ws_bytes / std::max<int64_t>(per_split, 1)));
      if (ns > 1) {
        const int32_t len = cdiv(cdiv(max_key, ns), kSplitAlign) * kSplitAlign;
        a.n_splits = cdiv(max_key, len);
        a.split_len = len;
        a.ws_acc = (float*)ws;
        a.ws_ml = a.ws_acc + (int64_t)a.n_splits * a.n_rows * p->d;
      }
    }
    if (p->timing && p->clk && (wide || pipe)) {
      hipError_t err = hipMemsetAsync(p->clk, 0, (size_t)p->clk_n * 4 * sizeof(uint64_t), st);
      if (err != hipSuccess) return hip_fail(err, "clock probe reset");
      a.clk = p->clk;
      a.clk_n = p->clk_n;
      p->clk_written = true;
    }
    hipError_t err = p->dtype == PGSR_F32    ? launch_attn_f32(a, st)
                     : wide                  ? launch_attn_bf16_wide(a, st)
                     : pipe                  ? launch_attn_bf16_pipe(a, st)
                     : p->dtype == PGSR_BF16 ? launch_attn_bf16(a, st)
                                             : launch_attn_fp8(a, st);
    if (err == hipSuccess && a.n_splits > 1) err = launch_split_combine(a, p->dtype == PGSR_F32, st);
    if (err != hipSuccess) return hip_fail(err, "attention launch");
  }

  if (p->timing) {
    hipError_t err = hipEventRecord(p->ev[3], st);
    if (err != hipSuccess) return hip_fail(err, "timing event");
    p->timed_call = true;
  }
  if (commit) {
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
      p->h_len[seqs[i]] += q_lens[i];
      total += q_lens[i];
    }
    if (recomputed) *recomputed += total;
  }
  return PGSR_OK;
}

// Restore (crop seqs[i] to crop_lens[i]; none when crop_lens is null) then the
// replay of q_lens on `layer`, validated together on the mirror before anything
// is launched.  The crop's device work rides in the append launch when that
// launch covers it: a bf16 pool with a fused kernel for its geometry, at most
// kMaxFusedSeqs sequences and kMaxFusedItems appended blocks, every sequence
// with work, and no kept partial tail block named by another row (so no
// copy-on-write).  Otherwise the crop is its own launch first.
int restore_replay(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                   const int32_t* crop_lens, const int32_t* q_lens, const void* q, const void* k,
                   const void* v, void* o, float scale, unsigned flags, int64_t* recomputed,
                   hipStream_t st) {
  int rc = check_seqs(p, n, seqs);
  if (rc) return rc;
  std::vector<int32_t> prefix(n), nalloc(n);
  int64_t free_after = p->h_top;
  if (crop_lens) {
    for (int32_t i = 0; i < n; ++i) {
      const int32_t L = crop_lens[i], len = p->h_len[seqs[i]];
      if (L < 0 || L > len)
        return fail(PGSR_ERANGE, "crop of sequence %d to %d tokens; it holds %d", seqs[i], L, len);
    }
    free_after += count_freed(p, n, seqs, crop_lens);
  }
  for (int32_t i = 0; i < n; ++i) {
    prefix[i] = crop_lens ? crop_lens[i] : p->h_len[seqs[i]];
    nalloc[i] = crop_lens ? cdiv(crop_lens[i], p->B) : p->h_nalloc[seqs[i]];
  }
  rc = check_replay(p, layer, n, seqs, q_lens, q, k, v, o, prefix, nalloc, (int32_t)free_after, scale);
  if (rc) return rc;
  if (!crop_lens || n == 0)
    return do_replay(p, layer, n, seqs, q_lens, q, k, v, o, scale, flags, recomputed, p->workspace,
                     p->workspace_bytes, st);
  bool fold = p->dtype == PGSR_BF16 && fused_append_supported(p->B, p->d) && n <= kMaxFusedSeqs;
  int64_t items = 0;
  for (int32_t i = 0; fold && i < n; ++i) {
    const int32_t L = crop_lens[i], S = q_lens[i];
    if (S <= 0) fold = false;
    items += cdiv((int64_t)L + S, p->B) - L / p->B;
    if (L % p->B != 0) {   // the kept partial tail block must be this row's alone
      const int32_t b = p->h_tab[(size_t)seqs[i] * p->max_bps + L / p->B];
      if (b < 0 || p->h_ref[b] != 1) fold = false;
    }
  }
  if (items > kMaxFusedItems) fold = false;
  if (!fold) {
    rc = do_crop(p, n, seqs, crop_lens, 0, st);
    if (rc) return rc;
    return do_replay(p, layer, n, seqs, q_lens, q, k, v, o, scale, flags, recomputed, p->workspace,
                     p->workspace_bytes, st);
  }
  FoldedCrop fc;
  fc.n = n;
  fc.top_before = p->h_top;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = seqs[i], L = crop_lens[i];
    CropEntry& e = fc.e[i];
    e.seq = s;
    e.new_len = L;
    e.keep = cdiv(L, p->B);
    e.nalloc = p->h_nalloc[s];
    mirror_crop(p, s, L);
    e.tail_private = 0;
  }
  return do_replay(p, layer, n, seqs, q_lens, q, k, v, o, scale, flags, recomputed, p->workspace,
                   p->workspace_bytes, st, &fc);
}

}  // namespace


namespace pgsr {
void set_error(const char* msg) { g_err = msg; }
void clear_error() { g_err.clear(); }
}  // namespace pgsr

extern "C" {

const char* pgsr_last_error(void) { return g_err.c_str(); }

int pgsr_abi_version(void) { return 2; }

int pgsr_pool_create(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                     int32_t block_size, int32_t dtype, int32_t n_blocks, int32_t max_seqs,
                     int32_t max_blocks_per_seq, void* k_cache, void* v_cache,
                     int32_t* block_tables, int32_t* seq_lens, int32_t* free_list,
                     int32_t* free_top, int32_t* ref_counts, void* workspace,
                     size_t workspace_bytes, const int32_t* init_free_order, void* stream,
                     pgsr_pool** out) {
  if (!out) return fail(PGSR_EINVAL, "out is null");
  *out = nullptr;
  if (n_layers <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_blocks <= 0 || max_seqs <= 0 ||
      max_blocks_per_seq <= 0)
    return fail(PGSR_EINVAL, "sizes must be positive");
  if (n_q_heads % n_kv_heads != 0)
    return fail(PGSR_EUNSUPPORTED, "n_q_heads %d is not a multiple of n_kv_heads %d", n_q_heads,
                n_kv_heads);
  if (dtype != PGSR_F32 && dtype != PGSR_BF16 && dtype != PGSR_FP8_E4M3)
    return fail(PGSR_EUNSUPPORTED, "dtype %d", dtype);
  if (head_dim != 64 && head_dim != 128)
    return fail(PGSR_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16 && block_size != 32 && block_size != 64)
    return fail(PGSR_EUNSUPPORTED, "block_size %d (supported: 16, 32, 64)", block_size);
  const int group = n_q_heads / n_kv_heads;
  if (dtype != PGSR_F32 && group > 32)
    return fail(PGSR_EUNSUPPORTED, "bf16 and fp8 kernels need n_q_heads / n_kv_heads <= 32");
  if ((int64_t)max_seqs * max_blocks_per_seq > INT32_MAX)
    return fail(PGSR_ERANGE, "block table larger than 2^31-1 entries");
  if (!k_cache || !v_cache || !block_tables || !seq_lens || !free_list || !free_top || !ref_counts)
    return fail(PGSR_EINVAL, "null device pointer");
  if (workspace == nullptr) workspace_bytes = 0;
  if (init_free_order) {
    std::vector<char> seen(n_blocks, 0);
    for (int32_t i = 0; i < n_blocks; ++i) {
      const int32_t id = init_free_order[i];
      if (id < 0 || id >= n_blocks || seen[id])
        return fail(PGSR_EINVAL, "init_free_order is not a permutation of 0..%d", n_blocks - 1);
      seen[id] = 1;
    }
  }
  hipStream_t st = (hipStream_t)stream;
  hipError_t err = launch_pool_init(block_tables, (int64_t)max_seqs * max_blocks_per_seq,
                                    seq_lens, max_seqs, init_free_order ? nullptr : free_list,
                                    n_blocks, free_top, ref_counts, st);
  if (err != hipSuccess) return hip_fail(err, "pool init launch");
  if (init_free_order) {
    err = hipMemcpyAsync(free_list, init_free_order, sizeof(int32_t) * n_blocks,
                         hipMemcpyHostToDevice, st);
    if (err != hipSuccess) return hip_fail(err, "copy of init_free_order");
  }
  err = hipStreamSynchronize(st);
  if (err != hipSuccess) return hip_fail(err, "pool init");
  pgsr_pool* p = new pgsr_pool{};
  p->n_layers = n_layers;
  p->hq = n_q_heads;
  p->hkv = n_kv_heads;
  p->d = head_dim;
  p->B = block_size;
  p->dtype = dtype;
  p->n_blocks = n_blocks;
  p->max_seqs = max_seqs;
  p->max_bps = max_blocks_per_seq;
  p->k_cache = k_cache;
  p->v_cache = v_cache;
  p->tables = block_tables;
  p->lens = seq_lens;
  p->free_list = free_list;
  p->free_top = free_top;
  p->refs = ref_counts;
  p->k_scale.assign(n_layers, 1.f);
  p->v_scale.assign(n_layers, 1.f);
  p->workspace = workspace;
  p->workspace_bytes = workspace_bytes;
  p->h_len.assign(max_seqs, 0);
  p->h_nalloc.assign(max_seqs, 0);
  p->h_tab.assign((size_t)max_seqs * max_blocks_per_seq, -1);
  p->h_free.resize(n_blocks);
  for (int32_t i = 0; i < n_blocks; ++i)
    p->h_free[i] = init_free_order ? init_free_order[i] : n_blocks - 1 - i;
  p->h_ref.assign(n_blocks, 0);
  p->h_top = n_blocks;
#ifdef PGSR_CHECKED
  err = hipMalloc((void**)&p->chk, sizeof(int32_t));
  if (err == hipSuccess) err = hipMemset(p->chk, 0, sizeof(int32_t));
  if (err != hipSuccess) {
    (void)hipFree(p->chk);
    delete p;
    return hip_fail(err, "checked build: flag allocation");
  }
#endif
  *out = p;
  return ok();
}

int pgsr_pool_destroy(pgsr_pool* pool) {
  if (pool) {
    for (hipEvent_t& e : pool->ev)
      if (e) (void)hipEventDestroy(e);
    if (pool->chk) (void)hipFree(pool->chk);
  }
  delete pool;
  return ok();
}

int pgsr_pool_set_kv_scales(pgsr_pool* p, const float* k_scales, const float* v_scales) {
  if (!p || !k_scales || !v_scales) return fail(PGSR_EINVAL, "null argument");
  if (p->dtype != PGSR_FP8_E4M3) return fail(PGSR_EINVAL, "KV scales apply to an FP8 pool only");
  for (int32_t l = 0; l < p->n_layers; ++l)
    for (const float x : {k_scales[l], v_scales[l]})
      if (!(x >= FLT_MIN && x <= FLT_MAX))
        return fail(PGSR_EINVAL, "scale of layer %d is not a positive normal float", l);
  p->k_scale.assign(k_scales, k_scales + p->n_layers);
  p->v_scale.assign(v_scales, v_scales + p->n_layers);
  return ok();
}

int pgsr_pool_enable_timing(pgsr_pool* p, int on) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (on && !p->ev[0]) {
    for (hipEvent_t& e : p->ev) {
      hipError_t err = hipEventCreate(&e);
      if (err != hipSuccess) return hip_fail(err, "hipEventCreate");
    }
  }
  p->timing = on != 0;
  p->timed_call = false;
  return ok();
}

int pgsr_pool_set_prefill_kernel(pgsr_pool* p, int kind) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (kind != PGSR_PREFILL_AUTO && kind != PGSR_PREFILL_FOUR_WAVE && kind != PGSR_PREFILL_PIPELINED)
    return fail(PGSR_EINVAL, "unknown prefill kernel %d", kind);
  p->prefill_kind = kind;
  return ok();
}

int pgsr_pool_last_times(pgsr_pool* p, float* append_ms, float* attention_ms) {
  if (!p || !append_ms || !attention_ms) return fail(PGSR_EINVAL, "null argument");
  if (!p->timed_call) return fail(PGSR_EINVAL, "no timed call since timing was enabled");
  hipError_t err = hipEventSynchronize(p->ev[3]);
  if (err == hipSuccess) err = hipEventElapsedTime(append_ms, p->ev[0], p->ev[1]);
  if (err == hipSuccess) err = hipEventElapsedTime(attention_ms, p->ev[2], p->ev[3]);
  if (err != hipSuccess) return hip_fail(err, "event timing");
  return ok();
}

int pgsr_pool_set_clock_buffer(pgsr_pool* p, void* buf, size_t bytes) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  const size_t n = buf ? bytes / (4 * sizeof(uint64_t)) : 0;
  p->clk = n ? (uint64_t*)buf : nullptr;
  p->clk_n = (int32_t)std::min<size_t>(n, INT32_MAX);
  p->clk_written = false;
  return ok();
}

int pgsr_pool_last_clock(pgsr_pool* p, void* stream, double* ghz, int64_t* cycles, int64_t* ticks) {
  if (!p || !ghz) return fail(PGSR_EINVAL, "null argument");
  if (!p->clk || !p->clk_written) return fail(PGSR_EINVAL, "no timed launch wrote the clock probe");
  std::vector<uint64_t> h((size_t)p->clk_n * 4);
  hipStream_t st = (hipStream_t)stream;
  hipError_t err = hipMemcpyAsync(h.data(), p->clk, h.size() * sizeof(uint64_t), hipMemcpyDeviceToHost, st);
  if (err == hipSuccess) err = hipStreamSynchronize(st);
  int dev = 0, khz = 0;
  if (err == hipSuccess) err = hipGetDevice(&dev);
  if (err == hipSuccess) err = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
  if (err != hipSuccess) return hip_fail(err, "clock probe read-back");
  uint64_t cyc = 0, tck = 0;
  for (int32_t b = 0; b < p->clk_n; ++b) {
    const uint64_t* c = &h[4 * (size_t)b];
    if (c[3] > c[2] && c[1] > c[0]) {
      cyc += c[1] - c[0];
      tck += c[3] - c[2];
    }
  }
  if (tck == 0 || khz <= 0) return fail(PGSR_EINVAL, "the clock probe holds no workgroup");
  *ghz = (double)cyc / (double)tck * (double)khz * 1e3 / 1e9;
  if (cycles) *cycles = (int64_t)cyc;
  if (ticks) *ticks = (int64_t)tck;
  return ok();
}

int pgsr_pool_refresh(pgsr_pool* p, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  hipStream_t st = (hipStream_t)stream;
  std::vector<int32_t> tables((size_t)p->max_seqs * p->max_bps), lens(p->max_seqs);
  std::vector<int32_t> free_list(p->n_blocks), refs(p->n_blocks);
  int32_t top = 0;
  hipError_t err = hipMemcpyAsync(tables.data(), p->tables, tables.size() * 4,
                                  hipMemcpyDeviceToHost, st);
  if (err == hipSuccess)
    err = hipMemcpyAsync(lens.data(), p->lens, lens.size() * 4, hipMemcpyDeviceToHost, st);
  if (err == hipSuccess)
    err = hipMemcpyAsync(free_list.data(), p->free_list, free_list.size() * 4, hipMemcpyDeviceToHost, st);
  if (err == hipSuccess)
    err = hipMemcpyAsync(refs.data(), p->refs, refs.size() * 4, hipMemcpyDeviceToHost, st);
  if (err == hipSuccess) err = hipMemcpyAsync(&top, p->free_top, 4, hipMemcpyDeviceToHost, st);
  if (err == hipSuccess) err = hipStreamSynchronize(st);
  if (err != hipSuccess) return hip_fail(err, "refresh copy");
  if (top < 0 || top > p->n_blocks) return fail(PGSR_ERANGE, "device free_top %d invalid", top);
  std::vector<int32_t> nalloc(p->max_seqs);
  for (int32_t s = 0; s < p->max_seqs; ++s) {
    int32_t na = 0;
    while (na < p->max_bps && tables[(size_t)s * p->max_bps + na] >= 0) ++na;
    if (lens[s] < 0 || cdiv(lens[s], p->B) > na)
      return fail(PGSR_ERANGE, "device length %d of sequence %d exceeds its blocks", lens[s], s);
    for (int32_t j = 0; j < na; ++j)
      if (tables[(size_t)s * p->max_bps + j] >= p->n_blocks)
        return fail(PGSR_ERANGE, "device table of sequence %d names block %d", s,
                    tables[(size_t)s * p->max_bps + j]);
    nalloc[s] = na;
  }
  p->h_nalloc = nalloc;
  p->h_len = lens;
  p->h_tab = tables;
  p->h_free = free_list;
  p->h_ref = refs;
  p->h_top = top;
  return ok();
}

int pgsr_seq_len(const pgsr_pool* p, int32_t seq, int32_t* len_out) {
  if (!p || !len_out) return fail(PGSR_EINVAL, "null argument");
  if (seq < 0 || seq >= p->max_seqs) return fail(PGSR_EINVAL, "sequence id %d", seq);
  *len_out = p->h_len[seq];
  return ok();
}

int pgsr_free_blocks(const pgsr_pool* p, int32_t* n_out) {
  if (!p || !n_out) return fail(PGSR_EINVAL, "null argument");
  *n_out = p->h_top;
  return ok();
}

size_t pgsr_workspace_bytes(int32_t n_q_heads, int32_t head_dim, int64_t max_total_q,
                            int32_t max_splits) {
  if (n_q_heads <= 0 || head_dim <= 0 || max_total_q <= 0 || max_splits <= 1) return 0;
  return (size_t)max_total_q * n_q_heads * max_splits * ((size_t)head_dim + 2) * sizeof(float);
}

int pgsr_kv_crop(pgsr_pool* p, int32_t n, const int32_t* seqs, const int32_t* new_lens,
                 unsigned flags, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (n < 0) return fail(PGSR_EINVAL, "n = %d", n);
  if (n == 0) return ok();
  if (!seqs || !new_lens) return fail(PGSR_EINVAL, "null seqs / new_lens");
  if (flags & ~(unsigned)PGSR_POISON) return fail(PGSR_EINVAL, "unknown crop flags 0x%x", flags);
  int rc = check_seqs(p, n, seqs);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t L = new_lens[i], len = p->h_len[seqs[i]];
    if (L < 0 || L > len)
      return fail(PGSR_ERANGE, "crop of sequence %d to %d tokens; it holds %d", seqs[i], L, len);
  }
  rc = do_crop(p, n, seqs, new_lens, flags, (hipStream_t)stream);
  if (!rc) rc = device_check(p, (hipStream_t)stream);
  return rc ? rc : ok();
}

int pgsr_kv_fork(pgsr_pool* p, int32_t n, const int32_t* srcs, const int32_t* dsts, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (n < 0) return fail(PGSR_EINVAL, "n = %d", n);
  if (n == 0) return ok();
  if (!srcs || !dsts) return fail(PGSR_EINVAL, "null srcs / dsts");
  int rc = check_seqs(p, n, dsts);
  if (rc) return rc;
  std::vector<char> is_dst(p->max_seqs, 0);
  for (int32_t i = 0; i < n; ++i) is_dst[dsts[i]] = 1;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = srcs[i], d = dsts[i];
    if (s < 0 || s >= p->max_seqs) return fail(PGSR_EINVAL, "source sequence id %d", s);
    if (is_dst[s]) return fail(PGSR_EINVAL, "sequence %d is both a source and a target", s);
    if (p->h_len[d] != 0 || p->h_nalloc[d] != 0)
      return fail(PGSR_EINVAL, "target sequence %d is not empty", d);
  }
  hipStream_t st = (hipStream_t)stream;
  for (int32_t base = 0; base < n; base += kMaxSeqsPerLaunch) {
    const int32_t cnt = std::min<int32_t>(kMaxSeqsPerLaunch, n - base);
    ForkArgs a{};
    a.tables = p->tables;
    a.lens = p->lens;
    a.refs = p->refs;
    a.chk = p->chk;
    a.max_bps = p->max_bps;
    a.n_blocks = p->n_blocks;
    a.n = cnt;
    for (int32_t i = 0; i < cnt; ++i) {
      const int32_t s = srcs[base + i], d = dsts[base + i];
      a.e[i] = {s, d, p->h_nalloc[s], p->h_len[s]};
      for (int32_t j = 0; j < p->h_nalloc[s]; ++j) {
        const int32_t b = p->h_tab[(size_t)s * p->max_bps + j];
        p->h_tab[(size_t)d * p->max_bps + j] = b;
        ++p->h_ref[b];
      }
      p->h_nalloc[d] = p->h_nalloc[s];
      p->h_len[d] = p->h_len[s];
    }
    hipError_t err = launch_fork(a, st);
    if (err != hipSuccess) return hip_fail(err, "fork launch");
  }
  rc = device_check(p, st);
  return rc ? rc : ok();
}

int pgsr_replay_prefill(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                        const int32_t* q_lens, const void* q, const void* k, const void* v,
                        void* o, float softmax_scale, unsigned flags,
                        int64_t* recomputed_tokens, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  return replay_prefill_ws(p, layer, n, seqs, q_lens, q, k, v, o, softmax_scale, flags,
                           recomputed_tokens, p->workspace, p->workspace_bytes, stream);
}

}  // extern "C"

namespace pgsr {

int replay_prefill_ws(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                      const int32_t* q_lens, const void* q, const void* k, const void* v, void* o,
                      float softmax_scale, unsigned flags, int64_t* recomputed_tokens, void* ws,
                      size_t ws_bytes, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (n < 0) return fail(PGSR_EINVAL, "n = %d", n);
  if (flags & ~(unsigned)PGSR_COMMIT) return fail(PGSR_EINVAL, "unknown replay flags 0x%x", flags);
  if (n > 0 && (!seqs || !q_lens)) return fail(PGSR_EINVAL, "null seqs / q_lens");
  int rc = check_seqs(p, n, seqs);
  if (rc) return rc;
  std::vector<int32_t> prefix(n), nalloc(n);
  for (int32_t i = 0; i < n; ++i) {
    prefix[i] = p->h_len[seqs[i]];
    nalloc[i] = p->h_nalloc[seqs[i]];
  }
  rc = check_replay(p, layer, n, seqs, q_lens, q, k, v, o, prefix, nalloc, p->h_top,
                    softmax_scale);
  if (rc) return rc;
  rc = do_replay(p, layer, n, seqs, q_lens, q, k, v, o, softmax_scale, flags, recomputed_tokens, ws,
                 ws_bytes, (hipStream_t)stream);
  if (!rc) rc = device_check(p, (hipStream_t)stream);
  return rc ? rc : ok();
}

int fail_with(int code, const char* msg) { return fail(code, "%s", msg); }

}  // namespace pgsr

extern "C" {

int pgsr_full_reset_prefill(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                            const int32_t* lens, const void* q, const void* k, const void* v,
                            void* o, float softmax_scale, unsigned flags,
                            int64_t* recomputed_tokens, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (n < 0) return fail(PGSR_EINVAL, "n = %d", n);
  if (flags & ~(unsigned)PGSR_COMMIT) return fail(PGSR_EINVAL, "unknown replay flags 0x%x", flags);
  if (n > 0 && (!seqs || !lens)) return fail(PGSR_EINVAL, "null seqs / lens");
  // layer 0: restore every sequence to 0 tokens, then replay the whole trajectory
  std::vector<int32_t> zeros(n, 0);
  int rc = restore_replay(p, layer, n, seqs, layer == 0 ? zeros.data() : nullptr, lens, q, k, v, o,
                          softmax_scale, flags, recomputed_tokens, (hipStream_t)stream);
  if (!rc) rc = device_check(p, (hipStream_t)stream);
  return rc ? rc : ok();
}

int pgsr_restore_replay_prefill(pgsr_pool* p, int32_t layer, int32_t n, const int32_t* seqs,
                                const int32_t* restore_lens, const int32_t* q_lens, const void* q,
                                const void* k, const void* v, void* o, float softmax_scale,
                                unsigned flags, int64_t* recomputed_tokens, void* stream) {
  if (!p) return fail(PGSR_EINVAL, "pool is null");
  if (n < 0) return fail(PGSR_EINVAL, "n = %d", n);
  if (flags & ~(unsigned)PGSR_COMMIT) return fail(PGSR_EINVAL, "unknown replay flags 0x%x", flags);
  if (n > 0 && (!seqs || !restore_lens || !q_lens)) return fail(PGSR_EINVAL, "null seqs / lens");
  int rc = restore_replay(p, layer, n, seqs, restore_lens, q_lens, q, k, v, o, softmax_scale, flags,
                          recomputed_tokens, (hipStream_t)stream);
  if (!rc) rc = device_check(p, (hipStream_t)stream);
  return rc ? rc : ok();
}

int pgsr_gemm_bf16(int32_t m, int32_t n, int32_t k, const void* x, const void* w, const void* r,
                   void* y, void* stream) {
  if (m < 0 || n < 0 || k < 0) return fail(PGSR_EINVAL, "negative size");
  if (n % 8 || k % 8) return fail(PGSR_EUNSUPPORTED, "n and k must be multiples of 8");
  if (m == 0 || n == 0) return ok();
  if (!x || !w || !y) return fail(PGSR_EINVAL, "null pointer");
  hipError_t err = launch_gemm_bf16(m, n, k, x, w, r, y, (hipStream_t)stream);
  if (err != hipSuccess) return hip_fail(err, "gemm launch");
  return ok();
}

// Vocabulary entries per sampling workgroup (a multiple of 4: Philox blocks
// never straddle two chunks).
constexpr int32_t kSampleChunk = 8192;

size_t pgsr_sample_workspace_bytes(int32_t n, int32_t vocab) {
  if (n <= 0 || vocab <= kSampleChunk) return 0;
  return (size_t)n * (size_t)cdiv(vocab, kSampleChunk) * sizeof(uint64_t);
}

int pgsr_sample_tokens(int32_t n, int32_t vocab, int32_t dtype, const void* logits, float temperature,
                       uint64_t seed, const int64_t* streams, const int64_t* positions, void* workspace,
                       size_t workspace_bytes, int32_t* tokens, void* stream) {
  if (n < 0 || vocab <= 0) return fail(PGSR_EINVAL, "n = %d, vocab = %d", n, vocab);
  if (dtype != PGSR_F32 && dtype != PGSR_BF16) return fail(PGSR_EUNSUPPORTED, "dtype %d", dtype);
  if (!(temperature >= 0.f) || temperature > 3.0e38f)
    return fail(PGSR_EINVAL, "temperature must be finite and >= 0");
  if (n == 0) return ok();
  if (!logits || !tokens || !streams || !positions) return fail(PGSR_EINVAL, "null pointer");
  const int32_t chunks = cdiv(vocab, kSampleChunk);
  const bool split = chunks > 1 && workspace &&
                     workspace_bytes >= (size_t)n * (size_t)chunks * sizeof(uint64_t);
  hipStream_t st = (hipStream_t)stream;
  SampleArgs a{};
  a.vocab = vocab;
  a.n_chunks = split ? chunks : 1;
  a.chunk_len = split ? kSampleChunk : ((vocab + 3) / 4) * 4;
  a.temperature = temperature;
  a.seed = seed;
  a.partial = split ? (uint64_t*)workspace : nullptr;
  for (int32_t r0 = 0; r0 < n; r0 += kMaxSeqsPerLaunch) {
    a.row0 = r0;
    a.n = std::min<int32_t>(kMaxSeqsPerLaunch, n - r0);
    for (int32_t i = 0; i < a.n; ++i) {
      a.stream[i] = streams[r0 + i];
      a.position[i] = positions[r0 + i];
    }
    hipError_t err = launch_sample(a, dtype, logits, tokens, st);
    if (err != hipSuccess) return hip_fail(err, "sample launch");
  }
  if (split) {
    hipError_t err = launch_sample_reduce(n, chunks, (const uint64_t*)workspace, tokens, st);
    if (err != hipSuccess) return hip_fail(err, "sample reduce launch");
  }
  return ok();
}

int pgsr_rmsnorm_bf16(int32_t n, int32_t d_model, const void* x, const void* gain, float eps, void* y,
                      void* stream) {
  if (n < 0 || d_model <= 0 || d_model % 8) return fail(PGSR_EINVAL, "n = %d, d_model = %d", n, d_model);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(PGSR_EINVAL, "eps must be finite and >= 0");
  if (n == 0) return ok();
  if (!x || !gain || !y) return fail(PGSR_EINVAL, "null pointer");
  hipError_t err = launch_rmsnorm(n, d_model, x, gain, eps, y, (hipStream_t)stream);
  return err == hipSuccess ? ok() : hip_fail(err, "rmsnorm launch");
}

int pgsr_rope_bf16(int32_t n, int32_t n_heads, int32_t head_dim, void* x, const int32_t* positions,
                   double theta, void* stream) {
  if (n < 0 || n_heads <= 0 || head_dim <= 0 || head_dim % 2)
    return fail(PGSR_EINVAL, "n = %d, heads = %d, head_dim = %d", n, n_heads, head_dim);
  if (!(theta > 1.0) || !std::isfinite(theta)) return fail(PGSR_EINVAL, "theta must be finite and > 1");
  if (n == 0) return ok();
  if (!x || !positions) return fail(PGSR_EINVAL, "null pointer");
  hipError_t err = launch_rope(n, n_heads, head_dim, x, positions, theta, (hipStream_t)stream);
  return err == hipSuccess ? ok() : hip_fail(err, "rope launch");
}

int pgsr_silu_mul_bf16(int32_t n, int32_t d_ff, const void* gate_up, void* out, void* stream) {
  if (n < 0 || d_ff <= 0 || d_ff % 8) return fail(PGSR_EINVAL, "n = %d, d_ff = %d", n, d_ff);
  if (n == 0) return ok();
  if (!gate_up || !out) return fail(PGSR_EINVAL, "null pointer");
  hipError_t err = launch_silu_mul(n, d_ff, gate_up, out, (hipStream_t)stream);
  return err == hipSuccess ? ok() : hip_fail(err, "silu_mul launch");
}

}  // extern "C"
