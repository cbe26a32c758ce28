// Paged KV pool kernels: initial state, restore-by-crop (block-table truncation
// and compaction of the released ids onto the free-list stack), NaN poisoning
// of released slots, and the reserve + append step of a replay.
//
// All of this is integer bookkeeping and bit copies: results are exact and do
// not depend on the launch shape.  Work per call is tiny (a crop touches at
// most a few KB of int32), so these kernels are launch-latency bound; they are
// written for clarity and coalescing, not occupancy.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace pgsr {

namespace {

__global__ void __launch_bounds__(256)
pool_init_kernel(int32_t* tables, int64_t n_table, int32_t* lens, int32_t max_seqs,
                 int32_t* free_list, int32_t n_blocks, int32_t* free_top) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_table; i += stride)
    tables[i] = -1;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < max_seqs; i += stride)
    lens[i] = 0;
  if (free_list)  // default stack: bottom n_blocks-1 ... top 0, so pops yield 0, 1, 2, ...
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_blocks; i += stride)
      free_list[i] = n_blocks - 1 - (int32_t)i;
  if (blockIdx.x == 0 && threadIdx.x == 0) *free_top = n_blocks;
}

// One workgroup per cropped sequence.  Entries j >= keep of the row move onto
// the stack at top_before + push_off + (j - keep), in ascending j.
__global__ void __launch_bounds__(256) crop_kernel(CropArgs a) {
  const CropEntry e = a.e[blockIdx.x];
  int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
  const int32_t n_free = e.nalloc - e.keep;
  int32_t* dst = a.free_list + a.top_before + e.push_off;
  for (int32_t j = threadIdx.x; j < n_free; j += blockDim.x) {
    dst[j] = row[e.keep + j];
    row[e.keep + j] = -1;
  }
  if (threadIdx.x == 0) {
    a.lens[e.seq] = e.new_len;
    if (blockIdx.x == 0) *a.free_top = a.top_after;
  }
}

template <typename T>
__device__ void fill_nan(T* p, int64_t n, T nan, int tid, int nthreads) {
  for (int64_t i = tid; i < n; i += nthreads) p[i] = nan;
}

// blockIdx.x: entry; blockIdx.y: layer.  Runs after crop_kernel on the same stream.
template <typename T>
__global__ void __launch_bounds__(256) poison_kernel(PoisonArgs a, T nan) {
  const CropEntry e = a.e[blockIdx.x];
  const int layer = blockIdx.y;
  const int64_t blk_elems = (int64_t)a.n_kv_heads * a.block_size * a.head_dim;
  T* kc = (T*)a.k_cache + (int64_t)layer * a.n_blocks * blk_elems;
  T* vc = (T*)a.v_cache + (int64_t)layer * a.n_blocks * blk_elems;
  const int32_t n_free = e.nalloc - e.keep;
  for (int32_t j = 0; j < n_free; ++j) {
    const int32_t id = a.free_list[a.top_before + e.push_off + j];
    fill_nan(kc + (int64_t)id * blk_elems, blk_elems, nan, threadIdx.x, blockDim.x);
    fill_nan(vc + (int64_t)id * blk_elems, blk_elems, nan, threadIdx.x, blockDim.x);
  }
  const int32_t tail = e.new_len % a.block_size;
  if (tail != 0) {  // slots tail .. B-1 of the kept partial block
    const int32_t id = a.tables[(int64_t)e.seq * a.max_bps + e.keep - 1];
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

// Reserve + append.  blockIdx.x enumerates (sequence, logical block) items,
// blockIdx.y the KV head.  The physical id of a newly reserved logical block
// lb is read straight from the stack (free_list[stack_before - 1 - k] for the
// k-th new block of the sequence), so no workgroup depends on another's table
// write; the kv-head-0 workgroup records it in the table.
//   K: token p -> k_cache[layer][id][h][p % B][:]      (row copy)
//   V: token p -> v_cache[layer][id][h][:][p % B]      (transposed via LDS)
template <typename T>
__global__ void __launch_bounds__(256) append_kernel(AppendArgs a) {
  __shared__ T vstage[64 * 128];  // [slot][d], block_size <= 64, head_dim <= 128
  const int item = blockIdx.x;
  int ei = 0;
  while (ei + 1 < a.n && a.e[ei + 1].item_start <= item) ++ei;
  const AppendEntry e = a.e[ei];
  const int B = a.block_size, D = a.head_dim, h = blockIdx.y;
  const int32_t lb = e.lb_first + (item - e.item_start);
  int32_t* row = a.tables + (int64_t)e.seq * a.max_bps;
  int32_t id;
  if (lb < e.nalloc_before) {
    id = row[lb];
  } else {
    id = a.free_list[e.stack_before - 1 - (lb - e.nalloc_before)];
    if (h == 0 && threadIdx.x == 0) row[lb] = id;
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
  const T* kin = (const T*)a.k_in;
  const T* vin = (const T*)a.v_in;
  T* kc = (T*)a.k_cache + blk * B * D;
  T* vc = (T*)a.v_cache + blk * D * B;
  for (int i = threadIdx.x; i < nt * D; i += blockDim.x) {
    const int t = i / D, c = i % D;
    const int64_t src = ((int64_t)(e.q_off + (p0 - e.prefix) + t) * a.n_kv_heads + h) * D + c;
    kc[(int64_t)(s0 + t) * D + c] = kin[src];
    vstage[t * D + c] = vin[src];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nt * D; i += blockDim.x) {
    const int c = i / nt, t = i % nt;
    vc[(int64_t)c * B + s0 + t] = vstage[t * D + c];
  }
}

}  // namespace

hipError_t launch_pool_init(int32_t* tables, int64_t n_table, int32_t* lens, int32_t max_seqs,
                            int32_t* free_list, int32_t n_blocks, int32_t* free_top,
                            hipStream_t s) {
  int64_t biggest = n_table > n_blocks ? n_table : n_blocks;
  if (max_seqs > biggest) biggest = max_seqs;
  int grid = (int)((biggest + 255) / 256);
  if (grid > 4096) grid = 4096;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL(pool_init_kernel, dim3(grid), dim3(256), 0, s, tables, n_table, lens,
                     max_seqs, free_list, n_blocks, free_top);
  return hipGetLastError();
}

hipError_t launch_crop(const CropArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(crop_kernel, dim3(a.n), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_poison(const PoisonArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.elem_bytes == 4)
    hipLaunchKernelGGL(poison_kernel<uint32_t>, dim3(a.n, a.n_layers), dim3(256), 0, s, a,
                       (uint32_t)0x7FC00000u);
  else
    hipLaunchKernelGGL(poison_kernel<uint16_t>, dim3(a.n, a.n_layers), dim3(256), 0, s, a,
                       (uint16_t)0x7FC0u);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, int elem_bytes, hipStream_t s) {
  if (a.n <= 0 || a.n_items <= 0) return hipSuccess;
  dim3 grid(a.n_items, a.n_kv_heads);
  if (elem_bytes == 4)
    hipLaunchKernelGGL(append_kernel<uint32_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(append_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace pgsr
