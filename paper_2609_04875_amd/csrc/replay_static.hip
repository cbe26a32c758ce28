// Replay prefill for callers that cannot allocate device memory (code under
// HIP graph capture, tight serving loops, harnesses that forbid allocation).
//
// The split-key and decode paths of the replay keep per-split partial softmax
// states (acc, m, l) in a workspace; pgsr_replay_prefill takes it from the
// pool (caller-allocated at pool creation).  This entry point runs the same
// call with the same kernels but puts the partials in `scratch`, a file-scope
// device array of PGSR_STATIC_SCRATCH_BYTES that every GPU the library runs
// on holds until the process ends.  Nothing is allocated per call.
//
// In host code the name `scratch` is a host-side stand-in, not a device
// address: its address on a device comes from hipGetSymbolAddress, taken once
// per device with that device current and kept in `g_scratch`; only that
// address is ever handed to a kernel.
//
// Every call on one GPU shares that GPU's array: calls whose work overlaps on
// one GPU (two streams, two host threads) race.  Nothing in it needs to start
// at zero: a split writes the partials of every query row it covers before
// the combine of the same call reads them, and the combine reads only splits
// that start at or before the row's position, which always cover it.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "internal.h"
#include "pgsr.h"

namespace {

constexpr size_t kScratchBytes = PGSR_STATIC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size");

static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};   // device address of `scratch`, per device

// Device of the stream the call runs on (the current device for the null
// stream), then the array's address there, resolved on first use with that
// device current.
int scratch_on_stream(hipStream_t st, void** out) {
  int dev = -1;
  hipError_t err = hipGetDevice(&dev);
  if (err == hipSuccess && st != nullptr) err = hipStreamGetDevice(st, &dev);
  if (err != hipSuccess) return pgsr::fail_with(PGSR_EHIP, hipGetErrorString(err));
  if (dev < 0 || dev >= kMaxDevices) return pgsr::fail_with(PGSR_EUNSUPPORTED, "device index past 63");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    int cur = -1;
    err = hipGetDevice(&cur);
    if (err == hipSuccess && cur != dev) err = hipSetDevice(dev);
    void* ptr = nullptr;
    if (err == hipSuccess) err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur >= 0 && cur != dev) {
      const hipError_t back = hipSetDevice(cur);
      if (err == hipSuccess) err = back;
    }
    if (err != hipSuccess || ptr == nullptr)
      return pgsr::fail_with(PGSR_EHIP, err != hipSuccess ? hipGetErrorString(err)
                                                          : "no device address for the static scratch");
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return PGSR_OK;
}

}  // namespace

extern "C" int pgsr_replay_prefill_static(pgsr_pool* pool, int32_t layer, int32_t n,
                                          const int32_t* seqs, const int32_t* q_lens, const void* q,
                                          const void* k, const void* v, void* o, float softmax_scale,
                                          unsigned flags, size_t scratch_bytes,
                                          int64_t* recomputed_tokens, void* stream) {
  if (!pool) return pgsr::fail_with(PGSR_EINVAL, "pool is null");
  if (scratch_bytes > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof msg, "scratch_bytes %zu exceeds the static scratch of %zu bytes", scratch_bytes,
             kScratchBytes);
    return pgsr::fail_with(PGSR_ERANGE, msg);
  }
  void* ws = nullptr;
  if (scratch_bytes > 0) {
    const int rc = scratch_on_stream((hipStream_t)stream, &ws);
    if (rc) return rc;
  }
  return pgsr::replay_prefill_ws(pool, layer, n, seqs, q_lens, q, k, v, o, softmax_scale, flags,
                                 recomputed_tokens, ws, scratch_bytes, stream);
}
