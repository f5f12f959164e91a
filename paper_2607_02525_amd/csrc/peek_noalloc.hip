// peek_queue_signals_noalloc: the queue signals with their scratch in a
// file-scope device array instead of a caller's workspace, for callers that
// cannot allocate device memory (code under graph capture, serving loops,
// harnesses that forbid hipMalloc).
//
// The array's name is a host-side stand-in in host code; its device address
// is looked up once per device with hipGetSymbolAddress and only that
// address is handed to the kernels. Every call on one device shares that
// device's array, so calls whose work overlaps on the device (different
// streams, or host threads racing) race on it; calls ordered on one stream
// are safe. Each call clears what its kernels expect zeroed, so what an
// earlier call left there is harmless.
#include <mutex>

#include "peek_internal.h"

namespace {

__device__ __align__(256) unsigned char scratch[PEEK_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];   // the array's device address, per device once looked up

// Address of the scratch array on the current device.
peek_status scratch_here(void** out) {
  int dev = 0;
  PEEK_HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return peek::fail(PEEK_ERR_UNSUPPORTED_DEVICE, "device %d is beyond the %d this library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return peek::fail(PEEK_ERR_DEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                        hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return PEEK_OK;
}

}  // namespace

extern "C" peek_status peek_queue_signals_noalloc(const peek_cache* c, int32_t n, const int32_t* d_tokens,
                                                  const int64_t* d_offsets, const int32_t* d_last_node,
                                                  const int32_t* d_match_len, int32_t threshold,
                                                  int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand,
                                                  void* stream) {
  return peek::guarded([&]() -> peek_status {
    peek::clear_error();
    if (n < 0) return peek::fail(PEEK_ERR_INVALID_ARGUMENT, "n must be >= 0 (got %d)", n);
    if (threshold < 1) return peek::fail(PEEK_ERR_INVALID_ARGUMENT, "threshold must be >= 1 (got %d)", threshold);
    const int64_t nn = c ? c->num_nodes : 0;
    const size_t need = peek::signals_workspace_bytes(n, nn);
    if (need > (size_t)PEEK_NOALLOC_SCRATCH_BYTES)
      return peek::fail(PEEK_ERR_WORKSPACE_TOO_SMALL,
                        "%d requests against %lld cache nodes need %zu bytes of scratch; the static scratch holds %zu "
                        "(use peek_queue_signals with a workspace)",
                        n, (long long)nn, need, (size_t)PEEK_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    const peek_status s = scratch_here(&ws);
    if (s != PEEK_OK) return s;
    return peek::signals_entry(c, n, d_tokens, d_offsets, d_last_node, d_match_len, threshold, d_cluster_id,
                               d_cluster_size, d_demand, nullptr, ws, PEEK_NOALLOC_SCRATCH_BYTES, stream, false);
  });
}
