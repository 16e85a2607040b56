// Exact top-1 retrieval for callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc): precog_retrieve_top1 with its workspace taken from a fixed
// device array of this library instead of a caller-supplied buffer.
//
// `scratch` is a file-scope device array.  In host code its name is only a
// host-side stand-in for the symbol, not a device address, so host code never
// passes it to a kernel or a copy: on the first call on each device (with
// that device current) its device address is looked up once with
// hipGetSymbolAddress and kept per device, and every launch uses that
// address.  Each device holds its own copy of the array until the process
// ends.  Every call on one device shares that device's copy, so two calls
// that overlap on one device (different streams, no ordering between them)
// race on it.  The retrieval kernels write every workspace entry they read
// within the same call (query operands, screen scores, block maxima, key
// norms), so nothing needs clearing between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "precog.h"
#include "precog_kernels.h"

namespace {

static __device__ __align__(256) unsigned char scratch[PRECOG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, null until looked up

// Device address of the current device's `scratch`, looked up on the first
// call on that device.
precog_status scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return PRECOG_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return PRECOG_ERR_ARCH;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return PRECOG_ERR_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return PRECOG_OK;
}

}  // namespace

extern "C" {

precog_status precog_retrieve_top1_noalloc(const float* query_emb, const float* index_emb,
                                           int64_t Q, int64_t M, int64_t E, int32_t* idx,
                                           void* stream) {
  // reject what precog_retrieve_top1 rejects, and workspaces past the array,
  // before touching the device
  if (Q < 0 || M < 0 || E < 4 || E > 4096) return PRECOG_ERR_SHAPE;
  if (E % 4 != 0) return PRECOG_ERR_ALIGN;
  if (Q > 0x7fffffffLL || M > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if ((M + 31) / 32 * ((Q + 127) / 128) > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (Q == 0) return PRECOG_OK;
  const size_t need = precog_retrieve_workspace_bytes(Q, M, E);
  if (need > PRECOG_NOALLOC_SCRATCH_BYTES) return PRECOG_ERR_WORKSPACE;
  if (!query_emb || !idx || (M > 0 && !index_emb)) return PRECOG_ERR_NULL;
  void* ws = nullptr;
  const precog_status st = scratch_address(&ws);
  if (st != PRECOG_OK) return st;
  return precog::retrieve_entry(query_emb, index_emb, nullptr, Q, M, E, 1, idx, nullptr, ws,
                                PRECOG_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
