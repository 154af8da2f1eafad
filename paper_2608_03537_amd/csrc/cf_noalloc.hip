// Allocation-free variant of cf_gemm_subgraph, for callers that cannot
// allocate device memory (code under stream capture, tight serving loops).
//
// The only scratch the subgraph path needs without the row-cluster exchange
// is the split-N path's per-tile partial statistics and fp32 pre-norm rows.
// Here they live in one file-scope device array of kScratchBytes, which each
// GPU the library runs on holds until the process ends.  Its device address
// is looked up once per device (hipGetSymbolAddress, with that device
// current) and only that address is handed to kernels: in host code the
// array's name stands for a host-side shadow, not device memory.
//
// Every call on one GPU shares that GPU's array, so calls that overlap in
// time on one GPU (two streams, two threads) race.  Nothing in the array has
// to start at zero: the split pass writes every partial and row it reads.
#include <hip/hip_runtime.h>

#include <mutex>

#include "comfuse.h"
#include "cf_internal.h"

namespace cf {
cf_status gemm_subgraph_scratch(const cf_subgraph_args* a, void* scratch, size_t scratch_bytes, void* hip_stream,
                                bool validate_only, bool* empty);
cf_status record_error(cf_status s, const char* what);
}  // namespace cf

namespace {
constexpr size_t kScratchBytes = size_t(32) << 20;   // 32 MiB per GPU
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::mutex g_mu;
void* g_scratch[kMaxDevices];   // device address of `scratch` on each device, once looked up

cf_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return cf::record_error(CF_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return cf::record_error(CF_ERR_HIP, "device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return cf::record_error(CF_ERR_HIP, "hipGetSymbolAddress of the scratch array failed");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return CF_OK;
}
}  // namespace

extern "C" cf_status cf_gemm_subgraph_noalloc(const cf_subgraph_args* a, void* hip_stream) {
  try {
    bool empty = false;
    cf_status s = cf::gemm_subgraph_scratch(a, nullptr, kScratchBytes, hip_stream, true, &empty);
    if (s != CF_OK || empty) return s;
    void* ws = nullptr;
    if ((s = scratch_address(&ws)) != CF_OK) return s;
    return cf::gemm_subgraph_scratch(a, ws, kScratchBytes, hip_stream, false, nullptr);
  } catch (...) {
    return cf::record_error(CF_ERR_HIP, "internal error");
  }
}
