// Back-to-back GEMM kernels (placeholder until the B2B kernels land).
#include <hip/hip_runtime.h>

#include "comfuse.h"

extern "C" cf_status cf_b2bgemm(const cf_b2b_args* a, void* workspace, size_t ws_bytes, void* hip_stream) {
  (void)a; (void)workspace; (void)ws_bytes; (void)hip_stream;
  return CF_ERR_UNSUPPORTED;
}
