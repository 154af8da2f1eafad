// 128-row tiles on the direct-to-LDS pipeline (W stored N x K).
#include "cf_gemm_tile.h"

namespace cf {

using S0 = TileShape<bf16_t, 2, 2, 2, 2, 128, 4>;
using S1 = TileShape<bf16_t, 2, 3, 2, 2, 128, 4>;
using S2 = TileShape<bf16_t, 2, 4, 2, 2, 128, 3>;
using S3 = TileShape<float, 2, 2, 2, 2, 128, 3>;
using S4 = TileShape<float, 2, 4, 2, 2, 128, 3>;

static const GemmKernel kTable[] = {
    CF_GEMM_ENTRY(S0, 1, 0),
    CF_GEMM_ENTRY(S0, 1, 1),
    CF_GEMM_ENTRY(S1, 1, 0),
    CF_GEMM_ENTRY(S1, 1, 1),
    CF_GEMM_ENTRY(S2, 1, 0),
    CF_GEMM_ENTRY(S2, 1, 1),
    CF_GEMM_ENTRY(S3, 1, 0),
    CF_GEMM_ENTRY(S3, 1, 1),
    CF_GEMM_ENTRY(S4, 1, 0),
    CF_GEMM_ENTRY(S4, 1, 1),
};

const GemmKernel* gemm_kernels_v2(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
