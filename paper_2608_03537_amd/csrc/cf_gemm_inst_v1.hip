// 128-row tiles on the register-staged loop (K x N weights, ragged K).
#include "cf_gemm_tile.h"

namespace cf {

using S0 = TileShape<bf16_t, 2, 2, 2, 2, 128, 0>;
using S1 = TileShape<bf16_t, 2, 4, 2, 2, 128, 0>;
using S2 = TileShape<float, 2, 2, 2, 2, 128, 0>;
using S3 = TileShape<float, 2, 4, 2, 2, 128, 0>;

static const GemmKernel kTable[] = {
    CF_GEMM_ENTRY(S0, 0, 0),
    CF_GEMM_ENTRY(S0, 0, 1),
    CF_GEMM_ENTRY(S1, 0, 0),
    CF_GEMM_ENTRY(S1, 0, 1),
    CF_GEMM_ENTRY(S2, 0, 0),
    CF_GEMM_ENTRY(S2, 0, 1),
    CF_GEMM_ENTRY(S3, 0, 0),
    CF_GEMM_ENTRY(S3, 0, 1),
};

const GemmKernel* gemm_kernels_v1(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
