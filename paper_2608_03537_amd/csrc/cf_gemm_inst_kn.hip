// 128-row tiles on the direct-to-LDS pipeline for bf16 W stored K x N (the
// A fragments come from transposing LDS reads).
#include "cf_gemm_tile.h"

namespace cf {

using S0 = TileShape<bf16_t, 2, 2, 2, 2, 128, 4>;
using S2 = TileShape<bf16_t, 2, 4, 2, 2, 128, 3>;

static const GemmKernel kTable[] = {
    CF_GEMM_ENTRY(S0, 2, 0), CF_GEMM_ENTRY(S0, 2, 1), CF_GEMM_ENTRY(S0, 2, 2),
    CF_GEMM_ENTRY(S2, 2, 0), CF_GEMM_ENTRY(S2, 2, 1), CF_GEMM_ENTRY(S2, 2, 2),
};

const GemmKernel* gemm_kernels_kn(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
