// The GEMM pass of the split-N path (stage 1, then fp32 x and per-tile
// (mean, M2) to the workspace), for every 128-row tile of both main loops.
#include "cf_gemm_tile.h"

namespace cf {

using V0 = TileShape<bf16_t, 2, 2, 2, 2, 128, 4>;
using V1 = TileShape<bf16_t, 2, 3, 2, 2, 128, 4>;
using V2 = TileShape<bf16_t, 2, 4, 2, 2, 128, 3>;
using V3 = TileShape<float, 2, 2, 2, 2, 128, 3>;
using V4 = TileShape<float, 2, 4, 2, 2, 128, 3>;
using R0 = TileShape<bf16_t, 2, 2, 2, 2, 128, 0>;
using R1 = TileShape<bf16_t, 2, 4, 2, 2, 128, 0>;
using R2 = TileShape<float, 2, 2, 2, 2, 128, 0>;
using R3 = TileShape<float, 2, 4, 2, 2, 128, 0>;

static const GemmKernel kTable[] = {
    CF_GEMM_ENTRY(V0, 1, 2), CF_GEMM_ENTRY(V1, 1, 2), CF_GEMM_ENTRY(V2, 1, 2),
    CF_GEMM_ENTRY(V3, 1, 2), CF_GEMM_ENTRY(V4, 1, 2), CF_GEMM_ENTRY(R0, 0, 2),
    CF_GEMM_ENTRY(R1, 0, 2), CF_GEMM_ENTRY(R2, 0, 2), CF_GEMM_ENTRY(R3, 0, 2),
};

const GemmKernel* gemm_kernels_split(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
