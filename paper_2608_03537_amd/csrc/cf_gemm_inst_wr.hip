// Whole-row tiles (TM 32): one workgroup owns complete rows.  The register-
// staged loop serves any layout and ragged K; the direct-to-LDS ring serves
// W stored N x K with K a multiple of the 128-byte stage.
#include "cf_gemm_tile.h"

namespace cf {

using S0 = TileShape<bf16_t, 1, 1, 1, 4, 64, 0>;
using S1 = TileShape<bf16_t, 1, 2, 1, 4, 64, 0>;
using S2 = TileShape<bf16_t, 1, 3, 1, 4, 64, 0>;
using S3 = TileShape<bf16_t, 1, 4, 1, 4, 64, 0>;
using S4 = TileShape<bf16_t, 1, 6, 1, 4, 64, 0>;
using S5 = TileShape<float, 1, 1, 1, 4, 64, 0>;
using S6 = TileShape<float, 1, 2, 1, 4, 64, 0>;
using S7 = TileShape<float, 1, 3, 1, 4, 64, 0>;
using S8 = TileShape<float, 1, 4, 1, 4, 64, 0>;
using S9 = TileShape<float, 1, 6, 1, 4, 64, 0>;
using D0 = TileShape<bf16_t, 1, 1, 1, 4, 128, 4>;
using D1 = TileShape<bf16_t, 1, 2, 1, 4, 128, 4>;
using D2 = TileShape<bf16_t, 1, 3, 1, 4, 128, 3>;
using D3 = TileShape<float, 1, 1, 1, 4, 128, 4>;
using D4 = TileShape<float, 1, 2, 1, 4, 128, 4>;

static const GemmKernel kTable[] = {
    CF_GEMM_ENTRY(S0, 0, 1),
    CF_GEMM_ENTRY(S1, 0, 1),
    CF_GEMM_ENTRY(S2, 0, 1),
    CF_GEMM_ENTRY(S3, 0, 1),
    CF_GEMM_ENTRY(S4, 0, 1),
    CF_GEMM_ENTRY(S5, 0, 1),
    CF_GEMM_ENTRY(S6, 0, 1),
    CF_GEMM_ENTRY(S7, 0, 1),
    CF_GEMM_ENTRY(S8, 0, 1),
    CF_GEMM_ENTRY(S9, 0, 1),
    CF_GEMM_ENTRY(D0, 1, 1),
    CF_GEMM_ENTRY(D1, 1, 1),
    CF_GEMM_ENTRY(D2, 1, 1),
    CF_GEMM_ENTRY(D3, 1, 1),
    CF_GEMM_ENTRY(D4, 1, 1),
};

const GemmKernel* gemm_kernels_wr(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
