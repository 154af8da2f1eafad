// 128-row tiles on the direct-to-LDS pipeline (W stored N x K).
#include "cf_gemm_tile.h"

namespace cf {

static const GemmKernel kTable[] = {
    {TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::TM, TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::TN, 0, 1, 0, TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 2, 2, 2, 128, 4>, 1, 0>)},
    {TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::TM, TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::TN, 0, 1, 1, TileShape<bf16_t, 2, 2, 2, 2, 128, 4>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 2, 2, 2, 128, 4>, 1, 1>)},
    {TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::TM, TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::TN, 0, 1, 0, TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 3, 2, 2, 128, 4>, 1, 0>)},
    {TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::TM, TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::TN, 0, 1, 1, TileShape<bf16_t, 2, 3, 2, 2, 128, 4>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 3, 2, 2, 128, 4>, 1, 1>)},
    {TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::TM, TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::TN, 0, 1, 0, TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 4, 2, 2, 128, 3>, 1, 0>)},
    {TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::TM, TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::TN, 0, 1, 1, TileShape<bf16_t, 2, 4, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 4, 2, 2, 128, 3>, 1, 1>)},
    {TileShape<float, 2, 2, 2, 2, 128, 3>::TM, TileShape<float, 2, 2, 2, 2, 128, 3>::TN, 1, 1, 0, TileShape<float, 2, 2, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 2, 2, 2, 128, 3>, 1, 0>)},
    {TileShape<float, 2, 2, 2, 2, 128, 3>::TM, TileShape<float, 2, 2, 2, 2, 128, 3>::TN, 1, 1, 1, TileShape<float, 2, 2, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 2, 2, 2, 128, 3>, 1, 1>)},
    {TileShape<float, 2, 4, 2, 2, 128, 3>::TM, TileShape<float, 2, 4, 2, 2, 128, 3>::TN, 1, 1, 0, TileShape<float, 2, 4, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 4, 2, 2, 128, 3>, 1, 0>)},
    {TileShape<float, 2, 4, 2, 2, 128, 3>::TM, TileShape<float, 2, 4, 2, 2, 128, 3>::TN, 1, 1, 1, TileShape<float, 2, 4, 2, 2, 128, 3>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 4, 2, 2, 128, 3>, 1, 1>)},
};

const GemmKernel* gemm_kernels_v2(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
