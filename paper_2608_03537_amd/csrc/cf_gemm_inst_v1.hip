// 128-row tiles on the register-staged loop (K x N weights, ragged K).
#include "cf_gemm_tile.h"

namespace cf {

static const GemmKernel kTable[] = {
    {TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::TM, TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::TN, 0, 0, 0, TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 2, 2, 2, 128, 0>, 0, 0>)},
    {TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::TM, TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::TN, 0, 0, 1, TileShape<bf16_t, 2, 2, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 2, 2, 2, 128, 0>, 0, 1>)},
    {TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::TM, TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::TN, 0, 0, 0, TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 4, 2, 2, 128, 0>, 0, 0>)},
    {TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::TM, TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::TN, 0, 0, 1, TileShape<bf16_t, 2, 4, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 2, 4, 2, 2, 128, 0>, 0, 1>)},
    {TileShape<float, 2, 2, 2, 2, 128, 0>::TM, TileShape<float, 2, 2, 2, 2, 128, 0>::TN, 1, 0, 0, TileShape<float, 2, 2, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 2, 2, 2, 128, 0>, 0, 0>)},
    {TileShape<float, 2, 2, 2, 2, 128, 0>::TM, TileShape<float, 2, 2, 2, 2, 128, 0>::TN, 1, 0, 1, TileShape<float, 2, 2, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 2, 2, 2, 128, 0>, 0, 1>)},
    {TileShape<float, 2, 4, 2, 2, 128, 0>::TM, TileShape<float, 2, 4, 2, 2, 128, 0>::TN, 1, 0, 0, TileShape<float, 2, 4, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 4, 2, 2, 128, 0>, 0, 0>)},
    {TileShape<float, 2, 4, 2, 2, 128, 0>::TM, TileShape<float, 2, 4, 2, 2, 128, 0>::TN, 1, 0, 1, TileShape<float, 2, 4, 2, 2, 128, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 2, 4, 2, 2, 128, 0>, 0, 1>)},
};

const GemmKernel* gemm_kernels_v1(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
