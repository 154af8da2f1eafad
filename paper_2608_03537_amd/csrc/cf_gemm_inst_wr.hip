// Whole-row tiles (TM 32): one workgroup owns complete rows.
#include "cf_gemm_tile.h"

namespace cf {

static const GemmKernel kTable[] = {
    {TileShape<bf16_t, 1, 1, 1, 4, 64, 0>::TM, TileShape<bf16_t, 1, 1, 1, 4, 64, 0>::TN, 0, 0, 1, TileShape<bf16_t, 1, 1, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 1, 1, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<bf16_t, 1, 2, 1, 4, 64, 0>::TM, TileShape<bf16_t, 1, 2, 1, 4, 64, 0>::TN, 0, 0, 1, TileShape<bf16_t, 1, 2, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 1, 2, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<bf16_t, 1, 3, 1, 4, 64, 0>::TM, TileShape<bf16_t, 1, 3, 1, 4, 64, 0>::TN, 0, 0, 1, TileShape<bf16_t, 1, 3, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 1, 3, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<bf16_t, 1, 4, 1, 4, 64, 0>::TM, TileShape<bf16_t, 1, 4, 1, 4, 64, 0>::TN, 0, 0, 1, TileShape<bf16_t, 1, 4, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 1, 4, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<bf16_t, 1, 6, 1, 4, 64, 0>::TM, TileShape<bf16_t, 1, 6, 1, 4, 64, 0>::TN, 0, 0, 1, TileShape<bf16_t, 1, 6, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<bf16_t, 1, 6, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<float, 1, 1, 1, 4, 64, 0>::TM, TileShape<float, 1, 1, 1, 4, 64, 0>::TN, 1, 0, 1, TileShape<float, 1, 1, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 1, 1, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<float, 1, 2, 1, 4, 64, 0>::TM, TileShape<float, 1, 2, 1, 4, 64, 0>::TN, 1, 0, 1, TileShape<float, 1, 2, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 1, 2, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<float, 1, 3, 1, 4, 64, 0>::TM, TileShape<float, 1, 3, 1, 4, 64, 0>::TN, 1, 0, 1, TileShape<float, 1, 3, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 1, 3, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<float, 1, 4, 1, 4, 64, 0>::TM, TileShape<float, 1, 4, 1, 4, 64, 0>::TN, 1, 0, 1, TileShape<float, 1, 4, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 1, 4, 1, 4, 64, 0>, 0, 1>)},
    {TileShape<float, 1, 6, 1, 4, 64, 0>::TM, TileShape<float, 1, 6, 1, 4, 64, 0>::TN, 1, 0, 1, TileShape<float, 1, 6, 1, 4, 64, 0>::NT,
     reinterpret_cast<const void*>(&gemm_rows_kernel<TileShape<float, 1, 6, 1, 4, 64, 0>, 0, 1>)},
};

const GemmKernel* gemm_kernels_wr(int* n) {
  *n = (int)(sizeof(kTable) / sizeof(kTable[0]));
  return kTable;
}

}  // namespace cf
