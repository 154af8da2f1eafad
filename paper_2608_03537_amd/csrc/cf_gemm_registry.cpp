// Registry of the compiled GEMM kernels and their launcher.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "cf_internal.h"

namespace cf {

static std::vector<GemmKernel>& table() {
  static std::vector<GemmKernel> t;
  static std::once_flag once;
  std::call_once(once, [] {
    for (auto get : {gemm_kernels_v2, gemm_kernels_v1, gemm_kernels_wr, gemm_kernels_split, gemm_kernels_kn}) {
      int n = 0;
      const GemmKernel* k = get(&n);
      t.insert(t.end(), k, k + n);
    }
  });
  return t;
}

int find_gemm_kernel(int in_f32, int tm, int tn, int loop, int epi) {
  const auto& t = table();
  for (size_t i = 0; i < t.size(); ++i)
    if (t[i].in_f32 == in_f32 && t[i].tm == tm && t[i].tn == tn && t[i].loop == loop && t[i].epi == epi)
      return (int)i;
  return -1;
}

const GemmKernel& gemm_kernel(int idx) { return table()[idx]; }

int resident_wgs(int idx) {
  static std::mutex mu;
  static std::vector<int> cache;
  std::lock_guard<std::mutex> lock(mu);
  if (cache.empty()) cache.assign(table().size(), 0);
  if (idx < 0 || idx >= (int)cache.size()) return 0;
  if (cache[idx]) return cache[idx];
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const GemmKernel& k = table()[idx];
  // Both forms must fit: the one-tile form runs when the grid is not capped.
  int per_cu_persist = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k.fn, k.threads, 0) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_persist, k.fn_persist, k.threads, 0) != hipSuccess)
    return 0;
  cache[idx] = cus * std::min(per_cu, per_cu_persist);
  return cache[idx];
}

hipError_t launch_gemm_rows(const GemmRowsParams& p, int idx, hipStream_t st) {
  const GemmKernel& k = table()[idx];
  dim3 grid((unsigned)(8 * p.slots * p.cn), (unsigned)p.batch), block((unsigned)k.threads);
  void* args[] = {const_cast<GemmRowsParams*>(&p)};
  // Without row clusters every tile has a workgroup of its own (grouped
  // order); with them, workgroups loop only when the grid was capped below
  // one slot per row block of each XCD.
  const bool persist = p.mode == ROWS_CLUSTER && (int64_t)p.slots * 8 < (int64_t)p.num_rb;
  return hipLaunchKernel(persist ? k.fn_persist : k.fn, grid, block, args, 0, st);
}

}  // namespace cf
