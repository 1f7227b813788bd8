// Contiguity of the retained sets (Sec. 4, "Selection trades coverage for contiguity";
// Table "Selection decomposition", column "run len."; App. "Diagnostic details"): for
// every (sequence, KV head), the number of maximal runs of consecutive positions among
// the selected past keys and their mean length.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kRunThreads = 256;

// One workgroup per (KV head, sequence).  The indices are ascending (as the selection
// writes them), so a run starts at r = 0 and wherever idx[r] != idx[r-1] + 1; the
// starts are summed per wavefront and then across the four wavefronts.
__global__ __launch_bounds__(kRunThreads) void retained_runs_kernel(const int32_t* idx,
                                                                    const int32_t* n_kept,
                                                                    int n_kv_heads, int n_select,
                                                                    int32_t* runs,
                                                                    float* mean_len) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int n = min(max(n_kept[b], 0), n_select);
  const int32_t* row = idx + ((int64_t)b * n_kv_heads + h) * n_select;
  int starts = 0;
  for (int r = threadIdx.x; r < n; r += kRunThreads)
    starts += (r == 0 || row[r] != row[r - 1] + 1) ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) starts += __shfl_xor(starts, o, kWave);
  __shared__ int part[kRunThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = starts;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
#pragma unroll
    for (int w = 0; w < kRunThreads / kWave; ++w) tot += part[w];
    runs[(int64_t)b * n_kv_heads + h] = tot;
    mean_len[(int64_t)b * n_kv_heads + h] = tot > 0 ? (float)n / (float)tot : 0.0f;
  }
}

}  // namespace

hipError_t launch_retained_runs(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                                int n_select, int32_t* runs, float* mean_len, hipStream_t st) {
  hipLaunchKernelGGL(retained_runs_kernel, dim3(g.n_kv_heads, g.batch), dim3(kRunThreads), 0, st,
                     idx, n_kept, g.n_kv_heads, n_select, runs, mean_len);
  return hipGetLastError();
}

}  // namespace dge
