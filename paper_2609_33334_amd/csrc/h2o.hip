// H2O accumulated attention (Table "Complexity and measured overhead", footnote a): the causal softmax of every
// cached row, summed down each key column and meaned over the GQA group,
//   colsum[h][j] = (1/G) sum_g sum_{p >= j} exp(q_{g,p} . k_j / sqrt(d) - lse_{g,p}).
//
// Two launches, both on the bf16 matrix cores:
//   lse    (skipped when the caller passes its own): one wavefront per 16 query rows
//          walks the keys j <= p with an online (max, sum) per row;
//   colsum : one wavefront per 16-key tile keeps its K fragment in registers and walks
//          the query rows p >= j of all G heads of its group; the column sum of P stays
//          in the lanes (each lane owns 4 rows of one key column) until the very end,
//          so the inner loop is MFMA + exp2 + add with no cross-lane traffic.
// Workgroups with the longest column (small j) are issued first.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int D = 128;
constexpr int NS = RowChunks<bf16_t, D>::kSteps;

struct H2oArgs {
  const bf16_t* q;      // [H_q][T][D]
  const bf16_t* k;      // [H_kv][stride]
  const float* lse;     // [H_q][T] natural log
  float* lse_out;       // workspace [H_q][T] (when computing)
  float* colsum;        // [H_kv][T]
  SeqOffsets offs;
  int64_t kv_head_stride;
  int64_t total_rows;
  int n_q_heads, n_kv_heads, G;
  float scale_log2;
  float inv_G;
};

__global__ __launch_bounds__(256) void h2o_lse_kernel(H2oArgs a) {
  const int rb = blockIdx.x, hq = blockIdx.y, b = blockIdx.z;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int r0 = rb * 64 + wv * 16;
  if (r0 >= N) return;
  const int h = hq / a.G;
  const bf16_t* qrow = a.q + (int64_t)hq * a.total_rows * D + (s0 + min(r0 + c16, N - 1)) * D;
  uint4 qf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) qf[s] = load16(qrow + chunk_elem<bf16_t, D>(s, g16));
  const bf16_t* kb = a.k + (int64_t)h * a.kv_head_stride + s0 * D;
  float m[4], sm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m[i] = -INFINITY; sm[i] = 0.0f; }
  const int last = min(r0 + 15, N - 1);
  for (int j0 = 0; j0 <= last; j0 += 16) {
    const int j = j0 + c16;
    const bf16_t* krow = kb + (int64_t)min(j, N - 1) * D;
    uint4 kf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) kf[s] = load16(krow + chunk_elem<bf16_t, D>(s, g16));
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) acc = mma_step(bf16_t{}, qf[s], kf[s], acc);
    const bool diag = j0 + 15 > r0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float x = acc[i] * a.scale_log2;
      const int p = r0 + 4 * g16 + i;
      if (!diag || j <= p) online_push(x, m[i], sm[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float mm = m[i], ss = sm[i];
    online_merge(mm, ss, shfl_xor_f<1>(mm), shfl_xor_f<1>(ss));
    online_merge(mm, ss, shfl_xor_f<2>(mm), shfl_xor_f<2>(ss));
    online_merge(mm, ss, shfl_xor_f<4>(mm), shfl_xor_f<4>(ss));
    online_merge(mm, ss, shfl_xor_f<8>(mm), shfl_xor_f<8>(ss));
    const int p = r0 + 4 * g16 + i;
    if (c16 == 0 && p < N)
      a.lse_out[(int64_t)hq * a.total_rows + s0 + p] = (mm + log2f(ss)) * 0.6931471805599453f;
  }
}

__global__ __launch_bounds__(256) void h2o_colsum_kernel(H2oArgs a, int n_blocks) {
  const int kbk = n_blocks - 1 - (int)blockIdx.x;   // longest columns first
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int j0 = kbk * 64 + wv * 16;
  if (j0 >= N) return;
  const int j = j0 + c16;
  const bf16_t* krow = a.k + (int64_t)h * a.kv_head_stride + (s0 + min(j, N - 1)) * D;
  uint4 kf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) kf[s] = load16(krow + chunk_elem<bf16_t, D>(s, g16));
  float colp = 0.0f;
  for (int g = 0; g < a.G; ++g) {
    const int hq = h * a.G + g;
    const bf16_t* qb = a.q + (int64_t)hq * a.total_rows * D + s0 * D;
    const float* lb = a.lse + (int64_t)hq * a.total_rows + s0;
    for (int p0 = j0; p0 < N; p0 += 16) {
      const bf16_t* qrow = qb + (int64_t)min(p0 + c16, N - 1) * D;
      uint4 qf[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[s] = load16(qrow + chunk_elem<bf16_t, D>(s, g16));
      float l2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) l2[i] = lb[min(p0 + 4 * g16 + i, N - 1)] * kLog2e;
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) acc = mma_step(bf16_t{}, qf[s], kf[s], acc);
      const bool edge = (p0 == j0) || (p0 + 15 >= N);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = p0 + 4 * g16 + i;
        float pr = exp2f(fmaf(acc[i], a.scale_log2, -l2[i]));
        if (edge) pr = (p < N && j <= p && j < N) ? pr : 0.0f;
        colp += pr;
      }
    }
  }
  colp += shfl_xor_f<16>(colp);
  colp += shfl_xor_f<32>(colp);
  if (g16 == 0 && j < N) a.colsum[(int64_t)h * a.total_rows + s0 + j] = colp * a.inv_G;
}

}  // namespace

size_t h2o_workspace_bytes(const dge_geom_t& g) {
  return (size_t)g.n_q_heads * (size_t)total_rows(g) * sizeof(float) + 256;
}

hipError_t launch_h2o(const dge_geom_t& g, const void* q_all, const void* k, const float* lse,
                      float* colsum, void* ws, hipStream_t st) {
  H2oArgs a{};
  a.q = reinterpret_cast<const bf16_t*>(q_all);
  a.k = reinterpret_cast<const bf16_t*>(k);
  a.colsum = colsum;
  a.offs = seq_offsets(g);
  a.kv_head_stride = g.kv_head_stride;
  a.total_rows = total_rows(g);
  a.n_q_heads = g.n_q_heads;
  a.n_kv_heads = g.n_kv_heads;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.scale_log2 = kLog2e / sqrtf((float)D);
  a.inv_G = 1.0f / (float)a.G;
  const int nblk = (int)((max_seq_rows(g) + 63) / 64);
  if (nblk == 0) return hipSuccess;
  if (lse == nullptr) {
    a.lse_out = reinterpret_cast<float*>(ws);
    hipLaunchKernelGGL(h2o_lse_kernel, dim3(nblk, g.n_q_heads, g.batch), dim3(256), 0, st, a);
    a.lse = a.lse_out;
  } else {
    a.lse = lse;
  }
  hipLaunchKernelGGL(h2o_colsum_kernel, dim3(nblk, g.n_kv_heads, g.batch), dim3(256), 0, st, a,
                     nblk);
  return hipGetLastError();
}

}  // namespace dge
