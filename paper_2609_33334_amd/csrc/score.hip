// Window / draft scoring of every cached key (Alg. 1 step B; app:diagnostics).
//
//   raw[h][j] = (1/G) sum_{g in group h} sum_r softmax_j(q_{g,r} . k_j / sqrt(d)),
//   softmax over keys j <= p_r (causal), fp32 throughout after the bf16/fp32 product.
//
// The column sums need every scoring row's global normaliser before any column can
// be summed, so a layer runs as three launches over the same split of the keys:
//   1. stats : each workgroup streams its chunk of K, forms the logits of all G*n_rows
//              query rows on the matrix cores and keeps an online (max, sum) per row;
//   2. reduce: one small workgroup per (sequence, KV head) merges the chunk partials
//              into c_r = log2 Z_r (log2 domain, max folded in);
//   3. colsum: each workgroup streams its chunk again, P = 2^(x - c_r), sums over the
//              rows of the group and writes raw[] for its keys.
// The second pass re-reads K; a layer's K slab (8-34 MB at Llama-3-8B geometry)
// stays in the 256 MB Infinity Cache between the two passes.
//
// Work split: a workgroup is 4 wavefronts; each wavefront owns 16-key tiles and ALL
// query rows of the group, so a key tile is loaded exactly once per pass, straight
// from HBM into matrix-core B fragments (16-byte loads per lane), and the column sum
// over rows stays inside the wavefront.  Query fragments (the A operand) stay in
// registers for the whole chunk.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

struct ScoreArgs {
  const void* q;
  const void* k;
  float* raw;
  float2* partial;   // [batch][H_kv][n_chunks][M_pad] (max, sum) per chunk, log2 domain
  float* rowc;       // [batch][H_kv][M_pad]  log2 of each row's softmax normaliser
  const int64_t* offs;
  int64_t kv_head_stride;   // elements
  int64_t q_head_stride;    // elements between query heads = batch * n_rows * D
  int64_t total_rows;       // T
  int n_kv_heads, G, n_rows, p0_from_end;
  int M, M_pad, groups, tiles_per_wave, chunk_keys, n_chunks;
  float scale_log2;         // log2(e) / sqrt(d)
  float inv_G;
};

template <typename T, int D, int MT>
__device__ __forceinline__ void load_q_frags(const ScoreArgs& a, int h, int b, int grp, int c16,
                                             int g16, uint4 (&qf)[MT][RowChunks<T, D>::kSteps]) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  const T* qb = reinterpret_cast<const T*>(a.q);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = (grp * MT + mt) * 16 + c16;   // A operand: lane supplies row l % 16
    if (m < a.M) {
      const int g = m / a.n_rows;
      const int r = m - g * a.n_rows;
      const T* row = qb + (int64_t)(h * a.G + g) * a.q_head_stride + (int64_t)(b * a.n_rows + r) * D;
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[mt][s] = load16(row + chunk_elem<T, D>(s, g16));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[mt][s] = make_uint4(0, 0, 0, 0);
    }
  }
}

template <typename T, int D, int MT>
__global__ __launch_bounds__(256) void score_stats_kernel(ScoreArgs a) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const T* kb = reinterpret_cast<const T*>(a.k) + (int64_t)h * a.kv_head_stride + s0 * D;

  __shared__ float2 red[4][MT * 16];

  for (int grp = 0; grp < a.groups; ++grp) {
    uint4 qf[MT][NS];
    load_q_frags<T, D, MT>(a, h, b, grp, c16, g16, qf);
    float mrow[MT][4], srow[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) { mrow[mt][i] = -INFINITY; srow[mt][i] = 0.0f; }

    for (int t = 0; t < a.tiles_per_wave; ++t) {
      const int j0 = c0 + 16 * (wv + 4 * t);
      if (j0 >= N) break;
      const int j = j0 + c16;
      const T* krow = kb + (int64_t)min(j, N - 1) * D;
      uint4 kf[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[s] = load16(krow + chunk_elem<T, D>(s, g16));
      // keys of this tile that some row cannot see, or that lie past the sequence
      const bool need_mask = (j0 + 15 > p0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s) acc = mma_step(T{}, qf[mt][s], kf[s], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = acc[i] * a.scale_log2;
          if (!need_mask) {
            online_push(x, mrow[mt][i], srow[mt][i]);
          } else {
            const int m = (grp * MT + mt) * 16 + 4 * g16 + i;
            const int pos = p0 + (m < a.M ? m % a.n_rows : 0);
            if (m < a.M && j < N && j <= pos) online_push(x, mrow[mt][i], srow[mt][i]);
          }
        }
      }
    }
    // merge the 16 lanes that hold the same rows (different key columns)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float m = mrow[mt][i], s = srow[mt][i];
        online_merge(m, s, shfl_xor_f<1>(m), shfl_xor_f<1>(s));
        online_merge(m, s, shfl_xor_f<2>(m), shfl_xor_f<2>(s));
        online_merge(m, s, shfl_xor_f<4>(m), shfl_xor_f<4>(s));
        online_merge(m, s, shfl_xor_f<8>(m), shfl_xor_f<8>(s));
        if (c16 == 0) red[wv][mt * 16 + 4 * g16 + i] = make_float2(m, s);
      }
    __syncthreads();
    for (int r = threadIdx.x; r < MT * 16; r += blockDim.x) {
      const int m = grp * MT * 16 + r;
      if (m < a.M) {
        float mm = red[0][r].x, ss = red[0][r].y;
        for (int w = 1; w < 4; ++w) online_merge(mm, ss, red[w][r].x, red[w][r].y);
        a.partial[((int64_t)(b * a.n_kv_heads + h) * a.n_chunks + chunk) * a.M_pad + m] =
            make_float2(mm, ss);
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void score_reduce_kernel(ScoreArgs a) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int N = (int)(a.offs[b + 1] - a.offs[b]);
  const int nch = (N + a.chunk_keys - 1) / a.chunk_keys;
  const int64_t base = (int64_t)(b * a.n_kv_heads + h);
  for (int m = threadIdx.x; m < a.M_pad; m += blockDim.x) {
    float out = INFINITY;   // padded rows: 2^(x - inf) = 0
    if (m < a.M) {
      float mm = -INFINITY, ss = 0.0f;
      for (int ch = 0; ch < nch; ++ch) {
        const float2 p = a.partial[(base * a.n_chunks + ch) * a.M_pad + m];
        online_merge(mm, ss, p.x, p.y);
      }
      out = mm + log2f(ss);
    }
    a.rowc[base * a.M_pad + m] = out;
  }
}

template <typename T, int D, int MT>
__global__ __launch_bounds__(256) void score_colsum_kernel(ScoreArgs a) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const T* kb = reinterpret_cast<const T*>(a.k) + (int64_t)h * a.kv_head_stride + s0 * D;
  const float* rowc = a.rowc + (int64_t)(b * a.n_kv_heads + h) * a.M_pad;

  uint4 qf[MT][NS];
  float cr[MT][4];
  int loaded = -1;
  for (int t = 0; t < a.tiles_per_wave; ++t) {
    const int j0 = c0 + 16 * (wv + 4 * t);
    if (j0 >= N) break;
    const int j = j0 + c16;
    const T* krow = kb + (int64_t)min(j, N - 1) * D;
    uint4 kf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) kf[s] = load16(krow + chunk_elem<T, D>(s, g16));
    const bool need_mask = (j0 + 15 > p0);
    float colp = 0.0f;
    for (int grp = 0; grp < a.groups; ++grp) {
      if (grp != loaded) {
        load_q_frags<T, D, MT>(a, h, b, grp, c16, g16, qf);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = (grp * MT + mt) * 16 + 4 * g16 + i;
            cr[mt][i] = m < a.M ? rowc[m] : INFINITY;   // padding rows contribute 2^-inf = 0
          }
        loaded = grp;
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s) acc = mma_step(T{}, qf[mt][s], kf[s], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float p = exp2f(fmaf(acc[i], a.scale_log2, -cr[mt][i]));
          if (need_mask) {
            const int m = (grp * MT + mt) * 16 + 4 * g16 + i;
            const int pos = p0 + (m < a.M ? m % a.n_rows : 0);
            p = (m < a.M && j < N && j <= pos) ? p : 0.0f;
          }
          colp += p;
        }
      }
    }
    // rows of a key column are spread over the 4 lane groups
    colp += shfl_xor_f<16>(colp);
    colp += shfl_xor_f<32>(colp);
    if (g16 == 0 && j < N) a.raw[(int64_t)h * a.total_rows + s0 + j] = colp * a.inv_G;
  }
}

template <typename T, int D, int MT>
hipError_t launch_typed(const ScoreArgs& a, const dge_geom_t& g, hipStream_t st) {
  dim3 grid(a.n_chunks, g.n_kv_heads, g.batch);
  hipLaunchKernelGGL((score_stats_kernel<T, D, MT>), grid, dim3(256), 0, st, a);
  hipLaunchKernelGGL(score_reduce_kernel, dim3(g.n_kv_heads, g.batch), dim3(256), 0, st, a);
  hipLaunchKernelGGL((score_colsum_kernel<T, D, MT>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_mt(const ScoreArgs& a, const dge_geom_t& g, int mt, hipStream_t st) {
  switch (mt) {
    case 1: return launch_typed<T, D, 1>(a, g, st);
    case 2: return launch_typed<T, D, 2>(a, g, st);
    case 3: return launch_typed<T, D, 3>(a, g, st);
    case 4: return launch_typed<T, D, 4>(a, g, st);
    case 5: return launch_typed<T, D, 5>(a, g, st);
    case 6: return launch_typed<T, D, 6>(a, g, st);
    case 7: return launch_typed<T, D, 7>(a, g, st);
    case 8: return launch_typed<T, D, 8>(a, g, st);
    case 9: return launch_typed<T, D, 9>(a, g, st);
    default: return hipErrorInvalidValue;
  }
}

// Register budget for query fragments: mt * steps <= 36 sixteen-byte chunks per lane.
int max_mt(const dge_geom_t& g) {
  const int steps = g.head_dim * (g.dtype == DGE_BF16 ? 2 : 4) / 64;
  int m = 36 / steps;
  return m > 9 ? 9 : m;
}

}  // namespace

int64_t total_rows(const dge_geom_t& g) { return g.kv_offsets_host[g.batch]; }

int64_t max_seq_rows(const dge_geom_t& g) {
  int64_t m = 0;
  for (int b = 0; b < g.batch; ++b) {
    const int64_t n = g.kv_offsets_host[b + 1] - g.kv_offsets_host[b];
    m = n > m ? n : m;
  }
  return m;
}

ScorePlan plan_score(const dge_geom_t& g, int rows_mode) {
  ScorePlan p{};
  switch (rows_mode) {
    case DGE_ROWS_DRAFT: p.n_rows = g.k_draft; p.p0_from_end = g.k_draft; break;
    case DGE_ROWS_WINDOW: p.n_rows = g.window; p.p0_from_end = g.k_draft + g.window; break;
    default: p.n_rows = g.window + g.k_draft; p.p0_from_end = g.window + g.k_draft; break;
  }
  const int G = g.n_q_heads / g.n_kv_heads;
  p.M = G * p.n_rows;
  p.M_pad = (p.M + 15) / 16 * 16;
  const int tiles = p.M_pad / 16;
  const int mtmax = max_mt(g);
  p.groups = tiles == 0 ? 1 : (tiles + mtmax - 1) / mtmax;
  p.mt = tiles == 0 ? 1 : (tiles + p.groups - 1) / p.groups;
  // Aim for ~512 workgroups over the whole layer (two per compute unit).
  const int64_t cols = (int64_t)g.n_kv_heads * total_rows(g);
  int64_t per_wg = (cols + 511) / 512;
  int tpw = (int)((per_wg + 63) / 64);
  tpw = tpw < 1 ? 1 : (tpw > 64 ? 64 : tpw);
  p.tiles_per_wave = tpw;
  p.chunk_keys = 64 * tpw;
  const int64_t nmax = max_seq_rows(g);
  p.n_chunks = (int)((nmax + p.chunk_keys - 1) / p.chunk_keys);
  if (p.n_chunks < 1) p.n_chunks = 1;
  return p;
}

size_t score_workspace_bytes(const dge_geom_t& g, const ScorePlan& p) {
  const size_t units = (size_t)g.batch * g.n_kv_heads;
  return units * p.n_chunks * p.M_pad * sizeof(float2) + units * p.M_pad * sizeof(float) + 256;
}

hipError_t launch_score(const dge_geom_t& g, const ScorePlan& p, const void* q, const void* k,
                        float* raw, void* ws, hipStream_t st) {
  ScoreArgs a{};
  a.q = q;
  a.k = k;
  a.raw = raw;
  const size_t units = (size_t)g.batch * g.n_kv_heads;
  a.partial = reinterpret_cast<float2*>(ws);
  a.rowc = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                    units * p.n_chunks * p.M_pad * sizeof(float2));
  a.offs = g.kv_offsets;
  a.kv_head_stride = g.kv_head_stride;
  a.q_head_stride = (int64_t)g.batch * p.n_rows * g.head_dim;
  a.total_rows = total_rows(g);
  a.n_kv_heads = g.n_kv_heads;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.n_rows = p.n_rows;
  a.p0_from_end = p.p0_from_end;
  a.M = p.M;
  a.M_pad = p.M_pad;
  a.groups = p.groups;
  a.tiles_per_wave = p.tiles_per_wave;
  a.chunk_keys = p.chunk_keys;
  a.n_chunks = p.n_chunks;
  a.scale_log2 = kLog2e / sqrtf((float)g.head_dim);
  a.inv_G = 1.0f / (float)a.G;
  if (g.dtype == DGE_BF16) {
    return g.head_dim == 128 ? launch_mt<bf16_t, 128>(a, g, p.mt, st)
                             : launch_mt<bf16_t, 64>(a, g, p.mt, st);
  }
  return g.head_dim == 128 ? launch_mt<float, 128>(a, g, p.mt, st)
                           : launch_mt<float, 64>(a, g, p.mt, st);
}

}  // namespace dge
