// Window / draft scoring of every cached key (Alg. 1 step B; App. "Diagnostic details").
//
//   raw[h][j] = (1/G) sum_{g in group h} sum_r softmax_j(q_{g,r} . k_j / sqrt(d)),
//   softmax over keys j <= p_r (causal), fp32 after the bf16/fp32 product.
//
// A column sum needs every scoring row's global normaliser first, so one layer runs
// as three launches over the same split of the keys into chunks:
//   1. stats : each workgroup streams its chunk of K and keeps, per query row, the
//              running (max, sum of 2^(x - max)) of its logits (log2 domain);
//   2. reduce: one wavefront per (row, sequence, KV head) merges the chunk partials
//              into c_r = log2 Z_r;
//   3. colsum: each workgroup streams its chunk again, P = 2^(x - c_r), sums over all
//              rows of the group and writes raw[] (the K slab of one layer, 8-34 MB at
//              Llama-3-8B geometry, is still in the 256 MB Infinity Cache).
//
// Workgroups are laid out XCD-aware (see xcd_unit): the chunks of one KV head share an
// XCD, so its query block is fetched into one L2, and the colsum pass finds each chunk
// in the L2 that streamed it during the stats pass.
//
// Work split inside a workgroup (4 wavefronts, one KV head, one chunk of keys):
// - The G * n_rows query rows form 16-row tiles; wavefront w owns tiles w, w+4, w+8...
//   Its query fragments stay in registers for the whole chunk (<= 48 VGPRs at
//   Llama-3-8B geometry), so several workgroups fit on a compute unit.
// - Each 64-key tile of K is read from HBM once per workgroup with 16-byte loads, one
//   coalesced row per 16 threads, and staged in LDS with the 16-byte units of row r
//   XOR-swizzled by r: the 16 lanes that read one fragment column hit 16 different
//   bank groups.  The next tile's global loads are in flight while the current tile
//   is on the matrix cores.
// - stats uses the transposed product (A = keys, B = query rows): a lane then holds
//   4 keys of ONE row, so the per-row max/sum is mostly in-lane and needs two
//   cross-lane steps per row tile at the end of the chunk.
// - colsum uses A = query rows, B = keys: a lane holds 4 rows of ONE key, the sum
//   over rows is in-lane, then across the 4 lane groups and the 4 wavefronts.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int KT = 64;          // keys per workgroup iteration
constexpr int kThreads = 256;

struct ScoreArgs {
  const void* q;
  const void* k;
  float* raw;
  float2* partial;   // [batch][H_kv][n_chunks][M_pad] (max, sum) per chunk, log2 domain
  float* rowc;       // [batch][H_kv][M_pad]  log2 of each row's softmax normaliser
  const float* lse_in;      // optional [H_q][batch * n_rows] natural-log row LSE
  SeqOffsets offs;
  int64_t kv_head_stride;   // elements
  int64_t q_head_stride;    // elements between query heads = batch * n_rows * D
  int64_t total_rows;       // T
  int n_kv_heads, batch, G, n_rows, p0_from_end;
  int M, M_pad, n_tiles, groups, iters, chunk_keys, n_chunks;
  float scale_log2;         // log2(e) / sqrt(d)
  float inv_G;
};

template <typename T, int D>
struct KTile {
  static constexpr int kRowBytes = D * Elem<T>::kBytes;
  static constexpr int kUnits = kRowBytes / 16;                // 16-byte units per row
  static constexpr int kPerThread = KT * kUnits / kThreads;    // units each thread stages
  static constexpr int kBytes = KT * kRowBytes;
};

// Issue the global loads of one 64-key tile (rows past the sequence are clamped to
// its last row; their logits are masked later).
template <typename T, int D>
__device__ __forceinline__ void ktile_load(const char* kb, int j0, int N, int tid,
                                           uint4 (&st)[KTile<T, D>::kPerThread]) {
  using KTl = KTile<T, D>;
#pragma unroll
  for (int i = 0; i < KTl::kPerThread; ++i) {
    const int e = tid + kThreads * i;
    const int r = e / KTl::kUnits, u = e % KTl::kUnits;
    const int j = min(j0 + r, N - 1);
    st[i] = load16(kb + (int64_t)j * KTl::kRowBytes + u * 16);
  }
}

template <typename T, int D>
__device__ __forceinline__ void ktile_store(char* lds, int tid,
                                            const uint4 (&st)[KTile<T, D>::kPerThread]) {
  using KTl = KTile<T, D>;
#pragma unroll
  for (int i = 0; i < KTl::kPerThread; ++i) {
    const int e = tid + kThreads * i;
    const int r = e / KTl::kUnits, u = e % KTl::kUnits;
    *reinterpret_cast<uint4*>(lds + r * KTl::kRowBytes + ((u ^ (r % KTl::kUnits)) * 16)) = st[i];
  }
}

// Fragment of key row r (0..63 within the tile) for chunk step s and lane group g16.
template <typename T, int D>
__device__ __forceinline__ uint4 ktile_frag(const char* lds, int r, int s, int g16) {
  using KTl = KTile<T, D>;
  const int u = s * 4 + g16;
  return *reinterpret_cast<const uint4*>(lds + r * KTl::kRowBytes + ((u ^ (r % KTl::kUnits)) * 16));
}

// Query fragments of the row tiles owned by wavefront wv in row group grp.
template <typename T, int D, int MTW>
__device__ __forceinline__ void load_q_frags(const ScoreArgs& a, int h, int b, int tile0, int wv,
                                             int c16, int g16,
                                             uint4 (&qf)[MTW][RowChunks<T, D>::kSteps]) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  const T* qb = reinterpret_cast<const T*>(a.q);
#pragma unroll
  for (int mt = 0; mt < MTW; ++mt) {
    const int m = (tile0 + wv + 4 * mt) * 16 + c16;   // lane supplies row l % 16
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

template <typename T, int D, int MTW>
__global__ __launch_bounds__(kThreads) void score_stats_kernel(ScoreArgs a) {
  using KTl = KTile<T, D>;
  constexpr int NS = RowChunks<T, D>::kSteps;
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  __shared__ __attribute__((aligned(16))) char lds[KTl::kBytes];

  for (int grp = 0; grp < a.groups; ++grp) {
    const int tile0 = grp * 4 * MTW;
    uint4 qf[MTW][NS];
    load_q_frags<T, D, MTW>(a, h, b, tile0, wv, c16, g16, qf);
    // this lane's row in each owned tile, and that row's position
    int pos[MTW];
    bool live[MTW];
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) {
      const int m = (tile0 + wv + 4 * mt) * 16 + c16;
      live[mt] = m < a.M;
      pos[mt] = p0 + (live[mt] ? m % a.n_rows : 0);
    }
    float mrow[MTW], srow[MTW];
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) { mrow[mt] = -INFINITY; srow[mt] = 0.0f; }

    // two K tiles in flight per workgroup: tile t+2 loads while tile t is consumed
    uint4 stA[KTl::kPerThread], stB[KTl::kPerThread];
    ktile_load<T, D>(kb, c0, N, tid, stA);
    if (c0 + KT < c1) ktile_load<T, D>(kb, c0 + KT, N, tid, stB);
    auto consume = [&](int j0) {
      // no key of this tile is past the sequence or beyond any row's position
      const bool need_mask = (j0 + KT - 1 > p0);
#pragma unroll 2
      for (int sub = 0; sub < KT / 16; ++sub) {
        uint4 kf[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, sub * 16 + c16, s, g16);
        // MTW independent accumulation chains, issued k-step-major
        f32x4_t acc[MTW];
#pragma unroll
        for (int mt = 0; mt < MTW; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int mt = 0; mt < MTW; ++mt) acc[mt] = mma_step(T{}, kf[s], qf[mt][s], acc[mt]);
        // acc[mt][t] = logit of key j0 + sub*16 + 4*g16 + t for this lane's row
#pragma unroll
        for (int mt = 0; mt < MTW; ++mt) {
          float x[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) x[t] = acc[mt][t] * a.scale_log2;
          if (need_mask) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int j = j0 + sub * 16 + 4 * g16 + t;
              x[t] = (live[mt] && j < N && j <= pos[mt]) ? x[t] : -INFINITY;
            }
          }
          const float mx = fmaxf(fmaxf(mrow[mt], fmaxf(x[0], x[1])), fmaxf(x[2], x[3]));
          const float base = mx == -INFINITY ? 0.0f : mx;
          srow[mt] = srow[mt] * fast_exp2(mrow[mt] - base) + fast_exp2(x[0] - base) +
                     fast_exp2(x[1] - base) + fast_exp2(x[2] - base) + fast_exp2(x[3] - base);
          mrow[mt] = mx;
        }
      }
    };
    for (int j0 = c0; j0 < c1; j0 += 2 * KT) {
      __syncthreads();
      ktile_store<T, D>(lds, tid, stA);
      __syncthreads();
      if (j0 + 2 * KT < c1) ktile_load<T, D>(kb, j0 + 2 * KT, N, tid, stA);
      consume(j0);
      if (j0 + KT >= c1) break;
      __syncthreads();
      ktile_store<T, D>(lds, tid, stB);
      __syncthreads();
      if (j0 + 3 * KT < c1) ktile_load<T, D>(kb, j0 + 3 * KT, N, tid, stB);
      consume(j0 + KT);
    }
    // merge the four lane groups that hold the same row
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) {
      float m = mrow[mt], s = srow[mt];
      const float mx = fmaxf(fmaxf(m, shfl_xor_f<16>(m)), fmaxf(shfl_xor_f<32>(m), shfl_xor_f<48>(m)));
      s *= rescale(m, mx);
      s += shfl_xor_f<16>(s);
      s += shfl_xor_f<32>(s);
      const int row = (tile0 + wv + 4 * mt) * 16 + c16;
      if (g16 == 0 && row < a.M)
        a.partial[((int64_t)(b * a.n_kv_heads + h) * a.n_chunks + chunk) * a.M_pad + row] =
            make_float2(mx, s);
    }
  }
}

// One wavefront per query row: merge that row's chunk partials.
__global__ __launch_bounds__(256) void score_reduce_kernel(ScoreArgs a) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int h = blockIdx.y, b = blockIdx.z;
  if (m >= a.M_pad) return;
  const int64_t base = (int64_t)(b * a.n_kv_heads + h);
  if (m >= a.M) {   // padding rows: 2^(x - inf) = 0
    if (lane == 0) a.rowc[base * a.M_pad + m] = INFINITY;
    return;
  }
  const int N = (int)(a.offs[b + 1] - a.offs[b]);
  const int nch = (N + a.chunk_keys - 1) / a.chunk_keys;
  float mm = -INFINITY, ss = 0.0f;
  for (int ch = lane; ch < nch; ch += 64) {
    const float2 p = a.partial[(base * a.n_chunks + ch) * a.M_pad + m];
    const float mx = fmaxf(mm, p.x);
    ss = ss * rescale(mm, mx) + p.y * rescale(p.x, mx);
    mm = mx;
  }
  float mx = mm;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  ss *= rescale(mm, mx);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) ss += __shfl_xor(ss, o, 64);
  if (lane == 0) a.rowc[base * a.M_pad + m] = mx + __log2f(ss);
}

template <typename T, int D, int MTW>
__global__ __launch_bounds__(kThreads) void score_colsum_kernel(ScoreArgs a) {
  using KTl = KTile<T, D>;
  constexpr int NS = RowChunks<T, D>::kSteps;
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  const float* rowc = a.rowc + (int64_t)(b * a.n_kv_heads + h) * a.M_pad;
  float* out = a.raw + (int64_t)h * a.total_rows + s0;
  __shared__ __attribute__((aligned(16))) char lds[KTl::kBytes];
  __shared__ float red[4][KT];

  for (int grp = 0; grp < a.groups; ++grp) {
    const int tile0 = grp * 4 * MTW;
    uint4 qf[MTW][NS];
    load_q_frags<T, D, MTW>(a, h, b, tile0, wv, c16, g16, qf);
    // normalisers and positions of this lane's 4 rows in each owned tile
    float cr[MTW][4];
    int pos[MTW][4];
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int m = (tile0 + wv + 4 * mt) * 16 + 4 * g16 + t;
        if (a.lse_in != nullptr) {
          const int g = m / a.n_rows, r = m - (m / a.n_rows) * a.n_rows;
          cr[mt][t] = m < a.M ? a.lse_in[(int64_t)(h * a.G + g) * (a.q_head_stride / D) +
                                         b * a.n_rows + r] * kLog2e
                              : INFINITY;
        } else {
          cr[mt][t] = m < a.M ? rowc[m] : INFINITY;
        }
        pos[mt][t] = p0 + (m < a.M ? m % a.n_rows : 0);
      }

    uint4 stA[KTl::kPerThread], stB[KTl::kPerThread];
    ktile_load<T, D>(kb, c0, N, tid, stA);
    if (c0 + KT < c1) ktile_load<T, D>(kb, c0 + KT, N, tid, stB);
    auto consume = [&](int j0) {
      const bool need_mask = (j0 + KT - 1 > p0);
#pragma unroll 2
      for (int sub = 0; sub < KT / 16; ++sub) {
        uint4 kf[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, sub * 16 + c16, s, g16);
        f32x4_t acc[MTW];
#pragma unroll
        for (int mt = 0; mt < MTW; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int mt = 0; mt < MTW; ++mt) acc[mt] = mma_step(T{}, qf[mt][s], kf[s], acc[mt]);
        // acc[mt][t] = logit of row (tile*16 + 4*g16 + t) for key j0 + sub*16 + c16
        const int j = j0 + sub * 16 + c16;
        float colp = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            float p = fast_exp2(fmaf(acc[mt][t], a.scale_log2, -cr[mt][t]));
            if (need_mask) p = (j < N && j <= pos[mt][t]) ? p : 0.0f;
            colp += p;
          }
        colp += shfl_xor_f<16>(colp);
        colp += shfl_xor_f<32>(colp);
        if (g16 == 0) red[wv][sub * 16 + c16] = colp;
      }
      __syncthreads();
      if (tid < KT && j0 + tid < c1) {
        const float v = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
        if (grp == 0) out[j0 + tid] = v * a.inv_G;
        else out[j0 + tid] += v * a.inv_G;
      }
    };
    for (int j0 = c0; j0 < c1; j0 += 2 * KT) {
      __syncthreads();
      ktile_store<T, D>(lds, tid, stA);
      __syncthreads();
      if (j0 + 2 * KT < c1) ktile_load<T, D>(kb, j0 + 2 * KT, N, tid, stA);
      consume(j0);
      if (j0 + KT >= c1) break;
      __syncthreads();
      ktile_store<T, D>(lds, tid, stB);
      __syncthreads();
      if (j0 + 3 * KT < c1) ktile_load<T, D>(kb, j0 + 3 * KT, N, tid, stB);
      consume(j0 + KT);
    }
    __syncthreads();
  }
}

template <typename T, int D, int MTW>
hipError_t launch_typed(const ScoreArgs& a, const dge_geom_t& g, hipStream_t st) {
  const dim3 grid(xcd_grid(a.n_chunks * g.n_kv_heads * g.batch));
  if (a.lse_in != nullptr) {   // normalisers supplied: one pass over K
    hipLaunchKernelGGL((score_colsum_kernel<T, D, MTW>), grid, dim3(kThreads), 0, st, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((score_stats_kernel<T, D, MTW>), grid, dim3(kThreads), 0, st, a);
  hipLaunchKernelGGL(score_reduce_kernel, dim3(a.M_pad / 4, g.n_kv_heads, g.batch), dim3(256), 0,
                     st, a);
  hipLaunchKernelGGL((score_colsum_kernel<T, D, MTW>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_mt(const ScoreArgs& a, const dge_geom_t& g, int mtw, hipStream_t st) {
  switch (mtw) {
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

// Register budget for query fragments: tiles-per-wavefront * steps <= 36 16-byte chunks.
int max_mtw(const dge_geom_t& g) {
  const int steps = g.head_dim * (g.dtype == DGE_BF16 ? 2 : 4) / 64;
  const int m = 36 / steps;
  return m > 9 ? 9 : m;
}

}  // namespace

SeqOffsets seq_offsets(const dge_geom_t& g) {
  SeqOffsets o{};
  o.dev = g.kv_offsets;
  o.batch = g.batch;
  if (g.batch <= kInlineSeqs)
    for (int b = 0; b <= g.batch; ++b) o.inl[b] = g.kv_offsets_host[b];
  return o;
}

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
  p.n_tiles = p.M_pad / 16;
  const int cap = max_mtw(g);
  const int per_wave = (p.n_tiles + 3) / 4;
  p.groups = per_wave <= cap ? 1 : (per_wave + cap - 1) / cap;
  p.mt = (per_wave + p.groups - 1) / p.groups;
  if (p.mt < 1) p.mt = 1;
  // About one resident round of workgroups (two per compute unit): every workgroup
  // loads its query fragments once and streams several 64-key tiles with two in flight.
  const int64_t tiles_total = (int64_t)g.n_kv_heads * ((total_rows(g) + KT - 1) / KT);
  int iters = (int)((tiles_total + 511) / 512);
  iters = iters < 1 ? 1 : (iters > 16 ? 16 : iters);
  p.tiles_per_wave = iters;
  p.chunk_keys = KT * iters;
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
                        const float* row_lse, float* raw, void* ws, hipStream_t st) {
  ScoreArgs a{};
  a.lse_in = row_lse;
  a.q = q;
  a.k = k;
  a.raw = raw;
  const size_t units = (size_t)g.batch * g.n_kv_heads;
  a.partial = reinterpret_cast<float2*>(ws);
  a.rowc = ws == nullptr ? nullptr
                         : reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                                    units * p.n_chunks * p.M_pad * sizeof(float2));
  a.offs = seq_offsets(g);
  a.kv_head_stride = g.kv_head_stride;
  a.q_head_stride = (int64_t)g.batch * p.n_rows * g.head_dim;
  a.total_rows = total_rows(g);
  a.n_kv_heads = g.n_kv_heads;
  a.batch = g.batch;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.n_rows = p.n_rows;
  a.p0_from_end = p.p0_from_end;
  a.M = p.M;
  a.M_pad = p.M_pad;
  a.n_tiles = p.n_tiles;
  a.groups = p.groups;
  a.iters = p.tiles_per_wave;
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
