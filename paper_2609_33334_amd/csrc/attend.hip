// Attention of query rows over a compacted cache: the continuation check of the
// evicted cache (Sec. 3 Eq. 1; the eviction-mass equation of App. "Why deferral can
// recover FullKV"; App. "Attention-matching loss").
//
// One workgroup per (query row of a sequence, KV head) handles the G query heads of
// the group, so each cache row is read once for all of them.  The attended rows are
// contiguous, [0, n_kept + visible tail), and go in chunks of 256 keys:
//   - thread t computes the G logits of key c0 + t (its K row in 16-byte loads, the
//     query rows broadcast from LDS), in the log2 domain;
//   - per head, the chunk maximum and the chunk sum of 2^(x - m) are reduced across the
//     4 wavefronts, and the running (m, sum, output) are rescaled (online softmax);
//   - the output update is lane-per-dimension: for each key of the chunk a wavefront
//     reads one V row with consecutive lanes on consecutive elements.
// This is a check kernel: it reads the compacted K/V once per query row and is bound by
// that traffic and by latency, not by arithmetic.
//
// The MASS variant reads only K: from the log-partition over the retained rows and the
// caller's full-cache log-partition it writes each observation row's evicted mass
// rho = 1 - Z_R / Z = -expm1(-(lse_full - lse_R)); a second launch averages rho and the
// deficit -log(1 - rho) over each (sequence, KV head)'s rows in a fixed order.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kAttThreads = 256;
constexpr int kChunk = kAttThreads;   // keys per chunk, one per thread
constexpr int kMaxAttG = 8;           // query heads per KV head

struct AttArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* n_kept;
  float* out;
  float* lse;
  const float* lse_full;              // MASS: [H_q][batch * n_q] natural log, full cache
  float* rho;                         // MASS: [H_q][batch * n_q] evicted mass per row
  float* beta;                        // MASS: [batch][H_kv] mean rho
  float* l_match;                     // MASS: [batch][H_kv] mean -log(1 - rho)
  int batch, n_kv_heads, G, n_q, q_from_end, n_select, n_tail, n_out;
  float scale_log2;                   // log2(e) / sqrt(d)
};

__device__ __forceinline__ float elem_f32(const uint16_t* p, int64_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}
__device__ __forceinline__ float elem_f32(const float* p, int64_t i) { return p[i]; }

// 16 bytes of a K row as floats (8 bf16 or 4 fp32 values)
__device__ __forceinline__ void row_chunk(const uint16_t* row, int e0, float (&x)[8]) {
  const uint4 u = load16(row + e0);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void row_chunk(const float* row, int e0, float (&x)[8]) {
  const uint4 u = load16(row + e0);
  x[0] = __uint_as_float(u.x); x[1] = __uint_as_float(u.y);
  x[2] = __uint_as_float(u.z); x[3] = __uint_as_float(u.w);
}

template <typename E, int D, bool MASS>
__global__ __launch_bounds__(kAttThreads) void cache_attention_kernel(AttArgs a) {
  constexpr int kPer16 = 16 / (int)sizeof(E);                 // elements per 16 bytes
  constexpr int kOwn = (kMaxAttG * D + kAttThreads - 1) / kAttThreads;
  const int row = blockIdx.x;                                 // b * n_q + r
  const int b = row / a.n_q, r = row - b * a.n_q;
  const int h = blockIdx.y;
  const int G = a.G;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  __shared__ float qs[kMaxAttG][D];
  __shared__ float ps[kMaxAttG][kChunk];
  __shared__ float redm[kMaxAttG][4], reds[kMaxAttG][4];

  const int64_t q_rows = (int64_t)a.batch * a.n_q;
  const E* qb = reinterpret_cast<const E*>(a.q);
  for (int i = tid; i < G * D; i += kAttThreads) {
    const int g = i / D, e = i - g * D;
    qs[g][e] = elem_f32(qb, ((int64_t)(h * G + g) * q_rows + row) * D + e);
  }
  const int nk = max(0, min(a.n_kept[b], a.n_select));
  const int nt = max(0, min(a.n_tail, a.n_tail - a.q_from_end + r + 1));
  const int n_vis = nk + nt;                                  // rows [0, n_vis) attended
  const int64_t row0 = ((int64_t)b * a.n_kv_heads + h) * a.n_out;
  const E* kc = reinterpret_cast<const E*>(a.k) + row0 * D;
  const E* vc = reinterpret_cast<const E*>(a.v) + row0 * D;

  // this thread's output elements: e = tid + kAttThreads * i (head e / D, dim e % D;
  // kAttThreads is a multiple of D, so the dim is the same for all of them)
  const int dim = tid % D;
  float o[kOwn];
#pragma unroll
  for (int i = 0; i < kOwn; ++i) o[i] = 0.0f;
  float m2[kMaxAttG], sum[kMaxAttG];                          // wave-uniform
#pragma unroll
  for (int g = 0; g < kMaxAttG; ++g) { m2[g] = -INFINITY; sum[g] = 0.0f; }
  __syncthreads();                                            // qs ready

  for (int c0 = 0; c0 < n_vis; c0 += kChunk) {
    const int j = c0 + tid;
    const bool valid = j < n_vis;
    float x[kMaxAttG];
#pragma unroll
    for (int g = 0; g < kMaxAttG; ++g) x[g] = 0.0f;
    if (valid) {
      const E* krow = kc + (int64_t)j * D;
      for (int e0 = 0; e0 < D; e0 += kPer16) {
        float kv[8];
        row_chunk(krow, e0, kv);
#pragma unroll
        for (int g = 0; g < kMaxAttG; ++g)
          if (g < G)
#pragma unroll
            for (int t = 0; t < kPer16; ++t) x[g] = fmaf(kv[t], qs[g][e0 + t], x[g]);
      }
    }
    // chunk maxima per head, across the 4 wavefronts
#pragma unroll
    for (int g = 0; g < kMaxAttG; ++g) {
      if (g >= G) break;
      x[g] = valid ? x[g] * a.scale_log2 : -INFINITY;
      float mx = x[g];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      if (lane == 0) redm[g][wv] = mx;
    }
    __syncthreads();
    float alpha[kMaxAttG];
#pragma unroll
    for (int g = 0; g < kMaxAttG; ++g) {
      if (g >= G) break;
      const float cm = fmaxf(fmaxf(redm[g][0], redm[g][1]), fmaxf(redm[g][2], redm[g][3]));
      const float nm = fmaxf(m2[g], cm);
      alpha[g] = rescale(m2[g], nm);
      m2[g] = nm;
      const float p = valid ? fast_exp2(x[g] - nm) : 0.0f;
      ps[g][tid] = p;
      float s = p;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
      if (lane == 0) reds[g][wv] = s;
    }
    __syncthreads();                                          // ps and reds complete
#pragma unroll
    for (int g = 0; g < kMaxAttG; ++g) {
      if (g >= G) break;
      sum[g] = sum[g] * alpha[g] + ((reds[g][0] + reds[g][1]) + (reds[g][2] + reds[g][3]));
    }
    if constexpr (MASS) {
      __syncthreads();                                        // redm, reds free
      continue;
    }
    // output: o[head][dim] = o * alpha + sum_t p[head][t] * V[c0 + t][dim]
    const int n_here = min(kChunk, n_vis - c0);
#pragma unroll
    for (int i = 0; i < kOwn; ++i) {
      const int g = (tid + kAttThreads * i) / D;
      if (g < G) o[i] *= alpha[g];
    }
    const E* vrow = vc + (int64_t)c0 * D + dim;
#pragma unroll 8
    for (int t = 0; t < n_here; ++t) {
      const float vv = elem_f32(vrow, (int64_t)t * D);
#pragma unroll
      for (int i = 0; i < kOwn; ++i) {
        const int g = (tid + kAttThreads * i) / D;
        if (g < G) o[i] = fmaf(ps[g][t], vv, o[i]);
      }
    }
    __syncthreads();                                          // ps, redm, reds free
  }

  if constexpr (MASS) {
    if (tid < G) {
      const int g = tid;
      const int64_t ri = (int64_t)(h * G + g) * q_rows + row;
      const float lse_r = n_vis > 0 ? (m2[g] + __log2f(sum[g])) * 0.6931471805599453f : -INFINITY;
      // deficit log Z - log Z_R >= 0 (rounding can leave it a hair below 0 when nothing of
      // the row's attention is evicted)
      const float dlt = fmaxf(a.lse_full[ri] - lse_r, 0.0f);
      a.rho[ri] = -expm1f(-dlt);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < kOwn; ++i) {
    const int e = tid + kAttThreads * i;
    const int g = e / D;
    if (g < G) {
      const int64_t oi = ((int64_t)(h * G + g) * q_rows + row) * D + dim;
      a.out[oi] = n_vis > 0 ? o[i] / sum[g] : 0.0f;
    }
  }
  if (tid < G) {
    const int g = tid;
    a.lse[(int64_t)(h * G + g) * q_rows + row] =
        n_vis > 0 ? (m2[g] + __log2f(sum[g])) * 0.6931471805599453f : -INFINITY;
  }
}

// beta[b][h] and l_match[b][h]: means of rho and -log(1 - rho) over the G * n_q rows of
// (sequence b, KV head h), one wavefront each, summed in a fixed order.
__global__ __launch_bounds__(64) void mass_reduce_kernel(AttArgs a) {
  const int b = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int n = a.G * a.n_q;
  const int64_t q_rows = (int64_t)a.batch * a.n_q;
  float s_rho = 0.0f, s_def = 0.0f;
  for (int i = lane; i < n; i += 64) {
    const int g = i / a.n_q, r = i - g * a.n_q;
    const float rho = a.rho[(int64_t)(h * a.G + g) * q_rows + b * a.n_q + r];
    s_rho += rho;
    s_def += -log1pf(-rho);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    s_rho += __shfl_xor(s_rho, off, 64);
    s_def += __shfl_xor(s_def, off, 64);
  }
  if (lane == 0) {
    a.beta[b * a.n_kv_heads + h] = s_rho / (float)n;
    a.l_match[b * a.n_kv_heads + h] = s_def / (float)n;
  }
}

template <typename E, int D, bool MASS>
hipError_t launch_att(const AttArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((cache_attention_kernel<E, D, MASS>), dim3(a.batch * a.n_q, a.n_kv_heads),
                     dim3(kAttThreads), 0, st, a);
  if constexpr (MASS)
    hipLaunchKernelGGL(mass_reduce_kernel, dim3(a.batch, a.n_kv_heads), dim3(64), 0, st, a);
  return hipGetLastError();
}

template <bool MASS>
hipError_t launch_att_typed(const dge_geom_t& g, const AttArgs& a, hipStream_t st) {
  if (g.dtype == DGE_BF16)
    return g.head_dim == 128 ? launch_att<uint16_t, 128, MASS>(a, st)
                             : launch_att<uint16_t, 64, MASS>(a, st);
  return g.head_dim == 128 ? launch_att<float, 128, MASS>(a, st) : launch_att<float, 64, MASS>(a, st);
}

}  // namespace

int cache_attention_max_group() { return kMaxAttG; }

hipError_t launch_cache_attention(const dge_geom_t& g, const void* q, int n_q, int q_from_end,
                                  const void* k_c, const void* v_c, int n_select, int n_tail,
                                  const int32_t* n_kept, float* out, float* lse,
                                  hipStream_t st) {
  AttArgs a{};
  a.q = q;
  a.k = k_c;
  a.v = v_c;
  a.n_kept = n_kept;
  a.out = out;
  a.lse = lse;
  a.batch = g.batch;
  a.n_kv_heads = g.n_kv_heads;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.n_q = n_q;
  a.q_from_end = q_from_end;
  a.n_select = n_select;
  a.n_tail = n_tail;
  a.n_out = n_select + n_tail;
  a.scale_log2 = kLog2e / sqrtf((float)g.head_dim);
  return launch_att_typed<false>(g, a, st);
}

hipError_t launch_evicted_mass(const dge_geom_t& g, const void* q, int n_q, int q_from_end,
                               const void* k_c, int n_select, int n_tail, const int32_t* n_kept,
                               const float* lse_full, float* rho, float* beta, float* l_match,
                               hipStream_t st) {
  AttArgs a{};
  a.q = q;
  a.k = k_c;
  a.n_kept = n_kept;
  a.lse_full = lse_full;
  a.rho = rho;
  a.beta = beta;
  a.l_match = l_match;
  a.batch = g.batch;
  a.n_kv_heads = g.n_kv_heads;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.n_q = n_q;
  a.q_from_end = q_from_end;
  a.n_select = n_select;
  a.n_tail = n_tail;
  a.n_out = n_select + n_tail;
  a.scale_log2 = kLog2e / sqrtf((float)g.head_dim);
  return launch_att_typed<true>(g, a, st);
}

}  // namespace dge
