// H2O accumulated attention (Table "Complexity and measured overhead", footnote a): the
// causal softmax of every cached row, summed down each key column and meaned over the
// GQA group,
//   colsum[h][j] = (1/G) sum_g sum_{p >= j} exp(q_{g,p} . k_j / sqrt(d) - lse_{g,p}).
//
// Two kernels on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16):
//
// lse (skipped when the caller supplies it): a workgroup owns a pair of 64-row blocks
//   (one from each end of the sequence, so every workgroup does the same causal work)
//   of one KV head; wavefront g is query head g of the group and keeps its 4 row tiles
//   of Q in registers.  64-key tiles of K stream through a ring of XOR-swizzled LDS
//   tiles (global->LDS copies, two in flight) and are read by all G wavefronts.  The
//   product is taken transposed (A = keys, B = query rows) so a lane holds 4 keys of one
//   row and keeps that row's (reference, sum) in registers.
//
// colsum: a workgroup owns a 128-key block and a 512-row segment of one KV head; each
//   wavefront keeps two 16-key tiles of K in registers.  For every query head of the
//   group, 64-row blocks of Q and their log-sum-exp are staged in LDS (double-buffered,
//   next block prefetched into registers) and shared by the four wavefronts.  With
//   A = query rows, a lane holds 4 rows of one key: P = 2^(x - lse) is summed in the
//   lane and crosses lanes once, at the end of the segment.  A small reduction adds
//   the segments' partial sums in a fixed order.
// No atomics: every partial column sum is owned by exactly one wavefront.
#include <type_traits>
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int D = 128;
constexpr int NS = RowChunks<bf16_t, D>::kSteps;   // 4 chunk steps of 32 elements
constexpr int RB = 64;                              // rows per Q block (colsum) / lse block
constexpr int KB = 128;                             // keys per colsum key block
constexpr int KTL = 64;                             // keys per K tile (lse)
constexpr int RowBytes = D * 2;
constexpr int kMaxG = 4;                            // lse kernel: one wavefront per head

struct H2oArgs {
  const bf16_t* q;      // [H_q][T][D]
  const bf16_t* k;      // [H_kv][stride]
  const float* lse;     // [H_q][T] natural log
  float* lse_out;       // workspace [H_q][T] (when computing)
  float* colsum;        // [H_kv][T]
  SeqOffsets offs;
  int64_t kv_head_stride;
  int64_t total_rows;
  int n_q_heads, n_kv_heads, G, batch;
  int n_pairs;          // block pairs per (sequence, KV head)
  float scale_log2;
  float inv_G;
};

// 64 rows x 256 B staged with the 16-byte unit u of row r at u ^ (r % 16).
__device__ __forceinline__ int swz(int r, int u) { return r * RowBytes + ((u ^ (r & 15)) * 16); }

__device__ __forceinline__ uint4 lds_frag(const char* lds, int r, int s, int g16) {
  return *reinterpret_cast<const uint4*>(lds + swz(r, s * 4 + g16));
}

// Global loads of a 64-row Q block of the colsum kernel (rows clamped to the sequence);
// 4 units per thread, unit
// u = tid % 16 of rows tid / 16 + 16 i.  The address is a wave-uniform base at row
// rb = min(r0, N - 1) plus a 32-bit lane offset below 16 KB (scalar-base loads): the row
// offset is clamped to lim = N - 1 - rb, so a load costs one min and one shift-add.
__device__ __forceinline__ void block_load(const char* base, int r0, int N, int tid, uint4 (&st)[4]) {
  const int rb = min(r0, N - 1);
  const int lim = N - 1 - rb;
  const char* b0 = base + (int64_t)rb * RowBytes;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t off = (uint32_t)(min((tid >> 4) + 16 * i, lim) * RowBytes + (tid & 15) * 16);
    st[i] = load16(b0 + off);
  }
}

// LDS stores of the block loaded above: the units of rows tid / 16 + 16 i sit 16 rows
// (4 KB) apart under the swizzle (which depends on the row mod 16 only), so one address
// serves the four stores through the instruction's offset field.
__device__ __forceinline__ void block_store(char* lds, int tid, const uint4 (&st)[4]) {
  char* p = lds + swz(tid >> 4, tid & 15);
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<uint4*>(p + 16 * RowBytes * i) = st[i];
}

// ------------------------------------------------------------------------------------
// Row log-sum-exp: one (row-block pair, KV head, sequence) per workgroup.
// ------------------------------------------------------------------------------------
// One 64-key tile for the wavefront's four 16-row tiles (rows r0 + rt*16 + c16): the
// transposed product (A = keys) puts 4 keys of one row in each lane, and each 16-key
// subtile's four logits per row go through rebase_lse_update (no maximum in the common
// path, one wave-uniform overflow check per subtile).
template <bool MASK>
__device__ __forceinline__ void lse_tile(const char* buf, int j0, int r0, int N, int c16,
                                         int g16, const uint4 (&qf)[4][NS], float scale,
                                         float (&m)[4], float (&sm)[4]) {
  // two subtiles per loop iteration: their fragment reads take immediate LDS offsets (a
  // full unroll runs out of registers at three wavefronts per SIMD)
#pragma unroll 2
  for (int sub = 0; sub < KTL / 16; ++sub) {
    uint4 kf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) kf[s] = lds_frag(buf, sub * 16 + c16, s, g16);
    f32x4_t acc[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) acc[rt] = mma_step(bf16_t{}, kf[s], qf[rt][s], acc[rt]);
    // acc[rt][i] = logit of key j0 + sub*16 + 4*g16 + i for row r0 + rt*16 + c16
    float x[4][4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[rt][i] = acc[rt][i];
        if constexpr (MASK) {
          const int p = r0 + rt * 16 + c16, j = j0 + sub * 16 + 4 * g16 + i;
          x[rt][i] = (j <= p && j < N) ? x[rt][i] : -INFINITY;
        }
      }
    rebase_lse_update<4, 4>(x, scale, m, sm);
  }
}

// K tiles of the row-LSE kernel stream through a ring of kLseStages 16 KB LDS tiles filled
// by global->LDS copies (kLseStages - 1 in flight while one is on the matrix cores; a copy
// past the last tile re-reads tile 0, so every wait has a fixed count).  Copy i of thread
// tid fills the 16 bytes at 1024 (4 wv + i) + 16 lane of a tile with the unit that belongs
// there under the swizzle (unit u of row r at u ^ (r % 16)); rows past the sequence read
// its last row (their logits are masked).
constexpr int kLseStages = 3;
constexpr int kLseCopies = KTL * RowBytes / (256 * 16);

__device__ __forceinline__ void lse_tile_copy(const char* kb, int j0, int N, uint32_t lds_tile,
                                              const uint32_t (&row)[kLseCopies],
                                              const uint32_t (&col)[kLseCopies]) {
  const uint32_t lim = (uint32_t)(N - 1 - j0);
  const char* base = kb + (int64_t)j0 * RowBytes;
#pragma unroll
  for (int i = 0; i < kLseCopies; ++i)
    dma16_sbase(base, min(row[i], lim) * RowBytes + col[i], lds_tile + i * 1024);
}

// Three workgroups per compute unit (168 registers): every block pair of the
// Llama-3-8B-shaped layer (65 pairs x 8 KV heads) is resident in one round.
__global__ __launch_bounds__(256, 3) void h2o_lse_kernel(H2oArgs a) {
  const int units = a.n_pairs * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int pair = unit % a.n_pairs, h = (unit / a.n_pairs) % a.n_kv_heads,
            b = unit / (a.n_pairs * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int nrb = (N + RB - 1) / RB;
  if (pair >= (nrb + 1) / 2) return;        // a shorter sequence of a ragged batch
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int wvu = __builtin_amdgcn_readfirstlane(wv);   // wave-uniform: scalar addresses
  const bool active = wvu < a.G;            // wavefront wv = query head h*G + wv
  const int hq = h * a.G + (active ? wvu : 0);
  const char* kb = reinterpret_cast<const char*>(a.k + (int64_t)h * a.kv_head_stride + s0 * D);
  const char* qb = reinterpret_cast<const char*>(a.q + (int64_t)hq * a.total_rows * D + s0 * D);
  __shared__ __attribute__((aligned(16))) char ring[kLseStages][KTL * RowBytes];
  uint32_t crow[kLseCopies], ccol[kLseCopies];
#pragma unroll
  for (int i = 0; i < kLseCopies; ++i) {
    const int o = ((wv * kLseCopies + i) * 64 + lane) * 16;
    const int r = o / RowBytes, pu = (o % RowBytes) / 16;
    crow[i] = (uint32_t)r;
    ccol[i] = (uint32_t)((pu ^ (r & 15)) * 16);
  }
  const uint32_t lds_wave = (uint32_t)(wvu * kLseCopies * 1024);

  for (int side = 0; side < 2; ++side) {
    const int rb = side == 0 ? pair : nrb - 1 - pair;
    if (side == 1 && rb == pair) break;     // odd count: the middle block once
    if (rb >= nrb || rb < 0) break;
    const int r0 = rb * RB;
    const int last = min(r0 + RB, N);       // keys [0, last) can be seen by this block
    const int ntile = (last + KTL - 1) / KTL;
    auto issue = [&](int t) {               // copies of tile t (t >= ntile: tile 0 again)
      lse_tile_copy(kb, t < ntile ? t * KTL : 0, N,
                    (uint32_t)(uintptr_t)(lds_ptr_t)ring[t % kLseStages] + lds_wave, crow, ccol);
    };
    lds_barrier();                          // the previous side is done with the ring
    // Q fragments of this wavefront's 4 row tiles (B operand: lane supplies row c16), from
    // asm so that no compiler wait drains the copies; they land with the first tile
    u32x4_t qa[4][NS];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const char* row = qb + (int64_t)min(r0 + rt * 16 + c16, N - 1) * RowBytes;
#pragma unroll
      for (int s = 0; s < NS; ++s) qa[rt][s] = async_load16(row + (s * 4 + g16) * 16);
    }
#pragma unroll
    for (int t = 0; t < kLseStages - 1; ++t) issue(t);
    asm_wait_vmcnt<(kLseStages - 2) * kLseCopies>();   // tile 0 (and the fragments) landed
    uint4 qf[4][NS];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        reg_fence(qa[rt][s]);
        qf[rt][s] = as_uint4(qa[rt][s]);
      }
    float m[4], sm[4];                      // reference and sum (rebase_lse_update)
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) { m[rt] = kLazyRefInit; sm[rt] = 0.0f; }
    for (int t = 0; t < ntile; ++t) {
      if (t > 0) asm_wait_vmcnt<(kLseStages - 2) * kLseCopies>();   // tile t landed (own copies)
      lds_barrier();                        // ... everyone's; slot (t - 1) % S is free
      issue(t + kLseStages - 1);
      const char* buf = ring[t % kLseStages];
      const int j0 = t * KTL;
      if (active) {
        // tiles that reach the block's diagonal (or the sequence end) run the masked body
        if (j0 + KTL > r0) lse_tile<true>(buf, j0, r0, N, c16, g16, qf, a.scale_log2, m, sm);
        else lse_tile<false>(buf, j0, r0, N, c16, g16, qf, a.scale_log2, m, sm);
      }
    }
    asm_wait_vmcnt<0>();                    // no copy still writes into the ring
    if (active) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        float mm = m[rt], ss = sm[rt];
        const float mx = fmaxf(fmaxf(mm, shfl_xor_f<16>(mm)), fmaxf(shfl_xor_f<32>(mm), shfl_xor_f<48>(mm)));
        ss *= rescale(mm, mx);
        ss += shfl_xor_f<16>(ss);
        ss += shfl_xor_f<32>(ss);
        const int p = r0 + rt * 16 + c16;
        if (g16 == 0 && p < N)
          a.lse_out[(int64_t)hq * a.total_rows + s0 + p] = (mx + __log2f(ss)) * 0.6931471805599453f;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Column sums.  Work unit = (128-key block kb, 512-row segment s, KV head, sequence):
// the rows p >= 128*kb of segment s, for all G query heads of the group.  Units whose
// segment ends before the key block starts, or starts past the sequence, exit at once;
// every other unit is at most SEG rows x G heads, so the ~half of a causal grid that
// has work is evenly loaded.  Each unit writes the partial column sums of its 128 keys
// to part[s][h][j]; h2o_reduce_kernel adds the segments in a fixed order.  Compiled for
// four wavefronts per SIMD (<= 128 registers; four workgroups and their 32 KB of staged
// query blocks per compute unit): 3.5% faster than three with the row LSE supplied.
// ------------------------------------------------------------------------------------
constexpr int SEG = 512;
constexpr int NKT = KB / 64;     // 16-key tiles of K per wavefront (4 wavefronts per key block)

__global__ __launch_bounds__(256, 4) void h2o_colsum_kernel(H2oArgs a, float* part, int nkb_max,
                                                         int nseg_max) {
  const int units = nkb_max * nseg_max * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int kblk = unit % nkb_max, seg = (unit / nkb_max) % nseg_max;
  const int h = (unit / (nkb_max * nseg_max)) % a.n_kv_heads,
            b = unit / (nkb_max * nseg_max * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int k0 = kblk * KB;
  const int seg_lo = seg * SEG, seg_hi = min(N, seg_lo + SEG);
  if (k0 >= N || seg_lo >= N || seg_hi <= k0) return;     // no rows p >= k0 here
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  __shared__ __attribute__((aligned(16))) char qlds[2][RB * RowBytes];
  __shared__ __attribute__((aligned(16))) float llds[2][RB];

  // this wavefront's NKT 16-key tiles of K (B operand: lane supplies key c16)
  int jk[NKT];
  uint4 kf[NKT][NS];
  {
    const bf16_t* kh = a.k + (int64_t)h * a.kv_head_stride + s0 * D;
#pragma unroll
    for (int t = 0; t < NKT; ++t) {
      jk[t] = k0 + wv * (16 * NKT) + 16 * t + c16;
      const char* rk = reinterpret_cast<const char*>(kh + (int64_t)min(jk[t], N - 1) * D);
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[t][s] = load16(rk + (s * 4 + g16) * 16);
    }
  }
  float col[NKT];
#pragma unroll
  for (int t = 0; t < NKT; ++t) col[t] = 0.0f;
  const int rlo = max(seg_lo, k0 / RB * RB);   // first 64-row block with rows >= k0
  const int per = (seg_hi - rlo + RB - 1) / RB;
  const int nblk = per * a.G;                  // (head, row block) iterations
  const int64_t qstride = a.total_rows * D;
  const bf16_t* qh = a.q + (int64_t)(h * a.G) * qstride + s0 * D;
  const float* lh = a.lse + (int64_t)(h * a.G) * a.total_rows + s0;
  uint4 st[4];
  float lst = 0.0f;
  block_load(reinterpret_cast<const char*>(qh), rlo, N, tid, st);
  if (tid < RB) lst = lh[min(rlo + tid, N - 1)];
  for (int it = 0; it < nblk; ++it) {
    const int cur = it & 1;
    block_store(qlds[cur], tid, st);
    if (tid < RB) llds[cur][tid] = lst * kLog2e;
    __syncthreads();
    const int r0 = rlo + (it % per) * RB;
    if (it + 1 < nblk) {
      const int g1 = (it + 1) / per, r1 = rlo + ((it + 1) % per) * RB;
      block_load(reinterpret_cast<const char*>(qh + (int64_t)g1 * qstride), r1, N, tid, st);
      if (tid < RB) lst = lh[(int64_t)g1 * a.total_rows + min(r1 + tid, N - 1)];
    }
    // rows that can be masked: below the key block, or past the segment / sequence
    const bool edge = (r0 < k0 + KB) || (r0 + RB > seg_hi);
    // masking only in the (rare) edge blocks: the common body has no branch per logit
    auto body = [&](auto edge_c) {
      constexpr bool EDGE = decltype(edge_c)::value;
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        uint4 qf[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) qf[s] = lds_frag(qlds[cur], rt * 16 + c16, s, g16);
        f32x4_t acc[NKT];
#pragma unroll
        for (int t = 0; t < NKT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int t = 0; t < NKT; ++t) acc[t] = mma_step(bf16_t{}, qf[s], kf[t][s], acc[t]);
        // acc[t][i] = logit of row r0 + rt*16 + 4*g16 + i for key jk[t]
        const float4 l4 = *reinterpret_cast<const float4*>(&llds[cur][rt * 16 + 4 * g16]);
        const float l2[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int t = 0; t < NKT; ++t) {
            float pv = fast_exp2(fmaf(acc[t][i], a.scale_log2, -l2[i]));
            if constexpr (EDGE) {
              const int p = r0 + rt * 16 + 4 * g16 + i;
              pv = (p < seg_hi && jk[t] <= p) ? pv : 0.0f;
            }
            col[t] += pv;
          }
      }
    };
    if (edge) body(std::true_type{});
    else body(std::false_type{});
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    col[t] += shfl_xor_f<16>(col[t]);
    col[t] += shfl_xor_f<32>(col[t]);
  }
  if (g16 == 0) {
    float* out = part + ((int64_t)seg * a.n_kv_heads + h) * a.total_rows + s0;
#pragma unroll
    for (int t = 0; t < NKT; ++t)
      if (jk[t] < N) out[jk[t]] = col[t];
  }
}

// colsum[h][j] = (1/G) * sum over the segments that hold rows >= j's key block, in order.
__global__ __launch_bounds__(256) void h2o_reduce_kernel(H2oArgs a, const float* part) {
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N) return;
  const int nseg = (N + SEG - 1) / SEG;
  float acc = 0.0f;
  for (int s = (j / KB) * KB / SEG; s < nseg; ++s)
    acc += part[((int64_t)s * a.n_kv_heads + h) * a.total_rows + s0 + j];
  a.colsum[(int64_t)h * a.total_rows + s0 + j] = acc * a.inv_G;
}

}  // namespace

size_t h2o_workspace_bytes(const dge_geom_t& g) {
  // row LSE [H_q][T] (when computed here) + segment partials [nseg][H_kv][T]
  const size_t T = (size_t)total_rows(g);
  const size_t nseg = (size_t)((max_seq_rows(g) + SEG - 1) / SEG);
  return (size_t)g.n_q_heads * T * sizeof(float) + nseg * g.n_kv_heads * T * sizeof(float) + 512;
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
  a.batch = g.batch;
  a.scale_log2 = kLog2e / sqrtf((float)D);
  a.inv_G = 1.0f / (float)a.G;
  const int64_t nmax = max_seq_rows(g);
  if (nmax == 0) return hipSuccess;
  if (lse == nullptr) {
    if (a.G > kMaxG) return hipErrorInvalidValue;
    a.lse_out = reinterpret_cast<float*>(ws);
    const int nrb = (int)((nmax + RB - 1) / RB);
    a.n_pairs = (nrb + 1) / 2;
    hipLaunchKernelGGL(h2o_lse_kernel, dim3(xcd_grid(a.n_pairs * g.n_kv_heads * g.batch)),
                       dim3(256), 0, st, a);
    a.lse = a.lse_out;
  } else {
    a.lse = lse;
  }
  const int nkb = (int)((nmax + KB - 1) / KB);
  const int nseg = (int)((nmax + SEG - 1) / SEG);
  const size_t lse_bytes = ((size_t)g.n_q_heads * (size_t)a.total_rows * sizeof(float) + 255) / 256 * 256;
  float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + lse_bytes);
  hipLaunchKernelGGL(h2o_colsum_kernel, dim3(xcd_grid(nkb * nseg * g.n_kv_heads * g.batch)),
                     dim3(256), 0, st, a, part, nkb, nseg);
  hipLaunchKernelGGL(h2o_reduce_kernel, dim3((unsigned)((nmax + 255) / 256), g.n_kv_heads, g.batch),
                     dim3(256), 0, st, a, part);
  return hipGetLastError();
}

}  // namespace dge
