// Query/key capture from a layer's input: out = RoPE(x W^T), the post-RoPE rows the scoring
// reads (App. "Draft-guided eviction implementation": queries recomputed post-RoPE from each
// layer's input by forward pre-hooks; rotate-half pairs (i, i + d/2) as in the
// compensation-token appendix; theta = 500,000 for the Table "Backbones" models).
//
// A bf16 matrix-core product with the rotation in its epilogue.  W is a Linear weight
// [n_heads * d][hidden] (rows = output features, K contiguous), x is [n_rows][hidden], so
// both operands stream along K with 16-byte loads, like Q and K in the scoring.
//
// Work split.  A workgroup owns 16 output columns that hold 8 complete rotation pairs,
// columns {8q .. 8q+7} and {d/2 + 8q .. d/2 + 8q+7} of one head, and a block of up to 64
// rows (as many 16-row tiles as the rows need); its eight wavefronts take an eighth of the
// hidden dimension each, with eight K steps of loads in flight, and their partial products
// are summed in LDS in a fixed order.  For the scoring rows (tens of rows) the product is
// bound by streaming W once (HBM); a Llama-3-8B query projection gives 4096 / 16 = 256
// workgroups, and a fused [W_q; W_k] weight (40 heads) 320 in one launch.  In a 16x16
// accumulator tile lane l holds column l % 16, so the partner of a low column sits eight
// lanes away and one shuffle pairs them.  The angle is formed and reduced modulo 2 pi in
// double (positions reach 32K and beyond), its sine and cosine and the rotation of the
// float32 sums in float, and the result is rounded once to bf16.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kProjUnroll = 8;               // K steps of 32 whose loads are issued together
constexpr int kMaxHalfProj = 64;

struct ProjArgs {
  const uint16_t* x;        // [n_rows][hidden] bf16
  const uint16_t* w;        // [n_heads * d][hidden] bf16
  const int32_t* pos;       // [n_rows]
  uint16_t* out;            // [n_heads][.. n_rows ..][d] bf16
  int64_t out_head_stride;  // elements between heads of out (n_rows * d, or more for a row range)
  int n_rows, hidden, n_heads, d, half;
  double inv_freq[kMaxHalfProj];
};

__device__ __forceinline__ uint16_t to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// MT row tiles per workgroup, WAVES wavefronts splitting the hidden dimension.
template <int MT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void project_rope_kernel(ProjArgs a) {
  const int groups = a.half / 8;                     // 8-pair column groups per head
  const int head = blockIdx.x / groups, grp = blockIdx.x % groups;
  const int row0 = blockIdx.y * (16 * MT);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, g16 = lane >> 4;
  // this lane's output column (low half for c16 < 8, its partner d/2 columns higher)
  const int pair = 8 * grp + (c16 & 7);
  const int col = head * a.d + (c16 < 8 ? pair : a.half + pair);
  const int kq = a.hidden / WAVES;                   // K range of this wavefront
  const int k_begin = wv * kq;
  const uint16_t* wrow = a.w + (int64_t)col * a.hidden + k_begin + 8 * g16;
  const uint16_t* xrow[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int r = min(row0 + 16 * i + c16, a.n_rows - 1);   // rows past the end repeat the last
    xrow[i] = a.x + (int64_t)r * a.hidden + k_begin + 8 * g16;
  }
  f32x4_t acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int steps = kq / 32;
  int s = 0;
  for (; s + kProjUnroll <= steps; s += kProjUnroll) {
    // every load of the unrolled steps in flight at once (asm loads: the compiler would
    // otherwise issue them one step at a time to save registers), one wait, then the
    // products
    u32x4_t bw[kProjUnroll], ax[kProjUnroll][MT];
#pragma unroll
    for (int u = 0; u < kProjUnroll; ++u) {
      bw[u] = async_load16(wrow + 32 * (s + u));
#pragma unroll
      for (int i = 0; i < MT; ++i) ax[u][i] = async_load16(xrow[i] + 32 * (s + u));
    }
    asm_wait_vmcnt<0>();
#pragma unroll
    for (int u = 0; u < kProjUnroll; ++u) {
      reg_fence(bw[u]);
#pragma unroll
      for (int i = 0; i < MT; ++i) reg_fence(ax[u][i]);
    }
#pragma unroll
    for (int u = 0; u < kProjUnroll; ++u)
#pragma unroll
      for (int i = 0; i < MT; ++i)
        acc[i] = mma_step(bf16_t{}, as_uint4(ax[u][i]), as_uint4(bw[u]), acc[i]);
  }
  for (; s < steps; ++s) {
    const uint4 bw = load16(wrow + 32 * s);
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = mma_step(bf16_t{}, load16(xrow[i] + 32 * s), bw, acc[i]);
  }
  // sum of the wavefronts' partial products in a fixed order, wavefront i finishing row
  // tile i
  __shared__ float part[WAVES][MT][4][64];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) part[wv][i][t][lane] = acc[i][t];
  __syncthreads();
  if (wv >= MT) return;
  const int i = wv;
  float v[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) sum += part[w][i][t][lane];
    v[t] = sum;
  }
  // rotation: lane c16 < 8 holds x_pair, lane c16 + 8 holds x_{pair + d/2}, same rows
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int r = row0 + 16 * i + 4 * g16 + t;
    const float other = __shfl_xor(v[t], 8, 64);
    if (r < a.n_rows) {
      // the angle in double, reduced to [-pi, pi] with a two-part 2 pi, then sine and cosine
      // in float: ~3e-7 of error, far below the bf16 rounding of the result
      const double ang = (double)a.pos[r] * a.inv_freq[pair];
      const double k = rint(ang * 0.15915494309189535);
      const double red = fma(-k, 2.4492935982947064e-16, fma(-k, 6.283185307179586, ang));
      float sn, cs;
      sincosf((float)red, &sn, &cs);
      const float lo = c16 < 8 ? v[t] : other;
      const float hi = c16 < 8 ? other : v[t];
      const float res = c16 < 8 ? fmaf(lo, cs, -hi * sn) : fmaf(hi, cs, lo * sn);
      const int dcol = c16 < 8 ? pair : a.half + pair;
      a.out[(int64_t)head * a.out_head_stride + (int64_t)r * a.d + dcol] = to_bf16_rne(res);
    }
  }
}

// ---------------------------------------------------------------------------------------
// Short row sets (the scoring rows): the hidden dimension split over KS workgroups.
// The whole x is smaller than nothing here -- 34 rows x 8 KB is ~2x a compute unit's share
// of W_q -- so every workgroup that covers all of K for 16 columns (above) reads ~3x more
// x than W through its compute unit's ~30 GB/s load path.  Here a workgroup covers 64
// columns (4 pair groups, one per wavefront) for 1/KS of K: it stages that K slice of x
// in LDS once (16-byte units XOR-swizzled by row, so the 16 rows of a fragment read hit
// different banks) and streams its W slice; float32 partial sums go to the workspace,
// [KS][n_rows][n_heads * d], and a second launch adds the KS slices in a fixed order,
// rotates and rounds.
// ---------------------------------------------------------------------------------------
constexpr int kSplitCols = 64;

// STEPS = kr / 32 K steps per wavefront (8 or 16): every W load of the slice and the x
// staging loads are issued before the first wait, so the workgroup pays one memory round
// trip (a chain of round trips is what a short workgroup costs).
template <int MT, int STEPS>
__global__ __launch_bounds__(256) void project_split_kernel(ProjArgs a, float* part) {
  constexpr int kr = 32 * STEPS;
  constexpr int units = kr / 8;                       // 16-byte units per staged row
  const int groups = a.half / 8;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, g16 = lane >> 4;
  const int ks = blockIdx.y;                          // K slice
  const int k_lo = ks * kr;
  const int pg = blockIdx.x * 4 + wv;                 // this wavefront's pair group
  const int head = pg / groups, grp = pg % groups;
  const int pair = 8 * grp + (c16 & 7);
  const int col = head * a.d + (c16 < 8 ? pair : a.half + pair);
  const int ncols = a.n_heads * a.d;
  __shared__ __attribute__((aligned(16))) char xs[16 * MT * kr * 2];   // [rows][kr] bf16, swizzled
  const uint16_t* wrow = a.w + (int64_t)col * a.hidden + k_lo + 8 * g16;
  u32x4_t bw[STEPS];
#pragma unroll
  for (int u = 0; u < STEPS; ++u) bw[u] = async_load16(wrow + 32 * u);
  // stage x[rows][k_lo, k_lo + kr) (rows past the end repeat the last row); the compiler's
  // wait before the LDS stores also covers the W loads issued above
  constexpr int kPer = (16 * MT * units + 255) / 256;
  uint4 xv[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = tid + 256 * i;
    const int r = min(e / units, 16 * MT - 1), u = e % units;
    xv[i] = load16(a.x + (int64_t)min(r, a.n_rows - 1) * a.hidden + k_lo + 8 * u);
  }
  asm_wait_vmcnt<0>();
#pragma unroll
  for (int u = 0; u < STEPS; ++u) reg_fence(bw[u]);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = tid + 256 * i;
    if (e < 16 * MT * units) {
      const int r = e / units, u = e % units;
      *reinterpret_cast<uint4*>(xs + ((r * units) + (u ^ (r & 15))) * 16) = xv[i];
    }
  }
  __syncthreads();
  f32x4_t acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < STEPS; ++u)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int r = 16 * i + c16, unit = 4 * u + g16;
      const uint4 ax = *reinterpret_cast<const uint4*>(xs + ((r * units) + (unit ^ (r & 15))) * 16);
      acc[i] = mma_step(bf16_t{}, ax, as_uint4(bw[u]), acc[i]);
    }
  // lane holds rows 16 i + 4 g16 + t of column col
  float* pk = part + (int64_t)ks * a.n_rows * ncols;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int r = 16 * i + 4 * g16 + t;
      if (r < a.n_rows) pk[(int64_t)r * ncols + col] = acc[i][t];
    }
}

// sum of the KS slices (fixed order), rotation, bf16: one thread per (row, head, pair).
// The slices' loads are issued kFinishBatch at a time before they are added (a loop that
// waits for each load before the next is a chain of KS memory round trips).
constexpr int kFinishBatch = 16;

__global__ __launch_bounds__(256) void project_finish_kernel(ProjArgs a, const float* part, int n_split) {
  const int half = a.half;
  const int64_t total = (int64_t)a.n_rows * a.n_heads * half;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int pair = (int)(t % half);
  const int head = (int)((t / half) % a.n_heads);
  const int r = (int)(t / ((int64_t)half * a.n_heads));
  const int ncols = a.n_heads * a.d;
  const int64_t o = (int64_t)r * ncols + head * a.d + pair;
  const int64_t slice = (int64_t)a.n_rows * ncols;
  float lo = 0.0f, hi = 0.0f;
  for (int k0 = 0; k0 < n_split; k0 += kFinishBatch) {
    float pl[kFinishBatch], ph[kFinishBatch];
#pragma unroll
    for (int k = 0; k < kFinishBatch; ++k) {
      const bool in = k0 + k < n_split;
      pl[k] = in ? part[(k0 + k) * slice + o] : 0.0f;
      ph[k] = in ? part[(k0 + k) * slice + o + half] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < kFinishBatch; ++k) {
      if (k0 + k < n_split) {
        lo += pl[k];
        hi += ph[k];
      }
    }
  }
  const double ang = (double)a.pos[r] * a.inv_freq[pair];
  const double kk = rint(ang * 0.15915494309189535);
  const double red = fma(-kk, 2.4492935982947064e-16, fma(-kk, 6.283185307179586, ang));
  float sn, cs;
  sincosf((float)red, &sn, &cs);
  uint16_t* orow = a.out + (int64_t)head * a.out_head_stride + (int64_t)r * a.d;
  orow[pair] = to_bf16_rne(fmaf(lo, cs, -hi * sn));
  orow[half + pair] = to_bf16_rne(fmaf(hi, cs, lo * sn));
}

template <int WAVES>
hipError_t launch_proj_waves(const ProjArgs& a, hipStream_t st) {
  // row tiles per workgroup: just enough for a short row set (the scoring rows), else 4
  const int mt = a.n_rows >= 64 ? 4 : (a.n_rows + 15) / 16;
  const dim3 grid(a.n_heads * (a.half / 8), (a.n_rows + 16 * mt - 1) / (16 * mt));
  const dim3 block(64 * WAVES);
  switch (mt) {
    case 1: hipLaunchKernelGGL((project_rope_kernel<1, WAVES>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((project_rope_kernel<2, WAVES>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((project_rope_kernel<3, WAVES>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((project_rope_kernel<4, WAVES>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

// ---------------------------------------------------------------------------------------
// Many rows (every prompt row of a layer, e.g. H2O's queries): a 128 x 128 output tile per
// workgroup over all of K.  x rows (A) and W rows (B, the output columns) stream through a
// 4-stage LDS ring of 32-wide K slices (8 KB + 8 KB per stage, 3 stages in flight) with
// global->LDS copies, as the scoring streams K.  Within a 64-byte row slice the 16-byte unit
// u of row r sits at u ^ ((r >> 1) & 3), so the 8 rows a fragment read serves together hit
// 8 different 16-byte bank groups.  Wavefront w computes rows 64 (w & 1) .. +64 and four
// 16-column tiles: two low tiles of rotation pairs and their partners d/2 columns higher,
// so each lane holds both halves of its pairs and the epilogue rotates in registers.
// ---------------------------------------------------------------------------------------
constexpr int kGT = 128;                       // rows and columns per workgroup
constexpr int kGBK = 32;                       // K per stage
constexpr int kGStages = 4;
constexpr int kGHalfBytes = kGT * kGBK * 2;    // A or B part of a stage: 8 KB
constexpr int kGStageBytes = 2 * kGHalfBytes;  // 16 KB
constexpr int kGCopies = kGStageBytes / (256 * 16);   // global->LDS copies per thread per stage

// Tile order: each XCD takes a contiguous range of tiles (xcd_unit), walked in groups of
// 8 row blocks across all column blocks, so the workgroups resident on one XCD share both
// x row blocks and W column blocks in its L2.
constexpr int kGGroup = 8;

__global__ __launch_bounds__(256, 2) void project_tile_kernel(ProjArgs a, int nrb, int ncb) {
  const int units = nrb * ncb;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int group = unit / (kGGroup * ncb), in_group = unit % (kGGroup * ncb);
  const int first = group * kGGroup, rows_g = min(nrb - first, kGGroup);
  const int rb = first + in_group % rows_g, cb = in_group / rows_g;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, g16 = lane >> 4;
  const int row0 = rb * kGT, col0 = cb * kGT;
  __shared__ __attribute__((aligned(16))) char ring[kGStages][kGStageBytes];
  // this thread's copies: wavefront wv's instruction i fills bytes [(4 wv + i) KB, +1 KB) of a
  // stage, lane l the 16 bytes at 16 l of that kilobyte; it fetches the unit that belongs there
  uint32_t goff[kGCopies];
  const int wvu = __builtin_amdgcn_readfirstlane(wv);        // wave-uniform copy of wv
  bool is_b[kGCopies];                                       // B part (W rows): wave-uniform
#pragma unroll
  for (int i = 0; i < kGCopies; ++i) {
    const int o = ((wv * kGCopies + i) * 64 + lane) * 16;    // byte offset in the stage
    is_b[i] = (wvu * kGCopies + i) * 1024 >= kGHalfBytes;
    const int ob = is_b[i] ? o - kGHalfBytes : o;
    const int r = ob / 64, pu = (ob % 64) / 16;               // row, physical unit
    const int u = pu ^ ((r >> 1) & 3);                        // logical unit (K offset 8u)
    const int grow = is_b[i] ? col0 + r : min(row0 + r, a.n_rows - 1);
    goff[i] = (uint32_t)(((int64_t)grow * a.hidden + 8 * u) * 2);
  }
  const uint32_t lds_wave = (uint32_t)(wvu * kGCopies * 1024);
  const int nk = a.hidden / kGBK;
  auto issue = [&](int t) {                    // copies of stage t (t >= nk: stage 0 again)
    const int te = t < nk ? t : 0;
    char* buf = ring[t % kGStages];
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_ptr_t)buf + lds_wave;
    const char* xa = reinterpret_cast<const char*>(a.x) + (int64_t)te * kGBK * 2;
    const char* wb = reinterpret_cast<const char*>(a.w) + (int64_t)te * kGBK * 2;
#pragma unroll
    for (int i = 0; i < kGCopies; ++i) dma16_sbase(is_b[i] ? wb : xa, goff[i], lds + i * 1024);
  };
  // the wavefront's tiles: row half rh, low column tiles lt[e] and partners lt[e] + P
  const int rh = wv & 1, j = wv >> 1;
  const int lpt = a.d / 32;                    // low 16-column tiles per head
  int ct[4];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int L = 2 * j + e;
    const int lo = (L / lpt) * (a.d / 16) + L % lpt;
    ct[e] = lo;
    ct[e + 2] = lo + lpt;
  }
  f32x4_t acc[4][4];                           // [row tile][column tile]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // fragment reads of stage t (LDS -> registers)
  auto frags = [&](int t, uint4 (&af)[4], uint4 (&bf)[4]) {
    const char* st = ring[t % kGStages];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = rh * 64 + i * 16 + c16;
      af[i] = *reinterpret_cast<const uint4*>(st + r * 64 + ((g16 ^ ((r >> 1) & 3)) * 16));
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = ct[e] * 16 + c16;
      bf[e] = *reinterpret_cast<const uint4*>(st + kGHalfBytes + r * 64 + ((g16 ^ ((r >> 1) & 3)) * 16));
    }
  };
  // Software-pipelined: the fragments of stage t + 1 are read while the products of stage
  // t run.  Stage t + 1 has landed for everyone after the wait and barrier at the top of
  // iteration t; the same barrier tells that every wavefront's reads of stage t (issued in
  // iteration t - 1) have completed, so its slot may take the copies of stage t + S.
#pragma unroll
  for (int t = 0; t < kGStages - 1; ++t) issue(t);
  asm_wait_vmcnt<(kGStages - 2) * kGCopies>();     // stage 0 has landed (this thread's part)
  lds_barrier();                                   // ... everyone's
  issue(kGStages - 1);
  // stage t: the next stage's fragments into (an, bn), then the products of (af, bf).  No
  // branch: the last stage reads a slot of dummy copies it never uses, so the products
  // wait only for their own fragments (a join of paths would make the compiler wait for
  // all LDS reads in flight).
  auto step = [&](int t, const uint4 (&af)[4], const uint4 (&bf)[4], uint4 (&an)[4], uint4 (&bn)[4]) {
    asm_wait_vmcnt<(kGStages - 2) * kGCopies>();   // stage t + 1 has landed (this thread's part)
    lds_barrier();                                 // ... everyone's; stage t's slot is free
    issue(t + kGStages);
    frags(t + 1, an, bn);
    // keep the reads above the products (the scheduler would otherwise sink them below,
    // serialising LDS latency and matrix cores again)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][e] = mma_step(bf16_t{}, af[i], bf[e], acc[i][e]);
  };
  uint4 a0[4], b0[4], a1[4], b1[4];              // two fragment sets, used in turn
  frags(0, a0, b0);
  for (int t = 0; t < nk; t += 2) {
    step(t, a0, b0, a1, b1);
    if (t + 1 < nk) step(t + 1, a1, b1, a0, b0);
  }
  asm_wait_vmcnt<0>();                         // no copy still writes into the ring
  // epilogue: lane holds rows 4 g16 + k of each row tile, column c16 of each column tile
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int colg = col0 + ct[e] * 16 + c16;  // global low column
    const int head = colg / a.d, pair = colg % a.d;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int r = row0 + rh * 64 + i * 16 + 4 * g16 + k;
        if (r < a.n_rows) {
          const double ang = (double)a.pos[r] * a.inv_freq[pair];
          const double kk = rint(ang * 0.15915494309189535);
          const double red = fma(-kk, 2.4492935982947064e-16, fma(-kk, 6.283185307179586, ang));
          float sn, cs;
          sincosf((float)red, &sn, &cs);
          const float lo = acc[i][e][k], hi = acc[i][e + 2][k];
          uint16_t* orow = a.out + (int64_t)head * a.out_head_stride + (int64_t)r * a.d;
          orow[pair] = to_bf16_rne(fmaf(lo, cs, -hi * sn));
          orow[a.half + pair] = to_bf16_rne(fmaf(hi, cs, lo * sn));
        }
      }
  }
}

// ---------------------------------------------------------------------------------------
// Large tiles for many rows: 256 x 256 per workgroup, eight wavefronts, each computing 128
// rows x 64 columns (eight row tiles; two low 16-column tiles and their partners, as
// above).  Per 32-wide K slice a workgroup copies 32 KB into LDS for 512 products, half
// the L2-to-LDS bytes per product of the 128 x 128 tiles; 3 stages (96 KB) leave one
// workgroup per compute unit.  Same LDS row format and swizzle as the 128 x 128 kernel.
// ---------------------------------------------------------------------------------------
constexpr int kHT = 256;                        // rows and columns per workgroup
constexpr int kHWaves = 8;
constexpr int kHStages = 3;
constexpr int kHHalfBytes = kHT * kGBK * 2;     // A or B part of a stage: 16 KB
constexpr int kHStageBytes = 2 * kHHalfBytes;   // 32 KB
constexpr int kHCopies = kHStageBytes / (64 * kHWaves * 16);   // copies per thread per stage

__global__ __launch_bounds__(64 * kHWaves, 1) void project_tile256_kernel(ProjArgs a, int nrb, int ncb) {
  const int units = nrb * ncb;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int group = unit / (kGGroup * ncb), in_group = unit % (kGGroup * ncb);
  const int first = group * kGGroup, rows_g = min(nrb - first, kGGroup);
  const int rb = first + in_group % rows_g, cb = in_group / rows_g;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, g16 = lane >> 4;
  const int row0 = rb * kHT, col0 = cb * kHT;
  __shared__ __attribute__((aligned(16))) char ring[kHStages][kHStageBytes];
  // wavefront wv's copy i fills bytes [(kHCopies wv + i) KB, +1 KB) of a stage: the A part
  // (x rows) for wavefronts 0-3, the B part (W rows) for 4-7
  const int wvu = __builtin_amdgcn_readfirstlane(wv);
  const bool is_b = wvu * kHCopies * 1024 >= kHHalfBytes;
  uint32_t goff[kHCopies];
#pragma unroll
  for (int i = 0; i < kHCopies; ++i) {
    const int o = ((wv * kHCopies + i) * 64 + lane) * 16 - (is_b ? kHHalfBytes : 0);
    const int r = o / 64, pu = (o % 64) / 16;
    const int u = pu ^ ((r >> 1) & 3);
    const int grow = is_b ? col0 + r : min(row0 + r, a.n_rows - 1);
    goff[i] = (uint32_t)(((int64_t)grow * a.hidden + 8 * u) * 2);
  }
  const uint32_t lds_wave = (uint32_t)(wvu * kHCopies * 1024);
  const int nk = a.hidden / kGBK;
  auto issue = [&](int t) {                     // copies of stage t (t >= nk: stage 0 again)
    const int te = t < nk ? t : 0;
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_ptr_t)ring[t % kHStages] + lds_wave;
    const char* src = reinterpret_cast<const char*>(is_b ? a.w : a.x) + (int64_t)te * kGBK * 2;
#pragma unroll
    for (int i = 0; i < kHCopies; ++i) dma16_sbase(src, goff[i], lds + i * 1024);
  };
  const int rh = wv & 1, j = wv >> 1;
  const int lpt = a.d / 32;                     // low 16-column tiles per head
  int ct[4];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int L = 2 * j + e;
    const int lo = (L / lpt) * (a.d / 16) + L % lpt;
    ct[e] = lo;
    ct[e + 2] = lo + lpt;
  }
  f32x4_t acc[8][4];                            // [row tile][column tile]
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[i][e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < kHStages - 1; ++t) issue(t);
  for (int t = 0; t < nk; ++t) {
    asm_wait_vmcnt<(kHStages - 2) * kHCopies>();   // stage t has landed (this thread's part)
    lds_barrier();                                 // ... everyone's; slot (t - 1) % S is free
    issue(t + kHStages - 1);
    const char* st = ring[t % kHStages];
    uint4 bf[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = ct[e] * 16 + c16;
      bf[e] = *reinterpret_cast<const uint4*>(st + kHHalfBytes + r * 64 + ((g16 ^ ((r >> 1) & 3)) * 16));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = rh * 128 + i * 16 + c16;
      const uint4 af = *reinterpret_cast<const uint4*>(st + r * 64 + ((g16 ^ ((r >> 1) & 3)) * 16));
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][e] = mma_step(bf16_t{}, af, bf[e], acc[i][e]);
    }
  }
  asm_wait_vmcnt<0>();                          // no copy still writes into the ring
  // epilogue: lane holds rows 4 g16 + k of each row tile, column c16 of each column tile
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int colg = col0 + ct[e] * 16 + c16;   // global low column
    const int head = colg / a.d, pair = colg % a.d;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int r = row0 + rh * 128 + i * 16 + 4 * g16 + k;
        if (r < a.n_rows) {
          const double ang = (double)a.pos[r] * a.inv_freq[pair];
          const double kk = rint(ang * 0.15915494309189535);
          const double red = fma(-kk, 2.4492935982947064e-16, fma(-kk, 6.283185307179586, ang));
          // the hardware sine and cosine on the reduced angle (error ~1e-6, far below the
          // bf16 rounding of the result): with the library sincosf the 64 rotations of a
          // lane are too large to unroll, and the accumulators then go to scratch memory
          float sn, cs;
          __sincosf((float)red, &sn, &cs);
          const float lo = acc[i][e][k], hi = acc[i][e + 2][k];
          uint16_t* orow = a.out + (int64_t)head * a.out_head_stride + (int64_t)r * a.d;
          orow[pair] = to_bf16_rne(fmaf(lo, cs, -hi * sn));
          orow[a.half + pair] = to_bf16_rne(fmaf(hi, cs, lo * sn));
        }
      }
  }
}

bool project_tiled(int n_rows, int hidden, int n_heads, int head_dim) {
  const int64_t ncols = (int64_t)n_heads * head_dim;
  return n_rows >= kGT && ncols % kGT == 0 && hidden % kGBK == 0 &&
         (int64_t)n_rows * hidden * 2 < ((int64_t)1 << 32) && ncols * hidden * 2 < ((int64_t)1 << 32);
}

// Hidden-dimension split of the short-row path: about 512 workgroups of 64 columns, K
// slices of 256 or 512 (8 or 16 K steps per wavefront, all in flight at once; the staged x
// slice, 16 MT x kr bf16, stays within 64 KB of LDS).  1 = no split.
int project_split(int n_rows, int hidden, int n_heads, int head_dim) {
  if (n_rows > 64 || hidden % 256 != 0) return 1;
  const int colblocks = n_heads * head_dim / kSplitCols;
  if (colblocks < 1 || (n_heads * head_dim) % kSplitCols != 0) return 1;
  int ks = 1;
  while (ks * 2 * colblocks <= 768 && hidden / (ks * 2) >= 256 && hidden % (ks * 2 * 256) == 0) ks *= 2;
  while (hidden / ks > 512 && hidden % (ks * 2 * 256) == 0) ks *= 2;
  return hidden / ks > 512 ? 1 : ks;
}

size_t project_workspace_bytes(int n_rows, int hidden, int n_heads, int head_dim) {
  const int ks = project_split(n_rows, hidden, n_heads, head_dim);
  return ks == 1 ? 0 : (size_t)ks * n_rows * n_heads * head_dim * sizeof(float);
}

hipError_t launch_project_rope(int n_rows, int hidden, const void* x, int n_heads, int head_dim,
                               const void* w, const int32_t* positions, double theta, void* out,
                               void* ws, hipStream_t st) {
  ProjArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.w = static_cast<const uint16_t*>(w);
  a.pos = positions;
  a.out = static_cast<uint16_t*>(out);
  a.out_head_stride = (int64_t)n_rows * head_dim;
  a.n_rows = n_rows;
  a.hidden = hidden;
  a.n_heads = n_heads;
  a.d = head_dim;
  a.half = head_dim / 2;
  for (int i = 0; i < a.half; ++i) a.inv_freq[i] = pow(theta, -2.0 * i / head_dim);
  const int ks = project_split(n_rows, hidden, n_heads, head_dim);
  if (ks > 1) {
    float* part = static_cast<float*>(ws);
    const int kr = hidden / ks;
    const int mt = (n_rows + 15) / 16;
    const dim3 grid(n_heads * head_dim / kSplitCols, ks);
#define DGE_SPLIT_LAUNCH(MT, STEPS) \
    hipLaunchKernelGGL((project_split_kernel<MT, STEPS>), grid, dim3(256), 0, st, a, part)
    if (kr == 256) {
      switch (mt) {
        case 1: DGE_SPLIT_LAUNCH(1, 8); break;
        case 2: DGE_SPLIT_LAUNCH(2, 8); break;
        case 3: DGE_SPLIT_LAUNCH(3, 8); break;
        default: DGE_SPLIT_LAUNCH(4, 8); break;
      }
    } else {
      switch (mt) {
        case 1: DGE_SPLIT_LAUNCH(1, 16); break;
        case 2: DGE_SPLIT_LAUNCH(2, 16); break;
        case 3: DGE_SPLIT_LAUNCH(3, 16); break;
        default: DGE_SPLIT_LAUNCH(4, 16); break;
      }
    }
#undef DGE_SPLIT_LAUNCH
    const int64_t total = (int64_t)n_rows * n_heads * a.half;
    hipLaunchKernelGGL(project_finish_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st,
                       a, part, ks);
    return hipGetLastError();
  }
  if (project_tiled(n_rows, hidden, n_heads, head_dim)) {
    // Whole tiles only (a partial block would cost as much as a full one, in a round of its
    // own at the end of a launch): 256-row blocks on the large tiles when the columns come
    // in 256s, then whole 128-row blocks, then the rest through the small-row kernel, each
    // launch on a row range of the same output.
    const int64_t ncols = (int64_t)n_heads * head_dim;
    auto range = [&](int r0, int n) {
      ProjArgs ar = a;
      ar.x = a.x + (int64_t)r0 * hidden;
      ar.pos = a.pos + r0;
      ar.out = a.out + (int64_t)r0 * head_dim;
      ar.n_rows = n;
      return ar;
    };
    int done = 0;
    if (ncols % kHT == 0 && n_rows >= kHT) {
      const int nrb = n_rows / kHT, ncb = (int)(ncols / kHT);
      hipLaunchKernelGGL(project_tile256_kernel, dim3(xcd_grid(nrb * ncb)), dim3(64 * kHWaves), 0, st,
                         range(0, nrb * kHT), nrb, ncb);
      done = nrb * kHT;
    }
    if (n_rows - done >= kGT) {
      const int nrb = (n_rows - done) / kGT, ncb = (int)(ncols / kGT);
      hipLaunchKernelGGL(project_tile_kernel, dim3(xcd_grid(nrb * ncb)), dim3(256), 0, st,
                         range(done, nrb * kGT), nrb, ncb);
      done += nrb * kGT;
    }
    if (done == n_rows) return hipGetLastError();
    const ProjArgs ar = range(done, n_rows - done);
    return hidden % 256 == 0 ? launch_proj_waves<8>(ar, st) : launch_proj_waves<4>(ar, st);
  }
  // eight wavefronts split the hidden dimension (each keeps 8 K steps of loads in flight),
  // four when it is not a multiple of 256
  return hidden % 256 == 0 ? launch_proj_waves<8>(a, st) : launch_proj_waves<4>(a, st);
}

}  // namespace dge
