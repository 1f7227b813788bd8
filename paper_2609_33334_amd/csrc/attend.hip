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

// ---------------------------------------------------------------------------------------
// Matrix-core path (bf16; d = 128, or d = 64 for the evicted mass; n_q <= 64).  One
// workgroup per (query head, sequence): wavefront w takes row tile w % 4 of the head's n_q
// rows and key pair w / 4 (keys 32 (w / 4) .. +31) of every tile (64 keys and 8 wavefronts
// for the attention, 128 keys and 16 for the mass), so several wavefronts per SIMD hide
// each other's latencies; at the end the key pairs of a row tile are merged in LDS in a
// fixed order.  The G workgroups of a KV head are
// consecutive units of the XCD-aware order, so they share one L2 and each compacted row
// leaves HBM once.  Tiles of the compacted K (and V) are loaded from asm into a ring of
// register slots (tiles in flight while one is computed; past the end the loads re-read
// the last row and those tiles are fully masked, so every wait has a fixed count) and
// stored into double-buffered LDS: K rows XOR-swizzled by row as in the scoring, V
// transposed to [dim][key] (four keys of one dimension per 8-byte unit, units swizzled by
// dimension) so that a lane reads the 8 keys of an MFMA operand with two 8-byte loads.
//   logits:  S^T = K Q^T per 16-key subtile (A = keys, B = query rows): a lane holds 4 keys
//            of one row; tiles below every row's first invisible key skip the mask;
//   softmax: per row a reference m, the same in the row's four lane groups, and a sum per
//            lane; m moves only when a sum reaches kSumLimit (then to the row's batch
//            maximum, the sums and outputs rescaled), so the common path is fma, exp2, add;
//   output:  O^T += V^T P^T per 32 keys (A = V^T from LDS, B = the lane's own 8 weights
//            from two subtiles), P split into a truncated bf16 high part and the bf16 of
//            the remainder (two products, ~15 bits of weight); a lane holds 4 dimensions of
//            its own row, so the rescale of a row is local to the lane.
// The evicted-mass variant stops after the sums.
// Tiles of 64 keys and 8 wavefronts (two key pairs) for the attention, whose output
// accumulators need the registers of two wavefronts per SIMD; 128 keys and 16 wavefronts
// (four key pairs) for the evicted mass.
template <int D, bool MASS>
struct AttMfma {
  static constexpr int kKT = MASS ? 128 : 64;              // keys per tile
  static constexpr int kSplit = kKT / 32;                  // key pairs: wavefronts per row tile
  static constexpr int kThreads = 4 * kSplit * kWave;
  static constexpr int kRowBytes = D * 2;
  static constexpr int kUnits = kRowBytes / 16;            // 16-byte units per K row
  static constexpr int kKBytes = kKT * kRowBytes;          // one K tile
  static constexpr int kKLoads = kKT * kUnits / kThreads;  // per thread
  static constexpr int kVBytes = D * kKT * 2;              // one transposed V tile
  static constexpr int kNS = D / 32;                       // MFMA steps over d
  static constexpr int kDT = D / 16;                       // 16-dimension output tiles
};

template <int D, bool MASS>
__global__ __launch_bounds__((AttMfma<D, MASS>::kThreads)) void cache_attention_mfma_kernel(AttArgs a) {
  using AT = AttMfma<D, MASS>;
  constexpr int kAttKT = AT::kKT, kAttSplit = AT::kSplit, kAttMfmaThreads = AT::kThreads;
  constexpr int NS = AT::kNS;
  static_assert(MASS || (D == 128 && kAttKT * 16 == 2 * kAttMfmaThreads),
                "the V transpose: 128 dimensions (16 x 8), a key pair per thread");
  static_assert(AT::kKLoads >= 1 && AT::kKLoads * kAttMfmaThreads == kAttKT * AT::kUnits, "K staging");
  const int units = a.batch * a.n_kv_heads * a.G;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int hq = unit % (a.n_kv_heads * a.G), b = unit / (a.n_kv_heads * a.G);
  const int h = hq / a.G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wvu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rt = wvu & 3, ks = wvu >> 2;                       // row tile, key pair
  const int g16 = lane >> 4, c16 = lane & 15;
  const bool own = rt * 16 < a.n_q;                            // wave-uniform
  const int64_t q_rows = (int64_t)a.batch * a.n_q;
  const int nk = max(0, min(a.n_kept[b], a.n_select));
  const int n_vis_max = nk + max(0, min(a.n_tail, a.n_tail - a.q_from_end + a.n_q));
  const int n_vis_min = nk + max(0, min(a.n_tail, a.n_tail - a.q_from_end + 1));
  const int64_t row0 = ((int64_t)b * a.n_kv_heads + h) * a.n_out;
  const char* kc = reinterpret_cast<const char*>(a.k) + row0 * AT::kRowBytes;
  const char* vc = MASS ? nullptr : reinterpret_cast<const char*>(a.v) + row0 * AT::kRowBytes;
  constexpr int kStageBytes = AT::kKBytes + (MASS ? 0 : AT::kVBytes);
  __shared__ __attribute__((aligned(16))) char lds[2 * kStageBytes];
  __shared__ float mfin[kAttSplit][4][16], sfin[kAttSplit][4][16];

  const int r = rt * 16 + c16;                                 // this lane's row
  if (n_vis_max == 0) {                                        // nothing visible: no loads
    if (ks == 0 && own && r < a.n_q) {
      const int64_t ri = (int64_t)hq * q_rows + (int64_t)b * a.n_q + r;
      if constexpr (MASS) {
        if (g16 == 0) a.rho[ri] = 1.0f;
      } else {
        if (g16 == 0) a.lse[ri] = -INFINITY;
        for (int e = 4 * g16; e < D; e += 16)
#pragma unroll
          for (int q = 0; q < 4; ++q) a.out[ri * D + e + q] = 0.0f;
      }
    }
    return;
  }
  const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.q) +
                         ((int64_t)hq * q_rows + (int64_t)b * a.n_q + min(r, a.n_q - 1)) * D;
  u32x4_t qf[NS];
#pragma unroll
  for (int st = 0; st < NS; ++st) qf[st] = async_load16(reinterpret_cast<const char*>(qrow) + (st * 4 + g16) * 16);
  const int lim = r < a.n_q ? nk + max(0, min(a.n_tail, a.n_tail - a.q_from_end + r + 1)) : 0;
  float m = kLazyRefInit, ssum = 0.0f;
  f32x4_t o[MASS ? 1 : AT::kDT];
#pragma unroll
  for (int dt = 0; dt < (MASS ? 1 : AT::kDT); ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // tile staging: K units (kKLoads per thread) and, for the attention, keys 2 (tid / 16),
  // +1 of V at dimensions 8 (tid % 16) .. +7, stored as the 4-byte halves of V^T units
  constexpr int PF = MASS ? 4 : 3;                             // tiles in flight
  constexpr int NV = MASS ? 0 : 2;
  constexpr int LPT = AT::kKLoads + NV;                        // loads per tile per thread
  u32x4_t kst[PF][AT::kKLoads], vst[PF][MASS ? 1 : NV];
  const int vp = tid >> 4, vo = tid & 15;
  auto stage_load = [&](int t, u32x4_t (&kr)[AT::kKLoads], u32x4_t (&vr)[MASS ? 1 : NV]) {
    const int j0 = t * kAttKT;
#pragma unroll
    for (int i = 0; i < AT::kKLoads; ++i) {
      const int e = tid + kAttMfmaThreads * i;
      const int rr = e / AT::kUnits, u = e % AT::kUnits;
      kr[i] = async_load16(kc + (int64_t)max(0, min(j0 + rr, n_vis_max - 1)) * AT::kRowBytes + u * 16);
    }
    if constexpr (!MASS) {
#pragma unroll
      for (int k = 0; k < 2; ++k)
        vr[k] = async_load16(vc + (int64_t)max(0, min(j0 + 2 * vp + k, n_vis_max - 1)) * AT::kRowBytes + vo * 16);
    }
  };
  auto stage_store = [&](int buf, u32x4_t (&kr)[AT::kKLoads], u32x4_t (&vr)[MASS ? 1 : NV]) {
    char* kl = lds + buf * kStageBytes;
#pragma unroll
    for (int i = 0; i < AT::kKLoads; ++i) {
      reg_fence(kr[i]);
      const int e = tid + kAttMfmaThreads * i;
      const int rr = e / AT::kUnits, u = e % AT::kUnits;
      *reinterpret_cast<uint4*>(kl + rr * AT::kRowBytes + ((u ^ (rr % AT::kUnits)) * 16)) = as_uint4(kr[i]);
    }
    if constexpr (!MASS) {
      char* vl = kl + AT::kKBytes;
      reg_fence(vr[0]);
      reg_fence(vr[1]);
      const int quad = vp >> 1, hpos = (vp & 1) * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int odd = 0; odd < 2; ++odd) {
          const int d = 8 * vo + 2 * i + odd;
          *reinterpret_cast<uint32_t*>(vl + d * (kAttKT * 2) + ((quad ^ (d & 15)) * 8) + hpos) =
              __builtin_amdgcn_perm(vr[1][i], vr[0][i], odd ? 0x07060302u : 0x05040100u);
        }
      }
    }
  };

  auto compute = [&](int t, int buf) {
    if (!own) return;
    const char* kl = lds + buf * kStageBytes;
    const int j0 = t * kAttKT + 32 * ks;                       // this wavefront's 32 keys
    const bool masked = j0 + 32 > n_vis_min;                    // uniform: some key may be hidden
    float x[8];
#pragma unroll
    for (int su = 0; su < 2; ++su) {
      const int kr = 32 * ks + 16 * su + c16;
      uint4 kf[NS];
#pragma unroll
      for (int st = 0; st < NS; ++st)
        kf[st] = *reinterpret_cast<const uint4*>(kl + kr * AT::kRowBytes + (((st * 4 + g16) ^ (kr % AT::kUnits)) * 16));
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < NS; ++st) acc = mma_step(bf16_t{}, kf[st], as_uint4(qf[st]), acc);
      // acc[q] = logit of key j0 + 16 su + 4 g16 + q for this lane's row
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = j0 + 16 * su + 4 * g16 + q;
        x[4 * su + q] = (!masked || j < lim) ? acc[q] : -INFINITY;
      }
    }
    float pv[8], ps = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      pv[q] = fast_exp2(fmaf(x[q], a.scale_log2, -m));
      ps += pv[q];
    }
    float ns = ssum + ps;
    // a row whose sum (in any of its lane groups) reaches kSumLimit moves its reference,
    // the same in all four lane groups
    int ov = !(ns < kSumLimit) ? 1 : 0;
    if (__any(ov)) {
      ov |= __shfl_xor(ov, 16, 64);
      ov |= __shfl_xor(ov, 32, 64);
      float mx = x[0];
#pragma unroll
      for (int q = 1; q < 8; ++q) mx = fmaxf(mx, x[q]);
      mx *= a.scale_log2;
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (ov) {
        const float nr = fmaxf(mx, m + kLazyBound);
        const float f = fast_exp2(m - nr);
        ps = 0.0f;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          pv[q] = fast_exp2(fmaf(x[q], a.scale_log2, -nr));
          ps += pv[q];
        }
        ns = ssum * f + ps;
        if constexpr (!MASS) {
#pragma unroll
          for (int dt = 0; dt < AT::kDT; ++dt)
#pragma unroll
            for (int q = 0; q < 4; ++q) o[dt][q] *= f;
        }
        m = nr;
      }
    }
    ssum = ns;
    if constexpr (!MASS) {
      // P ~ hi + lo: hi = the upper half of each float (a bf16 truncation), lo = the
      // remainder, also truncated; packed two weights per register
      uint32_t hb[4], lb[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t u0 = __float_as_uint(pv[2 * q]), u1 = __float_as_uint(pv[2 * q + 1]);
        const float l0 = pv[2 * q] - __uint_as_float(u0 & 0xffff0000u);
        const float l1 = pv[2 * q + 1] - __uint_as_float(u1 & 0xffff0000u);
        hb[q] = __builtin_amdgcn_perm(u1, u0, 0x07060302u);
        lb[q] = __builtin_amdgcn_perm(__float_as_uint(l1), __float_as_uint(l0), 0x07060302u);
      }
      const uint4 ph = make_uint4(hb[0], hb[1], hb[2], hb[3]);
      const uint4 pl = make_uint4(lb[0], lb[1], lb[2], lb[3]);
      const char* vl = kl + AT::kKBytes;
#pragma unroll
      for (int dt = 0; dt < AT::kDT; ++dt) {
        const int d = dt * 16 + c16;
        const char* vrow = vl + d * (kAttKT * 2);
        const uint2 v0 = *reinterpret_cast<const uint2*>(vrow + (((8 * ks + g16) ^ (d & 15)) * 8));
        const uint2 v1 = *reinterpret_cast<const uint2*>(vrow + (((8 * ks + 4 + g16) ^ (d & 15)) * 8));
        const uint4 vf = make_uint4(v0.x, v0.y, v1.x, v1.y);
        o[dt] = mma_step(bf16_t{}, vf, ph, o[dt]);
        o[dt] = mma_step(bf16_t{}, vf, pl, o[dt]);
      }
    }
  };

  // Whole rounds of PF tiles: the loads of tile t + PF are issued while tile t is computed,
  // so the PF - 1 younger tiles' loads are always in flight when tile t's are awaited and
  // every wait has a fixed count; the first wait also covers the query fragments.
  const int nt = (n_vis_max + kAttKT - 1) / kAttKT;
  const int rounds = (nt + PF - 1) / PF;
#pragma unroll
  for (int p = 0; p < PF; ++p) stage_load(p, kst[p], vst[p]);
  asm_wait_vmcnt<(PF - 1) * LPT>();
#pragma unroll
  for (int st = 0; st < NS; ++st) reg_fence(qf[st]);
  for (int rd = 0; rd < rounds; ++rd) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int t = rd * PF + p;
      if (p > 0) asm_wait_vmcnt<(PF - 1) * LPT>();        // tile t's loads have landed
      stage_store(t & 1, kst[p], vst[p]);
      __syncthreads();
      stage_load(t + PF, kst[p], vst[p]);
      compute(t, t & 1);
      __syncthreads();
    }
    asm_wait_vmcnt<(PF - 1) * LPT>();                    // the next round's first tile
  }
  asm_wait_vmcnt<0>();                                   // no load still writes a register

  // merge the four key pairs of each row: references and sums first, then the outputs
  // (through the staging buffers, which are free after the loop's last barrier)
  float st = ssum;
  st += __shfl_xor(st, 16, 64);
  st += __shfl_xor(st, 32, 64);
  if (own && g16 == 0) {
    mfin[ks][rt][c16] = m;
    sfin[ks][rt][c16] = st;
  }
  float* ofin = reinterpret_cast<float*>(lds);                 // [ks][rt][16 rows][D]
  static_assert(MASS || kAttSplit * 4 * 16 * D * 4 <= 2 * kStageBytes, "output merge area");
  if constexpr (!MASS) {
    if (own) {
#pragma unroll
      for (int dt = 0; dt < AT::kDT; ++dt)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          ofin[((ks * 4 + rt) * 16 + c16) * D + dt * 16 + 4 * g16 + q] = o[dt][q];
    }
  }
  __syncthreads();
  if (ks != 0 || !own || r >= a.n_q) return;
  float mf = mfin[0][rt][c16];
#pragma unroll
  for (int k = 1; k < kAttSplit; ++k) mf = fmaxf(mf, mfin[k][rt][c16]);
  float w[kAttSplit], sf = 0.0f;
#pragma unroll
  for (int k = 0; k < kAttSplit; ++k) {
    w[k] = rescale(mfin[k][rt][c16], mf);
    sf += sfin[k][rt][c16] * w[k];
  }
  const bool seen = sf > 0.0f;
  const float lse_r = seen ? (mf + __log2f(sf)) * 0.6931471805599453f : -INFINITY;
  const int64_t ri = (int64_t)hq * q_rows + (int64_t)b * a.n_q + r;
  if constexpr (MASS) {
    if (g16 == 0) {
      // deficit log Z - log Z_R >= 0 (rounding can leave it a hair below 0)
      const float dlt = fmaxf(a.lse_full[ri] - lse_r, 0.0f);
      a.rho[ri] = -expm1f(-dlt);
    }
  } else {
    if (g16 == 0) a.lse[ri] = lse_r;
    const float inv = seen ? 1.0f / sf : 0.0f;
#pragma unroll
    for (int dt = 0; dt < AT::kDT; ++dt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = dt * 16 + 4 * g16 + q;
        float acc = 0.0f;
#pragma unroll
        for (int k = 0; k < kAttSplit; ++k) acc += ofin[((k * 4 + rt) * 16 + c16) * D + e] * w[k];
        a.out[ri * D + e] = acc * inv;
      }
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

template <int D, bool MASS>
hipError_t launch_att_mfma(const AttArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((cache_attention_mfma_kernel<D, MASS>),
                     dim3(xcd_grid(a.batch * a.n_kv_heads * a.G)), dim3(AttMfma<D, MASS>::kThreads), 0,
                     st, a);
  if constexpr (MASS)
    hipLaunchKernelGGL(mass_reduce_kernel, dim3(a.batch, a.n_kv_heads), dim3(64), 0, st, a);
  return hipGetLastError();
}

template <bool MASS>
hipError_t launch_att_typed(const dge_geom_t& g, const AttArgs& a, hipStream_t st) {
  // the matrix-core path: bf16, at most 64 query rows (a row tile per wavefront), d = 128
  // (or 64 for the evicted mass)
  if (g.dtype == DGE_BF16 && a.n_q >= 1 && a.n_q <= 64) {
    if (g.head_dim == 128) return launch_att_mfma<128, MASS>(a, st);
    if constexpr (MASS) {
      if (g.head_dim == 64) return launch_att_mfma<64, true>(a, st);
    }
  }
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
