// Device-side helpers shared by the gfx950 kernels of the eviction step.
//
// Matrix-core fragments.  Every QK^T product here runs on the 16x16 MFMA tiles of
// CDNA4 with 64-lane wavefronts:
//   bf16: v_mfma_f32_16x16x32_bf16  (A 16x32, B 32x16, one 16-byte chunk per lane)
//   f32 : v_mfma_f32_16x16x4_f32    (four issues consume one 16-byte chunk per lane)
// Lane l supplies row (l % 16) of A and column (l % 16) of B; lane group g = l / 16
// supplies a contiguous run of the reduction dimension.  Because the same run is
// loaded for A (query rows) and B (key rows), the pairing of reduction indices
// inside the instruction never matters.  The accumulator tile is read as
//   D[4*g + t][l % 16], t = 0..3,
// i.e. a lane holds 4 query rows of one key column.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dge {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kWave = 64;

// Storage tags: bf16 elements are moved as raw 16-bit patterns.
struct bf16_t { uint16_t bits; };

template <typename T> struct Elem;
template <> struct Elem<bf16_t> { static constexpr int kBytes = 2; };
template <> struct Elem<float> { static constexpr int kBytes = 4; };

// Number of 16-byte chunk steps a wave needs to cover one row of D elements
// (each step covers 64 bytes of the row: 16 bytes from each lane group).
template <typename T, int D>
struct RowChunks {
  static constexpr int kElemsPerLane = 16 / Elem<T>::kBytes;   // per lane per step
  static constexpr int kElemsPerStep = 4 * kElemsPerLane;       // per wave per step
  static constexpr int kSteps = D / kElemsPerStep;
};

__device__ __forceinline__ uint4 load16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ f32x4_t mma_step(bf16_t, uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4_t mma_step(float, uint4 a, uint4 b, f32x4_t c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

// Element offset, within a row, of the 16 bytes lane group g loads at chunk step s.
template <typename T, int D>
__device__ __forceinline__ int chunk_elem(int s, int g) {
  return s * RowChunks<T, D>::kElemsPerStep + g * RowChunks<T, D>::kElemsPerLane;
}

// Online softmax statistics in the log2 domain: value m (running max) and
// s = sum 2^(x - m).  One exp2 per element: the larger of (x, m) becomes the max.
__device__ __forceinline__ void online_push(float x, float& m, float& s) {
  const float dlt = x - m;              // m == -inf on the first push gives +inf
  const float e = exp2f(-fabsf(dlt));
  const bool up = dlt > 0.0f;
  s = up ? fmaf(s, e, 1.0f) : s + e;
  m = up ? x : m;
}

__device__ __forceinline__ void online_merge(float& m, float& s, float m2, float s2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) { m = mx; s = 0.0f; return; }
  s = s * exp2f(m - mx) + s2 * exp2f(m2 - mx);
  m = mx;
}

template <int kMask>
__device__ __forceinline__ float shfl_xor_f(float v) {
  return __shfl_xor(v, kMask, kWave);
}

// 2^x on the transcendental unit (v_exp_f32); results below 2^-126 may flush to 0,
// far below anything a softmax score resolves.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Rescale factor 2^(m - mx) for merging a (max, sum) pair into a larger max mx,
// well defined when both are -inf (empty partial).
__device__ __forceinline__ float rescale(float m, float mx) {
  return m == mx ? 1.0f : fast_exp2(m - mx);
}

// Online sums of 2^(x*scale - m) (log2 domain) for R rows, NV logits of each per call,
// x unscaled logits and scale = log2(e)/sqrt(d).  The common path is fma + exp2 + add per
// logit against the current reference m, with no maximum: only when a row's sum reaches
// kSumLimit = 2^100 (a logit about 2^7 above m, or very many somewhat above it) does
// that row, in one wave-uniform branch, move its reference up to its batch maximum (and
// at least kLazyBound above the old one) and sum the batch again onto the rescaled old
// sum, which then stays below 2^37.  Accepted sums stay below 2^100, so merging a few
// of them (lane groups, wavefronts) cannot overflow.  m starts finite and very negative
// (kLazyRefInit): the first live batch of a row takes the branch, masked logits (-inf)
// add exactly 0, and the result merges with others like any (max, sum) pair.
constexpr float kLazyBound = 64.0f;
constexpr float kLazyRefInit = -1.0e30f;
constexpr float kSumLimit = 0x1p100f;
template <int R, int NV>
__device__ __forceinline__ void rebase_lse_update(const float (&x)[R][NV], float scale, float* m,
                                                  float* s) {
  auto batch = [&](int r, float ref) {
    float e[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) e[i] = fast_exp2(fmaf(x[r][i], scale, -ref));
#pragma unroll
    for (int w = 1; w < NV; w *= 2)
#pragma unroll
      for (int i = 0; i + w < NV; i += 2 * w) e[i] += e[i + w];
    return e[0];
  };
  // one wave-wide test for all R sums: their maximum against the limit (the sums are
  // never NaN: finite or masked (-inf) logits give exponentials in [0, inf])
  float ns[R];
  float big = 0.0f;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    ns[r] = s[r] + batch(r, m[r]);
    big = fmaxf(big, ns[r]);
  }
  if (__builtin_amdgcn_ballot_w64(!(big < kSumLimit)) != 0) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!(ns[r] < kSumLimit)) {
        float mx = x[r][0];
#pragma unroll
        for (int i = 1; i < NV; ++i) mx = fmaxf(mx, x[r][i]);
        const float nr = fmaxf(mx * scale, m[r] + kLazyBound);
        ns[r] = fmaf(s[r], fast_exp2(m[r] - nr), batch(r, nr));
        m[r] = nr;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) s[r] = ns[r];
}

// Sum of v over the four lane groups (lanes l, l^16, l^32, l^48), returned in every
// lane.  v_permlane32_swap exchanges the upper half of one copy with the lower half of
// the other, so the two results add to the sum over l and l^32; v_permlane16_swap does
// the same for odd/even rows of 16 lanes.  Both are VALU operations (no LDS round trip).
__device__ __forceinline__ float sum_lane_groups(float v) {
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  v = __uint_as_float(h[0]) + __uint_as_float(h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Reduce-scatter over the four lane groups: lane group g returns, for its position
// c = l % 16, the sum of v[g] over lanes c, c+16, c+32, c+48.  The first two swaps
// leave the half-sums of v[0] / v[1] in lanes 0-31 and of v[2] / v[3] in lanes 32-63;
// the row swap then pairs rows (0,1) and (2,3).
__device__ __forceinline__ float reduce_scatter_lane_groups(const float (&v)[4]) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[0]), __float_as_uint(v[2]),
                                                  false, false);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[1]), __float_as_uint(v[3]),
                                                  false, false);
  const float a = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const float b = __uint_as_float(q[0]) + __uint_as_float(q[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Waits and barriers for pipelines that keep global->LDS copies in flight across
// workgroup barriers (__syncthreads() would drain every outstanding load).
// s_waitcnt immediate on gfx9: vmcnt[3:0] + vmcnt[5:4] at [15:14], expcnt[6:4],
// lgkmcnt[11:8]; fields not waited on are set to their maximum.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}
// Workgroup barrier for LDS traffic only: this wave's LDS reads/writes are done, then
// s_barrier.  Outstanding global loads (including global->LDS copies) stay in flight.
// The empty asm statements keep the compiler from moving memory accesses across the
// barrier (the s_barrier builtin itself is not a memory operation to the optimiser).
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void lds_barrier() {
  wait_lgkmcnt0();
  wg_barrier();
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) const void* global_ptr_t;

// 16 bytes per lane from global memory straight into LDS: lane l of the wavefront
// writes lds_wave_base + 16 * l (lds_wave_base must be the same for the whole wave).
// Issued from asm so that the compiler's own wait insertion, which cannot tell the
// ring buffers apart, does not drain every copy in flight before each LDS read; the
// callers order these copies with explicit vmcnt waits and workgroup barriers.  M0
// (the LDS base) is saved and restored around the copy; the s_nop covers the wait
// state required between an M0 write and an LDS-DMA load.
__device__ __forceinline__ void dma16(const void* g, void* lds_wave_base) {
  const uint32_t base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(lds_ptr_t)lds_wave_base);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(base)
      : "memory");
}

// As dma16, with the global address split into a wave-uniform base (an SGPR pair) and a
// 32-bit per-lane byte offset (the saddr form of the instruction): no 64-bit address
// arithmetic per lane.  lds_wave_base must already be wave-uniform.
__device__ __forceinline__ void dma16_sbase(const void* sbase, uint32_t voff,
                                            uint32_t lds_wave_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "s"(lds_wave_base)
      : "memory");
}

// Register loads issued from asm, for kernels that keep global->LDS copies in flight
// with explicit vmcnt waits: the compiler does not track these loads, so it inserts no
// wait of its own (which would also drain the copies).  The caller waits (vmcnt) and
// then passes the values through reg_fence() before any use, so that nothing reads the
// registers while the load is outstanding.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4_t async_load16(const void* p) {
  u32x4_t v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ float async_load4(const void* p) {
  float v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void reg_fence(u32x4_t& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ uint4 as_uint4(const u32x4_t& v) { return __builtin_bit_cast(uint4, v); }
__device__ __forceinline__ void reg_fence(float& v) { asm volatile("" : "+v"(v)); }
// vmcnt wait as an asm statement, ordered with the loads and fences above.
template <int N>
__device__ __forceinline__ void asm_wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// XCD-aware work mapping.  The command processor hands workgroups to the 8 XCDs of an
// MI355X round-robin by linear block id, and each XCD has its own L2.  Grids that use
// this mapping are 1-D with a multiple of 8 blocks; block L runs on XCD L % 8 and takes
// unit (L % 8) * per + L / 8, so every XCD owns one contiguous range of units (units
// that share inputs -- the chunks of one KV head -- then share one L2).  Units at or
// beyond `total` belong to no work and exit.
constexpr int kXcds = 8;
__host__ __device__ __forceinline__ int xcd_per(int total) { return (total + kXcds - 1) / kXcds; }
__host__ __device__ __forceinline__ int xcd_grid(int total) { return kXcds * xcd_per(total); }
__device__ __forceinline__ int xcd_unit(int total) {
  const int L = (int)blockIdx.x;
  return (L % kXcds) * xcd_per(total) + L / kXcds;
}

// Sequence offsets as a kernel argument: up to kInlineSeqs sequences whose offsets fit
// in 31 bits travel by value in the argument block (as 32-bit values); otherwise the
// kernel reads the device array.  The inline values are picked by a select chain over
// values held in scalar registers (not an indexed load: that would add a dependent
// round trip at kernel start), and the result is wave-uniform.
constexpr int kInlineSeqs = 16;
struct SeqOffsets {
  const int64_t* dev;
  int32_t inl[kInlineSeqs + 1];
  int batch;
  int use_inline;
  // i must be the same for the whole wavefront
  __device__ __forceinline__ int64_t operator[](int i) const {
    if (use_inline) {
      int32_t v = inl[0];
      asm volatile("" : "+s"(v));
#pragma unroll
      for (int k = 1; k <= kInlineSeqs; ++k) {
        int32_t w = inl[k];
        asm volatile("" : "+s"(w));
        v = i == k ? w : v;
      }
      return v;
    }
    const int64_t v = dev[i];
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
  }
};

// Makes the given kernel arguments resident in scalar registers at this point, so that
// they are fetched together (one round trip) instead of one dependent load at a time
// after each early-exit branch.
template <typename T>
__device__ __forceinline__ void prefetch_arg(const T& x) {
  asm volatile("" : : "s"(x));
}
__device__ __forceinline__ void prefetch_arg(const SeqOffsets& o) {
  prefetch_arg(o.use_inline);
  prefetch_arg(o.dev);
#pragma unroll
  for (int k = 0; k <= kInlineSeqs; ++k) prefetch_arg(o.inl[k]);
}
template <typename... Ts>
__device__ __forceinline__ void prefetch_args(const Ts&... xs) {
  (prefetch_arg(xs), ...);
}

}  // namespace dge
